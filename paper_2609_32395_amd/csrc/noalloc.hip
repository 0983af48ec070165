// Reader decode whose split partials live in a library-held device array, for
// callers that cannot allocate (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc) and for stores whose workspace they
// want left untouched.
//
// `scratch` is a file-scope device array: every GPU the library runs on holds
// its own copy, at its own address, until the process ends.  Host code never
// uses the array's name as a device address (on the host it is only a
// stand-in symbol); the first call on a device looks the device address up
// with hipGetSymbolAddress, with that device current, and keeps it.
//
// Every call on one GPU shares that GPU's array and leaves the last call's
// partials in it.  Nothing in it has to start at zero: a call writes every
// split record before its merge reads it.  Calls that overlap on one GPU
// (different streams, or several host threads without ordering) race on the
// array; calls ordered on one stream do not.
#include <mutex>

#include "common.h"

namespace smem {

// 16 MiB of split partials: (dh + 4) floats per split of each (sequence,
// head).  The 410M-shaped decode (64 sequences x 16 heads, 9 splits, dh 64)
// takes 2.4 MiB, the 1.5B-shaped stress decode (16 x 16, 65 splits, dh 128)
// 8.4 MiB.
constexpr size_t kStaticScratchFloats = (size_t)4 << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) float scratch[kStaticScratchFloats];

namespace {

std::mutex g_mu;
float* g_ptr[kMaxDevices] = {};

// Device address of this GPU's scratch array (the current device's).
smem_status scratch_of_current_device(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(SMEM_EHIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return set_error(SMEM_EINVAL, "device ordinal beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) return set_error(SMEM_EHIP, "hipGetSymbolAddress(scratch) failed");
    g_ptr[dev] = (float*)p;
  }
  *out = g_ptr[dev];
  return SMEM_OK;
}

}  // namespace
}  // namespace smem

extern "C" smem_status smem_reader_decode_static(smem_store* st, int32_t n_seq, const int32_t* seq_ids,
                                                 const int32_t* query_block, const int32_t* pos, const void* q,
                                                 const void* k_new, const void* v_new, void* k_cache,
                                                 void* v_cache, const void* null_kv, void* out, hipStream_t s) {
  float* ws = nullptr;
  const smem_status r = smem::scratch_of_current_device(&ws);
  if (r != SMEM_OK) return r;
  return smem::decode_impl(st, nullptr, n_seq, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv,
                           out, ws, smem::kStaticScratchFloats, s);
}
