// Store kernels: device metadata (block table and dense live lists), row
// insert into a page, page scrub and canonical export.
//
// The memory is the multiset of all blocks' rows, listed by block index
// (Section 2, "Model").  Device metadata per sequence:
//   table[seq][j]     page holding block j, or -1
//   live_blk[seq][i]  i-th present block index, ascending
//   live_page[seq][i] its page
//   n_live[seq]
// An edit sets table entries, then the sequence's dense lists are rebuilt
// from the table by a stream compaction: indices move, rows never do
// (Theorem 1: deleting a block leaves the other blocks' rows and indices
// untouched).
#include "common.h"

namespace smem {

__global__ void k_init_meta(int32_t* __restrict__ table, int32_t* __restrict__ n_live, size_t n_table, int n_seq) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t j = i; j < n_table; j += stride) table[j] = -1;
  for (size_t j = i; j < (size_t)n_seq; j += stride) n_live[j] = 0;
}

hipError_t launch_init_meta(int32_t* table, int32_t* n_live, size_t n_table, int n_seq, hipStream_t s) {
  size_t work = n_table > (size_t)n_seq ? n_table : (size_t)n_seq;
  unsigned grid = (unsigned)((work + 255) / 256);
  if (grid > 4096) grid = 4096;
  if (grid == 0) grid = 1;
  hipLaunchKernelGGL(k_init_meta, dim3(grid), dim3(256), 0, s, table, n_live, n_table, n_seq);
  return hipGetLastError();
}

// One workgroup per (sequence, table chunk) item: apply this launch's edits
// that fall in the chunk to the table, then write the chunk's live blocks,
// in index order, into the dense lists from the position the host computed
// for it (the live blocks of the earlier chunks, after the edits).  Each
// thread takes kMetaPerThread consecutive entries; offsets inside the chunk
// come from wave prefix sums (shuffles) and wave totals in LDS.
constexpr int kMetaPerThread = kMetaChunk / 256;

__global__ void __launch_bounds__(256) k_meta(MetaArgs a) {
  const int it = blockIdx.x;
  const int seq = a.i_seq[it];
  const int j0 = a.i_chunk[it] * kMetaChunk;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t* trow = a.table + (size_t)seq * a.max_blocks;
  for (int e = tid; e < a.n_edits; e += 256)
    if (a.e_seq[e] == seq && a.e_blk[e] >= j0 && a.e_blk[e] < j0 + kMetaChunk) trow[a.e_blk[e]] = a.e_page[e];
  __syncthreads();

  __shared__ int wave_tot[4];
  int32_t* lp = a.live_page + (size_t)seq * a.max_blocks;
  int32_t* lb = a.live_blk + (size_t)seq * a.max_blocks;
  const int jt = j0 + tid * kMetaPerThread;
  int32_t v[kMetaPerThread];
  int cnt = 0;
#pragma unroll
  for (int e = 0; e < kMetaPerThread; ++e) {
    const int j = jt + e;
    v[e] = (j < a.max_blocks) ? trow[j] : -1;
    cnt += v[e] >= 0 ? 1 : 0;
  }
  int incl = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wave_tot[wave] = incl;
  __syncthreads();
  int off = a.i_base[it] + incl - cnt;
  for (int w = 0; w < wave; ++w) off += wave_tot[w];
#pragma unroll
  for (int e = 0; e < kMetaPerThread; ++e) {
    if (v[e] >= 0) {
      lp[off] = v[e];
      lb[off] = jt + e;
      ++off;
    }
  }
  if (a.i_last[it] && tid == 0)
    a.n_live[seq] = a.i_base[it] + wave_tot[0] + wave_tot[1] + wave_tot[2] + wave_tot[3];
}

hipError_t launch_meta(const MetaArgs& a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_meta, dim3(a.n_items), dim3(256), 0, s, a);
  return hipGetLastError();
}

// Insert one block's rows: src rows [b][H][dh] -> key plane [b][dh] and
// transposed value plane [dh][b] of every head.  One workgroup per head;
// 16-byte loads and stores throughout, the value tile transposed through LDS.
template <typename T>
__global__ void __launch_bounds__(256) k_put_rows(PutArgs a) {
  constexpr int E = 16 / sizeof(T);
  extern __shared__ unsigned char smem_raw[];
  T* tile = reinterpret_cast<T*>(smem_raw);  // [b][dh + 1]
  const int h = blockIdx.x, i = blockIdx.y;
  const int H = a.H, b = a.b, dh = a.dh;
  T* kp = (T*)a.pages + page_head_offset(a.page[i], h, H, b, dh);
  T* vp = kp + (size_t)b * dh;
  const T* k_rows = (const T*)a.k_rows + (size_t)i * b * H * dh;
  const T* v_rows = (const T*)a.v_rows + (size_t)i * b * H * dh;
  const int cpr = dh / E;
  for (int j = threadIdx.x; j < b * cpr; j += blockDim.x) {
    const int r = j / cpr, c = j % cpr;
    const size_t src = ((size_t)r * H + h) * dh + c * E;
    *(u32x4*)(kp + r * dh + c * E) = *(const u32x4*)(k_rows + src);
    const u32x4 vv = *(const u32x4*)(v_rows + src);
    T vals[E];
    __builtin_memcpy(vals, &vv, 16);
#pragma unroll
    for (int e = 0; e < E; ++e) tile[r * (dh + 1) + c * E + e] = vals[e];
  }
  __syncthreads();
  const int cpv = b / E;
  for (int j = threadIdx.x; j < dh * cpv; j += blockDim.x) {
    const int d = j / cpv, kc = j % cpv;
    T vals[E];
#pragma unroll
    for (int e = 0; e < E; ++e) vals[e] = tile[(kc * E + e) * (dh + 1) + d];
    u32x4 out;
    __builtin_memcpy(&out, vals, 16);
    *(u32x4*)(vp + d * b + kc * E) = out;
  }
}

hipError_t launch_put_blocks(int dtype, const PutArgs& a, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const size_t es = dtype == F32 ? 4 : 2;
  const size_t lds = (size_t)a.b * (a.dh + 1) * es;
  if (dtype == F32) hipLaunchKernelGGL(k_put_rows<float>, dim3(a.H, n), dim3(256), lds, s, a);
  else hipLaunchKernelGGL(k_put_rows<uint16_t>, dim3(a.H, n), dim3(256), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_put_rows(int dtype, void* pages, int page, int H, int b, int dh,
                           const void* k_rows, const void* v_rows, hipStream_t s) {
  PutArgs a;
  a.pages = pages; a.k_rows = k_rows; a.v_rows = v_rows;
  a.H = H; a.b = b; a.dh = dh;
  a.page[0] = page;
  return launch_put_blocks(dtype, a, 1, s);
}

__global__ void k_scrub(uint4* __restrict__ p, size_t n16) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  const uint4 z = make_uint4(0, 0, 0, 0);
  for (; i < n16; i += stride) p[i] = z;
}

hipError_t launch_scrub(void* page_base, size_t bytes, hipStream_t s) {
  char* base = (char*)page_base;     // a page is a multiple of 16 bytes
  size_t n16 = bytes / 16;
  unsigned grid = (unsigned)((n16 + 255) / 256);
  if (grid > 1024) grid = 1024;
  hipLaunchKernelGGL(k_scrub, dim3(grid), dim3(256), 0, s, (uint4*)base, n16);
  return hipGetLastError();
}

// Canonical export: live entry i, head h -> rows [i*b, (i+1)*b) of k_out and
// v_out ([rows][H][dh]).  Every global access is a whole 16-byte chunk: the
// key plane is copied row chunk by row chunk (a key row is contiguous in the
// page and in the output); the value plane [dh][b] goes through LDS, where
// chunk rc of value row d sits at slot rc ^ ((d / E) mod (b / E)), so the
// gather of one output chunk (E dims of one row) by neighbouring lanes
// (neighbouring chunks of the row) spreads over the banks.
template <typename T>
__global__ void __launch_bounds__(256) k_export(const T* __restrict__ pages, const int32_t* __restrict__ live_page,
                                                 int H, int b, int dh, T* __restrict__ k_out, T* __restrict__ v_out) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  T* tile = reinterpret_cast<T*>(smem_raw);  // [dh][b], 16-byte slots permuted per row
  constexpr int E = 16 / sizeof(T);          // elements per 16-byte chunk
  const int i = blockIdx.x, h = blockIdx.y;
  const T* kp = pages + page_head_offset(live_page[i], h, H, b, dh);
  const T* vp = kp + (size_t)b * dh;
  const int CR = dh / E, CB = b / E;         // chunks per output row, per value row
  const size_t rs = (size_t)H * dh;          // output row stride
  T* ko = k_out + ((size_t)i * b * H + h) * dh;
  T* vo = v_out + ((size_t)i * b * H + h) * dh;
  for (int q = threadIdx.x; q < b * CR; q += blockDim.x) {
    const int r = q / CR, cc = q % CR;
    *(u32x4*)(ko + r * rs + cc * E) = *(const u32x4*)(kp + r * dh + cc * E);
  }
  for (int q = threadIdx.x; q < dh * CB; q += blockDim.x) {
    const int d = q / CB, rc = q % CB;
    *(u32x4*)(tile + d * b + ((rc ^ ((d / E) % CB)) * E)) = *(const u32x4*)(vp + d * b + rc * E);
  }
  __syncthreads();
  for (int q = threadIdx.x; q < b * CR; q += blockDim.x) {
    const int r = q / CR, cc = q % CR;
    const int off = ((r / E) ^ (cc % CB)) * E + r % E;
    union {
      u32x4 u;
      T e[E];
    } v;
#pragma unroll
    for (int j = 0; j < E; ++j) v.e[j] = tile[(cc * E + j) * b + off];
    *(u32x4*)(vo + r * rs + cc * E) = v.u;
  }
}

hipError_t launch_export(int dtype, const void* pages, const int32_t* live_page_seq, int n_live,
                         int H, int b, int dh, void* k_out, void* v_out, hipStream_t s) {
  if (n_live <= 0) return hipSuccess;
  if (dtype == F32) {
    hipLaunchKernelGGL(k_export<float>, dim3(n_live, H), dim3(256), (size_t)dh * b * sizeof(float), s,
                       (const float*)pages, live_page_seq, H, b, dh, (float*)k_out, (float*)v_out);
  } else {
    hipLaunchKernelGGL(k_export<uint16_t>, dim3(n_live, H), dim3(256), (size_t)dh * b * sizeof(uint16_t), s,
                       (const uint16_t*)pages, live_page_seq, H, b, dh, (uint16_t*)k_out, (uint16_t*)v_out);
  }
  return hipGetLastError();
}

__global__ void __launch_bounds__(256) k_copy16(u32x4* __restrict__ dst, const u32x4* __restrict__ src, size_t n16) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n16; i += stride) dst[i] = src[i];
}

hipError_t launch_copy16(void* dst, const void* src, size_t bytes, hipStream_t s) {
  const size_t n16 = bytes / 16;
  unsigned grid = (unsigned)((n16 + 255) / 256);
  if (grid > 1024) grid = 1024;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy16, dim3(grid), dim3(256), 0, s, (u32x4*)dst, (const u32x4*)src, n16);
  return hipGetLastError();
}

// The same copy through LDS by DMA (global_load_lds_dwordx4, the way the
// attention kernels bring pages in): each workgroup moves 16 KiB tiles, the
// four waves loading 4 KiB each into LDS, then storing them from LDS.
// bytes is a multiple of 16 KiB.
__global__ void __launch_bounds__(256) k_copy_dma(uint8_t* __restrict__ dst, const uint8_t* __restrict__ src,
                                                  size_t n_tiles) {
  __shared__ __attribute__((aligned(1024))) uint8_t buf[16384];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t lds0 = (uint32_t)(uintptr_t)buf + (uint32_t)(wave * 4096);
  for (size_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
    const uint8_t* s = src + t * 16384 + wave * 4096 + lane * 16;
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16(s + i * 1024, __builtin_amdgcn_readfirstlane(lds0 + i * 1024));
    wait_vm<0>();
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *(u32x4*)(dst + t * 16384 + (i * 256 + tid) * 16) = *(const u32x4*)(buf + (i * 256 + tid) * 16);
    __syncthreads();
  }
}

hipError_t launch_copy_dma(void* dst, const void* src, size_t bytes, hipStream_t s) {
  const size_t n_tiles = bytes / 16384;
  if (n_tiles == 0) return hipSuccess;
  const unsigned grid = (unsigned)(n_tiles < 2048 ? n_tiles : 2048);
  hipLaunchKernelGGL(k_copy_dma, dim3(grid), dim3(256), 0, s, (uint8_t*)dst, (const uint8_t*)src, n_tiles);
  return hipGetLastError();
}

// Rotary table (the SMem+RoPE composite): entry (p, k) = (cos, sin) of
// p * base^(-2k/dh), evaluated in fp64 and stored as fp32.
__global__ void __launch_bounds__(256) k_rope_table(float* __restrict__ tab, int dh, int n_phases, double base) {
  const int half = dh / 2;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n_phases * half) return;
  const int p = i / half, k = i % half;
  const double ang = (double)p * pow(base, -2.0 * (double)k / (double)dh);
  double sn, cs;
  sincos(ang, &sn, &cs);
  *(f32x2*)(tab + 2 * (size_t)i) = f32x2{(float)cs, (float)sn};
}

hipError_t launch_rope_table(float* table, int dh, int n_phases, double base, hipStream_t s) {
  const int n = n_phases * (dh / 2);
  if (n <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, s, table, dh, n_phases, base);
  return hipGetLastError();
}

}  // namespace smem
