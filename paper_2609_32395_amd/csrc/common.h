// Shared definitions of the SMem HIP library (gfx950): element conversions,
// the device layout of a store, kernel argument blocks and launcher
// declarations.  Host code (smem_api.cpp) and the kernel files include it.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "smem.h"

namespace smem {

// ---------------------------------------------------------------- constants

// Per-launch capacity of the argument arrays carried by value in kernel
// arguments (sequence ids, block counts, positions).  Larger batches are
// split into several launches by the host.
constexpr int kMaxSlots = 128;
// Edits applied by one metadata launch, and its (sequence, table chunk) work
// items: each item is one workgroup that applies the edits falling in its
// chunk of kMetaChunk table entries and writes the chunk's live blocks into
// the dense lists at a position the host computes.
constexpr int kMaxEdits = 128;
constexpr int kMaxMetaItems = 128;
constexpr int kMetaChunk = 1024;
// Split-K: memory pages of one (query, head) are cut into at most kSplitCap
// splits of whole pages, plus possibly one split for the null row and the
// in-block keys.
constexpr int kSplitCap = 64;
constexpr int kSplitStride = kSplitCap + 1;
// Minimum pages per split and split caps (decode / VALU reader, MFMA prefill).
// A prefill split's partial output is b rows of dh+4 floats, so prefill uses
// fewer, longer splits to keep the partials small next to the pages read.
constexpr int kMinPagesDecode = 8;
// Minimum pages per split of a VALU reader launch: 4 at d_h <= 32, where a
// page is half the bytes (measured on the 410M and 1.5B model decode cells:
// up to 2.5% faster than 8; 16 was slower), else 8 (the 410M decode
// headline: 4 / 8 / 16 pages 167.4 / 162.9 / 179.3 us per step).
inline int min_pages_decode(int dh) { return dh <= 32 ? 4 : kMinPagesDecode; }
constexpr int kMinPagesPrefill = 4;
constexpr int kSplitCapPrefill = 32;
// Memory splits of one prefill (query block, head): enough that a single
// query block fills the chip (about 512 workgroups over the H heads), no more,
// since every split writes a b x (d_h + 4) partial that the merge reads back.
// A function of the store's H alone, so a block's result never depends on the
// batch it is read in.
#ifndef SMEM_PREFILL_WG_TARGET
#define SMEM_PREFILL_WG_TARGET 512
#endif
inline int prefill_split_cap(int H) {
  const int c = SMEM_PREFILL_WG_TARGET / (H > 0 ? H : 1);
  return c < 1 ? 1 : (c > kSplitCapPrefill ? kSplitCapPrefill : c);
}
// An MFMA prefill launch runs one workgroup per (query block, head) pair that
// reads the pair's splits in turn and folds them itself when it has at least
// kFoldPairs pairs (the pairs fill the chip, and the split partials would
// cost more than the longest pair's serial read), or when its longest pair
// reads at most kFoldSerial / max(d_h, 64) pages (16 pages up to d_h = 64: a
// short serial read beats a second launch and the split workgroups' own
// set-up; measured, a single block over 31 pages is faster split).
// Otherwise one workgroup per split and a merge.  Either way the splits and
// their fold are the same, so the choice never changes a result.
// (Decode keeps the split launch and the merge: its one-query workgroups
// stream a page per wave at a time, and folding them was measured slower.)
#ifndef SMEM_FOLD_PAIRS
#define SMEM_FOLD_PAIRS 512
#endif
#ifndef SMEM_FOLD_SERIAL
#define SMEM_FOLD_SERIAL 1024
#endif
constexpr int kFoldPairs = SMEM_FOLD_PAIRS;
constexpr int kFoldSerial = SMEM_FOLD_SERIAL;
inline bool fold_in_workgroup(long n_pairs, int max_pages, int dh) {
  return n_pairs >= kFoldPairs || (long)max_pages * (dh > 64 ? dh : 64) <= kFoldSerial;
}
// A folding launch of at most kParPairs pairs at d_h <= 64 whose reads have
// at most four memory splits runs the few-pair variant instead: one wave
// group per split, the four read at once, each pair's query rows split over
// two workgroups (same splits, same fold, same bits).
#ifndef SMEM_PAR_PAIRS
#define SMEM_PAR_PAIRS 128
#endif
constexpr int kParPairs = SMEM_PAR_PAIRS;
constexpr int kParSplits = 4;
// Query slots whose prefill partials the workspace must hold at once.
constexpr int kPrefillSlotChunk = 16;
// Row-plane decode: pages per split max(kMinPagesRows, ceil(n_read /
// kRowsSplitCap)), and at most kRowsPartials split partials per launch.
constexpr int kMinPagesRows = 8;
constexpr int kRowsSplitCap = 32;
constexpr int kRowsPartials = 1024;

// Pages per split: a function of the number of memory pages read only, so a
// query's split boundaries (and hence its rounding) never depend on the
// batch it is in or on the physical page numbers.
inline int pages_per_split(int n_read, int min_pages, int cap = kSplitCap) {
  int p = (n_read + cap - 1) / cap;
  return p < min_pages ? min_pages : p;
}
// Splits of one (query, head): ceil(n_read / pps) memory splits, then one
// split for the null row and the in-block keys.
__host__ __device__ inline int total_splits(int n_read, int pps) { return (n_read + pps - 1) / pps + 1; }

enum Dtype : int32_t { F32 = 0, BF16 = 1 };

// Native vector types (kept in registers by the compiler; used for every
// 16- and 8-byte load, store and register stage).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Streamed page data is read once per call: non-temporal loads keep it from
// displacing reused lines in the caches.
__device__ __forceinline__ u32x4 load_stream(const void* p) {
  return __builtin_nontemporal_load((const u32x4*)p);
}

// ---------------------------------------------------------------- LDS DMA

// s_waitcnt with only the vector-memory counter limited to n (0..63).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// One 16-byte-per-lane global -> LDS load: lane l's 16 bytes land at LDS
// byte address lds + 16*l (M0 holds the uniform base).  Issued as assembly
// so that the compiler does not tie later LDS reads or barriers to it with a
// full vector-memory wait; completion is waited for explicitly (wait_vm).
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(g), "s"(lds) : "memory", "m0");
}

// Barrier for LDS hand-offs between waves: this wave's LDS writes complete
// (lgkmcnt 0), then s_barrier; vector-memory loads (the DMA ring) stay in
// flight.  The empty asm statements keep the compiler from moving memory
// operations across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" : : : "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // vmcnt 63, expcnt 7, lgkmcnt 0
  __builtin_amdgcn_s_barrier();
  asm volatile("" : : : "memory");
}

// ---------------------------------------------------------------- conversions

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t x) { return __uint_as_float(x << 16); }

// float -> bf16 bits, round to nearest even (the gfx950 conversion instruction).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  const __bf16 h = (__bf16)f;
  return __builtin_bit_cast(uint16_t, h);
}

// 2^x for softmax weights, x <= 0: the hardware exponential.  Arguments below
// -126 come out as 0 or a denormal, a weight that is negligible next to the
// maximum's weight of 1; 2^-inf = 0 exactly.
__device__ __forceinline__ float exp2w(float x) { return __builtin_amdgcn_exp2f(x); }

// Split partials of one (query, head) -- running maximum m (log2 units), sum
// of weights l, unnormalised output o -- are combined in split order by a
// running rescale, starting from split 0's triple as it is:
//   M' = max(M, m_s), alpha = 2^(M - M'), beta = 2^(m_s - M'),
//   L <- fma(l_s, beta, L alpha), O <- fma(o_s, beta, O alpha), M <- M'.
// The split merge and the one-workgroup prefill both call these two
// functions, so a (query, head) gets the same bits whichever of them
// combines its splits.  An empty split (m_s = -inf, l_s = 0, o_s = 0) leaves
// the state unchanged; M stays finite because split 0 reads memory rows.
struct FoldScale {
  float alpha, beta;
};
__device__ __forceinline__ FoldScale fold_scale(float& M, float m_s) {
  const float Mn = fmaxf(M, m_s);
  const FoldScale c{exp2w(M - Mn), exp2w(m_s - Mn)};
  M = Mn;
  return c;
}
__device__ __forceinline__ float fold_value(float acc, const FoldScale& c, float x) {
  return __builtin_fmaf(x, c.beta, acc * c.alpha);
}

// 16-byte chunk -> E floats (E = 4 for fp32, 8 for bf16).
template <typename T> struct Chunk;
template <> struct Chunk<float> {
  static constexpr int E = 4;
  __device__ __forceinline__ static void unpack(const u32x4& c, float* f) {
    f[0] = __uint_as_float(c.x); f[1] = __uint_as_float(c.y);
    f[2] = __uint_as_float(c.z); f[3] = __uint_as_float(c.w);
  }
};
template <> struct Chunk<uint16_t> {
  static constexpr int E = 8;
  __device__ __forceinline__ static void unpack(const u32x4& c, float* f) {
    f[0] = __uint_as_float(c.x << 16); f[1] = __uint_as_float(c.x & 0xffff0000u);
    f[2] = __uint_as_float(c.y << 16); f[3] = __uint_as_float(c.y & 0xffff0000u);
    f[4] = __uint_as_float(c.z << 16); f[5] = __uint_as_float(c.z & 0xffff0000u);
    f[6] = __uint_as_float(c.w << 16); f[7] = __uint_as_float(c.w & 0xffff0000u);
  }
};

// ---------------------------------------------------------------- rotary phases

// Rotary table: row p (p = 0 .. n_phases-1) holds, for each adjacent pair k
// of a head's dh dimensions, (cos, sin) of the angle p * base^(-2k/dh) as
// fp32; a row is dh floats.  rope_turn rotates E consecutive elements
// (E/2 pairs starting at pair k0, k0 even) by the phase of one row:
// (x0, x1) -> (x0 cos - x1 sin, x0 sin + x1 cos).
template <int E>
__device__ __forceinline__ void rope_turn(float (&x)[E], const float* __restrict__ row, int k0) {
  static_assert(E % 4 == 0, "two pairs per 16-byte table read");
#pragma unroll
  for (int m = 0; m < E / 4; ++m) {
    const f32x4 cs = *(const f32x4*)(row + 2 * k0 + 4 * m);
    const float a0 = x[4 * m], a1 = x[4 * m + 1], b0 = x[4 * m + 2], b1 = x[4 * m + 3];
    x[4 * m] = a0 * cs.x - a1 * cs.y;
    x[4 * m + 1] = a0 * cs.y + a1 * cs.x;
    x[4 * m + 2] = b0 * cs.z - b1 * cs.w;
    x[4 * m + 3] = b0 * cs.w + b1 * cs.z;
  }
}

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t x) { return bf16_bits_to_f32(x); }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float x) { return f32_to_bf16_bits(x); }

// ---------------------------------------------------------------- device layout

// A page holds one block's rows for every head: for head h, a key plane
// [b][dh] (row-major, one key per row) followed by a value plane stored
// transposed, [dh][b] (one value dimension per row, keys contiguous).  The
// (page, head) pair is one contiguous 2*b*dh run.
__host__ __device__ inline size_t page_head_offset(int page, int h, int H, int b, int dh) {
  return ((size_t)page * H + h) * 2 * (size_t)b * dh;
}

struct DevLayout {
  size_t off_table, off_live_page, off_live_blk, off_n_live, off_ws, off_pages, total;
  size_t ws_floats;    // split partials
  // row stores only: absorbed queries, in-block partials, projected null row,
  // row-split partials (part_cap of them)
  size_t off_qabs, off_intra, off_null_kv, off_sw, off_part;
  int32_t part_cap;
};

// ---------------------------------------------------------------- kernel args

// Reader launch (VALU reader and MFMA prefill): one slot per query row group.
//   prefill: a slot is one (sequence, query block); nq = b queries
//   decode : a slot is one sequence; nq = 1
//   encoder (no memory): a slot is one block; nq = b
struct ReaderArgs {
  const void* q;          // query of (slot i, row t, head h) at ((i*nq + t)*H + h)*dh
  const void* k_in;       // in-block keys: row r of slot i at ((i*b + r)*H + h)*dh (NULL: none)
  const void* v_in;
  const void* k_new;      // decode: key/value of the new token, [slot][H][dh]
  const void* v_new;
  void* k_cache_w;        // decode: the new token is also written to row pos of these
  void* v_cache_w;
  const void* null_kv;    // [2][H][dh] or NULL
  const void* pages;      // page pool
  const int32_t* live_page;  // [n_seq][max_blocks] dense live list -> page
  float* ws;              // split partials, (dh+4) floats each: split k of (query row qr, head h)
                          // at ws + ((qr*H + h)*ws_stride + k)*(dh+4)
  void* out;              // output, same indexing as q
  void* page_sink;        // encoder (fp32): also write O as key and value rows of page aux[i]
  int32_t max_blocks;
  int32_t H;
  int32_t b;
  int32_t nq;
  int32_t intra_mode;     // 0: all b keys (bidirectional), 1: keys 0..t (causal), 2: decode, keys 0..pos
  int32_t n_slots;
  float scale_log2;       // log2(e)/sqrt(dh)
  int32_t seq[kMaxSlots];     // sequence of the slot (its live list)
  int32_t n_read[kMaxSlots];  // memory pages the slot reads (live blocks j < J)
  int32_t pps[kMaxSlots];     // pages per split
  int32_t aux[kMaxSlots];     // decode: pos; fp32 encoder: sink page or -1
  // SMem+RoPE composite (NULL rope: no rotary phases)
  const float* rope;          // rotary table, rows of dh floats
  const int32_t* live_blk;    // [n_seq][max_blocks] dense live list -> block index
  int32_t rope_clip;          // W: a block-j key read from block J is turned by min(J - j, W)
  int32_t qblk[kMaxSlots];    // query block J of the slot
  int32_t intra_partial;      // 1: the in-block / null split always writes a compact partial
                              //    ws[(qs*H + h)*(dh+4)] (row-plane decode merges it)
  // MFMA prefill, one workgroup per (slot, head) reading every split in turn
  // and folding them as the merge would (no partials, no merge launch);
  // workgroup z takes slot order[z] (slots with the most pages first).
  // fuse = 2: the 16-wave variant that reads up to four splits at once.
  int32_t fuse;
  int16_t order[kMaxSlots];
  int32_t ws_stride;          // split records per (query row, head) in ws (>= the launch's most splits)
};

// Row-plane decode (bf16): rows of width d, absorbed queries, split partials.
// Heads are read in tiles of 16 (one MFMA row tile): ht = ceil(H / 16) tiles,
// head h in tile h / 16, padded heads zero.
struct RowsArgs {
  const uint16_t* pages;      // row pages [n_pages][b][d]
  const int32_t* live_page;   // [n_seq][max_blocks]
  const uint16_t* qabs;       // absorbed queries [slot][ht*16][d]
  float* part;                // split partials per (slot, split, tile): U[16][d], m[16], l[16]
  const float* intra;         // in-block / null partials [slot][H][dh+4]
  const uint16_t* w_v;        // value map [H*dh][d]
  uint16_t* ubuf;             // combined weighted rows [slot][ht*16][d] (bf16)
  float* sw;                  // in-block weight / L per [slot][ht*16]
  uint16_t* out;              // [slot][H][dh]
  // in-block keys and the mapped null row (the split after the row splits)
  const uint16_t* q;          // [slot][H][dh]
  const uint16_t* k_new;      // [slot][H][dh] or NULL (no in-block keys)
  const uint16_t* v_new;
  uint16_t* k_cache;          // [slot*b + r][H][dh], row pos written
  uint16_t* v_cache;
  const uint16_t* null_kv;    // [2][H][dh] or NULL
  float* intra_w;             // in-block / null partials written here ([slot][H][dh+4])
  float scale_log2;
  int32_t max_blocks;
  int32_t b;
  int32_t H;
  int32_t ht;                 // head tiles
  int32_t max_split;          // row splits of the launch's longest read
  int32_t n_slots;
  int32_t seq[kMaxSlots];
  int32_t n_read[kMaxSlots];
  int32_t pps[kMaxSlots];
  int32_t pbase[kMaxSlots];   // first partial of the slot; split k, tile t at pbase + k*ht + t
  int32_t pos[kMaxSlots];     // in-block position of the new token
};
constexpr int kRowsMaxHeads = 64;

struct RowsPrepArgs {
  const uint16_t* q;          // [slot][H][dh]
  const uint16_t* w_k;        // key map [H*dh][d]
  const uint16_t* w_v;
  const uint16_t* null_row;   // [d] or NULL
  uint16_t* qabs;             // [slot][ht*16][d]
  uint16_t* null_kv;          // [2][H][dh]
  int32_t d;
  int32_t H;
  int32_t ht;
  int32_t n_slots;
  float scale_log2;
};

struct MetaArgs {
  int32_t* table;
  int32_t* live_page;
  int32_t* live_blk;
  int32_t* n_live;
  int32_t max_blocks;
  int32_t n_edits;
  int32_t n_items;                // work items (one workgroup each)
  int32_t e_seq[kMaxEdits];
  int32_t e_blk[kMaxEdits];
  int32_t e_page[kMaxEdits];      // -1: delete
  int32_t i_seq[kMaxMetaItems];   // item: sequence
  int32_t i_chunk[kMaxMetaItems]; //       table entries i_chunk*kMetaChunk ..
  int32_t i_base[kMaxMetaItems];  //       list position of the chunk's first live block
  int8_t i_last[kMaxMetaItems];   //       1: the last chunk that can hold a live block (writes n_live)
};

// ---------------------------------------------------------------- launchers

hipError_t launch_init_meta(int32_t* table, int32_t* n_live, size_t n_table, int n_seq, hipStream_t s);
hipError_t launch_meta(const MetaArgs& a, hipStream_t s);
hipError_t launch_put_rows(int dtype, void* pages, int page, int H, int b, int dh,
                           const void* k_rows, const void* v_rows, hipStream_t s);
// Row insert of n <= kMaxSlots blocks: block i's rows (k_rows/v_rows + i*b*H*dh) into page a.page[i].
struct PutArgs {
  void* pages;
  const void* k_rows;
  const void* v_rows;
  int32_t H, b, dh;
  int32_t page[kMaxSlots];
};
hipError_t launch_put_blocks(int dtype, const PutArgs& a, int n, hipStream_t s);
hipError_t launch_scrub(void* page_base, size_t bytes, hipStream_t s);
hipError_t launch_export(int dtype, const void* pages, const int32_t* live_page_seq, int n_live,
                         int H, int b, int dh, void* k_out, void* v_out, hipStream_t s);

// VALU reader: every split of every (slot, query, head), then the merge.
hipError_t launch_reader_valu(int dtype, int b, int dh, const ReaderArgs& a, hipStream_t s);
// Merge the split partials of every (query row, head) in split order.
hipError_t launch_merge(int dtype, int dh, const ReaderArgs& a, hipStream_t s);
// MFMA (bf16, b = 64) encoder and prefill.
// rope: rotary table (in-block phases), or NULL.
hipError_t launch_encoder_mfma(int b, int dh, const void* q, const void* k, const void* v, void* out,
                               void* pages, const int32_t* sink_pages, int n_blocks, int H, int mask,
                               float scale_log2, const float* rope, hipStream_t s);
hipError_t launch_prefill_mfma(int b, int dh, const ReaderArgs& a, hipStream_t s);
// Row-plane decode: stage 0 = absorbed queries (+ null row projection),
// stage 1 = row reader + merge.
hipError_t launch_rows(int d, int dh, const RowsArgs& a, const RowsPrepArgs& pa, int stage, hipStream_t s);
// Plain device copy (16-byte multiples), and the same through LDS by DMA
// (16 KiB multiples).
hipError_t launch_copy16(void* dst, const void* src, size_t bytes, hipStream_t s);
hipError_t launch_copy_dma(void* dst, const void* src, size_t bytes, hipStream_t s);
// Reader decode (smem_reader_decode and its variants).  ws_ext == NULL: split
// partials in the store's workspace; otherwise in ws_ext, which holds
// ws_ext_floats floats (the call is rejected if its partials do not fit).
smem_status decode_impl(smem_store* st, const smem_rope* rope, int32_t n_seq, const int32_t* seq_ids,
                        const int32_t* query_block, const int32_t* pos, const void* q, const void* k_new,
                        const void* v_new, void* k_cache, void* v_cache, const void* null_kv, void* out,
                        float* ws_ext, size_t ws_ext_floats, hipStream_t s);
// Record a failure for smem_last_error() (defined with the C ABI); returns st.
smem_status set_error(smem_status st, const char* msg);
// Rotary table of n_phases rows for heads of width dh, computed in fp64.
hipError_t launch_rope_table(float* table, int dh, int n_phases, double base, hipStream_t s);

}  // namespace smem
