// MFMA (bf16, fp32 accumulation) encoder and reader-prefill attention for
// blocks of b = 64 tokens.
//
// Encoder (Section 2, "Model"; Appendix A, "Encoder"): one workgroup per
// (block, head); the whole 64 x 64 score tile fits, so the softmax is exact
// in one pass.  Reader prefill (Section 3.1, block-skip serving): one
// workgroup per (query block, head, split); it streams whole memory pages of
// its split with an online softmax, and the split after the memory holds the
// null row and the in-block causal tile.  Splits merge in split order -- by
// the merge launch, or, in a launch of many query blocks or short reads, by
// one workgroup per (query block, head) that reads all its splits and folds
// them with the merge's own arithmetic.
//
// Both compute S^T = K Q^T and O^T = V^T P^T with
// __builtin_amdgcn_mfma_f32_16x16x32_bf16 (A: 16 rows x 32 k, B: 32 k x 16
// columns, D: 16 x 16).  Lane l of a wave supplies A row l%16 and B column
// l%16; its 8 k-values per operand are k-slots (l/16, 0..7), and A and B pair
// the same slot (checked on gfx950).  D element (4*(l/16)+i, l%16) lands in
// lane l, value i.  With keys as the rows of S^T, every lane owns one query
// column: the softmax statistics and the output rescale are per-lane
// scalars, and P^T reaches the second product straight from the score
// accumulators -- key tile 2c gives k-slots j<4 and tile 2c+1 gives j>=4, and
// the A operand (transposed values) reads the same keys in the same slots.
// The store keeps value planes transposed ([dh][b], keys contiguous) so that
// operand is two contiguous 8-byte reads per lane.
//
// SMem+RoPE composite (ROPE = true; Section 3, "SMem composes with RoPE"):
// queries and keys take rotary phases, values never do.  Inside a block the
// phase is the in-block offset (query row turned when its fragments are
// loaded, key rows when the tile passes through registers).  A memory page of
// block j read from block J turns the query by min(J - j, W) against the
// stored keys (the same turn for all b rows, so the fragments are re-turned
// only when it changes); the null row is a key of index 0.
#include "common.h"
#include "attn_ring.h"

namespace smem {

// ------------------------------------------------------------------ encoder

struct EncArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* out;        // may be NULL
  uint16_t* pages;      // may be NULL
  int32_t H;
  int32_t n_blocks;
  int32_t causal;
  float scale_log2;
  const float* rope;         // rotary table (in-block phases) or NULL
  int32_t sink[kMaxSlots];   // page of block i, or -1
};

// One workgroup per (block, head) tile, heads fastest: neighbouring
// workgroups read neighbouring head slices of the same token rows.  Every
// tile's loads are issued at once; with all tiles resident, tiles whose data
// arrive first compute while the rest are still loading.  The tile sits in
// LDS in the page layout, so the operand reads are the prefill's.
template <int DH, bool CAUSAL, bool ROPE>
__global__ void __launch_bounds__(256) k_encoder_mfma(EncArgs a) {
  using R = PageRing<DH>;
  __shared__ __attribute__((aligned(1024))) uint8_t T[R::TILE];
  const int h = blockIdx.x, blk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t rs = (size_t)a.H * DH;
  const size_t base = (size_t)blk * BT * rs + (size_t)h * DH;
  const int qrow = wave * 16 + (lane & 15);
  bf16x8 qf[DH / 32];
  load_q<DH>(qf, a.q + base + (size_t)wave * 16 * rs, rs, lane);
  if constexpr (ROPE) rope_q<DH>(qf, qf, a.rope + (size_t)qrow * DH, lane);
  intra_ring_store<DH, 256>(T, a.k + base, a.v + base, rs, tid, ROPE ? a.rope : nullptr);
  __syncthreads();
  floatx4 s4[4];
  scores_ring<DH>(s4, T, qf, lane);
  floatx4 o[DH / 16];
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  online_step<DH, CAUSAL>(s4, m, l, o, lane, qrow, a.scale_log2);
  pv_ring<DH>(o, T, s4, lane);
  l = qsum(l);
  const float inv = 1.f / l;
  const int pg = a.sink[blk];
  uint16_t* kp = (a.pages && pg >= 0) ? a.pages + page_head_offset(pg, h, a.H, BT, DH) : nullptr;
  // The block's output rows go through LDS (the key plane's space and
  // layout) so that global stores are whole 16-byte chunks of consecutive
  // rows: a lane's fragment is 4 dims of one query row, 8 bytes scattered
  // over 64 rows.  An 8-byte write serves 16 consecutive lanes (16 rows, one
  // dim group) per pass over 128 bytes of banks, and the key swizzle maps two
  // of those rows to the same 16-byte slot modulo 128 bytes (rows q and q ^ 1
  // at d_h = 64, rows whose slots differ in byte-address bit 7 at d_h = 128,
  // q and q + 8 at d_h = 32); a slot whose address bit SWB (7, or 9 at d_h =
  // 32) is set therefore stores its two 8-byte halves swapped (swapped back
  // when read), which gives the 16 lanes 16 distinct 8-byte places.  A page insert writes the key plane from the
  // same rows and the transposed value plane by gathering each chunk's 8 rows
  // (the lanes of one instruction read one row).
  __syncthreads();                           // every wave is done with the key and value tiles
  constexpr int SWB = DH == 32 ? 9 : 7;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    const int d0 = dt * 16 + (lane >> 4) * 4;
    uint16_t rr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) rr[i] = f32_to_bf16_bits(o[dt][i] * inv);
    const int slot = qrow * R::KRB + (((d0 >> 3) ^ R::kswz(qrow)) << 4);
    const int half = ((d0 >> 2) & 1) ^ ((slot >> SWB) & 1);  // halves swapped where bit SWB is set
    *(u32x2*)(T + slot + half * 8) =
        u32x2{(uint32_t)rr[0] | ((uint32_t)rr[1] << 16), (uint32_t)rr[2] | ((uint32_t)rr[3] << 16)};
  }
  __syncthreads();
  for (int c = tid; c < BT * DH / 8; c += 256) {
    const int row = c / (DH / 8), c8 = c % (DH / 8);
    const int slot = row * R::KRB + ((c8 ^ R::kswz(row)) << 4);
    u32x4 v16 = *(const u32x4*)(T + slot);
    if ((slot >> SWB) & 1) v16 = u32x4{v16.z, v16.w, v16.x, v16.y};
    if (a.out) *(u32x4*)(a.out + ((size_t)blk * BT + row) * rs + (size_t)h * DH + c8 * 8) = v16;
    if (kp) *(u32x4*)(kp + row * DH + c8 * 8) = v16;
  }
  if (kp) {
    for (int c = tid; c < DH * BT / 8; c += 256) {
      const int d = c % DH, r8 = c / DH;
      auto at = [&](int r) {
        const int slot = r * R::KRB + (((d >> 3) ^ R::kswz(r)) << 4);
        return (uint32_t) * (const uint16_t*)(T + slot + (((d & 7) * 2) ^ (((slot >> SWB) & 1) * 8)));
      };
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = at(r8 * 8 + 2 * j) | (at(r8 * 8 + 2 * j + 1) << 16);
      *(u32x4*)(kp + BT * DH + d * BT + r8 * 8) = u32x4{w[0], w[1], w[2], w[3]};
    }
  }
}

template <int DH>
static hipError_t launch_enc(const EncArgs& a, int n_blocks, hipStream_t s) {
  const dim3 grid(a.H, n_blocks);
  if (a.rope) {
    if (a.causal) hipLaunchKernelGGL((k_encoder_mfma<DH, true, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_encoder_mfma<DH, false, true>), grid, dim3(256), 0, s, a);
  } else {
    if (a.causal) hipLaunchKernelGGL((k_encoder_mfma<DH, true, false>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_encoder_mfma<DH, false, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_encoder_mfma(int b, int dh, const void* q, const void* k, const void* v, void* out, void* pages,
                               const int32_t* sink_pages, int n_blocks, int H, int mask, float scale_log2,
                               const float* rope, hipStream_t s) {
  if (b != BT || n_blocks > kMaxSlots) return hipErrorInvalidValue;
  if (n_blocks <= 0) return hipSuccess;
  EncArgs a;
  a.q = (const uint16_t*)q;
  a.k = (const uint16_t*)k;
  a.v = (const uint16_t*)v;
  a.out = (uint16_t*)out;
  a.pages = (uint16_t*)pages;
  a.H = H;
  a.n_blocks = n_blocks;
  a.causal = mask;
  a.scale_log2 = scale_log2;
  a.rope = rope;
  for (int i = 0; i < kMaxSlots; ++i) a.sink[i] = i < n_blocks ? sink_pages[i] : -1;
  if (dh == 32) return launch_enc<32>(a, n_blocks, s);
  if (dh == 64) return launch_enc<64>(a, n_blocks, s);
  if (dh == 128) return launch_enc<128>(a, n_blocks, s);
  return hipErrorInvalidValue;
}

// ------------------------------------------------------------------ reader prefill

// Rotary rows a memory split keeps in LDS: the turns of one split form a
// contiguous range (turn = min(J - j, W) falls as j rises); a split whose range
// fits reads its cos/sin from LDS, so re-turning the query inside the page loop
// never waits on a global load issued behind the in-flight pages.
constexpr int kRopeRows = 24;

// The final split's in-block tile uses the ring's first stage (split
// workgroups leave the ring unused; the folding one has drained it).
template <int DH, bool ROPE>
struct PrefillLds {
  __attribute__((aligned(1024))) uint8_t ring[PageRing<DH>::NS * PageRing<DH>::TILE];
};
template <int DH>
struct PrefillLds<DH, true> {
  __attribute__((aligned(1024))) uint8_t ring[PageRing<DH>::NS * PageRing<DH>::TILE];
  float rows[kRopeRows * DH];                          // turns d_lo .. d_lo + kRopeRows - 1
};

template <int N>
__device__ __forceinline__ void wait_pages(int ahead) {
  if (ahead >= 3) wait_vm<3 * N < 63 ? 3 * N : 63>();
  else if (ahead == 2) wait_vm<2 * N>();
  else if (ahead == 1) wait_vm<N>();
  else wait_vm<0>();
}

// The null row, one always-visible key/value pair per head, as the first key
// of the final split (m, l, o start empty).
// nkh, nvh: the head's null key and value vectors (global memory or LDS).
template <int DH, bool ROPE>
__device__ __forceinline__ void null_row_at(const uint16_t* nkh, const uint16_t* nvh, const ReaderArgs& a, int slot,
                                            const bf16x8 (&qf)[DH / 32], int lane, float& m, float& l,
                                            floatx4 (&o)[DH / 16]) {
  const uint16_t* nk = nkh + (lane >> 4) * 8;
  const uint16_t* nv = nvh;
  bf16x8 qn[DH / 32];
  if constexpr (ROPE) {
    rope_q<DH>(qn, qf, a.rope + (size_t)min(a.qblk[slot], a.rope_clip) * DH, lane);
  } else {
#pragma unroll
    for (int kk = 0; kk < DH / 32; ++kk) qn[kk] = qf[kk];
  }
  float x = 0.f;
#pragma unroll
  for (int kk = 0; kk < DH / 32; ++kk) {
    const u32x4 kr = *(const u32x4*)(nk + kk * 32);
    float kf[8];
    Chunk<uint16_t>::unpack(kr, kf);
#pragma unroll
    for (int j = 0; j < 8; ++j) x += (float)qn[kk][j] * kf[j];
  }
  x = qsum(x) * a.scale_log2;
  m = x;
  l = ((lane >> 4) == 0) ? 1.f : 0.f;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) o[dt][i] = bf16_bits_to_f32(nv[dt * 16 + (lane >> 4) * 4 + i]);
  }
}

template <int DH, bool ROPE>
__device__ __forceinline__ void null_row(const ReaderArgs& a, int slot, int h, const bf16x8 (&qf)[DH / 32], int lane,
                                         float& m, float& l, floatx4 (&o)[DH / 16]) {
  null_row_at<DH, ROPE>((const uint16_t*)a.null_kv + (size_t)h * DH, (const uint16_t*)a.null_kv + ((size_t)a.H + h) * DH,
                        a, slot, qf, lane, m, l, o);
}

// Fold one split's (m, l, o) into the running state (fm, fl, acc) -- the
// merge's arithmetic -- and start the next split empty.  l is this lane's
// share; the split's weight sum is its sum over the four lanes of the query.
template <int DH>
__device__ __forceinline__ void fold_split(bool first, float& m, float& l, floatx4 (&o)[DH / 16], float& fm,
                                           float& fl, floatx4 (&acc)[DH / 16]) {
  const float ls = qsum(l);
  if (first) {
    fm = m;
    fl = ls;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) acc[dt] = o[dt];
  } else {
    const FoldScale c = fold_scale(fm, m);
    fl = fold_value(fl, c, ls);
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[dt][i] = fold_value(acc[dt][i], c, o[dt][i]);
  }
  m = -INFINITY;
  l = 0.f;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
}

// Output rows of one wave: o * (1 / l) as bf16, l the weight sum (0 -> 0).
template <int DH>
__device__ __forceinline__ void store_out(uint16_t* orow, const floatx4 (&o)[DH / 16], float l, int lane) {
  const float inv = (l > 0.f) ? 1.f / l : 0.f;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    const int d0 = dt * 16 + (lane >> 4) * 4;
    uint16_t r4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) r4[i] = f32_to_bf16_bits(o[dt][i] * inv);
    *(u32x2*)(orow + d0) = u32x2{(uint32_t)r4[0] | ((uint32_t)r4[1] << 16), (uint32_t)r4[2] | ((uint32_t)r4[3] << 16)};
  }
}

// One (query block, head) over its splits.  FUSE = false: workgroup
// (h, split, slot) reads one split and writes its partial (m, l, o) -- or,
// with no memory split, the output.  FUSE = true: workgroup (h, 0, z) reads
// every split of slot order[z] in split order, the memory pages through one
// DMA ring, and folds each split's (m, l, o) into a running state as the
// merge does (fold_scale / fold_value), so both modes produce the same bits.
template <int DH, bool ROPE, bool FUSE>
__device__ __forceinline__ void prefill_body(const ReaderArgs& a, PrefillLds<DH, ROPE>& L) {
  static_assert(!(FUSE && ROPE), "the one-workgroup mode has no rotary variant");
  // heads fastest: neighbouring workgroups stream the adjacent head tiles of
  // the same pages
  const int h = blockIdx.x;
  const int split = FUSE ? 0 : (int)blockIdx.y;
  const int slot = FUSE ? (int)a.order[blockIdx.z] : (int)blockIdx.z;
  const int n_read = a.n_read[slot], pps = a.pps[slot];
  const int nms = (n_read + pps - 1) / pps;
  if (split > nms) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t rs = (size_t)a.H * DH;
  const int qrow = wave * 16 + (lane & 15);

  bf16x8 qf[DH / 32];
  load_q<DH>(qf, (const uint16_t*)a.q + ((size_t)slot * BT + wave * 16) * rs + (size_t)h * DH, rs, lane);
  floatx4 o[DH / 16];
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  // FUSE: the folded state of the splits read so far
  [[maybe_unused]] floatx4 acc[DH / 16];
  [[maybe_unused]] float fm = 0.f, fl = 0.f;

  if (split < nms) {
    using R = PageRing<DH>;
    const int p0 = split * pps, p1 = FUSE ? n_read : min(n_read, p0 + pps);
    const __attribute__((address_space(4))) int32_t* lpc =
        (const __attribute__((address_space(4))) int32_t*)(a.live_page + (size_t)a.seq[slot] * a.max_blocks);
    // this lane's 16 bytes of each DMA instruction: LDS byte (wave*IPW + i)*1024 + 16*lane of
    // the stage, read from the tile byte that the slot permutation puts there
    uint32_t src[R::IPW];
#pragma unroll
    for (int i = 0; i < R::IPW; ++i) {
      const int byte = (wave * R::IPW + i) * 1024 + lane * 16;
      if (byte < R::KBYTES) {
        const int r = byte / R::KRB, sl = (byte % R::KRB) >> 4;
        src[i] = r * R::KRB + ((sl ^ R::kswz(r)) << 4);
      } else {
        const int vb = byte - R::KBYTES, d = vb >> 7, sl = (vb & 127) >> 4;
        src[i] = R::KBYTES + d * 128 + ((sl ^ R::vswz(d)) << 4);
      }
    }
    const uint8_t* gpages = (const uint8_t*)a.pages;
    const uint32_t lds0 = (uint32_t)(uintptr_t)L.ring;
    auto issue = [&](int pi, int stage) {
      const uint8_t* t = gpages + page_head_offset(lpc[pi], h, a.H, BT, DH) * 2;
      const uint32_t d0 = lds0 + (uint32_t)(stage * R::TILE + wave * R::IPW * 1024);
#pragma unroll
      for (int i = 0; i < R::IPW; ++i) dma16(t + src[i], __builtin_amdgcn_readfirstlane(d0 + i * 1024));
    };
    // Rotary phases: a page of block j turns the query by min(J - j, W); the
    // turns of one split form a contiguous range, whose table rows are copied
    // to LDS when few enough (they are then read behind the DMA ring without
    // a load-counter wait); the unturned query fragments stay in registers.
    [[maybe_unused]] const __attribute__((address_space(4))) int32_t* lbc =
        (const __attribute__((address_space(4))) int32_t*)(a.live_blk + (size_t)a.seq[slot] * a.max_blocks);
    [[maybe_unused]] int turned = -1, d_lo = 0;
    [[maybe_unused]] bool rows_lds = false;
    [[maybe_unused]] bf16x8 qu[DH / 32];
    if constexpr (ROPE) {
      const int J = a.qblk[slot];
      const int d_hi = min(J - lbc[p0], a.rope_clip);
      d_lo = min(J - lbc[p1 - 1], a.rope_clip);
      rows_lds = d_hi - d_lo < kRopeRows;
      if (rows_lds) {
        const int n4 = (d_hi - d_lo + 1) * DH / 4;
        const f32x4* rsrc = (const f32x4*)(a.rope + (size_t)d_lo * DH);
        for (int i = tid; i < n4; i += 256) ((f32x4*)L.rows)[i] = rsrc[i];
      }
#pragma unroll
      for (int kk = 0; kk < DH / 32; ++kk) qu[kk] = qf[kk];
    }
    wait_vm<0>();                          // query fragments and rotary rows, before any DMA is in flight
#pragma unroll
    for (int k = 0; k < R::NS - 1; ++k)
      if (p0 + k < p1) issue(p0 + k, k);
    [[maybe_unused]] int split_end = p0 + pps;
    for (int pi = p0; pi < p1; ++pi) {
      const int k = pi - p0;
      wait_pages<R::IPW>(min(R::NS - 2, p1 - 1 - pi));
      lds_barrier();                       // page pi is in LDS; every wave is done with page pi - 1
      if (pi + R::NS - 1 < p1) issue(pi + R::NS - 1, (k + R::NS - 1) % R::NS);
      if constexpr (ROPE) {
        const int dlt = min(a.qblk[slot] - lbc[pi], a.rope_clip);
        if (dlt != turned) {
          rope_q<DH>(qf, qu, rows_lds ? L.rows + (dlt - d_lo) * DH : a.rope + (size_t)dlt * DH, lane);
          turned = dlt;
        }
      }
      const uint8_t* tile = L.ring + (k % R::NS) * R::TILE;
      floatx4 s[4];
      scores_ring<DH>(s, tile, qf, lane);
      online_step<DH, false>(s, m, l, o, lane, qrow, a.scale_log2);
      pv_ring<DH>(o, tile, s, lane);
      if constexpr (FUSE) {
        if (pi + 1 == split_end || pi + 1 == p1) {
          fold_split<DH>(split_end == pps, m, l, o, fm, fl, acc);
          split_end += pps;
        }
      }
    }
    if constexpr (FUSE) __syncthreads();   // every wave is done with the ring before the tiles reuse it
  }
  if (FUSE || split == nms) {
    if (a.null_kv != nullptr) null_row<DH, ROPE>(a, slot, h, qf, lane, m, l, o);
    if (a.k_in != nullptr) {
      const size_t base = (size_t)slot * BT * rs + (size_t)h * DH;
      if constexpr (ROPE) rope_q<DH>(qf, qf, a.rope + (size_t)qrow * DH, lane);
      intra_ring_store<DH, 256>(L.ring, (const uint16_t*)a.k_in + base, (const uint16_t*)a.v_in + base, rs, tid,
                                ROPE ? a.rope : nullptr);
      __syncthreads();
      floatx4 s[4];
      scores_ring<DH>(s, L.ring, qf, lane);
      online_step<DH, true>(s, m, l, o, lane, qrow, a.scale_log2);
      pv_ring<DH>(o, L.ring, s, lane);
    }
  }
  const size_t qs = (size_t)slot * BT + qrow;
  if (FUSE && nms > 0) {
    fold_split<DH>(false, m, l, o, fm, fl, acc);
    store_out<DH>((uint16_t*)a.out + qs * rs + (size_t)h * DH, acc, fl, lane);
    return;
  }
  l = qsum(l);
  if (nms == 0) {
    store_out<DH>((uint16_t*)a.out + qs * rs + (size_t)h * DH, o, l, lane);
  } else {
    float* part = a.ws + ((qs * a.H + h) * a.ws_stride + split) * (DH + 4);
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) {
      const int d0 = dt * 16 + (lane >> 4) * 4;
      *(f32x4*)(part + d0) = o[dt];
    }
    if ((lane >> 4) == 0) {
      part[DH] = m;
      part[DH + 1] = l;
    }
  }
}

// ------------------------------------------------------------------ few-pair prefill

// Launches with few (query block, head) pairs and at most four memory splits
// each.  A pair's 64 query rows go to 4/QW workgroups of 4 x QW waves (QW = 2,
// the one launched: two workgroups of 32 rows, launched 8 indices apart so
// both run on one XCD and the second fetch of each page hits its L2).
// Wave group g (QW waves of 16 rows each) reads memory split g through a DMA
// ring of its own, so four page streams and four MFMA -> softmax -> MFMA
// chains run on the CU at once; the groups step through their pages
// together, one workgroup barrier per page.  The in-block tile (in the ring's
// layout) and the null row are staged in LDS at the start; the final split
// (null row, then the in-block keys) is read by a group that has no page at
// that step.  At the end every group puts its split's state (m, l, o) into
// the ring's LDS, and the waves fold them in split order, the final split
// last, with the merge's functions, each wave one 16-wide dimension tile of
// its rows: every split is computed as in the split launch and the folding
// launch, so all three give the same bits.
template <int DH, int QW>
struct ParLds {
  using R = PageRing<DH>;
  static constexpr int G = 4;                          // split groups
  static constexpr int NSP = DH == 32 ? 4 : 2;         // ring stages per group
  static constexpr int IPW = R::TILE / 1024 / QW;      // DMA instructions per wave per page
  static constexpr int THREADS = 64 * G * QW;
  static constexpr int ROWS = 16 * QW;                 // query rows per workgroup
  static constexpr int RING = G * NSP * R::TILE;
  static constexpr int OFF_IN = RING;                  // in-block tile, ring layout
  static constexpr int OFF_NULL = OFF_IN + R::TILE;    // null key, then null value (bf16)
  static constexpr int BYTES = OFF_NULL + 4 * DH;
  // a split state per (slot, wave): o as DH/16 float4 planes of 64 lanes, then (m, l) pairs;
  // slots 0..3 hold memory splits 0..3, slot 4 the final split
  static constexpr int STATE = (DH / 16) * 1024 + 64 * 8;
  static_assert((G + 1) * QW * STATE <= RING, "split states fit in the ring");
  static_assert(BYTES <= 160 * 1024, "LDS");
  static_assert(NSP >= 2 && NSP <= 4 && 3 * IPW < 64, "wait_pages covers up to 3 pages ahead");
};

template <int DH>
__device__ __forceinline__ void state_put(uint8_t* st, const floatx4 (&o)[DH / 16], float m, float l, int lane) {
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) *(floatx4*)(st + (dt * 64 + lane) * 16) = o[dt];
  *(f32x2*)(st + (DH / 16) * 1024 + lane * 8) = f32x2{m, l};
}

// Workgroups of a few-pair launch: 4/QW parts per pair, 8 pairs per round of
// 8 x (4/QW) launch indices.
inline int par_grid(int n_pairs, int qw) { return ((n_pairs + 7) / 8) * 8 * (4 / qw); }

template <int DH, int QW>
__global__ void __launch_bounds__(64 * 4 * QW) k_prefill_mfma_par(ReaderArgs a) {
  using P = ParLds<DH, QW>;
  using R = PageRing<DH>;
  constexpr int NPART = 4 / QW;
  __shared__ __attribute__((aligned(1024))) uint8_t L[P::BYTES];
  const int n = blockIdx.x;
  const int pair = (n / (8 * NPART)) * 8 + (n % 8), part = (n / 8) % NPART;
  if (pair >= a.n_slots * a.H) return;   // padding of the last round (whole workgroup)
  const int slot = pair / a.H, h = pair % a.H;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = wave / QW, qw = wave % QW;
  const int n_read = a.n_read[slot], pps = a.pps[slot];
  const int nms = (n_read + pps - 1) / pps;
  const size_t rs = (size_t)a.H * DH;
  const int row0 = part * P::ROWS + qw * 16;             // this wave's first query row
  const int qrow = row0 + (lane & 15);
  const int p0 = g * pps, p1 = min(n_read, p0 + pps);    // this group's split (empty when g >= nms)
  // the final split is read by group fg at step fstep, when fg has no page
  const int fg = nms < P::G ? nms : P::G - 1;
  const int fstep = nms < P::G ? 0 : n_read - (P::G - 1) * pps;
  const int steps = max(nms > 0 ? pps : 0, fstep + 1);

  // ---- page DMA of this group's split: the whole ring at once
  const __attribute__((address_space(4))) int32_t* lpc =
      (const __attribute__((address_space(4))) int32_t*)(a.live_page + (size_t)a.seq[slot] * a.max_blocks);
  uint32_t src[P::IPW];
#pragma unroll
  for (int i = 0; i < P::IPW; ++i) {
    const int byte = (qw * P::IPW + i) * 1024 + lane * 16;
    if (byte < R::KBYTES) {
      const int r = byte / R::KRB, sl = (byte % R::KRB) >> 4;
      src[i] = r * R::KRB + ((sl ^ R::kswz(r)) << 4);
    } else {
      const int vb = byte - R::KBYTES, d = vb >> 7, sl = (vb & 127) >> 4;
      src[i] = R::KBYTES + d * 128 + ((sl ^ R::vswz(d)) << 4);
    }
  }
  const uint8_t* gpages = (const uint8_t*)a.pages;
  const uint32_t lds0 = (uint32_t)(uintptr_t)L + (uint32_t)(g * P::NSP * R::TILE + qw * P::IPW * 1024);
  auto issue_page = [&](int page, int stage) {
    const uint8_t* t = gpages + page_head_offset(page, h, a.H, BT, DH) * 2;
    const uint32_t d0 = lds0 + (uint32_t)(stage * R::TILE);
#pragma unroll
    for (int i = 0; i < P::IPW; ++i) dma16(t + src[i], __builtin_amdgcn_readfirstlane(d0 + i * 1024));
  };
  // A page number is the same for the whole wave: looked up with a
  // wave-uniform index it is a scalar load, which no vector-memory wait covers.
  auto page_of = [&](int pi) { return lpc[__builtin_amdgcn_readfirstlane(pi)]; };
  auto issue = [&](int pi, int stage) { issue_page(page_of(pi), stage); };
  if (p0 < p1) issue(p0, 0);              // the first page; the rest of the ring after the loads below

  // ---- query fragments; the in-block tile (ring layout) and the null row into LDS
  bf16x8 qf[DH / 32];
  load_q<DH>(qf, (const uint16_t*)a.q + ((size_t)slot * BT + row0) * rs + (size_t)h * DH, rs, lane);
  uint8_t* tin = L + P::OFF_IN;
  uint16_t* nul = (uint16_t*)(L + P::OFF_NULL);
  constexpr int CPR = DH / 8;                            // 16-byte chunks per row
  if (a.k_in != nullptr) {
    const size_t base = (size_t)slot * BT * rs + (size_t)h * DH;
    intra_ring_store<DH, P::THREADS>(tin, (const uint16_t*)a.k_in + base, (const uint16_t*)a.v_in + base, rs, tid);
  }
  if (a.null_kv != nullptr && tid < 2 * CPR) {
    const uint16_t* nsrc = (const uint16_t*)a.null_kv + (tid < CPR ? (size_t)h * DH + tid * 8
                                                                   : ((size_t)a.H + h) * DH + (tid - CPR) * 8);
    *(u32x4*)(nul + tid * 8) = *(const u32x4*)nsrc;
  }
  // The loads above are waited for here, with the first page (the compiler
  // waits for every vector-memory load before their first use, the page DMA
  // included); the rest of the ring is issued only now, so that wait does
  // not cover it.
  wait_vm<0>();
#pragma unroll 1
  for (int k = 1; k < P::NSP; ++k)
    if (p0 + k < p1) issue(p0 + k, k);

  // ---- memory pages (all groups step together) and the final split
  floatx4 o[DH / 16], of[DH / 16];
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    of[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  float m = -INFINITY, l = 0.f, mf = -INFINITY, lf = 0.f;
  for (int k = 0; k < steps; ++k) {
    const int pi = p0 + k;
    // the page this step refills the ring with: its number is looked up
    // before the waits below, so the lookup overlaps them
    const bool refill = k > 0 && pi + P::NSP - 1 < p1;
    const int next_page = refill ? page_of(pi + P::NSP - 1) : 0;
    wait_pages<P::IPW>(pi < p1 ? min(k == 0 ? P::NSP - 1 : P::NSP - 2, p1 - 1 - pi) : 0);
    lds_barrier();                       // page k of every group is in LDS; every wave is done with page k - 1
    if (refill) issue_page(next_page, (k + P::NSP - 1) % P::NSP);
    if (pi < p1) {
      const uint8_t* tile = L + (g * P::NSP + k % P::NSP) * R::TILE;
      floatx4 s[4];
      scores_ring<DH>(s, tile, qf, lane);
      online_step<DH, false>(s, m, l, o, lane, qrow, a.scale_log2);
      pv_ring<DH>(o, tile, s, lane);
    } else if (g == fg && k == fstep) {
      if (a.null_kv != nullptr) null_row_at<DH, false>(nul, nul + DH, a, slot, qf, lane, mf, lf, of);
      if (a.k_in != nullptr) {
        floatx4 s[4];
        scores_ring<DH>(s, tin, qf, lane);
        online_step<DH, true>(s, mf, lf, of, lane, qrow, a.scale_log2);
        pv_ring<DH>(of, tin, s, lane);
      }
    }
  }
  lds_barrier();                         // the ring is free
  // every split's state into LDS: slot j*QW + qw for memory split j, slot
  // G*QW + qw for the final split
  if (g < nms) state_put<DH>(L + (g * QW + qw) * P::STATE, o, m, l, lane);
  if (g == fg) state_put<DH>(L + (P::G * QW + qw) * P::STATE, of, mf, lf, lane);
  lds_barrier();
  // Wave (g, qw) folds dimension tile g of its 16 rows over the splits in
  // split order (per element the merge's arithmetic, so the split launch's
  // bits) and stores that tile: the fold runs on DH/16 waves at once.
  constexpr int NT = DH / 16;
  if (g < NT) {
    auto get = [&](int sl, floatx4& ot, float& ms, float& ls) {
      const uint8_t* st = L + (sl * QW + qw) * P::STATE;
      ot = *(const floatx4*)(st + (g * 64 + lane) * 16);
      const f32x2 ml = *(const f32x2*)(st + NT * 1024 + lane * 8);
      ms = ml.x;
      ls = qsum(ml.y);
    };
    floatx4 acc;
    float fm, fl;
    get(nms > 0 ? 0 : P::G, acc, fm, fl);
    for (int j = 1; j <= nms; ++j) {     // memory splits 1 .. nms-1, then the final split
      floatx4 ot;
      float ms, ls;
      get(j < nms ? j : P::G, ot, ms, ls);
      const FoldScale c = fold_scale(fm, ms);
      fl = fold_value(fl, c, ls);
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = fold_value(acc[i], c, ot[i]);
    }
    const float inv = (fl > 0.f) ? 1.f / fl : 0.f;
    uint16_t* orow = (uint16_t*)a.out + ((size_t)slot * BT + qrow) * rs + (size_t)h * DH;
    const int d0 = g * 16 + (lane >> 4) * 4;
    uint16_t r4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) r4[i] = f32_to_bf16_bits(acc[i] * inv);
    *(u32x2*)(orow + d0) = u32x2{(uint32_t)r4[0] | ((uint32_t)r4[1] << 16), (uint32_t)r4[2] | ((uint32_t)r4[3] << 16)};
  }
}

template <int DH>
__global__ void __launch_bounds__(256) k_prefill_mfma(ReaderArgs a) {
  __shared__ PrefillLds<DH, false> L;
  prefill_body<DH, false, false>(a, L);
}

template <int DH>
__global__ void __launch_bounds__(256) k_prefill_mfma_fused(ReaderArgs a) {
  __shared__ PrefillLds<DH, false> L;
  prefill_body<DH, false, true>(a, L);
}

// The rotary variant asks for at least two waves per SIMD: left free, the
// compiler spends registers on the query turn and falls to one wave at
// dh = 128 (it fits two without spilling).
template <int DH>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_prefill_mfma_rope(ReaderArgs a) {
  __shared__ PrefillLds<DH, true> L;
  prefill_body<DH, true, false>(a, L);
}

template <int DH>
static hipError_t launch_pre(const ReaderArgs& a, hipStream_t s) {
  int max_split = 0;
  for (int i = 0; i < a.n_slots; ++i) {
    const int ns = total_splits(a.n_read[i], a.pps[i]) - 1;
    if (ns > max_split) max_split = ns;
  }
  if (a.fuse == 2) {
    constexpr int D = DH > 64 ? 64 : DH;                 // (no few-pair variant at d_h 128)
    if (a.rope || DH > 64 || max_split > ParLds<D, 4>::G) return hipErrorInvalidValue;
    const int n_pairs = a.n_slots * a.H;
    hipLaunchKernelGGL((k_prefill_mfma_par<D, 2>), dim3(par_grid(n_pairs, 2)), dim3(512), 0, s, a);
    return hipGetLastError();
  }
  if (a.fuse) {
    if (a.rope) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_prefill_mfma_fused<DH>), dim3(a.H, 1, a.n_slots), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const dim3 grid(a.H, max_split + 1, a.n_slots);
  if (a.rope) hipLaunchKernelGGL((k_prefill_mfma_rope<DH>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((k_prefill_mfma<DH>), grid, dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || max_split == 0) return e;
  return launch_merge(BF16, DH, a, s);
}

hipError_t launch_prefill_mfma(int b, int dh, const ReaderArgs& a, hipStream_t s) {
  if (b != BT || a.nq != BT) return hipErrorInvalidValue;
  if (a.n_slots <= 0) return hipSuccess;
  if (dh == 32) return launch_pre<32>(a, s);
  if (dh == 64) return launch_pre<64>(a, s);
  if (dh == 128) return launch_pre<128>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace smem
