// Decode from the memory rows themselves (Appendix K, recomputing K/V from
// the memory rows; Appendix A, "Positions and memory": the rows are shared by
// all D reader layers, each layer projecting them with its own key and value
// maps).
//
// A row store page holds one block's b rows of width d.  Instead of forming
// K = mu W_K and V = mu W_V for every row read, the projections are folded
// into the query and the output (both exact identities):
//   score(q_h, row r) = <q_h, W_K^h^T mu_r> = <W_K^h q_h, mu_r>
//   sum_r a_r W_V^h^T mu_r = W_V^h^T (sum_r a_r mu_r)
// so the reader streams each row once for all heads: per 16-row chunk,
// S = Q' mu^T (heads x rows, MFMA over d) and U += P mu (heads x d, MFMA over
// the rows), with an online softmax per head.  The merge combines the splits'
// U in split order, applies W_V^h once per (query, head) and adds the
// in-block / null-row partial (dh-wide, from the VALU reader).
#include "common.h"

namespace smem {

typedef __bf16 bf16x8r __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kRowChunk = 16;     // rows per chunk (one MFMA column tile)

// Chunks stream global -> LDS by DMA (global_load_lds, 16 bytes per lane)
// through a ring of NS stages, so no register holds them in transit.
#ifndef SMEM_ROWS_STAGES
#define SMEM_ROWS_STAGES 2
#endif
template <int D>
struct RowsCfg {
  // LDS row pitch (elements): a 32-byte pad, so the pitch is 32 bytes past a
  // multiple of 256 (D = 512 .. 2048): the score reads (16 rows, 16 bytes
  // each) and the transposing value reads (16 rows, 4 lanes x 8 bytes each)
  // then touch every bank once (a 16-byte pad left both 2-way conflicted;
  // measured with a one-wave bank probe)
  static constexpr int MP = D + 16;
  // ring stages (LDS: NS * 16 rows * MP * 2 bytes; at most 2 at d = 2048)
  static constexpr int NS = D >= 2048 ? 2 : SMEM_ROWS_STAGES;
  static constexpr int RI = (D + 511) / 512;          // DMA instructions per row (the last partial at d = 768)
  static constexpr int KW = kRowChunk * RI / 4;        // DMA instructions per wave per chunk
  static constexpr int DW = D / 4;                 // dims per wave (score reduction, U ownership)
  static constexpr int NT = DW / 16;               // U tiles per wave
};

// TG head tiles per workgroup: wave group g (4 waves) takes tile g of the
// workgroup's TG; the row chunks in LDS serve every group.
template <int D, int TG>
struct RowsLds {
  alignas(16) uint16_t mu[RowsCfg<D>::NS][kRowChunk * RowsCfg<D>::MP];
  float sred[TG][4][256];                   // per-wave partial scores
  uint16_t p[TG][16 * 16];                  // P[head][row], bf16
  float alpha[TG][16];
  int rescale[TG];                          // some head's reference maximum moved this chunk
};

// Lazy rescaling: a head's reference maximum moves only when a score exceeds
// it by more than kLazy (log2 units), so P <= 2^kLazy and the accumulated U
// needs rescaling only in those chunks.  Every weight and U share the
// reference, so the result is the same up to rounding.
constexpr float kLazy = 8.f;

// Wave `wave` moves rows 4*wave .. 4*wave+3 of chunk c into stage st: each
// row is D*2 bytes, DMA instructions of 1 KiB (512 elements) and, at
// d = 768, one of 512 bytes (the lanes past the row's end stay idle).
template <int D, int TG>
__device__ __forceinline__ void chunk_dma(RowsLds<D, TG>& L, int st, const uint16_t* __restrict__ src, int wave,
                                          int lane) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = wave * 4 + r;
#pragma unroll
    for (int hk = 0; hk < RowsCfg<D>::RI; ++hk) {
      const uint16_t* g = src + (size_t)row * D + hk * 512 + lane * 8;
      const uint32_t l = (uint32_t)(uintptr_t)&L.mu[st][row * RowsCfg<D>::MP + hk * 512];
      if (hk * 512 + 512 <= D || hk * 512 + lane * 8 < D) dma16(g, __builtin_amdgcn_readfirstlane(l));
    }
  }
}

// Wait until this wave's DMA for the current chunk is done, with `ahead`
// later chunks (0 .. NS-1) allowed to stay in flight.
template <int D>
__device__ __forceinline__ void wait_chunk(int ahead) {
  constexpr int K = RowsCfg<D>::KW;
  if (ahead >= 3) wait_vm<(3 * K < 63 ? 3 * K : 63)>();
  else if (ahead == 2) wait_vm<2 * K>();
  else if (ahead == 1) wait_vm<K>();
  else wait_vm<0>();
}

// The splits after the row splits: the query's in-block keys 0..pos (the
// new key/value pair at pos, also written into the cache) and the mapped
// null row, under the query's own scale.  Workgroup g of them takes heads
// 4g .. 4g+3, one per wave: a lane scores one in-block row, then the lanes
// take the value dimensions (weights read back from LDS).  Writes the
// compact partial (acc[dh], max, sum) of each head.
template <int DHq>
__device__ __forceinline__ void rows_intra(const RowsArgs& a, int slot, int h, int lane, float* pw, float* red,
                                           float& M_out, float& L_out) {
  const int H = a.H, pos = a.pos[slot];
  const int n_in = a.k_new ? pos + 1 : 0;
  const size_t tok = (size_t)H * DHq;
  const uint16_t* qh = a.q + ((size_t)slot * H + h) * DHq;
  auto dot = [&](const uint16_t* kr) {   // the query is re-read per chunk (cached), not held
    float x = 0.f;
#pragma unroll 4
    for (int c8 = 0; c8 < DHq / 8; ++c8) {
      float kf[8], qf[8];
      Chunk<uint16_t>::unpack(*(const u32x4*)(kr + c8 * 8), kf);
      Chunk<uint16_t>::unpack(*(const u32x4*)(qh + c8 * 8), qf);
#pragma unroll
      for (int e = 0; e < 8; ++e) x += qf[e] * kf[e];
    }
    return x * a.scale_log2;
  };
  const uint16_t* knew = a.k_new ? a.k_new + ((size_t)slot * H + h) * DHq : nullptr;
  const uint16_t* vnew = a.v_new ? a.v_new + ((size_t)slot * H + h) * DHq : nullptr;
  float sc = -INFINITY;
  if (lane < n_in) sc = dot(lane == pos ? knew : a.k_cache + ((size_t)slot * a.b + lane) * tok + (size_t)h * DHq);
  const float sn = a.null_kv ? dot(a.null_kv + (size_t)h * DHq) : -INFINITY;
  float M = sc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) M = fmaxf(M, __shfl_xor(M, o));
  M = fmaxf(M, sn);
  const float p = (lane < n_in) ? exp2w(sc - M) : 0.f;
  const float pn = a.null_kv ? exp2w(sn - M) : 0.f;
  float Lsum = p;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) Lsum += __shfl_xor(Lsum, o);
  Lsum += pn;
  pw[lane] = p;                            // this wave's row of weights
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  float* part = a.intra_w + ((size_t)slot * H + h) * (DHq + 4);
  const uint16_t* vc = a.v_cache + (size_t)slot * a.b * tok + (size_t)h * DHq;
  // cached values (rows below pos): lane (g, c) sums rows g, g + RG, ... of
  // its 8-dim chunk c with 16-byte loads, all issued at once; the RG group
  // sums then meet in LDS and are added in group order
  constexpr int C = DHq / 8, RG = 64 / C;
  const int rg = lane / C, c8 = lane % C;
  const int nr = min(pos, n_in);
  float a8[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) a8[e] = 0.f;
#pragma unroll
  for (int i = 0; i < 64 / RG; ++i) {
    const int r = rg + RG * i;
    if (r < nr) {
      float vf[8];
      Chunk<uint16_t>::unpack(*(const u32x4*)(vc + (size_t)r * tok + c8 * 8), vf);
      const float w = pw[r];
#pragma unroll
      for (int e = 0; e < 8; ++e) a8[e] += w * vf[e];
    }
  }
  *(f32x4*)(red + rg * DHq + c8 * 8) = f32x4{a8[0], a8[1], a8[2], a8[3]};
  *(f32x4*)(red + rg * DHq + c8 * 8 + 4) = f32x4{a8[4], a8[5], a8[6], a8[7]};
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
  for (int dd = 0; dd < (DHq + 63) / 64; ++dd) {
    const int d = lane + dd * 64;
    if (d < DHq) {
      float acc = a.null_kv ? pn * bf16_bits_to_f32(a.null_kv[((size_t)H + h) * DHq + d]) : 0.f;
      if (n_in > 0) acc += pw[pos] * bf16_bits_to_f32(vnew[d]);
#pragma unroll
      for (int g = 0; g < RG; ++g) acc += red[g * DHq + d];
      part[d] = acc;
    }
  }
  M_out = M;
  L_out = Lsum;
  if (n_in > 0 && lane < DHq / 8) {         // the new pair into the cache at row pos
    const size_t off = ((size_t)slot * a.b + pos) * tok + (size_t)h * DHq + lane * 8;
    *(u32x4*)(a.k_cache + off) = *(const u32x4*)(knew + lane * 8);
    *(u32x4*)(a.v_cache + off) = *(const u32x4*)(vnew + lane * 8);
  }
}

// One workgroup per (sequence slot, split, group of TG head tiles), 4 waves
// per tile: the chunks of rows are moved into LDS once for the TG tiles.
// The tile groups of one (slot, split) read the same rows: their launch
// indices are 8 apart, so they run on one XCD (workgroups are dealt to the 8
// XCDs in turn) and share its L2.  Wave w of a group reduces dims
// [w*D/4, (w+1)*D/4) of its tile's scores and owns the same dims of U.
inline int rows_grid(int units, int groups) { return ((units + 7) / 8) * 8 * groups; }

template <int D, int DHq, int TG>
__global__ void __launch_bounds__(256 * TG) k_reader_rows(RowsArgs a) {
  using C = RowsCfg<D>;
  __shared__ RowsLds<D, TG> L;
  const int n_groups = a.ht / TG;
  const int n = blockIdx.x;
  const int unit = (n / (8 * n_groups)) * 8 + n % 8, tgi = (n / 8) % n_groups;
  const int slot = unit / a.max_split, split = unit % a.max_split;
  if (slot >= a.n_slots) return;            // padding of the last round (whole workgroup)
  const int n_read = a.n_read[slot], pps = a.pps[slot];
  const int nsp = (n_read + pps - 1) / pps;
  if (split >= nsp) return;
  const int tid_all = threadIdx.x, lane = tid_all & 63, wave_all = tid_all >> 6;
  const int grp = wave_all / 4, wave = wave_all % 4, tid = tid_all % 256;
  const int tile = tgi * TG + grp;
  constexpr int MP = C::MP, DW = C::DW, NT = C::NT, NS = C::NS;
  const int b = a.b;

  // absorbed-query fragments of this wave's dims stay in registers (A operand)
  u32x4 qa[DW / 32];
  {
    const uint16_t* qs = a.qabs + ((size_t)(slot * a.ht + tile) * 16 + (lane & 15)) * D + wave * DW + (lane >> 4) * 8;
#pragma unroll
    for (int kk = 0; kk < DW / 32; ++kk) qa[kk] = *(const u32x4*)(qs + kk * 32);
  }
  // softmax role of this thread: (head, row) of one score
  const int sl = tid >> 2, si = tid & 3;
  const int s_head = 4 * (sl >> 4) + si, s_row = sl & 15;
  float m_h = -INFINITY, l_h = 0.f;
  f32x4 u[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) u[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int p0 = split * pps, p1 = min(n_read, p0 + pps);
  const int cpp = b / kRowChunk;            // chunks per page
  const int n_chunks = (p1 - p0) * cpp;
  // The live list is read-only while a reader runs: reading it through the
  // constant address space keeps each lookup a scalar load (a vector load
  // would be waited for together with the chunk DMA in flight).
  const __attribute__((address_space(4))) int32_t* lpc =
      (const __attribute__((address_space(4))) int32_t*)(a.live_page + (size_t)a.seq[slot] * a.max_blocks);
  auto chunk_src = [&](int c) {
    const int pg = lpc[p0 + c / cpp];
    return a.pages + ((size_t)pg * b + (size_t)(c % cpp) * kRowChunk) * D;
  };
  wait_vm<0>();                             // the query fragments
  // the first group's waves move the chunks
#pragma unroll
  for (int c = 0; c < NS - 1; ++c)
    if (grp == 0 && c < n_chunks) chunk_dma<D, TG>(L, c, chunk_src(c), wave, lane);

  for (int c = 0; c < n_chunks; ++c) {
    const int st = c % NS;
    lds_barrier();                        // every wave is done with chunk c-1 (its stage, sred, p)
    const int nxt = c + NS - 1;
    if (grp == 0 && nxt < n_chunks) chunk_dma<D, TG>(L, nxt % NS, chunk_src(nxt), wave, lane);
    wait_chunk<D>(min(NS - 1, n_chunks - 1 - c));
    lds_barrier();                        // chunk c is in LDS for every wave
    // S partial over this wave's dims: D[m = head][n = row]
    const uint16_t* mu = L.mu[st];
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < DW / 32; kk += 2) {
      const int k0 = wave * DW + kk * 32 + (lane >> 4) * 8;
      const u32x4 m0 = *(const u32x4*)&mu[(lane & 15) * MP + k0];
      const u32x4 m1 = *(const u32x4*)&mu[(lane & 15) * MP + k0 + 32];
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8r, qa[kk]),
                                                   __builtin_bit_cast(bf16x8r, m0), s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8r, qa[kk + 1]),
                                                   __builtin_bit_cast(bf16x8r, m1), s1, 0, 0, 0);
    }
    *(f32x4*)&L.sred[grp][wave][lane * 4] = s0 + s1;
    if (tid == 0) L.rescale[grp] = 0;
    lds_barrier();
    // online softmax per head over the chunk's 16 rows, lazily rescaled
    {
      const float x = L.sred[grp][0][tid] + L.sred[grp][1][tid] + L.sred[grp][2][tid] + L.sred[grp][3][tid];
      float mx = x;
      mx = fmaxf(mx, __shfl_xor(mx, 4));
      mx = fmaxf(mx, __shfl_xor(mx, 8));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      float al = 1.f;
      if (mx > m_h + kLazy) {               // the same for the 16 threads of a head
        al = exp2w(m_h - mx);
        m_h = mx;
        if (s_row == 0) L.rescale[grp] = 1;
      }
      const float p = exp2w(x - m_h);
      float ps = p;
      ps += __shfl_xor(ps, 4);
      ps += __shfl_xor(ps, 8);
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      l_h = l_h * al + ps;
      L.p[grp][s_head * 16 + s_row] = f32_to_bf16_bits(p);
      if (s_row == 0) L.alpha[grp][s_head] = al;
    }
    lds_barrier();
    // U = U * alpha + P mu over this wave's dims
    {
      if (L.rescale[grp]) {
        float al4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) al4[i] = L.alpha[grp][4 * (lane >> 4) + i];
#pragma unroll
        for (int n = 0; n < NT; ++n) {
#pragma unroll
          for (int i = 0; i < 4; ++i) u[n][i] *= al4[i];
        }
      }
      const u32x2 pa = *(const u32x2*)&L.p[grp][(lane & 15) * 16 + (lane >> 4) * 4];
      const s16x4 A = __builtin_bit_cast(s16x4, pa);
      // B[k][n] = chunk row k, dim d0 + n for lane (n = l%16, k = 4(l/16) + i):
      // one transposing read per tile.  ds_read_b64_tr_b16 hands lane j of
      // each 16-lane group element i of the 8 bytes that lane 4i + j/4 of
      // the group addressed, element j%4; so lane l addresses row l/4,
      // dims d0 + 4(l%4) .. +3.
      const uint16_t* trow = mu + (lane >> 2) * MP + 4 * (lane & 3);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int d0 = wave * DW + n * 16;
        const s16x4 B = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(trow + d0));
        u[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(A, B, u[n], 0, 0, 0);
      }
    }
  }
  // partial: U[16][D], then m[16], l[16]
  float* part = a.part + (size_t)(a.pbase[slot] + split * a.ht + tile) * (16 * D + 32);
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const int dim = wave * DW + n * 16 + (lane & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) part[(size_t)(4 * (lane >> 4) + i) * D + dim] = u[n][i];
  }
  if (s_row == 0) {
    part[16 * D + s_head] = m_h;
    part[16 * D + 16 + s_head] = l_h;
  }
}

// Absorbed queries: qabs[slot][h][c] = scale_log2 * sum_j W_K[h*dh + j][c] q[slot][h][j]
// (bf16; zero rows for the padded heads H <= h < ht*16).  The maps are [H*dh][d] (a linear
// layer's out x in layout), so a thread per c reads them coalesced; a
// workgroup serves kAbsorbSlots query slots, the j loop unrolled so several
// map loads are in flight.
constexpr int kAbsorbSlots = 4;
template <int DHq>
__global__ void __launch_bounds__(256) k_rows_absorb_q(RowsPrepArgs a) {
  const int c = blockIdx.x * 256 + threadIdx.x, h = blockIdx.y, s0 = blockIdx.z * kAbsorbSlots;
  const int ns = min(kAbsorbSlots, a.n_slots - s0);
  __shared__ float qs[kAbsorbSlots][DHq];
  if (h < a.H) {
    for (int e = threadIdx.x; e < kAbsorbSlots * DHq; e += 256) {
      const int sl = e / DHq, j = e % DHq;
      qs[sl][j] = sl < ns ? bf16_bits_to_f32(a.q[((size_t)(s0 + sl) * a.H + h) * DHq + j]) : 0.f;
    }
  }
  __syncthreads();
  if (c >= a.d) return;
  float acc[kAbsorbSlots];
#pragma unroll
  for (int sl = 0; sl < kAbsorbSlots; ++sl) acc[sl] = 0.f;
  if (h < a.H) {
    const uint16_t* w = a.w_k + (size_t)h * DHq * a.d + c;
#pragma unroll 8
    for (int j = 0; j < DHq; ++j) {
      const float wj = bf16_bits_to_f32(w[(size_t)j * a.d]);
#pragma unroll
      for (int sl = 0; sl < kAbsorbSlots; ++sl) acc[sl] += wj * qs[sl][j];
    }
  }
#pragma unroll
  for (int sl = 0; sl < kAbsorbSlots; ++sl)
    if (sl < ns) a.qabs[((size_t)(s0 + sl) * a.ht * 16 + h) * a.d + c] = f32_to_bf16_bits(acc[sl] * a.scale_log2);
}

// The null row through each head's key and value maps:
// null_kv[m][h][j] = sum_c row[c] W_m[h*dh + j][c].  One workgroup per
// (head, map); each wave takes every fourth j, its lanes split the sum over c.
template <int DHq>
__global__ void __launch_bounds__(256) k_rows_null(RowsPrepArgs a) {
  const int h = blockIdx.x, which = blockIdx.y;
  const uint16_t* w = which == 0 ? a.w_k : a.w_v;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int j = wave; j < DHq; j += 4) {
    const uint16_t* wr = w + ((size_t)h * DHq + j) * a.d;
    float acc = 0.f;
    for (int c = lane; c < a.d; c += 64) acc += bf16_bits_to_f32(a.null_row[c]) * bf16_bits_to_f32(wr[c]);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) acc += __shfl_xor(acc, o);
    if (lane == 0) a.null_kv[((size_t)which * a.H + h) * DHq + j] = f32_to_bf16_bits(acc);
  }
}

// Per (slot, head): wave 0 reads the in-block keys and the null row
// (rows_intra) while waves 1-3 combine the row splits in split order against
// their own maximum Mr: u' = sum_k 2^(m_k - Mr) U_k, l' likewise.  Then with
// M = max(Mr, m_i): u = u' 2^(Mr - M) / L (bf16, into ubuf) and the in-block
// weight 2^(m_i - M) / L (into sw), L = l' 2^(Mr - M) + l_i 2^(m_i - M).
template <int D, int DHq>
__global__ void __launch_bounds__(256) k_rows_combine(RowsArgs a) {
  const int slot = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const int n_read = a.n_read[slot], pps = a.pps[slot];
  const int nsp = n_read > 0 ? (n_read + pps - 1) / pps : 0;
  __shared__ float w_sh[4][kRowsSplitCap];
  __shared__ __attribute__((aligned(16))) float u_sh[D];
  __shared__ float pw[64];
  __shared__ __attribute__((aligned(16))) float ired[512];   // in-block value sums of the row groups
  __shared__ float stat[4];   // m_i, l_i, Mr, l'
  __shared__ float fin[1];    // scale of u' (times 1/L)
  const int tile = h / 16, hh = h % 16;     // the head's tile and its row in the tile
  const size_t ustride = (size_t)a.ht * (16 * D + 32);    // one split of the slot to the next
  const float* pb = a.part + (size_t)(a.pbase[slot] + tile) * (16 * D + 32);
  const int lane = tid & 63, wave = tid >> 6;
  if (wave == 0) {
    float mi, li;
    rows_intra<DHq>(a, slot, h, lane, pw, ired, mi, li);
    if (lane == 0) {
      stat[0] = mi;
      stat[1] = li;
    }
  } else {
    // each of waves 1-3 derives the split weights itself (no block barrier)
    const float mk = lane < nsp ? pb[(size_t)lane * ustride + 16 * D + hh] : -INFINITY;
    float Mr = mk;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) Mr = fmaxf(Mr, __shfl_xor(Mr, o));
    if (lane < nsp) w_sh[wave][lane] = (mk == -INFINITY) ? 0.f : exp2w(mk - Mr);
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (wave == 1 && lane == 0) {
      float l = 0.f;
      for (int k = 0; k < nsp; ++k) l += w_sh[1][k] * pb[(size_t)k * ustride + 16 * D + 16 + hh];
      stat[2] = Mr;
      stat[3] = l;
    }
    // At d >= 2048 four consecutive elements per thread (16-byte loads),
    // the splits' loads of a batch of four issued before their products
    // (added in split order): 1.5B row-plane decode 11.1k -> 11.9k tok/s.
    // At d = 1024 that form measured slower (the 410M row-plane step 132.8
    // -> 136.8 us), so narrower rows keep one element per thread.
    if constexpr (D < 2048) {
      for (int c = (wave - 1) * 64 + lane; c < D; c += 192) {
        float x = 0.f;
        for (int k = 0; k < nsp; ++k) x += w_sh[wave][k] * pb[(size_t)k * ustride + (size_t)hh * D + c];
        u_sh[c] = x;
      }
    } else {
      for (int c4 = (wave - 1) * 64 + lane; c4 < D / 4; c4 += 192) {
        const float* pc = pb + (size_t)hh * D + c4 * 4;
        f32x4 x = {0.f, 0.f, 0.f, 0.f};
        int k = 0;
        for (; k + 4 <= nsp; k += 4) {
          f32x4 v[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = *(const f32x4*)(pc + (size_t)(k + j) * ustride);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float w = w_sh[wave][k + j];
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] += w * v[j][i];
          }
        }
        for (; k < nsp; ++k) {
          const f32x4 v = *(const f32x4*)(pc + (size_t)k * ustride);
          const float w = w_sh[wave][k];
#pragma unroll
          for (int i = 0; i < 4; ++i) x[i] += w * v[i];
        }
        *(f32x4*)(u_sh + c4 * 4) = x;
      }
    }
  }
  __syncthreads();
  if (tid == 0) {
    const float mi = stat[0], Mr = stat[2];
    const float M = fmaxf(mi, Mr);
    const float wr = (Mr == -INFINITY) ? 0.f : exp2w(Mr - M);
    const float wi = (mi == -INFINITY) ? 0.f : exp2w(mi - M);
    const float L = wr * stat[3] + wi * stat[1];
    const float inv = (L > 0.f) ? 1.f / L : 0.f;
    fin[0] = wr * inv;
    a.sw[(size_t)slot * a.ht * 16 + h] = wi * inv;
  }
  __syncthreads();
  const float sc = fin[0];
  for (int c = tid; c < D; c += 256) a.ubuf[((size_t)slot * a.ht * 16 + h) * D + c] = f32_to_bf16_bits(u_sh[c] * sc);
}

// out[s][h][j] = sum_c u[s][h][c] W_V[h*dh + j][c] + (w_i/L)[s][h] acc_i[s][h][j]:
// per head a (slots x d) x (d x dh) product on MFMA, one 16 x 16 tile per
// workgroup, its four waves splitting d (A: u rows, B: W_V rows, both
// contiguous in c), partial tiles summed in LDS.
template <int D, int DHq>
__global__ void __launch_bounds__(256) k_rows_project(RowsArgs a) {
  const int h = blockIdx.x, s0 = blockIdx.y * 16, j0 = blockIdx.z * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int srow = s0 + (lane & 15);
  const bool valid = srow < a.n_slots;
  const uint16_t* ua = a.ubuf + ((size_t)(valid ? srow : 0) * a.ht * 16 + h) * D + (lane >> 4) * 8;
  const uint16_t* wb = a.w_v + ((size_t)h * DHq + j0 + (lane & 15)) * D + (lane >> 4) * 8;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k0 = wave * (D / 4); k0 < (wave + 1) * (D / 4); k0 += 32) {
    u32x4 av = *(const u32x4*)(ua + k0);
    if (!valid) av = u32x4{0u, 0u, 0u, 0u};
    const u32x4 bv = *(const u32x4*)(wb + k0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8r, av), __builtin_bit_cast(bf16x8r, bv),
                                                  acc, 0, 0, 0);
  }
  __shared__ f32x4 red[4][64];
  red[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  acc = red[0][lane] + red[1][lane] + red[2][lane] + red[3][lane];
  const int j = j0 + (lane & 15);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int s = s0 + 4 * (lane >> 4) + i;
    if (s < a.n_slots) {
      const float* ip = a.intra + ((size_t)s * a.H + h) * (DHq + 4);
      const float o = acc[i] + a.sw[(size_t)s * a.ht * 16 + h] * ip[j];
      a.out[((size_t)s * a.H + h) * DHq + j] = f32_to_bf16_bits(o);
    }
  }
}

template <int D, int DHq>
static hipError_t launch_rows_dd(const RowsArgs& a, const RowsPrepArgs& pa, int max_split, int stage,
                                 hipStream_t s) {
  if (stage == 0) {   // absorbed queries (and the null row's keys and values)
    hipLaunchKernelGGL((k_rows_absorb_q<DHq>),
                       dim3((D + 255) / 256, pa.ht * 16, (pa.n_slots + kAbsorbSlots - 1) / kAbsorbSlots), dim3(256),
                       0, s, pa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || pa.null_row == nullptr) return e;
    hipLaunchKernelGGL((k_rows_null<DHq>), dim3(pa.H, 2), dim3(256), 0, s, pa);
    return hipGetLastError();
  }
  if (max_split > 0) {
    RowsArgs r = a;
    r.max_split = max_split;
    // Two head tiles per workgroup (one chunk stream for both) at d = 2048,
    // when the tiles pair up: there one tile's workgroup fills a CU's LDS and
    // runs one wave per SIMD, so the second tile's waves come for free.  At
    // the narrower widths several workgroups already share a CU and the
    // measured decode cells were as fast or faster with one tile each.
    if (D >= 2048 && a.ht % 2 == 0)
      hipLaunchKernelGGL((k_reader_rows<D, DHq, 2>), dim3(rows_grid(a.n_slots * max_split, a.ht / 2)), dim3(512), 0, s,
                         r);
    else
      hipLaunchKernelGGL((k_reader_rows<D, DHq, 1>), dim3(rows_grid(a.n_slots * max_split, a.ht)), dim3(256), 0, s, r);
  }
  hipLaunchKernelGGL((k_rows_combine<D, DHq>), dim3(a.n_slots, a.H), dim3(256), 0, s, a);
  hipLaunchKernelGGL((k_rows_project<D, DHq>), dim3(a.H, (a.n_slots + 15) / 16, DHq / 16), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_rows_d(int dh, const RowsArgs& a, const RowsPrepArgs& pa, int max_split, int stage,
                                hipStream_t s) {
  if (dh == 32) return launch_rows_dd<D, 32>(a, pa, max_split, stage, s);
  if (dh == 64) return launch_rows_dd<D, 64>(a, pa, max_split, stage, s);
  if (dh == 128) return launch_rows_dd<D, 128>(a, pa, max_split, stage, s);
  return hipErrorInvalidValue;
}

hipError_t launch_rows(int d, int dh, const RowsArgs& a, const RowsPrepArgs& pa, int stage, hipStream_t s) {
  if (a.n_slots <= 0) return hipSuccess;
  int max_split = 0;
  for (int i = 0; i < a.n_slots; ++i) {
    const int ns = a.n_read[i] > 0 ? (a.n_read[i] + a.pps[i] - 1) / a.pps[i] : 0;
    if (ns > max_split) max_split = ns;
  }
  if (d == 512) return launch_rows_d<512>(dh, a, pa, max_split, stage, s);
  if (d == 768) return launch_rows_d<768>(dh, a, pa, max_split, stage, s);
  if (d == 1024) return launch_rows_d<1024>(dh, a, pa, max_split, stage, s);
  if (d == 2048) return launch_rows_d<2048>(dh, a, pa, max_split, stage, s);
  return hipErrorInvalidValue;
}

}  // namespace smem
