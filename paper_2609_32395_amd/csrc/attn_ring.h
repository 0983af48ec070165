// Attention building blocks shared by the attention kernels and the model
// runtime's fused self-attention: MFMA operand packing, the query
// fragments, the online-softmax step, and the 64-key tile in LDS (key
// plane and transposed value plane) with its score and value products.
// The operand layout of the 16x16x32 bf16 MFMA these assume is described
// at the top of attn_mfma.hip.
#pragma once

#include "common.h"

namespace smem {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef f32x4 floatx4;

constexpr int BT = 64;         // block / page size handled here

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) {
  bf16x8 r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}

__device__ __forceinline__ bf16x8 pack_p(const floatx4& a, const floatx4& b) {
  bf16x8 r;
  r[0] = (__bf16)a[0]; r[1] = (__bf16)a[1]; r[2] = (__bf16)a[2]; r[3] = (__bf16)a[3];
  r[4] = (__bf16)b[0]; r[5] = (__bf16)b[1]; r[6] = (__bf16)b[2]; r[7] = (__bf16)b[3];
  return r;
}

__device__ __forceinline__ u32x4 pack8(const float (&x)[8]) {
  u32x4 r;
  r.x = (uint32_t)f32_to_bf16_bits(x[0]) | ((uint32_t)f32_to_bf16_bits(x[1]) << 16);
  r.y = (uint32_t)f32_to_bf16_bits(x[2]) | ((uint32_t)f32_to_bf16_bits(x[3]) << 16);
  r.z = (uint32_t)f32_to_bf16_bits(x[4]) | ((uint32_t)f32_to_bf16_bits(x[5]) << 16);
  r.w = (uint32_t)f32_to_bf16_bits(x[6]) | ((uint32_t)f32_to_bf16_bits(x[7]) << 16);
  return r;
}

// Query fragments of one wave (B operand of S^T = K Q^T): query row
// wave*16 + l%16, dims kk*32 + (l/16)*8 .. +8.
template <int DH>
__device__ __forceinline__ void load_q(bf16x8 (&qf)[DH / 32], const uint16_t* __restrict__ q, size_t row_stride,
                                       int lane) {
  const uint16_t* qr = q + (size_t)(lane & 15) * row_stride + (lane >> 4) * 8;
#pragma unroll
  for (int kk = 0; kk < DH / 32; ++kk) qf[kk] = as_bf16x8(*(const u32x4*)(qr + kk * 32));
}

// Query fragments turned by one phase row: dst = R(phase) src.
template <int DH>
__device__ __forceinline__ void rope_q(bf16x8 (&dst)[DH / 32], const bf16x8 (&src)[DH / 32],
                                       const float* __restrict__ row, int lane) {
#pragma unroll
  for (int kk = 0; kk < DH / 32; ++kk) {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)src[kk][j];
    rope_turn<8>(x, row, kk * 16 + (lane >> 4) * 4);
#pragma unroll
    for (int j = 0; j < 8; ++j) dst[kk][j] = (__bf16)x[j];
  }
}

// Max / sum over the four lanes that hold one query column (lanes l, l^16,
// l^32, l^48).  permlane16/32_swap of a value with itself leaves, in the
// pair it returns, the lane's own value and its partner's (l^16, l^32), so
// op(pair) is the two-lane reduction -- a VALU exchange instead of an LDS
// permute; both operations are commutative, so every lane gets the same bits.
// The exchanged values are already canonical floats (maxima of MFMA results),
// so the maximum is taken with a plain v_max_f32: fmaxf would first
// canonicalise both operands (two more instructions per exchange).
__device__ __forceinline__ float max_plain(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ float xor16_op_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max_plain(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_op_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max_plain(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor16_op_sum(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_op_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float qmax(float x) { return xor32_op_max(xor16_op_max(x)); }
__device__ __forceinline__ float qsum(float x) { return xor32_op_sum(xor16_op_sum(x)); }


// One online-softmax step over a 64-key tile for the lane's query.
// valid(kt, i) says whether key kt*16 + 4*(lane/16) + i is visible.
template <int DH, bool CAUSAL>
__device__ __forceinline__ void online_step(floatx4 (&s)[4], float& m, float& l, floatx4 (&o)[DH / 16], int lane,
                                            int qrow, float scale_log2) {
  // The maximum is taken over the raw scores and scaled once (the scale is
  // positive and rounding is monotone, so this is the maximum of the scaled
  // scores); each weight is then 2^(s*scale - max) with the scale and the
  // shift in one fused multiply-add.
  float mx = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float x = s[kt][i];
      if (CAUSAL) {
        const int key = kt * 16 + (lane >> 4) * 4 + i;
        if (key > qrow) x = -INFINITY;
      }
      s[kt][i] = x;
      mx = fmaxf(mx, x);
    }
  }
  mx = qmax(mx) * scale_log2;
  // When no query of the wave raises its maximum, the rescale factor is
  // exactly 1: l and o are left as they are (the same bits as multiplying).
  if (__all(mx <= m)) {
    float ps = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = (CAUSAL && s[kt][i] == -INFINITY) ? 0.f : exp2w(__builtin_fmaf(s[kt][i], scale_log2, -m));
        s[kt][i] = p;
        ps += p;
      }
    }
    l += ps;
    return;
  }
  const float mn = fmaxf(m, mx);
  // Without the causal mask every score is finite, so mn is finite and
  // 2^(m - mn) = 2^-inf = 0 on the first tile: the guards are only needed
  // when masked (-inf) scores can make mn = -inf.
  const float alpha = (CAUSAL && m == -INFINITY) ? 0.f : exp2w(m - mn);
  float ps = 0.f;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = (CAUSAL && s[kt][i] == -INFINITY) ? 0.f : exp2w(__builtin_fmaf(s[kt][i], scale_log2, -mn));
      s[kt][i] = p;
      ps += p;
    }
  }
  l = l * alpha + ps;
  m = mn;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) o[dt][i] *= alpha;
  }
}

// ------------------------------------------------------------------ LDS tile layout

// A 64-key tile in LDS -- a memory page's (page, head) tile, or a block's own
// keys and values -- keeps the page layout: the key plane [b][d_h] followed by
// the transposed value plane [d_h][b], with the 16-byte slots of each row
// permuted (key row r: slot = chunk ^ kswz(r); value row d: slot = chunk ^
// vswz(d)), so the rows one MFMA operand read touches fall on distinct banks
// (measured on gfx950: no bank conflicts for the key and value operand reads).
// Memory pages of the non-rotary prefill move global -> LDS by DMA
// (global_load_lds_dwordx4, 16 bytes per lane) through a ring of NS page
// stages, so NS - 1 pages are in flight while one is read and no register
// holds a page in transit.
#ifndef SMEM_PREFILL_STAGES32
#define SMEM_PREFILL_STAGES32 4
#endif
#ifndef SMEM_PREFILL_STAGES64
#define SMEM_PREFILL_STAGES64 4
#endif
#ifndef SMEM_PREFILL_STAGES128
#define SMEM_PREFILL_STAGES128 2
#endif
template <int DH>
struct PageRing {
  static constexpr int TILE = 2 * BT * DH * 2;         // bytes per (page, head)
  static constexpr int KBYTES = BT * DH * 2;           // key plane bytes
  static constexpr int KRB = DH * 2;                   // key row bytes
  static constexpr int KCH = DH / 8;                   // 16-byte chunks per key row
  static constexpr int NS = DH == 32 ? SMEM_PREFILL_STAGES32 : DH == 64 ? SMEM_PREFILL_STAGES64 : SMEM_PREFILL_STAGES128;
  static constexpr int IPW = TILE / 1024 / 4;          // DMA instructions per wave per page
  static_assert(NS >= 2 && NS <= 5, "wait_pages covers up to 3 pages ahead");
  // key rows: slot = chunk ^ kswz(r).  Chosen by measurement (a one-wave LDS
  // bank probe of the score reads): r / 2 for 64-byte rows (r / 4 left them
  // 2-way conflicted), r / 2 for 128-byte rows, r for 256-byte rows.
  __device__ static constexpr int kswz(int r) { return (DH == 32 ? r / 2 : r / (256 / KRB)) % KCH; }
  // the 16-row group (d >> 4) enters the value permutation so that the
  // reads of rows d and d + 16 are never a fixed distance apart: merged into
  // one read2 instruction, their two halves fell on the same banks
  __device__ static constexpr int vswz(int d) { return ((d >> 1) ^ (d >> 4)) & 7; }
};

// S^T for this wave's 16 queries against the 64 keys of a tile.
template <int DH>
__device__ __forceinline__ void scores_ring(floatx4 (&s)[4], const uint8_t* tile, const bf16x8 (&qf)[DH / 32],
                                            int lane) {
  using R = PageRing<DH>;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    const int r = kt * 16 + (lane & 15);
#pragma unroll
    for (int kk = 0; kk < DH / 32; ++kk) {
      const int c = kk * 4 + (lane >> 4);
      const u32x4 kf = *(const u32x4*)(tile + r * R::KRB + ((c ^ R::kswz(r)) << 4));
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf), qf[kk], acc, 0, 0, 0);
    }
    s[kt] = acc;
  }
}

// O^T += V^T P^T over the 64 keys of a tile: lane reads keys
// 4 (l/16) + 16 q .. +3 of value row dt*16 + l%16, q = 0..3.
template <int DH>
__device__ __forceinline__ void pv_ring(floatx4 (&o)[DH / 16], const uint8_t* tile, const floatx4 (&p)[4],
                                        int lane) {
  using R = PageRing<DH>;
  const bf16x8 p0 = pack_p(p[0], p[1]);
  const bf16x8 p1 = pack_p(p[2], p[3]);
  const int g = lane >> 4;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    const int d = dt * 16 + (lane & 15);
    const uint8_t* row = tile + R::KBYTES + d * 128 + (g & 1) * 8;
    u32x2 x[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = *(const u32x2*)(row + ((((g >> 1) + 2 * q) ^ R::vswz(d)) << 4));
    const u32x4 a0 = u32x4{x[0].x, x[0].y, x[1].x, x[1].y};
    const u32x4 a1 = u32x4{x[2].x, x[2].y, x[3].x, x[3].y};
    o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a0), p0, o[dt], 0, 0, 0);
    o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a1), p1, o[dt], 0, 0, 0);
  }
}


// A block's own keys and values from token-major tensors ([row][H][dh], row
// stride rs) into an LDS tile in the layout above, by NT threads: a key job
// is one 16-byte chunk of a row; a value job is one chunk of a row pair,
// written transposed as 32-bit pairs of consecutive keys.  tab: rotary table
// (keys turned by their in-block offsets), or NULL.
template <int DH, int NT>
__device__ __forceinline__ void intra_ring_store(uint8_t* tile, const uint16_t* __restrict__ kin,
                                                 const uint16_t* __restrict__ vin, size_t rs, int tid,
                                                 const float* __restrict__ tab = nullptr) {
  using R = PageRing<DH>;
  constexpr int CPR = DH / 8, NK = BT * CPR, NJ = NK + (BT / 2) * CPR, NIT = (NJ + NT - 1) / NT;
  // every global load first, then the LDS writes
  u32x4 ra[NIT], rb[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int j = tid + it * NT;
    if (j < NK) {                                      // key chunk (row, c8)
      ra[it] = *(const u32x4*)(kin + (j / CPR) * rs + (j % CPR) * 8);
    } else if (j < NJ) {                               // value rows (2 pr, 2 pr + 1), chunk c8
      const int pr = (j - NK) / CPR, c8 = (j - NK) % CPR;
      ra[it] = *(const u32x4*)(vin + (2 * pr) * rs + c8 * 8);
      rb[it] = *(const u32x4*)(vin + (2 * pr + 1) * rs + c8 * 8);
    }
  }
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int j = tid + it * NT;
    if (j < NK) {
      const int row = j / CPR, c8 = j % CPR;
      u32x4 kv = ra[it];
      if (tab) {
        float x[8];
        Chunk<uint16_t>::unpack(kv, x);
        rope_turn<8>(x, tab + (size_t)row * DH, c8 * 4);
        kv = pack8(x);
      }
      *(u32x4*)(tile + row * R::KRB + ((c8 ^ R::kswz(row)) << 4)) = kv;
    } else if (j < NJ) {
      const int pr = (j - NK) / CPR, c8 = (j - NK) % CPR;
      const uint32_t a4[4] = {ra[it].x, ra[it].y, ra[it].z, ra[it].w};
      const uint32_t b4[4] = {rb[it].x, rb[it].y, rb[it].z, rb[it].w};
      const int key = 2 * pr;
      // odd chunks write the odd dimension of each pair first: the lanes of
      // one write then cover both parities of rows (the two bank halves)
      const int flip = c8 & 1;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int d = c8 * 8 + 2 * q;
        const uint32_t lo = (a4[q] & 0xffffu) | (b4[q] << 16), hi = (a4[q] >> 16) | (b4[q] & 0xffff0000u);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int dd = d + (k ^ flip);
          *(uint32_t*)(tile + R::KBYTES + dd * 128 + (key & 7) * 2 + (((key >> 3) ^ R::vswz(dd)) << 4)) =
              (k ^ flip) ? hi : lo;
        }
      }
    }
  }
}

}  // namespace smem
