// Linear maps y = x W^T (W stored [out, in], a linear layer's layout) on
// MFMA for the whole-model runtime: a few-row kernel and an LDS-tiled GEMM
// that share one reduction order, and the host dispatch between them.
// Both MFMA operands run along the reduction dimension, so a lane's 8
// k-values are 16 contiguous bytes of an x row and of a W row.
#pragma once

#include <algorithm>

#include "common.h"

namespace smem {

typedef __bf16 bf16x8m __attribute__((ext_vector_type(8)));

enum LinEpi : int { kLinStore = 0, kLinGelu = 1, kLinResid = 2, kLinF32 = 3, kLinSplit = 4 };

struct LinArgs {
  const uint16_t* x;   // [M][ldx], K used
  const uint16_t* w;   // output rows n < n2: w + n*K
  const uint16_t* w2;  // output rows n >= n2: w2 + (n - n2)*K
  const uint16_t* res; // residual [M][ldy] (kLinResid; may equal y)
  uint16_t* y;         // [M][ldy]
  uint16_t* y1;        // kLinSplit: columns [ns, 2ns) -> y1, [2ns, 3ns) -> y2 (each [M][ns])
  uint16_t* y2;
  float* yf;           // kLinF32: [M][ldy]
  const uint16_t* lng; // y = LN(x) W^T when set: LayerNorm gain and bias [K]
  const uint16_t* lnb;
  uint16_t* lnout;     // many rows: LN(x) written here ([M][K]) before the map
  int32_t M, N, K, ldx, ldy, n2, ns;
};

// erf by Abramowitz and Stegun, Handbook of Mathematical Functions, formula
// 7.1.26: erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),
// t = 1 / (1 + p x), x >= 0, absolute error <= 1.5e-7 (odd extension for
// x < 0); far below the bf16 rounding of the activations it feeds.
__device__ __forceinline__ float erf_as(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(1.f + 0.3275911f * ax);
  const float poly = ((((1.061405429f * t - 1.453152027f) * t + 1.421413741f) * t - 0.284496736f) * t + 0.254829592f) * t;
  const float e = __builtin_amdgcn_exp2f(-ax * ax * 1.4426950408889634f);
  return copysignf(1.f - poly * e, x);
}

// GELU, exact (erf) form: x * Phi(x) = x/2 * (1 + erf(x / sqrt 2)).
__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.f + erf_as(x * 0.70710678118654752f)); }

// Reduction order of every linear map, whatever kernel computes it: the
// K-range is cut into chunks of lin_chunk(K) (a multiple of 256); inside a
// chunk, one 16x16x32 bf16 MFMA per 32-wide k step accumulates from zero in
// ascending k; the chunk sums are then added in ascending chunk order to a
// total that starts at zero.  Each output element therefore sees the same
// operations in the same order for any M and any tiling, which keeps a
// row's result independent of the other rows in the call (block-skip serving
// reproduces the cold pass bit for bit).
__host__ __device__ constexpr int lin_chunk(int K) { return 256 * ((K + 256 * 16 - 1) / (256 * 16)); }

// LayerNorm of a row of width d (d % 64 == 0, d <= 2048), eps 1e-5, with the
// statistics summed in one fixed order, so the stand-alone kernel below and
// the few-row map that normalizes its own x rows give the same bits.  The row
// is cut as a linear map cuts K: chunks of 256, each of 32-wide steps, each
// step of four 8-wide groups.  The partial of (chunk, group) adds its values
// in ascending k; a chunk's four partials add as (g0 + g1) + (g2 + g3); the
// chunk totals add in ascending chunk order from zero.  mean = total / d; the
// second moment sums (x - mean)^2 the same way; rstd = 1 / sqrt(m2 / d + eps).
__device__ __forceinline__ float ln_sum8(const u32x4& c, float s) {
  float f[8];
  Chunk<uint16_t>::unpack(c, f);
#pragma unroll
  for (int e = 0; e < 8; ++e) s += f[e];
  return s;
}
__device__ __forceinline__ float ln_sq8(const u32x4& c, float mean, float s) {
  float f[8];
  Chunk<uint16_t>::unpack(c, f);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float t = f[e] - mean;
    s += t * t;
  }
  return s;
}
__device__ __forceinline__ float ln_rstd(float m2, int d) { return 1.f / sqrtf(m2 / d + 1e-5f); }
__device__ __forceinline__ u32x4 ln_apply8(const u32x4& x, const u32x4& g, const u32x4& b, float mean, float rstd) {
  float xf[8], gf[8], bf[8];
  Chunk<uint16_t>::unpack(x, xf);
  Chunk<uint16_t>::unpack(g, gf);
  Chunk<uint16_t>::unpack(b, bf);
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float y0 = (xf[2 * e] - mean) * rstd * gf[2 * e] + bf[2 * e];
    const float y1 = (xf[2 * e + 1] - mean) * rstd * gf[2 * e + 1] + bf[2 * e + 1];
    w[e] = (uint32_t)f32_to_bf16_bits(y0) | ((uint32_t)f32_to_bf16_bits(y1) << 16);
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

// Stand-alone LayerNorm (rows x[row * ldx .. + d) -> y[row * ldy ..)): a
// row takes 4 n_chunks lanes, lane 4c + g holding group g of chunk c, and a
// wave holds 64 / (4 n_chunks) rows (4 at d = 1024), so every lane sums; the
// gain and bias are loaded with the row.
__host__ __device__ constexpr int ln_rows_per_wave(int d) { return 64 / (4 * ((d / 32 + 7) / 8)); }

__global__ void __launch_bounds__(64) k_ln_rows(const uint16_t* __restrict__ x, int ldx,
                                                const uint16_t* __restrict__ g, const uint16_t* __restrict__ b,
                                                uint16_t* __restrict__ y, int ldy, int rows, int d) {
  const int KS = d / 32, NC = (KS + 7) / 8, LPR = 4 * NC, R = 64 / LPR;
  const int lane = threadIdx.x, rl = lane / LPR, base = rl * LPR, l = lane - base;
  const int row = blockIdx.x * R + rl;
  if (rl >= R || row >= rows) return;
  const int c = l >> 2, k0 = 256 * c + 8 * (l & 3);
  const int nt = min(8, KS - 8 * c);
  const uint16_t* xr = x + (size_t)row * ldx + k0;
  u32x4 v[8], gv[8], bv[8];
#pragma unroll
  for (int t = 0; t < 8; ++t)
    if (t < nt) v[t] = *(const u32x4*)(xr + 32 * t);
#pragma unroll
  for (int t = 0; t < 8; ++t)
    if (t < nt) {
      gv[t] = *(const u32x4*)(g + k0 + 32 * t);
      bv[t] = *(const u32x4*)(b + k0 + 32 * t);
    }
  float s = 0.f;
#pragma unroll
  for (int t = 0; t < 8; ++t)
    if (t < nt) s = ln_sum8(v[t], s);
  s += __shfl_xor(s, 1);
  s += __shfl_xor(s, 2);
  float tot = 0.f;
  for (int q = 0; q < NC; ++q) tot += __shfl(s, base + 4 * q);
  const float mean = tot / d;
  float m2 = 0.f;
#pragma unroll
  for (int t = 0; t < 8; ++t)
    if (t < nt) m2 = ln_sq8(v[t], mean, m2);
  m2 += __shfl_xor(m2, 1);
  m2 += __shfl_xor(m2, 2);
  float tot2 = 0.f;
  for (int q = 0; q < NC; ++q) tot2 += __shfl(m2, base + 4 * q);
  const float rstd = ln_rstd(tot2, d);
  uint16_t* yr = y + (size_t)row * ldy + k0;
#pragma unroll
  for (int t = 0; t < 8; ++t)
    if (t < nt) *(u32x4*)(yr + 32 * t) = ln_apply8(v[t], gv[t], bv[t], mean, rstd);
}

template <int EPI>
__device__ __forceinline__ void lin_store(const LinArgs& a, int m, int n, float v) {
  if constexpr (EPI == kLinF32) {
    a.yf[(size_t)m * a.ldy + n] = v;
  } else if constexpr (EPI == kLinGelu) {
    a.y[(size_t)m * a.ldy + n] = f32_to_bf16_bits(gelu_erf(v));
  } else if constexpr (EPI == kLinResid) {
    const size_t o = (size_t)m * a.ldy + n;
    a.y[o] = f32_to_bf16_bits(v + bf16_bits_to_f32(a.res[o]));
  } else if constexpr (EPI == kLinSplit) {
    const int g = n / a.ns, c = n - g * a.ns;
    uint16_t* dst = g == 0 ? a.y : (g == 1 ? a.y1 : a.y2);
    dst[(size_t)m * a.ns + c] = f32_to_bf16_bits(v);
  } else {
    a.y[(size_t)m * a.ldy + n] = f32_to_bf16_bits(v);
  }
}

// Four consecutive outputs n .. n+3 of row m (n % 4 == 0; bf16 rows have
// ldy % 4 == 0, so the four share one 8-byte word; a split's column groups
// are multiples of 4 wide).  Columns >= N are dropped.
template <int EPI>
__device__ __forceinline__ void lin_store4(const LinArgs& a, int m, int n, const f32x4& v) {
  if constexpr (EPI == kLinF32) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (n + e < a.N) a.yf[(size_t)m * a.ldy + n + e] = v[e];
  } else {
    if (n + 3 >= a.N) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < a.N) lin_store<EPI>(a, m, n + e, v[e]);
      return;
    }
    float o[4];
    uint16_t* dst;
    if constexpr (EPI == kLinSplit) {
      const int g = n / a.ns, c = n - g * a.ns;
      dst = (g == 0 ? a.y : (g == 1 ? a.y1 : a.y2)) + (size_t)m * a.ns + c;
    } else {
      dst = a.y + (size_t)m * a.ldy + n;
    }
    if constexpr (EPI == kLinResid) {
      const u32x2 r = *(const u32x2*)(a.res + (size_t)m * a.ldy + n);
      o[0] = v[0] + bf16_bits_to_f32(r.x & 0xffffu);
      o[1] = v[1] + bf16_bits_to_f32(r.x >> 16);
      o[2] = v[2] + bf16_bits_to_f32(r.y & 0xffffu);
      o[3] = v[3] + bf16_bits_to_f32(r.y >> 16);
    } else if constexpr (EPI == kLinGelu) {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = gelu_erf(v[e]);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = v[e];
    }
    *(u32x2*)dst = u32x2{(uint32_t)f32_to_bf16_bits(o[0]) | ((uint32_t)f32_to_bf16_bits(o[1]) << 16),
                         (uint32_t)f32_to_bf16_bits(o[2]) | ((uint32_t)f32_to_bf16_bits(o[3]) << 16)};
  }
}

__device__ __forceinline__ const uint16_t* lin_wrow(const LinArgs& a, int n) {
  return n < a.n2 ? a.w + (size_t)n * a.K : a.w2 + (size_t)(n - a.n2) * a.K;
}

// One 16x16x32 step with the W tile as the MFMA's row operand and the x
// tile as its column operand: lane l then holds outputs (x row l % 16,
// W rows 4 (l / 16) .. +3), four consecutive output columns of one row.
__device__ __forceinline__ f32x4 mfma16(const u32x4& A, const u32x4& B, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8m, A), __builtin_bit_cast(bf16x8m, B), c,
                                                 0, 0, 0);
}

// Launch order -> work item.  Workgroups are dealt to the 8 XCDs round-robin
// (workgroup i to XCD i mod 8); the grid is padded to a multiple of 8 and
// item p = (i mod 8) * (T8 / 8) + i / 8, so each XCD takes one contiguous
// range of items and neighbouring items share that XCD's L2.  Padding
// workgroups get -1 and exit.
__device__ __forceinline__ int xcd_order(int i, int T) {
  const int T8 = (T + 7) & ~7;
  const int p = (i & 7) * (T8 >> 3) + (i >> 3);
  return p < T ? p : -1;
}
__host__ __device__ constexpr int xcd_grid(int T) { return (T + 7) & ~7; }

// Few rows (one or two blocks): the weights stream from HBM once and the
// time is load latency, so the reduction chunks run side by side.  A
// workgroup owns RT x 16 rows and G x 16 output columns and has one wave per
// chunk; each wave keeps U steps of operands (RT tiles of x, G tiles of W) in
// flight and leaves its chunk sums in LDS, where they are added in chunk
// order.  Launch order puts the row tiles of one column group next to each
// other on one XCD, so their W tiles are read from HBM once.
// Dynamic LDS: n_chunks x RT x G x 1 KiB <= 64 KiB.
template <int RT_, int G_, int U_>
struct SkinnyCfg {
  static constexpr int RT = RT_, G = G_, U = U_;
};

template <int EPI, class C>
__global__ void __launch_bounds__(1024) k_linear_skinny(LinArgs a, int row_tiles, int col_groups) {
  constexpr int RT = C::RT, G = C::G, U = C::U, W16 = 16 * G;
  extern __shared__ float part[];   // [n_chunks][16 RT][16 G]
  const int pid = xcd_order(blockIdx.x, row_tiles * col_groups);
  if (pid < 0) return;
  const int m0 = (pid % row_tiles) * 16 * RT, n0 = (pid / row_tiles) * W16;
  const int lane = threadIdx.x & 63, c = threadIdx.x >> 6;       // wave c computes chunk c
  const int kofs = (lane >> 4) * 8;
  const int KS = a.K / 32, CS = lin_chunk(a.K) / 32, NC = (KS + CS - 1) / CS;
  const uint16_t* ap[RT];
  const uint16_t* bp[G];
#pragma unroll
  for (int i = 0; i < RT; ++i) ap[i] = a.x + (size_t)min(m0 + i * 16 + (lane & 15), a.M - 1) * a.ldx + kofs;
#pragma unroll
  for (int j = 0; j < G; ++j) bp[j] = lin_wrow(a, min(n0 + j * 16 + (lane & 15), a.N - 1)) + kofs;
  const int s0 = c * CS, s1 = min(KS, s0 + CS);
  f32x4 acc[RT][G];
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int j = 0; j < G; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int u0 = s0; u0 < s1; u0 += U) {
    u32x4 A[U][RT], B[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int st = min(u0 + u, s1 - 1) * 32;
#pragma unroll
      for (int j = 0; j < G; ++j) B[u][j] = *(const u32x4*)(bp[j] + st);
#pragma unroll
      for (int i = 0; i < RT; ++i) A[u][i] = *(const u32x4*)(ap[i] + st);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u0 + u < s1) {
#pragma unroll
        for (int i = 0; i < RT; ++i)
#pragma unroll
          for (int j = 0; j < G; ++j) acc[i][j] = mfma16(B[u][j], A[u][i], acc[i][j]);
      }
    }
  }
  float* pc = part + c * (256 * RT * G);
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int j = 0; j < G; ++j)
      *(f32x4*)(pc + (i * 16 + (lane & 15)) * W16 + j * 16 + 4 * (lane >> 4)) = acc[i][j];
  __syncthreads();
  for (int q = threadIdx.x; q < 64 * RT * G; q += blockDim.x) {
    const int row = q / (4 * G), c0 = (q % (4 * G)) * 4;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    for (int ch = 0; ch < NC; ++ch) v += *(const f32x4*)(part + ch * (256 * RT * G) + row * W16 + c0);
    const int m = m0 + row;
    if (m < a.M) lin_store4<EPI>(a, m, n0 + c0, v);
  }
}

// Few rows with the LayerNorm fused (y = LN(x) W^T, K <= 2048, so every
// chunk is 256 wide, 8 steps): each wave loads its chunk of the x rows whole,
// the chunk partials of the row statistics meet in LDS in the fixed order of
// the stand-alone kernel, and the rows are normalized in registers before the
// MFMAs; the first U steps of W, issued with the x loads, are in flight
// meanwhile, and each step's W registers are refilled with step t + U once
// its MFMAs are issued.  The sums
// are the same as k_linear_skinny's on LN(x) rows, so the output is bitwise
// the unfused pair's.
// Dynamic LDS: gain and bias (4 K bytes) and two statistics planes of
// n_chunks x 16 RT floats, then, in the same space, n_chunks x RT x G KiB of
// partial sums.
// An empty asm that claims to rewrite the packed x rows, so the compiler
// unpacks them again where they are next used instead of keeping 8 floats
// per register live across the statistics barriers.
template <int T, int R>
__device__ __forceinline__ void opaque(u32x4 (&X)[T][R]) {
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < R; ++i) asm volatile("" : "+v"(X[t][i]));
}

template <int EPI, class C>
__global__ void __launch_bounds__(512) k_linear_skinny_ln(LinArgs a, int row_tiles, int col_groups) {
  constexpr int RT = C::RT, G = C::G, U = C::U, W16 = 16 * G;
  extern __shared__ float part[];   // [n_chunks][16 RT][16 G]
  const int pid = xcd_order(blockIdx.x, row_tiles * col_groups);
  if (pid < 0) return;
  const int m0 = (pid % row_tiles) * 16 * RT, n0 = (pid / row_tiles) * W16;
  const int lane = threadIdx.x & 63;
  const int c = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave c computes chunk c
  const int kofs = (lane >> 4) * 8;
  const int KS = a.K / 32, NC = (KS + 7) / 8;
  uint16_t* gb = (uint16_t*)part;                                // gain [K], bias [K] (until the MFMAs)
  float* st0 = (float*)(gb + 2 * a.K);                           // [n_chunks][16 RT] sums, then second moments
  float* st1 = st0 + NC * 16 * RT;
  const int s0 = c * 8, ns = min(8, KS - s0);
  const uint16_t* ap[RT];
  const uint16_t* bp[G];
#pragma unroll
  for (int i = 0; i < RT; ++i) ap[i] = a.x + (size_t)min(m0 + i * 16 + (lane & 15), a.M - 1) * a.ldx + kofs;
#pragma unroll
  for (int j = 0; j < G; ++j) bp[j] = lin_wrow(a, min(n0 + j * 16 + (lane & 15), a.N - 1)) + kofs;
  u32x4 X[8][RT], B[U][G];
#pragma unroll
  for (int t = 0; t < 8; ++t)
#pragma unroll
    for (int i = 0; i < RT; ++i) X[t][i] = *(const u32x4*)(ap[i] + (s0 + min(t, ns - 1)) * 32);
  const int q8 = threadIdx.x * 8;
  u32x4 g16 = {0, 0, 0, 0}, b16 = {0, 0, 0, 0};
  if (q8 < a.K) {
    g16 = *(const u32x4*)(a.lng + q8);
    b16 = *(const u32x4*)(a.lnb + q8);
  }
#pragma unroll
  for (int t = 0; t < U; ++t)
#pragma unroll
    for (int j = 0; j < G; ++j) B[t][j] = *(const u32x4*)(bp[j] + (s0 + min(t, ns - 1)) * 32);
  if (q8 < a.K) {
    *(u32x4*)(gb + q8) = g16;
    *(u32x4*)(gb + a.K + q8) = b16;
  }
  float mean[RT], rstd[RT];
#pragma unroll
  for (int i = 0; i < RT; ++i) {
    float v = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t)
      if (t < ns) v = ln_sum8(X[t][i], v);
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (lane < 16) st0[c * 16 * RT + i * 16 + lane] = v;
  }
  opaque(X);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < RT; ++i) {
    float tot = 0.f;
    for (int q = 0; q < NC; ++q) tot += st0[q * 16 * RT + i * 16 + (lane & 15)];
    mean[i] = tot / a.K;
    float v = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t)
      if (t < ns) v = ln_sq8(X[t][i], mean[i], v);
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (lane < 16) st1[c * 16 * RT + i * 16 + lane] = v;
  }
  opaque(X);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < RT; ++i) {
    float tot = 0.f;
    for (int q = 0; q < NC; ++q) tot += st1[q * 16 * RT + i * 16 + (lane & 15)];
    rstd[i] = ln_rstd(tot, a.K);
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const int k = (s0 + min(t, ns - 1)) * 32 + kofs;
    const u32x4 g8 = *(const u32x4*)(gb + k), b8 = *(const u32x4*)(gb + a.K + k);
#pragma unroll
    for (int i = 0; i < RT; ++i) X[t][i] = ln_apply8(X[t][i], g8, b8, mean[i], rstd[i]);
  }
  __syncthreads();                       // gain, bias and statistics are read; part may be written
  f32x4 acc[RT][G];
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int j = 0; j < G; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    if (t < ns) {
#pragma unroll
      for (int i = 0; i < RT; ++i)
#pragma unroll
        for (int j = 0; j < G; ++j) acc[i][j] = mfma16(B[t % U][j], X[t][i], acc[i][j]);
    }
    if (t + U < 8) {                     // refill this step's W registers with step t + U
#pragma unroll
      for (int j = 0; j < G; ++j) B[t % U][j] = *(const u32x4*)(bp[j] + (s0 + min(t + U, ns - 1)) * 32);
    }
  }
  float* pc = part + c * (256 * RT * G);
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int j = 0; j < G; ++j)
      *(f32x4*)(pc + (i * 16 + (lane & 15)) * W16 + j * 16 + 4 * (lane >> 4)) = acc[i][j];
  __syncthreads();
  for (int q = threadIdx.x; q < 64 * RT * G; q += blockDim.x) {
    const int row = q / (4 * G), c0 = (q % (4 * G)) * 4;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    for (int ch = 0; ch < NC; ++ch) v += *(const f32x4*)(part + ch * (256 * RT * G) + row * W16 + c0);
    const int m = m0 + row;
    if (m < a.M) lin_store4<EPI>(a, m, n0 + c0, v);
  }
}

template <int EPI, class C>
static void launch_skinny_cfg(const LinArgs& a, int nc, hipStream_t s) {
  const int rt = (a.M + 16 * C::RT - 1) / (16 * C::RT), cg = (a.N + 16 * C::G - 1) / (16 * C::G);
  hipLaunchKernelGGL((k_linear_skinny<EPI, C>), dim3(xcd_grid(rt * cg)), dim3(64 * nc), (size_t)nc * 1024 * C::RT * C::G, s,
                     a, rt, cg);
}

// The widest tile that still gives at least 192 workgroups (one row tile
// when M <= 16, where a second row tile is padding only): every workgroup
// reads its rows of x and its columns of W whole, and reads issued at the
// same time by several workgroups each cost close to a full read, so wider
// tiles (fewer duplicated reads) win until too few workgroups remain to keep
// the loads in flight (measured on the 64-row maps of the three model
// scales).  Partial sums need n_chunks x RT x G KiB of LDS (at most 64).  All
// tilings compute every output in the same order.
template <int EPI>
static void launch_skinny(const LinArgs& a, hipStream_t s) {
  const int nc = (a.K + lin_chunk(a.K) - 1) / lin_chunk(a.K);
  auto fits = [&](int rt, int g) {
    const long wgs = (long)((a.M + 16 * rt - 1) / (16 * rt)) * ((a.N + 16 * g - 1) / (16 * g));
    return wgs >= 192 && nc * rt * g <= 64 && (rt == 1 || a.M > 16);
  };
  if (fits(2, 4)) launch_skinny_cfg<EPI, SkinnyCfg<2, 4, 4>>(a, nc, s);
  else if (fits(2, 2)) launch_skinny_cfg<EPI, SkinnyCfg<2, 2, 4>>(a, nc, s);
  else if (fits(1, 2)) launch_skinny_cfg<EPI, SkinnyCfg<1, 2, 8>>(a, nc, s);
  else launch_skinny_cfg<EPI, SkinnyCfg<1, 1, 8>>(a, nc, s);
}

inline size_t skinny_ln_lds(int nc, int rt, int g, int K) {
  return std::max((size_t)nc * 1024 * rt * g, (size_t)4 * K + (size_t)2 * nc * 16 * rt * 4);
}

template <int EPI, class C>
static void launch_skinny_ln_cfg(const LinArgs& a, int nc, hipStream_t s) {
  const int rt = (a.M + 16 * C::RT - 1) / (16 * C::RT), cg = (a.N + 16 * C::G - 1) / (16 * C::G);
  hipLaunchKernelGGL((k_linear_skinny_ln<EPI, C>), dim3(xcd_grid(rt * cg)), dim3(64 * nc),
                     skinny_ln_lds(nc, C::RT, C::G, a.K), s, a, rt, cg);
}

// The tiling rule of launch_skinny, with the LayerNorm's LDS counted; at
// K <= 1024 one row tile of 2 column groups goes first (measured at 64 rows,
// weights out of the last-level cache: 1024 -> 3072 10.4 against 11.0 us for
// 2 x 2, 1024 -> 4096 10.5 against 11.2, 768 -> 3072 9.3 against 9.9).
template <int EPI>
static void launch_skinny_ln(const LinArgs& a, hipStream_t s) {
  const int nc = (a.K + 255) / 256;
  auto fits = [&](int rt, int g) {
    const long wgs = (long)((a.M + 16 * rt - 1) / (16 * rt)) * ((a.N + 16 * g - 1) / (16 * g));
    return wgs >= 192 && skinny_ln_lds(nc, rt, g, a.K) <= 65536 && (rt == 1 || a.M > 16);
  };
  if (a.K <= 1024 && fits(1, 2)) launch_skinny_ln_cfg<EPI, SkinnyCfg<1, 2, 8>>(a, nc, s);
  else if (fits(2, 4)) launch_skinny_ln_cfg<EPI, SkinnyCfg<2, 4, 4>>(a, nc, s);
  else if (fits(2, 2)) launch_skinny_ln_cfg<EPI, SkinnyCfg<2, 2, 8>>(a, nc, s);
  else if (fits(1, 2)) launch_skinny_ln_cfg<EPI, SkinnyCfg<1, 2, 8>>(a, nc, s);
  else launch_skinny_ln_cfg<EPI, SkinnyCfg<1, 1, 8>>(a, nc, s);
}

// Many rows: BM x BN tiles, WAVES_M x WAVES_N waves (each (BM/WAVES_M) x
// (BN/WAVES_N) as 16x16 MFMA tiles), K in BK-wide stages moved global -> LDS
// by DMA through a ring of NS stages, so no register holds an operand in
// transit and NS - 1 stages are in flight during each stage's MFMAs.  An LDS
// row is BK bf16 = BK/8 chunks of 16 B; chunk c of row r sits at slot
// c ^ swz(r), so the 16 rows one MFMA operand read touches cover every bank
// once.  Tiles are visited in groups of 8 row tiles, and consecutive groups
// of the launch order land on one XCD, so the A and W tiles a group shares
// stay in that XCD's L2.
template <int BM_, int BN_, int BK_, int NS_, int WAVES_M, int WAVES_N>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, NS = NS_;
  static constexpr int NW = WAVES_M * WAVES_N, NT = 64 * NW;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N, TM = WM / 16, TN = WN / 16;
  static constexpr int CPR = BK / 8;                 // 16-byte chunks per LDS row
  static constexpr int RPI = 1024 / (BK * 2);        // rows per DMA instruction (1 KiB)
  static constexpr int R256 = 256 / (BK * 2);        // rows per 256 bytes
  static constexpr int IA = BM / RPI / NW, IB = BN / RPI / NW;
  static constexpr int STAGE = (BM + BN) * BK;       // elements per stage
  static_assert(IA * RPI * NW == BM && IB * RPI * NW == BN, "DMA rows must tile the stage");
  static_assert(NS >= 2 && NS <= 5, "ring depth");
  __device__ static constexpr int swz(int r) { return (r / R256) % CPR; }
};

template <int N>
__device__ __forceinline__ void wait_stages(int ahead) {
  if (ahead >= 3) wait_vm<3 * N < 63 ? 3 * N : 63>();
  else if (ahead == 2) wait_vm<2 * N>();
  else if (ahead == 1) wait_vm<N>();
  else wait_vm<0>();
}

template <int EPI, class C>
__global__ void __launch_bounds__(C::NT, 2 * 4 / C::NW) k_gemm(LinArgs a, int tiles_m, int tiles_n) {
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, NS = C::NS, WM = C::WM, WN = C::WN;
  constexpr int TM = C::TM, TN = C::TN, IA = C::IA, IB = C::IB, STAGE = C::STAGE;
  __shared__ __attribute__((aligned(1024))) uint16_t lds[NS * STAGE];
  // launch order -> tile: consecutive pids of one XCD, then groups of 8 row tiles
  const int pid = xcd_order(blockIdx.x, tiles_m * tiles_n);
  if (pid < 0) return;
  const int per_group = 8 * tiles_n, g0 = (pid / per_group) * 8, gsz = min(tiles_m - g0, 8);
  const int tm = g0 + (pid % per_group) % gsz, tn = (pid % per_group) / gsz;
  const int n0 = tn * BN, m0 = tm * BM;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave % (BM / WM), wn = wave / (BM / WM);
  const int KT = a.K / BK, CT = lin_chunk(a.K) / BK;
  const uint16_t* ga[IA];
  const uint16_t* gb[IB];
#pragma unroll
  for (int i = 0; i < IA; ++i) {
    const int r = (wave * IA + i) * C::RPI + lane / C::CPR, c = (lane % C::CPR) ^ C::swz(r);
    ga[i] = a.x + (size_t)min(m0 + r, a.M - 1) * a.ldx + c * 8;
  }
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int r = (wave * IB + i) * C::RPI + lane / C::CPR, c = (lane % C::CPR) ^ C::swz(r);
    gb[i] = lin_wrow(a, min(n0 + r, a.N - 1)) + c * 8;
  }
  const uint32_t lbase = (uint32_t)(uintptr_t)lds;
  auto issue = [&](int kt) {
    const uint32_t sb = lbase + (uint32_t)((kt % NS) * STAGE * 2);
#pragma unroll
    for (int i = 0; i < IA; ++i)
      dma16(ga[i] + kt * BK, __builtin_amdgcn_readfirstlane(sb + (wave * IA + i) * 1024));
#pragma unroll
    for (int i = 0; i < IB; ++i)
      dma16(gb[i] + kt * BK, __builtin_amdgcn_readfirstlane(sb + BM * BK * 2 + (wave * IB + i) * 1024));
  };
  f32x4 acc[TM][TN], tot[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = tot[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < NS - 1 && p < KT; ++p) issue(p);
  for (int kt = 0; kt < KT; ++kt) {
    wait_stages<IA + IB>(min(NS - 2, KT - 1 - kt));
    lds_barrier();                       // stage kt is in LDS; every wave is done with stage kt - 1
    if (kt + NS - 1 < KT) issue(kt + NS - 1);
    const uint16_t* sa = lds + (kt % NS) * STAGE;
    const uint16_t* sb = sa + BM * BK;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      const int c = ks * 4 + (lane >> 4);
      u32x4 B[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WN + j * 16 + (lane & 15);
        B[j] = *(const u32x4*)(sb + r * BK + ((c ^ C::swz(r)) << 3));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WM + i * 16 + (lane & 15);
        const u32x4 A = *(const u32x4*)(sa + r * BK + ((c ^ C::swz(r)) << 3));
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(B[j], A, acc[i][j]);
      }
    }
    if ((kt + 1) % CT == 0 || kt + 1 == KT) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          tot[i][j] += acc[i][j];
          acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + wm * WM + i * 16 + (lane & 15);
    if (m < a.M) {
#pragma unroll
      for (int j = 0; j < TN; ++j) lin_store4<EPI>(a, m, n0 + wn * WN + j * 16 + 4 * (lane >> 4), tot[i][j]);
    }
  }
}

// Few rows by a very wide map (the output head: tens of thousands of
// columns): the x rows (at most 64 when K <= 1024, 32 at K = 2048) are
// loaded into LDS once per workgroup and stay there, and each wave computes
// two 16-column tiles side by side, streaming their weights a reduction
// chunk (8 steps) at a time with the next chunk's loads (16 KB) issued
// before the current chunk's MFMAs; each x fragment read from LDS feeds both
// tiles.  The weights are read from HBM once and x once per workgroup, where
// the few-row kernel re-reads x once per column group.  A wave sums every
// chunk of its tiles itself -- one MFMA per 32-wide step from zero inside a
// chunk, the chunk sums added in chunk order -- the reduction order of every
// linear map.  LDS rows are padded by 16 bytes so the 16 rows one operand
// read touches start on different banks.
template <int NCH, int RT>
__global__ void __launch_bounds__(512) k_linear_wide(LinArgs a, int n_tiles) {
  constexpr int K = 256 * NCH, XP = K + 8;
  __shared__ __attribute__((aligned(16))) uint16_t xs[RT * 16 * XP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int q = tid; q < RT * 16 * (K / 8); q += 512) {
    const int r = q / (K / 8), c8 = q % (K / 8);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < a.M) v = *(const u32x4*)(a.x + (size_t)r * a.ldx + c8 * 8);
    *(u32x4*)(xs + r * XP + c8 * 8) = v;     // rows M .. 16 RT - 1 are zero
  }
  __syncthreads();                           // the only barrier
  const int t0 = (blockIdx.x * 8 + wave) * 2;
  if (t0 >= n_tiles) return;
  const bool second = t0 + 1 < n_tiles;      // else the second tile re-reads the first and is not stored
  const int kofs = (lane >> 4) * 8;
  auto wrow = [&](int t) { return lin_wrow(a, min(t * 16 + (lane & 15), a.N - 1)) + kofs; };
  const uint16_t* wp[2] = {wrow(t0), wrow(second ? t0 + 1 : t0)};
  u32x4 W[2][2][8];                          // [chunk parity][tile][step]
  auto fetch = [&](u32x4 (&Wd)[2][8], int c) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int j = 0; j < 2; ++j) Wd[j][u] = *(const u32x4*)(wp[j] + c * 256 + u * 32);
  };
  fetch(W[0], 0);
  f32x4 tot[2][RT];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < RT; ++i) tot[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (c + 1 < NCH) fetch(W[(c + 1) & 1], c + 1);
    __builtin_amdgcn_sched_barrier(0);     // the next chunk's loads go out before this chunk's MFMAs
    // an opaque copy of the x offset keeps the compiler from holding x
    // fragments in registers across chunks (an offset, not a pointer, so
    // the reads stay LDS reads)
    int xv = (lane & 15) * XP + kofs + c * 256;
    asm volatile("" : "+v"(xv));
    const uint16_t* xt = xs + xv;
    f32x4 acc[2][RT];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < RT; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 8; ++st)
#pragma unroll
      for (int i = 0; i < RT; ++i) {
        const u32x4 xf = *(const u32x4*)(xt + i * 16 * XP + st * 32);
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[j][i] = mfma16(W[c & 1][j][st], xf, acc[j][i]);
      }
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < RT; ++i) tot[j][i] += acc[j][i];
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (j == 1 && !second) break;
#pragma unroll
    for (int i = 0; i < RT; ++i) {
      const int m = i * 16 + (lane & 15);
      if (m < a.M) lin_store4<kLinF32>(a, m, (t0 + j) * 16 + 4 * (lane >> 4), tot[j][i]);
    }
  }
}

// The wide kernel serves fp32 maps of at most 64 rows with K a multiple of
// 256 up to 2048 whose x rows fit in LDS (16 row tiles of K + 8 bf16 each:
// 64 rows up to K = 1024, 32 rows at K = 2048) and at least 8192 columns.
constexpr int kWideLds = 160 * 1024;
__host__ __device__ constexpr int wide_lds(int rt, int k) { return rt * 16 * (k + 8) * 2; }
inline bool wide_fits(const LinArgs& a) {
  return !a.lng && a.M >= 1 && a.M <= 64 && a.K % 256 == 0 && a.K <= 2048 && a.N >= 8192 && a.ldx % 8 == 0 &&
         wide_lds((a.M + 15) / 16, a.K) <= kWideLds;
}

template <int NCH, int RT>
static void launch_wide_rt(const LinArgs& a, int n_tiles, dim3 grid, hipStream_t s) {
  if constexpr (wide_lds(RT, 256 * NCH) <= kWideLds)
    hipLaunchKernelGGL((k_linear_wide<NCH, RT>), grid, dim3(512), 0, s, a, n_tiles);
}

template <int NCH>
static void launch_wide_nch(const LinArgs& a, hipStream_t s) {
  const int n_tiles = (a.N + 15) / 16;
  const dim3 grid((n_tiles + 15) / 16);                      // 8 waves of two tiles each
  switch ((a.M + 15) / 16) {
    case 1: launch_wide_rt<NCH, 1>(a, n_tiles, grid, s); break;
    case 2: launch_wide_rt<NCH, 2>(a, n_tiles, grid, s); break;
    case 3: launch_wide_rt<NCH, 3>(a, n_tiles, grid, s); break;
    default: launch_wide_rt<NCH, 4>(a, n_tiles, grid, s); break;
  }
}

static void launch_wide(const LinArgs& a, hipStream_t s) {
  switch (a.K / 256) {
    case 1: launch_wide_nch<1>(a, s); break;
    case 2: launch_wide_nch<2>(a, s); break;
    case 3: launch_wide_nch<3>(a, s); break;
    case 4: launch_wide_nch<4>(a, s); break;
    case 5: launch_wide_nch<5>(a, s); break;
    case 6: launch_wide_nch<6>(a, s); break;
    case 7: launch_wide_nch<7>(a, s); break;
    default: launch_wide_nch<8>(a, s); break;
  }
}

template <int EPI, class C>
static void launch_gemm(const LinArgs& a, hipStream_t s) {
  const int tm = (a.M + C::BM - 1) / C::BM, tn = (a.N + C::BN - 1) / C::BN;
  hipLaunchKernelGGL((k_gemm<EPI, C>), dim3(xcd_grid(tm * tn)), dim3(C::NT), 0, s, a, tm, tn);
}

#ifndef GEMM_BIG
#define GEMM_BIG GemmCfg<128, 128, 64, 2, 2, 2>
#endif
#ifndef GEMM_MID
#define GEMM_MID GemmCfg<64, 64, 64, 2, 2, 2>
#endif
// Mid tiles over a long reduction (K >= 3072): with one or two workgroups per
// CU the stage wait is the critical path, so four stages are kept in flight
// (measured 24.8 against 31.8 us for 1024 x 1024 x 4096; for K <= 2048 the
// deeper ring's prologue and LDS cost more than it saves).
#ifndef GEMM_MID_DEEP
#define GEMM_MID_DEEP GemmCfg<64, 64, 64, 4, 2, 2>
#endif
using GemmBig = GEMM_BIG;
using GemmMid = GEMM_MID;
using GemmMidDeep = GEMM_MID_DEEP;

template <int EPI>
static hipError_t linear(const LinArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.K <= 0 || a.K % 64) return hipErrorInvalidValue;
  if (EPI != kLinF32 && (a.ldy % 4 || (EPI == kLinSplit && a.ns % 4))) return hipErrorInvalidValue;
  if (a.lng) {
    if (!a.lnb || a.K > 2048 || a.ldx % 8) return hipErrorInvalidValue;
    if (a.M <= 128) {
      launch_skinny_ln<EPI>(a, s);
      return hipGetLastError();
    }
    if (!a.lnout) return hipErrorInvalidValue;
    const int rpw = ln_rows_per_wave(a.K);
    hipLaunchKernelGGL(k_ln_rows, dim3((a.M + rpw - 1) / rpw), dim3(64), 0, s, a.x, a.ldx, a.lng, a.lnb, a.lnout, a.K,
                       a.M, a.K);
    LinArgs n = a;
    n.x = a.lnout;
    n.ldx = a.K;
    n.lng = n.lnb = nullptr;
    return linear<EPI>(n, s);
  }
  if (EPI == kLinF32 && wide_fits(a)) {
    launch_wide(a, s);
  } else if (a.M <= 128) {
    launch_skinny<EPI>(a, s);
  } else if ((size_t)((a.N + GemmBig::BN - 1) / GemmBig::BN) * ((a.M + GemmBig::BM - 1) / GemmBig::BM) >= 256) {
    launch_gemm<EPI, GemmBig>(a, s);
  } else if (a.K >= 3072) {
    launch_gemm<EPI, GemmMidDeep>(a, s);
  } else {
    launch_gemm<EPI, GemmMid>(a, s);
  }
  return hipGetLastError();
}

}  // namespace smem
