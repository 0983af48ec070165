// VALU reader attention: one query per workgroup, split-K over memory pages.
//
// Reader attention (Section 2, "Model"; Appendix A, "Reader"), joint form: a
// query at in-block position t of block J reads, under one softmax,
//   [null row] ++ memory rows of live blocks j < J (ascending j) ++ in-block keys 0..t.
// This kernel is the decode path (one query per sequence, bandwidth bound,
// no MFMA), and also serves fp32 prefill and the fp32 encoder (a reader with
// no memory whose in-block keys are the block itself).
//
// Work decomposition (deterministic): the slot's n_read memory pages are cut
// into splits of pps whole pages (pps depends on n_read only); split index
// nms = ceil(n_read/pps) holds the null row and the in-block keys.  Inside a
// memory split, wave w streams pages w, w+4, ... with its own online-softmax
// state; the four wave states are combined in wave order, and the splits are
// combined in split order by k_merge.  Nothing depends on the batch, on
// physical page numbers or on timing, so equal inputs give equal bits.
//
// Memory page tiles (per page and head): key plane [b][dh] row-major, value
// plane transposed [dh][b].  Key rows are read 16 bytes per lane, LPR lanes
// per row (a wave reads 1 KiB contiguous per instruction); the row dot
// product is finished with xor-shuffles.  Softmax weights go through a
// per-wave LDS row so each lane can weight a 16-byte chunk of the
// transposed value plane (contiguous keys).
//
// SMem+RoPE composite (ROPE = true; Section 3, "SMem composes with RoPE"):
// rows carry no position, so the rotary phases are applied here.  A memory
// key of block j read from block J scores as <R(J) q, R(j') k> with
// j' = max(j, J - W), i.e. the query turned by min(J - j, W) against the
// stored key; the null row is a key of index 0; in-block keys score as
// <R(t) q, R(t') k> with t, t' the in-block offsets.  Values are never
// turned.  Every row of one page shares a turn, so the query is re-turned
// only when the turn changes from one page to the next.
#include "common.h"

namespace smem {

template <typename T, int DH, int B>
struct RCfg {
  static constexpr int E = Chunk<T>::E;   // elements per 16-byte chunk
  static constexpr int LPR = DH / E;      // lanes per key row
  static constexpr int RPL = 64 / LPR;    // key rows per wave load
  static constexpr int KLOADS = B / RPL;  // wave loads per page of keys
  static constexpr int LPV = B / E;       // lanes per transposed value row
  static constexpr int DPL = 64 / LPV;    // value dims per wave load
  static constexpr int VLOADS = DH / DPL; // wave loads per page of values
  static_assert(LPR >= 1 && LPR <= 64 && RPL * LPR == 64 && KLOADS * RPL == B, "key tiling");
  static_assert(LPV >= 1 && LPV <= 64 && DPL * LPV == 64 && VLOADS * DPL == DH, "value tiling");
};

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) x += __shfl_xor(x, o);
  return x;
}

// MEM = false: a launch in which no slot reads a memory page (every
// workgroup runs the null row and in-block keys only, e.g. a model layer's
// self-attention over its in-block cache): the page path is compiled out,
// so the kernel holds fewer registers and more workgroups run at once; the
// arithmetic of the split it runs is the same.
template <typename T, int DH, int B, bool ROPE, bool MEM = true>
__global__ void __launch_bounds__(256) k_reader_valu(ReaderArgs a) {
  using C = RCfg<T, DH, B>;
  constexpr int E = C::E;
  // heads fastest: neighbouring workgroups stream the adjacent head tiles of
  // the same pages
  const int h = blockIdx.x, split = blockIdx.y, qs = blockIdx.z;
  const int slot = qs / a.nq, t = qs % a.nq;
  const int n_read = a.n_read[slot], pps = a.pps[slot];
  const int nms = (n_read + pps - 1) / pps;
  if (split > nms) return;  // whole workgroup

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ float p_sh[4][B];
  __shared__ float wm[4], wl[4];
  __shared__ float wacc[4][DH];

  const int c = lane % C::LPR, rg = lane / C::LPR;
  float qf[E];
  {
    const T* qp = (const T*)a.q + ((size_t)qs * a.H + h) * DH + c * E;
    Chunk<T>::unpack(*(const u32x4*)qp, qf);
#pragma unroll
    for (int e = 0; e < E; ++e) qf[e] *= a.scale_log2;
  }
  [[maybe_unused]] float qb[E];   // the unturned query (rotary phases only)
  if constexpr (ROPE) {
#pragma unroll
    for (int e = 0; e < E; ++e) qb[e] = qf[e];
  }
  float m = -INFINITY, l = 0.f;

  if (MEM && split < nms) {
    // ------------------------------------------------ memory pages of this split
    float acc[C::VLOADS];
#pragma unroll
    for (int v = 0; v < C::VLOADS; ++v) acc[v] = 0.f;
    const int dr = lane / C::LPV, kc = lane % C::LPV;
    const int p0 = split * pps;
    const int p1 = min(n_read, p0 + pps);
    const int32_t* lp = a.live_page + (size_t)a.seq[slot] * a.max_blocks;
    [[maybe_unused]] const int32_t* lb = a.live_blk + (size_t)a.seq[slot] * a.max_blocks;
    [[maybe_unused]] int turned = -1;
    for (int pi = p0 + wave; pi < p1; pi += 4) {
      const int pg = lp[pi];
      if constexpr (ROPE) {
        const int dlt = min(a.qblk[slot] - lb[pi], a.rope_clip);
        if (dlt != turned) {
#pragma unroll
          for (int e = 0; e < E; ++e) qf[e] = qb[e];
          rope_turn<E>(qf, a.rope + (size_t)dlt * DH, c * (E / 2));
          turned = dlt;
        }
      }
      const T* Kt = (const T*)a.pages + page_head_offset(pg, h, a.H, B, DH);
      const T* VT = Kt + B * DH;
      u32x4 kraw[C::KLOADS];
      u32x4 vraw[C::VLOADS];
#pragma unroll
      for (int i = 0; i < C::KLOADS; ++i) kraw[i] = load_stream(Kt + (i * C::RPL + rg) * DH + c * E);
#pragma unroll
      for (int v = 0; v < C::VLOADS; ++v) vraw[v] = load_stream(VT + (v * C::DPL + dr) * B + kc * E);
      float s[C::KLOADS];
#pragma unroll
      for (int i = 0; i < C::KLOADS; ++i) {
        float kf[E];
        Chunk<T>::unpack(kraw[i], kf);
        float x = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) x += qf[e] * kf[e];
        s[i] = x;
      }
#pragma unroll
      for (int i = 0; i < C::KLOADS; ++i) {
#pragma unroll
        for (int o = 1; o < C::LPR; o <<= 1) s[i] += __shfl_xor(s[i], o);
      }
      float mx = s[0];
#pragma unroll
      for (int i = 1; i < C::KLOADS; ++i) mx = fmaxf(mx, s[i]);
#pragma unroll
      for (int o = C::LPR; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const float mn = fmaxf(m, mx);
      const float alpha = exp2w(m - mn);
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < C::KLOADS; ++i) {
        const float p = exp2w(s[i] - mn);
        if (c == 0) {
          p_sh[wave][i * C::RPL + rg] = p;
          ps += p;
        }
      }
      l = l * alpha + ps;
      m = mn;
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      float pv[E];
#pragma unroll
      for (int e = 0; e < E; ++e) pv[e] = p_sh[wave][kc * E + e];
#pragma unroll
      for (int v = 0; v < C::VLOADS; ++v) {
        float vf[E];
        Chunk<T>::unpack(vraw[v], vf);
        float x = acc[v] * alpha;
#pragma unroll
        for (int e = 0; e < E; ++e) x += pv[e] * vf[e];
        acc[v] = x;
      }
      __builtin_amdgcn_wave_barrier();
    }
#pragma unroll
    for (int v = 0; v < C::VLOADS; ++v) {
#pragma unroll
      for (int o = 1; o < C::LPV; o <<= 1) acc[v] += __shfl_xor(acc[v], o);
    }
    l = wave_sum(l);
    if (kc == 0) {
#pragma unroll
      for (int v = 0; v < C::VLOADS; ++v) wacc[wave][v * C::DPL + dr] = acc[v];
    }
    if (lane == 0) { wm[wave] = m; wl[wave] = l; }
  } else {
    // ------------------------------------------------ null row + in-block keys
    float acc2[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc2[e] = 0.f;
    if (a.null_kv != nullptr && wave == 0) {
      const T* nk = (const T*)a.null_kv + (size_t)h * DH + c * E;
      const T* nv = (const T*)a.null_kv + ((size_t)a.H + h) * DH + c * E;
      float kf[E], vf[E];
      Chunk<T>::unpack(*(const u32x4*)nk, kf);
      Chunk<T>::unpack(*(const u32x4*)nv, vf);
      float qn[E];
#pragma unroll
      for (int e = 0; e < E; ++e) qn[e] = qf[e];
      if constexpr (ROPE) rope_turn<E>(qn, a.rope + (size_t)min(a.qblk[slot], a.rope_clip) * DH, c * (E / 2));
      float x = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) x += qn[e] * kf[e];
#pragma unroll
      for (int o = 1; o < C::LPR; o <<= 1) x += __shfl_xor(x, o);
      m = x;
      l = (lane == 0) ? 1.f : 0.f;
      if (rg == 0) {
#pragma unroll
        for (int e = 0; e < E; ++e) acc2[e] = vf[e];
      }
    }
    int n_in;
    const bool decode = a.intra_mode == 2;
    const int pos = decode ? a.aux[slot] : 0;
    if (decode) n_in = (a.k_new != nullptr) ? pos + 1 : 0;
    else if (a.k_in == nullptr) n_in = 0;
    else n_in = (a.intra_mode == 0) ? B : t + 1;
    if constexpr (ROPE) rope_turn<E>(qf, a.rope + (size_t)(decode ? pos : t) * DH, c * (E / 2));
    for (int r0 = wave * C::RPL; r0 < n_in; r0 += 4 * C::RPL) {
      const int r = r0 + rg;
      const bool valid = r < n_in;
      float kf[E], vf[E];
#pragma unroll
      for (int e = 0; e < E; ++e) { kf[e] = 0.f; vf[e] = 0.f; }
      if (valid) {
        const T* ks;
        const T* vs;
        if (decode && r == pos) {
          ks = (const T*)a.k_new + ((size_t)slot * a.H + h) * DH;
          vs = (const T*)a.v_new + ((size_t)slot * a.H + h) * DH;
        } else {
          ks = (const T*)a.k_in + (((size_t)slot * B + r) * a.H + h) * DH;
          vs = (const T*)a.v_in + (((size_t)slot * B + r) * a.H + h) * DH;
        }
        Chunk<T>::unpack(*(const u32x4*)(ks + c * E), kf);
        Chunk<T>::unpack(*(const u32x4*)(vs + c * E), vf);
        if constexpr (ROPE) rope_turn<E>(kf, a.rope + (size_t)r * DH, c * (E / 2));
      }
      float x = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) x += qf[e] * kf[e];
#pragma unroll
      for (int o = 1; o < C::LPR; o <<= 1) x += __shfl_xor(x, o);
      const float sc = valid ? x : -INFINITY;
      float mx = sc;
#pragma unroll
      for (int o = C::LPR; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const float mn = fmaxf(m, mx);       // row r0 is valid, so mn is finite
      const float alpha = exp2w(m - mn);
      const float p = valid ? exp2w(sc - mn) : 0.f;
      l = l * alpha + ((c == 0) ? p : 0.f);
#pragma unroll
      for (int e = 0; e < E; ++e) acc2[e] = acc2[e] * alpha + p * vf[e];
      m = mn;
    }
    if (decode && a.k_cache_w != nullptr && wave == 0 && rg == 0) {
      // write the new token's key/value into the in-block cache at row pos
      const size_t src = ((size_t)slot * a.H + h) * DH + c * E;
      const size_t dst = (((size_t)slot * B + pos) * a.H + h) * DH + c * E;
      *(u32x4*)((T*)a.k_cache_w + dst) = *(const u32x4*)((const T*)a.k_new + src);
      *(u32x4*)((T*)a.v_cache_w + dst) = *(const u32x4*)((const T*)a.v_new + src);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) {
#pragma unroll
      for (int o = C::LPR; o < 64; o <<= 1) acc2[e] += __shfl_xor(acc2[e], o);
    }
    l = wave_sum(l);
    if (rg == 0) {
#pragma unroll
      for (int e = 0; e < E; ++e) wacc[wave][c * E + e] = acc2[e];
    }
    if (lane == 0) { wm[wave] = m; wl[wave] = l; }
  }
  __syncthreads();

  if (tid < DH) {
    const float M = fmaxf(fmaxf(wm[0], wm[1]), fmaxf(wm[2], wm[3]));
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float wgt = (wm[w] == -INFINITY) ? 0.f : exp2w(wm[w] - M);
      L += wgt * wl[w];
      A += wgt * wacc[w][tid];
    }
    if (nms == 0 && !a.intra_partial) {
      const float o = (L > 0.f) ? A / L : 0.f;
      const T ov = from_f32<T>(o);
      ((T*)a.out)[((size_t)qs * a.H + h) * DH + tid] = ov;
      if (a.page_sink != nullptr && a.aux[slot] >= 0) {
        T* kp = (T*)a.page_sink + page_head_offset(a.aux[slot], h, a.H, B, DH);
        kp[t * DH + tid] = ov;
        kp[B * DH + tid * B + t] = ov;
      }
    } else {
      float* part = a.intra_partial ? a.ws + ((size_t)qs * a.H + h) * (DH + 4)
                                    : a.ws + (((size_t)qs * a.H + h) * a.ws_stride + split) * (DH + 4);
      part[tid] = A;
      if (tid == 0) { part[DH] = M; part[DH + 1] = L; }
    }
  }
}

// Merge the splits of one (query row, head) in split order by the running
// rescale of fold_scale / fold_value: the split statistics are loaded in
// parallel, one thread walks them for the per-split scales (kept in LDS) and
// the weight sum, and each thread folds one output dimension over the splits.
template <typename T, int DH>
__global__ void __launch_bounds__(128) k_merge(ReaderArgs a) {
  const int qs = blockIdx.x, h = blockIdx.y;
  const int slot = qs / a.nq;
  const int S = total_splits(a.n_read[slot], a.pps[slot]);
  if (S == 1) return;
  __shared__ float m_sh[kSplitStride];
  __shared__ float l_sh[kSplitStride];
  __shared__ FoldScale c_sh[kSplitStride];
  __shared__ float inv_sh;
  const int tid = threadIdx.x;
  const float* base = a.ws + ((size_t)qs * a.H + h) * a.ws_stride * (DH + 4);
  if (tid < S) {
    m_sh[tid] = base[(size_t)tid * (DH + 4) + DH];
    l_sh[tid] = base[(size_t)tid * (DH + 4) + DH + 1];
  }
  __syncthreads();
  if (tid == 0) {
    float M = m_sh[0], L = l_sh[0];
    for (int k = 1; k < S; ++k) {
      const FoldScale c = fold_scale(M, m_sh[k]);
      c_sh[k] = c;
      L = fold_value(L, c, l_sh[k]);
    }
    inv_sh = (L > 0.f) ? 1.f / L : 0.f;
  }
  __syncthreads();
  for (int d = tid; d < DH; d += 128) {
    float A = base[d];
#pragma unroll 8
    for (int k = 1; k < S; ++k) A = fold_value(A, c_sh[k], base[(size_t)k * (DH + 4) + d]);
    ((T*)a.out)[((size_t)qs * a.H + h) * DH + d] = from_f32<T>(A * inv_sh);
  }
}

template <typename T>
static hipError_t launch_merge_t(int dh, const ReaderArgs& a, hipStream_t s) {
  const dim3 grid(a.n_slots * a.nq, a.H);
  if (dh == 32) hipLaunchKernelGGL((k_merge<T, 32>), grid, dim3(128), 0, s, a);
  else if (dh == 64) hipLaunchKernelGGL((k_merge<T, 64>), grid, dim3(128), 0, s, a);
  else if (dh == 128) hipLaunchKernelGGL((k_merge<T, 128>), grid, dim3(128), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_merge(int dtype, int dh, const ReaderArgs& a, hipStream_t s) {
  return dtype == F32 ? launch_merge_t<float>(dh, a, s) : launch_merge_t<uint16_t>(dh, a, s);
}

template <typename T, int DH, int B>
static hipError_t launch_rv(const ReaderArgs& a, hipStream_t s) {
  int max_split = 0;
  for (int i = 0; i < a.n_slots; ++i) {
    const int ns = total_splits(a.n_read[i], a.pps[i]) - 1;
    if (ns > max_split) max_split = ns;
  }
  dim3 grid(a.H, max_split + 1, a.n_slots * a.nq);
  if (a.rope != nullptr)
    hipLaunchKernelGGL((k_reader_valu<T, DH, B, true>), grid, dim3(256), 0, s, a);
  else if (max_split == 0)   // no slot reads a memory page
    hipLaunchKernelGGL((k_reader_valu<T, DH, B, false, false>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_reader_valu<T, DH, B, false>), grid, dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || max_split == 0) return e;
  return launch_merge(sizeof(T) == 4 ? F32 : BF16, DH, a, s);
}

template <typename T, int DH>
static hipError_t launch_rv_b(int b, const ReaderArgs& a, hipStream_t s) {
  if (b == 16) return launch_rv<T, DH, 16>(a, s);
  if (b == 64) return launch_rv<T, DH, 64>(a, s);
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t launch_rv_d(int b, int dh, const ReaderArgs& a, hipStream_t s) {
  if (dh == 32) return launch_rv_b<T, 32>(b, a, s);
  if (dh == 64) return launch_rv_b<T, 64>(b, a, s);
  if (dh == 128) return launch_rv_b<T, 128>(b, a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_reader_valu(int dtype, int b, int dh, const ReaderArgs& a, hipStream_t s) {
  if (a.n_slots <= 0) return hipSuccess;
  if (dtype == F32) return launch_rv_d<float>(b, dh, a, s);
  return launch_rv_d<uint16_t>(b, dh, a, s);
}

}  // namespace smem
