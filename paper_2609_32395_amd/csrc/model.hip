// The whole SMem model at given weights (Section 2, "Model"; Appendix A):
// the encoder stack producing memory rows, one key/value store per reader
// layer, the reader stack and the output head, driven from the host on the
// caller's stream.  Attention runs on the library's kernels (block-local
// encoder kernel for the encoder and the readers' self-attention, the
// block-skip reader for their cross-attention); the linear maps run on the
// kernels of linear.h, LayerNorm and the embedding on the kernels below.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <set>
#include <vector>

#include "attn_ring.h"
#include "common.h"
#include "linear.h"
#include "smem.h"

namespace smem {

struct EmbArgs {
  const int32_t* tokens;   // [rows]
  const uint16_t* tok_emb; // [vocab][d]
  const uint16_t* pos_emb; // [n_pos][d] or NULL
  uint16_t* x;             // [rows][d]
  int32_t rows, d, b, vocab, slots;
  int32_t per_row;         // 0: rows are whole blocks (row r: block blk[r / b], offset r % b);
                           // 1: one row per entry (row r: block blk[r], offset off[r])
  int32_t blk[kMaxSlots];  // block index of each b-row group, or of each row
  int32_t off[kMaxSlots];  // in-block offset of each row (per_row)
};

// x[r] = tok_emb[token] + pos_emb[min(block, slots-1)*b + offset]; one wave per
// row.  A token id outside [0, vocab) reads row 0 (it cannot read past the table).
__global__ void __launch_bounds__(256) k_embed(EmbArgs a) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= a.rows) return;
  int tok = a.tokens[r];
  if (tok < 0 || tok >= a.vocab) tok = 0;
  const int t = a.per_row ? a.off[r] : r % a.b;
  const int pos = min(a.blk[a.per_row ? r : r / a.b], a.slots - 1) * a.b + t;
  for (int c = lane * 8; c < a.d; c += 512) {
    float e[8], p[8];
    Chunk<uint16_t>::unpack(*(const u32x4*)(a.tok_emb + (size_t)tok * a.d + c), e);
    if (a.pos_emb) {
      Chunk<uint16_t>::unpack(*(const u32x4*)(a.pos_emb + (size_t)pos * a.d + c), p);
#pragma unroll
      for (int i = 0; i < 8; ++i) e[i] += p[i];
    }
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f32_to_bf16_bits(e[2 * i]) | ((uint32_t)f32_to_bf16_bits(e[2 * i + 1]) << 16);
    *(u32x4*)(a.x + (size_t)r * a.d + c) = u32x4{w[0], w[1], w[2], w[3]};
  }
}


// ---------------------------------------------------------------- fused self-attention

// The attention part of a self-attention sub-layer for d_h = 32 (Section 2,
// "Model"; Appendix A, "Encoder" and "Reader"): o = Attn(q, k, v) per
// (block, head) with q | k | v = LN(x) W_qkv^T, in one workgroup per
// (block, head) instead of a linear-map launch followed by the block-local
// attention launch.  Two waves per reduction chunk (256 wide), 32 rows each,
// compute the chunk's share of the head's 64 x 96 tile (its q, k and v
// columns) exactly as the few-row map computes a chunk: the rows normalized in registers with the
// statistics met in LDS in the LayerNorm's fixed order, one 16x16x32 MFMA
// per 32-wide step from zero, the W tile as the row operand; the chunk sums
// are added in chunk order from zero and rounded to bf16 into LDS.  Four
// waves then run the block-local attention kernel's steps on that tile
// (the same helpers in the same order), so q, k, v and the output carry the
// bits of the unfused pair.  PRE: x already holds LN(x) (many rows: one
// LayerNorm pass serves every head) and the normalization is skipped.
struct QkvAttnArgs {
  const uint16_t* x;    // [n_blocks * 64][d]: rows, or normalized rows (PRE)
  const uint16_t* lng;  // LayerNorm gain and shift [d] (not read with PRE)
  const uint16_t* lnb;
  const uint16_t* w;    // [3d][d]: q rows [0, d), k rows [d, 2d), v rows [2d, 3d)
  uint16_t* out;        // [n_blocks * 64][d]: head h in columns [32 h, 32 h + 32)
  float scale_log2;     // log2(e) / sqrt(d_h)
};

constexpr int kQkvDh = 32, kQkvCols = 3 * kQkvDh, kQkvMaxChunks = 4;

template <int NC, bool CAUSAL, bool PRE>
__global__ void __launch_bounds__(512) k_qkv_attn(QkvAttnArgs a) {
  // wave w < 2 NC: chunk w / 2, row tiles 2 (w % 2) and 2 (w % 2) + 1
  constexpr int DH = kQkvDh, NCOL = kQkvCols, CT = NCOL / 16, D = 256 * NC, U = 4, RT = 2;
  using R = PageRing<DH>;
  __shared__ __attribute__((aligned(1024))) uint8_t T[R::TILE];
  __shared__ __attribute__((aligned(16))) float part[NC * BT * NCOL];   // [chunk][row][column] sums
  __shared__ __attribute__((aligned(16))) uint16_t stage[BT * NCOL];    // q | k | v rows, bf16
  __shared__ __attribute__((aligned(16))) uint16_t gb[PRE ? 8 : 2 * D]; // gain, then shift
  __shared__ float st0[PRE ? 1 : NC * BT], st1[PRE ? 1 : NC * BT];      // [chunk][row] statistics
  const int h = blockIdx.x, blk = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = w >> 1, r0 = (w & 1) * RT * 16;                        // chunk, first row
  const int kofs = (lane >> 4) * 8;
  const bool worker = c < NC;

  u32x4 X[8][RT], B[U][CT];
  const uint16_t* wr[CT];
  if (worker) {
    const uint16_t* xr = a.x + ((size_t)blk * BT + r0 + (lane & 15)) * D + c * 256 + kofs;
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int i = 0; i < RT; ++i) X[t][i] = *(const u32x4*)(xr + (size_t)i * 16 * D + t * 32);
#pragma unroll
    for (int j = 0; j < CT; ++j)
      wr[j] = a.w + ((size_t)(j >> 1) * D + h * DH + (j & 1) * 16 + (lane & 15)) * D + c * 256 + kofs;
#pragma unroll
    for (int t = 0; t < U; ++t)
#pragma unroll
      for (int j = 0; j < CT; ++j) B[t][j] = *(const u32x4*)(wr[j] + t * 32);
  }
  if constexpr (!PRE) {
    const int q8 = tid * 8;
    if (q8 < D) {
      *(u32x4*)(gb + q8) = *(const u32x4*)(a.lng + q8);
      *(u32x4*)(gb + D + q8) = *(const u32x4*)(a.lnb + q8);
    }
    float mean[RT], rstd[RT];
    if (worker) {
#pragma unroll
      for (int i = 0; i < RT; ++i) {
        float v = 0.f;
#pragma unroll
        for (int t = 0; t < 8; ++t) v = ln_sum8(X[t][i], v);
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (lane < 16) st0[c * BT + r0 + i * 16 + lane] = v;
      }
      opaque(X);
    }
    __syncthreads();
    if (worker) {
#pragma unroll
      for (int i = 0; i < RT; ++i) {
        float tot = 0.f;
        for (int q = 0; q < NC; ++q) tot += st0[q * BT + r0 + i * 16 + (lane & 15)];
        mean[i] = tot / D;
        float v = 0.f;
#pragma unroll
        for (int t = 0; t < 8; ++t) v = ln_sq8(X[t][i], mean[i], v);
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (lane < 16) st1[c * BT + r0 + i * 16 + lane] = v;
      }
      opaque(X);
    }
    __syncthreads();
    if (worker) {
#pragma unroll
      for (int i = 0; i < RT; ++i) {
        float tot = 0.f;
        for (int q = 0; q < NC; ++q) tot += st1[q * BT + r0 + i * 16 + (lane & 15)];
        rstd[i] = ln_rstd(tot, D);
      }
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int k = c * 256 + t * 32 + kofs;
        const u32x4 g8 = *(const u32x4*)(gb + k), b8 = *(const u32x4*)(gb + D + k);
#pragma unroll
        for (int i = 0; i < RT; ++i) X[t][i] = ln_apply8(X[t][i], g8, b8, mean[i], rstd[i]);
      }
    }
  }
  if (worker) {
    f32x4 acc[RT][CT];
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int j = 0; j < CT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 8; ++t) {
#pragma unroll
      for (int i = 0; i < RT; ++i)
#pragma unroll
        for (int j = 0; j < CT; ++j) acc[i][j] = mfma16(B[t % U][j], X[t][i], acc[i][j]);
      if (t + U < 8) {
#pragma unroll
        for (int j = 0; j < CT; ++j) B[t % U][j] = *(const u32x4*)(wr[j] + (t + U) * 32);
      }
    }
    // lane: row r0 + i*16 + l%16, columns j*16 + 4 (l/16) .. +3
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int j = 0; j < CT; ++j)
        *(f32x4*)(part + (c * BT + r0 + i * 16 + (lane & 15)) * NCOL + j * 16 + 4 * (lane >> 4)) = acc[i][j];
  }
  __syncthreads();
  for (int q = tid; q < BT * NCOL / 4; q += 512) {
    const int row = q / (NCOL / 4), c0 = (q % (NCOL / 4)) * 4;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    for (int ch = 0; ch < NC; ++ch) v += *(const f32x4*)(part + (ch * BT + row) * NCOL + c0);
    *(u32x2*)(stage + row * NCOL + c0) =
        u32x2{(uint32_t)f32_to_bf16_bits(v[0]) | ((uint32_t)f32_to_bf16_bits(v[1]) << 16),
              (uint32_t)f32_to_bf16_bits(v[2]) | ((uint32_t)f32_to_bf16_bits(v[3]) << 16)};
  }
  __syncthreads();
  // block-local attention: waves 0..3 take 16 query rows each
  intra_ring_store<DH, 512>(T, stage + DH, stage + 2 * DH, NCOL, tid);
  __syncthreads();
  if (w >= 4) return;                    // no barrier follows
  const int qrow = w * 16 + (lane & 15);
  bf16x8 qf[DH / 32];
  load_q<DH>(qf, stage + w * 16 * NCOL, NCOL, lane);
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
  uint16_t* orow = a.out + ((size_t)blk * BT + qrow) * D + h * DH;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    const int d0 = dt * 16 + (lane >> 4) * 4;
    uint16_t r4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) r4[i] = f32_to_bf16_bits(o[dt][i] * inv);
    *(u32x2*)(orow + d0) = u32x2{(uint32_t)r4[0] | ((uint32_t)r4[1] << 16), (uint32_t)r4[2] | ((uint32_t)r4[3] << 16)};
  }
}

template <int NC>
static void launch_qkv_attn_nc(const QkvAttnArgs& a, int H, int nb, bool causal, bool pre, hipStream_t s) {
  const dim3 grid(H, nb);
  if (causal) {
    if (pre) hipLaunchKernelGGL((k_qkv_attn<NC, true, true>), grid, dim3(512), 0, s, a);
    else hipLaunchKernelGGL((k_qkv_attn<NC, true, false>), grid, dim3(512), 0, s, a);
  } else {
    if (pre) hipLaunchKernelGGL((k_qkv_attn<NC, false, true>), grid, dim3(512), 0, s, a);
    else hipLaunchKernelGGL((k_qkv_attn<NC, false, false>), grid, dim3(512), 0, s, a);
  }
}

// d = 32 H with d a multiple of 256 up to 1024 (the LDS of the chunk sums
// bounds the chunk count); nb blocks of 64 rows.
bool qkv_attn_fits(int d, int H) { return d == kQkvDh * H && d % 256 == 0 && d / 256 <= kQkvMaxChunks; }

hipError_t launch_qkv_attn(const QkvAttnArgs& a, int d, int H, int nb, bool causal, bool pre, hipStream_t s) {
  if (!qkv_attn_fits(d, H) || nb <= 0 || nb > 65535) return hipErrorInvalidValue;
  switch (d / 256) {
    case 1: launch_qkv_attn_nc<1>(a, H, nb, causal, pre, s); break;
    case 2: launch_qkv_attn_nc<2>(a, H, nb, causal, pre, s); break;
    case 3: launch_qkv_attn_nc<3>(a, H, nb, causal, pre, s); break;
    default: launch_qkv_attn_nc<4>(a, H, nb, causal, pre, s); break;
  }
  return hipGetLastError();
}

}  // namespace smem

using namespace smem;

// ---------------------------------------------------------------- host runtime

struct smem_model {
  smem_model_desc d;
  std::vector<const uint16_t*> W;
  std::vector<smem_store*> stores;   // one per reader layer (key/value layers)
  smem_store* rows = nullptr;        // row plane: the memory rows, shared by every reader layer
  smem_store* blockless = nullptr;   // row plane: an empty store for the decode's in-block self-attention
  char* pool = nullptr;
  uint16_t *x = nullptr, *h = nullptr, *q = nullptr, *k = nullptr, *v = nullptr, *o = nullptr, *f = nullptr;
  uint16_t* null_kv = nullptr;       // [D][2][d]
  uint16_t* cache = nullptr;         // decode: in-block keys/values [D][2][n_seq][b][d]
};

namespace {

smem_status mfail(smem_status st, const char* msg) { return set_error(st, msg); }

size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

int n_weights(const smem_model_desc* d) { return 2 + 8 * d->E + 3 + 14 * d->D + 3; }

bool desc_ok(const smem_model_desc* d) {
  if (!d) return false;
  if (d->row_plane != 0 && d->row_plane != 1) return false;
  if (d->row_plane && !(d->d == 512 || d->d == 768 || d->d == 1024 || d->d == 2048)) return false;
  if (d->E < 0 || d->D < 1 || d->b != 64 || d->H < 1 || !(d->dh == 32 || d->dh == 64 || d->dh == 128)) return false;
  if (d->d != d->H * d->dh || d->d % 64 || d->d > 2048) return false;
  if (d->vocab < 1 || d->n_pos < 0 || d->n_pos % d->b) return false;
  if (d->n_seq < 1 || d->max_blocks < 1 || d->n_pages < 1) return false;
  if (d->max_tokens < d->b || d->max_tokens % d->b || d->max_tokens > kMaxSlots * d->b) return false;
  return true;
}

smem_store_desc store_desc(const smem_model_desc* d) {
  return smem_store_desc{d->n_seq, d->max_blocks, d->n_pages, d->b, d->H, d->dh, SMEM_BF16};
}
// Row plane: the rows, and a store that holds no block (a decode read of
// block 0 through it is the in-block self-attention alone).
smem_rows_desc rows_desc(const smem_model_desc* d) {
  return smem_rows_desc{d->n_seq, d->max_blocks, d->n_pages, d->b, d->d, SMEM_BF16};
}
smem_store_desc blockless_desc(const smem_model_desc* d) {
  return smem_store_desc{d->n_seq, 1, 1, d->b, d->H, d->dh, SMEM_BF16};
}

struct Layout {
  size_t store_bytes, off_ws, off_null, off_cache, total;
  size_t rows_bytes;    // row plane: the row store, then the blockless store (store_bytes)
};

bool layout(const smem_model_desc* d, Layout* L) {
  if (!desc_ok(d)) return false;
  size_t off;
  if (d->row_plane) {
    const smem_rows_desc rd = rows_desc(d);
    const smem_store_desc bd = blockless_desc(d);
    L->rows_bytes = a256(smem_rows_bytes(&rd));
    L->store_bytes = a256(smem_store_bytes(&bd));
    if (L->rows_bytes == 0 || L->store_bytes == 0) return false;
    off = L->rows_bytes + L->store_bytes;
  } else {
    const smem_store_desc sd = store_desc(d);
    L->rows_bytes = 0;
    L->store_bytes = a256(smem_store_bytes(&sd));
    if (L->store_bytes == 0) return false;
    off = L->store_bytes * d->D;
  }
  L->off_ws = off;
  off += a256((size_t)d->max_tokens * d->d * 2) * 6 + a256((size_t)d->max_tokens * 4 * d->d * 2);
  L->off_null = off;
  off += a256((size_t)d->D * 2 * d->d * 2);
  L->off_cache = off;
  off += a256((size_t)d->D * 2 * d->n_seq * d->b * d->d * 2);
  L->total = off;
  return true;
}

// weight pointers by role
struct Wts {
  const smem_model* m;
  const uint16_t* at(int i) const { return m->W[i]; }
  const uint16_t* tok() const { return at(0); }
  const uint16_t* pos() const { return m->d.n_pos ? at(1) : nullptr; }
  const uint16_t* enc(int l, int i) const { return at(2 + 8 * l + i); }
  int base_mem() const { return 2 + 8 * m->d.E; }
  const uint16_t* mem_g() const { return at(base_mem()); }
  const uint16_t* mem_b() const { return at(base_mem() + 1); }
  const uint16_t* null_row() const { return at(base_mem() + 2); }
  const uint16_t* dec(int l, int i) const { return at(base_mem() + 3 + 14 * l + i); }
  int base_fin() const { return base_mem() + 3 + 14 * m->d.D; }
  const uint16_t* fin_g() const { return at(base_fin()); }
  const uint16_t* fin_b() const { return at(base_fin() + 1); }
  const uint16_t* head() const { return at(base_fin() + 2); }
};
enum { E_LN1G, E_LN1B, E_QKV, E_O, E_LN2G, E_LN2B, E_FF1, E_FF2 };
enum { R_LN1G, R_LN1B, R_QKV, R_O, R_LN2G, R_LN2B, R_Q, R_K, R_V, R_OC, R_LN3G, R_LN3B, R_FF1, R_FF2 };

hipError_t lnorm(const uint16_t* x, const uint16_t* g, const uint16_t* b, uint16_t* y, int rows, int d, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int rpw = ln_rows_per_wave(d);
  hipLaunchKernelGGL(k_ln_rows, dim3((rows + rpw - 1) / rpw), dim3(64), 0, s, x, d, g, b, y, d, rows, d);
  return hipGetLastError();
}

LinArgs lin(const uint16_t* x, int ldx, const uint16_t* w, int M, int N, int K, uint16_t* y, int ldy) {
  LinArgs a;
  memset(&a, 0, sizeof a);
  a.x = x; a.ldx = ldx; a.w = w; a.w2 = w; a.n2 = N;
  a.M = M; a.N = N; a.K = K; a.y = y; a.ldy = ldy;
  return a;
}

// y = LN(x) W^T: the few-row maps normalize their own rows; many rows go
// through the LayerNorm kernel into h first.
LinArgs lin_ln(const smem_model* m, const uint16_t* g, const uint16_t* b, const uint16_t* w, int M, int N,
               uint16_t* y, int ldy) {
  LinArgs a = lin(m->x, m->d.d, w, M, N, m->d.d, y, ldy);
  a.lng = g; a.lnb = b; a.lnout = m->h;
  return a;
}

#define MCHECK(expr, what)                                   \
  do {                                                       \
    hipError_t e_ = (expr);                                  \
    if (e_ != hipSuccess) return mfail(SMEM_EHIP, what);     \
  } while (0)
#define MSTATUS(expr)                                        \
  do {                                                       \
    smem_status r_ = (expr);                                 \
    if (r_ != SMEM_OK) return r_;                            \
  } while (0)

// embed one chunk of nb blocks (tokens [nb*b] on the device) into m->x
smem_status embed(smem_model* m, int nb, const int32_t* blocks, const int32_t* tokens, hipStream_t s) {
  const auto& d = m->d;
  Wts w{m};
  EmbArgs a;
  memset(&a, 0, sizeof a);
  a.tokens = tokens; a.tok_emb = w.tok(); a.pos_emb = w.pos(); a.x = m->x;
  a.rows = nb * d.b; a.d = d.d; a.b = d.b; a.vocab = d.vocab; a.slots = d.n_pos ? d.n_pos / d.b : 1;
  for (int i = 0; i < nb; ++i) a.blk[i] = blocks[i];
  hipLaunchKernelGGL(k_embed, dim3((a.rows + 3) / 4), dim3(256), 0, s, a);
  MCHECK(hipGetLastError(), "embedding");
  return SMEM_OK;
}

// x += attention-sublayer / feed-forward sublayer helpers
smem_status ffn(smem_model* m, int rows, const uint16_t* g, const uint16_t* b, const uint16_t* w1, const uint16_t* w2,
                hipStream_t s) {
  const int D = m->d.d;
  MCHECK(linear<kLinGelu>(lin_ln(m, g, b, w1, rows, 4 * D, m->f, 4 * D), s), "ffn up");
  LinArgs a = lin(m->f, 4 * D, w2, rows, D, 4 * D, m->x, D);
  a.res = m->x;
  MCHECK(linear<kLinResid>(a, s), "ffn down");
  return SMEM_OK;
}

// The attention part of a self-attention sub-layer: out = Attn(q, k, v) per
// (block, head) with q | k | v = LN(x) W_qkv^T.  path 1 (also path 0, the
// model's choice): the q|k|v map (its few-row or tiled kernel) into q, k, v,
// then the block-local attention launch; path 2: the fused kernel (d_h = 32,
// d <= 1024), whose rows above 128 are normalized by one LayerNorm pass into
// hn first.  Both paths give the same bits.  The fused kernel measured slower
// at every block count: a workgroup per (block, head) pulls the head's
// weights and the block's rows through one CU, where the map spreads them
// over hundreds of workgroups, and at many blocks its 64 x 96 tile re-reads
// the weights per block.
smem_status attn_sublayer(int nb, int d, int H, const uint16_t* x, const uint16_t* g, const uint16_t* b,
                          const uint16_t* wqkv, int mask, int path, uint16_t* out, uint16_t* hn, uint16_t* q,
                          uint16_t* k, uint16_t* v, hipStream_t s) {
  const int rows = nb * BT;
  if (path == 2) {
    const bool pre = rows > 128;
    if (pre) MCHECK(lnorm(x, g, b, hn, rows, d, s), "self-attention layernorm");
    QkvAttnArgs f;
    f.x = pre ? hn : x;
    f.lng = g; f.lnb = b; f.w = wqkv; f.out = out;
    f.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)kQkvDh));
    MCHECK(launch_qkv_attn(f, d, H, nb, mask == SMEM_MASK_CAUSAL, pre, s), "fused q|k|v and self-attention");
    return SMEM_OK;
  }
  LinArgs a = lin(x, d, wqkv, rows, 3 * d, d, q, d);
  a.lng = g; a.lnb = b; a.lnout = hn;
  a.y1 = k; a.y2 = v; a.ns = d;
  MCHECK(linear<kLinSplit>(a, s), "qkv");
  const smem_attn_desc shape{BT, H, d / H, SMEM_BF16};
  return smem_encode_blocks(nullptr, &shape, nb, nullptr, nullptr, q, k, v, out, mask, s);
}

smem_status self_attn(smem_model* m, int rows, int nb, const uint16_t* g, const uint16_t* b, const uint16_t* wqkv,
                      const uint16_t* wo, int mask, hipStream_t s) {
  const int D = m->d.d;
  MSTATUS(attn_sublayer(nb, D, m->d.H, m->x, g, b, wqkv, mask, 0, m->o, m->h, m->q, m->k, m->v, s));
  LinArgs o = lin(m->o, D, wo, rows, D, D, m->x, D);
  o.res = m->x;
  MCHECK(linear<kLinResid>(o, s), "attention out");
  return SMEM_OK;
}

// Reader stack over one chunk of nb query blocks (rows = nb*b <= max_tokens).
// With logits, the final LayerNorm and the head run on chunk rows [h0, rows)
// and logits row 0 is chunk row h0; without, they are skipped.
smem_status read_chunk(smem_model* m, int seq, int nb, const int32_t* qblk, const int32_t* tokens, float* logits,
                       int h0, hipStream_t s) {
  const auto& d = m->d;
  Wts w{m};
  const int rows = nb * d.b, D = d.d;
  MSTATUS(embed(m, nb, qblk, tokens, s));
  std::vector<int32_t> seqs(nb, seq);
  for (int l = 0; l < d.D; ++l) {
    MSTATUS(self_attn(m, rows, nb, w.dec(l, R_LN1G), w.dec(l, R_LN1B), w.dec(l, R_QKV), w.dec(l, R_O),
                      SMEM_MASK_CAUSAL, s));
    // cross-attention into the memory of strictly earlier blocks, with the null row
    MCHECK(linear<kLinStore>(lin_ln(m, w.dec(l, R_LN2G), w.dec(l, R_LN2B), w.dec(l, R_Q), rows, D, m->q, D), s),
           "cross-attention query");
    MSTATUS(smem_reader_prefill_block(m->stores[l], nb, seqs.data(), qblk, m->q, nullptr, nullptr,
                                      m->null_kv + (size_t)l * 2 * D, m->o, s));
    LinArgs o = lin(m->o, D, w.dec(l, R_OC), rows, D, D, m->x, D);
    o.res = m->x;
    MCHECK(linear<kLinResid>(o, s), "cross-attention out");
    MSTATUS(ffn(m, rows, w.dec(l, R_LN3G), w.dec(l, R_LN3B), w.dec(l, R_FF1), w.dec(l, R_FF2), s));
  }
  if (!logits) return SMEM_OK;
  const int hr = rows - h0;
  MCHECK(lnorm(m->x + (size_t)h0 * D, w.fin_g(), w.fin_b(), m->h + (size_t)h0 * D, hr, D, s), "final layernorm");
  LinArgs hd = lin(m->h + (size_t)h0 * D, D, w.head(), hr, d.vocab, D, nullptr, d.vocab);
  hd.yf = logits;
  MCHECK(linear<kLinF32>(hd, s), "output head");
  return SMEM_OK;
}

// One decode step for sequences first .. first + n - 1 (n <= kMaxSlots):
// rows are single tokens; each reader layer's self-attention reads the
// sequence's in-block cache (the new key/value written at pos first), its
// cross-attention the memory of the live blocks below J with the null row.
smem_status decode_chunk(smem_model* m, int first, int n, const int32_t* qblk, const int32_t* pos,
                         const int32_t* tokens, float* logits, hipStream_t s) {
  const auto& d = m->d;
  Wts w{m};
  const int D = d.d;
  {
    EmbArgs e;
    memset(&e, 0, sizeof e);
    e.tokens = tokens; e.tok_emb = w.tok(); e.pos_emb = w.pos(); e.x = m->x;
    e.rows = n; e.d = D; e.b = d.b; e.vocab = d.vocab; e.slots = d.n_pos ? d.n_pos / d.b : 1; e.per_row = 1;
    for (int i = 0; i < n; ++i) {
      e.blk[i] = qblk[i];
      e.off[i] = pos[i];
    }
    hipLaunchKernelGGL(k_embed, dim3((n + 3) / 4), dim3(256), 0, s, e);
    MCHECK(hipGetLastError(), "embedding");
  }
  std::vector<int32_t> seqs(n), zero(n, 0);
  for (int i = 0; i < n; ++i) seqs[i] = first + i;
  const size_t plane = (size_t)d.n_seq * d.b * D;              // one layer's key (or value) cache
  for (int l = 0; l < d.D; ++l) {
    uint16_t* kc = m->cache + (size_t)l * 2 * plane + (size_t)first * d.b * D;
    uint16_t* vc = kc + plane;
    // self-attention over the block's cached tokens 0..pos
    LinArgs a = lin_ln(m, w.dec(l, R_LN1G), w.dec(l, R_LN1B), w.dec(l, R_QKV), n, 3 * D, m->q, D);
    a.y1 = m->k; a.y2 = m->v; a.ns = D;
    MCHECK(linear<kLinSplit>(a, s), "qkv");
    smem_store* sa = m->d.row_plane ? m->blockless : m->stores[l];
    MSTATUS(smem_reader_decode(sa, n, seqs.data(), zero.data(), pos, m->q, m->k, m->v, kc, vc, nullptr, m->o, s));
    LinArgs o = lin(m->o, D, w.dec(l, R_O), n, D, D, m->x, D);
    o.res = m->x;
    MCHECK(linear<kLinResid>(o, s), "attention out");
    // cross-attention into the memory of strictly earlier blocks, with the null row
    MCHECK(linear<kLinStore>(lin_ln(m, w.dec(l, R_LN2G), w.dec(l, R_LN2B), w.dec(l, R_Q), n, D, m->q, D), s),
           "cross-attention query");
    if (m->d.row_plane) {
      // the shared rows through this layer's key and value maps (folded into
      // the query and the output), the null row mapped once at creation
      const smem_rows_layer layer{d.H, d.dh, w.dec(l, R_K), w.dec(l, R_V), nullptr, m->null_kv + (size_t)l * 2 * D};
      MSTATUS(smem_reader_decode_rows(m->rows, &layer, n, seqs.data(), qblk, nullptr, m->q, nullptr, nullptr,
                                      nullptr, nullptr, m->o, s));
    } else {
      MSTATUS(smem_reader_decode(m->stores[l], n, seqs.data(), qblk, pos, m->q, nullptr, nullptr, nullptr, nullptr,
                                 m->null_kv + (size_t)l * 2 * D, m->o, s));
    }
    LinArgs oc = lin(m->o, D, w.dec(l, R_OC), n, D, D, m->x, D);
    oc.res = m->x;
    MCHECK(linear<kLinResid>(oc, s), "cross-attention out");
    MSTATUS(ffn(m, n, w.dec(l, R_LN3G), w.dec(l, R_LN3B), w.dec(l, R_FF1), w.dec(l, R_FF2), s));
  }
  MCHECK(lnorm(m->x, w.fin_g(), w.fin_b(), m->h, n, D, s), "final layernorm");
  LinArgs hd = lin(m->h, D, w.head(), n, d.vocab, D, nullptr, d.vocab);
  hd.yf = logits;
  MCHECK(linear<kLinF32>(hd, s), "output head");
  return SMEM_OK;
}

}  // namespace

extern "C" {

size_t smem_model_bytes(const smem_model_desc* desc) {
  Layout L;
  return layout(desc, &L) ? L.total : 0;
}

int32_t smem_model_n_weights(const smem_model_desc* desc) { return desc_ok(desc) ? n_weights(desc) : 0; }

smem_status smem_model_create(const smem_model_desc* desc, const void* const* weights, void* dev_pool,
                              size_t pool_bytes, hipStream_t s, smem_model** out) {
  if (!out) return mfail(SMEM_EINVAL, "out is NULL");
  *out = nullptr;
  Layout L;
  if (!layout(desc, &L))
    return mfail(SMEM_EINVAL, "invalid model descriptor (b = 64; dh in {32,64,128}; d = H*dh, a multiple of 64, "
                              "<= 2048; n_pos a multiple of b; max_tokens a multiple of b, <= 128*b)");
  if (!weights || !dev_pool) return mfail(SMEM_EINVAL, "weights and dev_pool are required");
  if (((uintptr_t)dev_pool & 255u) != 0) return mfail(SMEM_EINVAL, "dev_pool must be 256-byte aligned");
  if (pool_bytes < L.total) return mfail(SMEM_ENOMEM, "pool too small for the model");
  const int nw = n_weights(desc);
  for (int i = 0; i < nw; ++i) {
    if (i == 1 && desc->n_pos == 0) continue;
    if (!weights[i] || ((uintptr_t)weights[i] & 15u)) return mfail(SMEM_EINVAL, "a weight pointer is NULL or not 16-byte aligned");
  }
  smem_model* m = new (std::nothrow) smem_model();
  if (!m) return mfail(SMEM_ENOMEM, "host allocation failed");
  m->d = *desc;
  m->pool = (char*)dev_pool;
  for (int i = 0; i < nw; ++i) m->W.push_back((const uint16_t*)weights[i]);
  if (desc->row_plane) {
    const smem_rows_desc rd = rows_desc(desc);
    const smem_store_desc bd = blockless_desc(desc);
    smem_status r = smem_rows_create(&rd, m->pool, L.rows_bytes, s, &m->rows);
    if (r == SMEM_OK) r = smem_store_create(&bd, m->pool + L.rows_bytes, L.store_bytes, s, &m->blockless);
    if (r != SMEM_OK) {
      smem_model_destroy(m);
      return r;
    }
  } else {
    const smem_store_desc sd = store_desc(desc);
    for (int l = 0; l < desc->D; ++l) {
      smem_store* st = nullptr;
      smem_status r = smem_store_create(&sd, m->pool + L.store_bytes * l, L.store_bytes, s, &st);
      if (r != SMEM_OK) {
        smem_model_destroy(m);
        return r;
      }
      m->stores.push_back(st);
    }
  }
  const size_t T = desc->max_tokens, D = desc->d;
  char* ws = m->pool + L.off_ws;
  uint16_t** bufs[6] = {&m->x, &m->h, &m->q, &m->k, &m->v, &m->o};
  for (int i = 0; i < 6; ++i) {
    *bufs[i] = (uint16_t*)ws;
    ws += a256(T * D * 2);
  }
  m->f = (uint16_t*)ws;
  m->null_kv = (uint16_t*)(m->pool + L.off_null);
  m->cache = (uint16_t*)(m->pool + L.off_cache);
  // the null row through every reader layer's key and value maps, once
  Wts w{m};
  for (int l = 0; l < desc->D; ++l) {
    LinArgs a = lin(w.null_row(), (int)D, w.dec(l, R_K), 1, 2 * (int)D, (int)D, m->null_kv + (size_t)l * 2 * D, 2 * (int)D);
    a.w2 = w.dec(l, R_V);
    a.n2 = (int)D;
    if (linear<kLinStore>(a, s) != hipSuccess) {
      smem_model_destroy(m);
      return mfail(SMEM_EHIP, "null row maps");
    }
  }
  *out = m;
  return SMEM_OK;
}

smem_status smem_model_destroy(smem_model* m) {
  if (!m) return SMEM_OK;
  for (smem_store* st : m->stores) smem_store_destroy(st);
  smem_store_destroy(m->rows);
  smem_store_destroy(m->blockless);
  delete m;
  return SMEM_OK;
}

smem_status smem_model_encode_blocks(smem_model* m, int32_t n_blocks, const int32_t* seq_ids,
                                     const int32_t* block_idx, const int32_t* tokens, hipStream_t s) {
  if (!m) return mfail(SMEM_EINVAL, "model is NULL");
  const auto& d = m->d;
  if (n_blocks < 0) return mfail(SMEM_EINVAL, "n_blocks < 0");
  if (n_blocks == 0) return SMEM_OK;
  if (!seq_ids || !block_idx || !tokens) return mfail(SMEM_EINVAL, "seq_ids, block_idx and tokens are required");
  std::set<std::pair<int32_t, int32_t>> seen;
  for (int i = 0; i < n_blocks; ++i) {
    if (seq_ids[i] < 0 || seq_ids[i] >= d.n_seq) return mfail(SMEM_EINVAL, "seq out of range");
    if (block_idx[i] < 0 || block_idx[i] >= d.max_blocks) return mfail(SMEM_EINVAL, "block index out of range");
    if (!seen.insert({seq_ids[i], block_idx[i]}).second) return mfail(SMEM_EEXIST, "a block is given twice");
  }
  // every layer's store holds the same blocks: check occupancy and space on the first
  smem_store* mem = m->d.row_plane ? m->rows : m->stores[0];
  {
    std::set<int32_t> seqs_in;
    for (int i = 0; i < n_blocks; ++i) seqs_in.insert(seq_ids[i]);
    std::vector<int32_t> live(d.max_blocks);
    for (int32_t q : seqs_in) {
      int32_t n_live = 0;
      MSTATUS(m->d.row_plane ? smem_rows_export(mem, q, live.data(), &n_live, nullptr, s)
                             : smem_store_export(mem, q, live.data(), &n_live, nullptr, nullptr, s));
      for (int i = 0; i < n_live; ++i)
        if (seen.count({q, live[i]})) return mfail(SMEM_EEXIST, "a block index is occupied");
    }
    int32_t used = 0, free_pages = 0;
    MSTATUS(smem_store_stats(mem, &used, &free_pages));
    if (free_pages < n_blocks) return mfail(SMEM_ENOMEM, "not enough free pages");
  }
  Wts w{m};
  const int cb = d.max_tokens / d.b, D = d.d;
  for (int i0 = 0; i0 < n_blocks; i0 += cb) {
    const int nb = std::min(cb, n_blocks - i0), rows = nb * d.b;
    MSTATUS(embed(m, nb, block_idx + i0, tokens + (size_t)i0 * d.b, s));
    for (int l = 0; l < d.E; ++l) {
      MSTATUS(self_attn(m, rows, nb, w.enc(l, E_LN1G), w.enc(l, E_LN1B), w.enc(l, E_QKV), w.enc(l, E_O),
                        SMEM_MASK_BIDIR, s));
      MSTATUS(ffn(m, rows, w.enc(l, E_LN2G), w.enc(l, E_LN2B), w.enc(l, E_FF1), w.enc(l, E_FF2), s));
    }
    MCHECK(lnorm(m->x, w.mem_g(), w.mem_b(), m->h, rows, D, s), "memory layernorm");
    if (d.row_plane) {          // the rows themselves, once for every layer
      for (int i = 0; i < nb; ++i)
        MSTATUS(smem_rows_put_block(m->rows, seq_ids[i0 + i], block_idx[i0 + i], m->h + (size_t)i * d.b * D, s));
      continue;
    }
    for (int l = 0; l < d.D; ++l) {
      LinArgs a = lin(m->h, D, w.dec(l, R_K), rows, 2 * D, D, m->q, D);
      a.w2 = w.dec(l, R_V); a.n2 = D; a.y1 = m->k; a.ns = D;
      MCHECK(linear<kLinSplit>(a, s), "memory key/value maps");
      MSTATUS(smem_store_put_blocks(m->stores[l], nb, seq_ids + i0, block_idx + i0, m->q, m->k, s));
    }
  }
  return SMEM_OK;
}

smem_status smem_model_encode(smem_model* m, int32_t seq, int32_t n_blocks, const int32_t* block_idx,
                              const int32_t* tokens, hipStream_t s) {
  if (n_blocks < 0) return mfail(SMEM_EINVAL, "n_blocks < 0");
  const std::vector<int32_t> seqs(n_blocks, seq);
  return smem_model_encode_blocks(m, n_blocks, seqs.data(), block_idx, tokens, s);
}

smem_status smem_model_read(smem_model* m, int32_t seq, int32_t n_blocks, const int32_t* query_block,
                            const int32_t* tokens, float* logits, hipStream_t s) {
  if (!m) return mfail(SMEM_EINVAL, "model is NULL");
  const auto& d = m->d;
  if (n_blocks < 0) return mfail(SMEM_EINVAL, "n_blocks < 0");
  if (n_blocks == 0) return SMEM_OK;
  if (!query_block || !tokens || !logits) return mfail(SMEM_EINVAL, "query_block, tokens and logits are required");
  if (d.row_plane) return mfail(SMEM_EINVAL, "a row-plane model decodes; block reads need the key/value layers");
  if (seq < 0 || seq >= d.n_seq) return mfail(SMEM_EINVAL, "seq out of range");
  for (int i = 0; i < n_blocks; ++i)
    if (query_block[i] < 0 || query_block[i] > d.max_blocks) return mfail(SMEM_EINVAL, "query block out of range");
  const int cb = d.max_tokens / d.b;
  for (int i0 = 0; i0 < n_blocks; i0 += cb) {
    const int nb = std::min(cb, n_blocks - i0);
    MSTATUS(read_chunk(m, seq, nb, query_block + i0, tokens + (size_t)i0 * d.b, logits + (size_t)i0 * d.b * d.vocab,
                       0, s));
  }
  return SMEM_OK;
}

smem_status smem_model_prefill(smem_model* m, int32_t seq, int32_t first_block, int32_t n_blocks,
                               const int32_t* tokens, float* logits, hipStream_t s) {
  if (!m) return mfail(SMEM_EINVAL, "model is NULL");
  const auto& d = m->d;
  if (n_blocks < 1) return mfail(SMEM_EINVAL, "n_blocks < 1");
  if (!tokens || !logits) return mfail(SMEM_EINVAL, "tokens and logits are required");
  if (d.row_plane) return mfail(SMEM_EINVAL, "a row-plane model decodes; block reads need the key/value layers");
  if (first_block < 0 || (int64_t)first_block + n_blocks > d.max_blocks)
    return mfail(SMEM_EINVAL, "blocks first_block .. first_block + n_blocks - 1 out of range");
  std::vector<int32_t> blocks(n_blocks);
  for (int i = 0; i < n_blocks; ++i) blocks[i] = first_block + i;
  MSTATUS(smem_model_encode(m, seq, n_blocks, blocks.data(), tokens, s));
  const int cb = d.max_tokens / d.b;
  for (int i0 = 0; i0 < n_blocks; i0 += cb) {
    const int nb = std::min(cb, n_blocks - i0);
    const bool last = i0 + nb == n_blocks;
    MSTATUS(read_chunk(m, seq, nb, blocks.data() + i0, tokens + (size_t)i0 * d.b, last ? logits : nullptr,
                       (nb - 1) * d.b, s));
  }
  return SMEM_OK;
}

smem_status smem_model_decode(smem_model* m, int32_t first_seq, int32_t n_seq, const int32_t* query_block,
                              const int32_t* pos, const int32_t* tokens, float* logits, hipStream_t s) {
  if (!m) return mfail(SMEM_EINVAL, "model is NULL");
  const auto& d = m->d;
  if (n_seq < 0) return mfail(SMEM_EINVAL, "n_seq < 0");
  if (n_seq == 0) return SMEM_OK;
  if (!query_block || !pos || !tokens || !logits) return mfail(SMEM_EINVAL, "query_block, pos, tokens and logits are required");
  if (first_seq < 0 || (int64_t)first_seq + n_seq > d.n_seq) return mfail(SMEM_EINVAL, "sequences out of range");
  for (int i = 0; i < n_seq; ++i) {
    if (query_block[i] < 0 || query_block[i] > d.max_blocks) return mfail(SMEM_EINVAL, "query block out of range");
    if (pos[i] < 0 || pos[i] >= d.b) return mfail(SMEM_EINVAL, "pos out of range [0, b)");
  }
  const int chunk = std::min(kMaxSlots, (int)d.max_tokens);
  for (int i0 = 0; i0 < n_seq; i0 += chunk) {
    const int n = std::min(chunk, n_seq - i0);
    MSTATUS(decode_chunk(m, first_seq + i0, n, query_block + i0, pos + i0, tokens + i0,
                         logits + (size_t)i0 * d.vocab, s));
  }
  return SMEM_OK;
}

smem_status smem_model_delete_block(smem_model* m, int32_t seq, int32_t block_idx, hipStream_t s) {
  if (!m) return mfail(SMEM_EINVAL, "model is NULL");
  if (m->d.row_plane) return smem_delete_block(m->rows, seq, block_idx, 0, s);
  for (smem_store* st : m->stores) MSTATUS(smem_delete_block(st, seq, block_idx, 0, s));
  return SMEM_OK;
}

smem_status smem_self_attention(int32_t n_blocks, int32_t d, int32_t H, const void* x, const void* ln_g,
                                const void* ln_b, const void* w_qkv, int32_t mask, int32_t path, void* out, void* work,
                                hipStream_t s) {
  if (n_blocks < 0 || H < 1 || d < 64 || d % 64 || d > 2048 || d % H) return mfail(SMEM_EINVAL, "bad shape");
  const int dh = d / H;
  if (dh != 32 && dh != 64 && dh != 128) return mfail(SMEM_EINVAL, "d / H must be 32, 64 or 128");
  if (mask != SMEM_MASK_BIDIR && mask != SMEM_MASK_CAUSAL) return mfail(SMEM_EINVAL, "bad mask");
  if (path < 0 || path > 2) return mfail(SMEM_EINVAL, "path is 0 (the model's choice), 1 (unfused) or 2 (fused)");
  if (path == 2 && !qkv_attn_fits(d, H))
    return mfail(SMEM_EINVAL, "the fused path needs d / H = 32 and d a multiple of 256 up to 1024");
  if (n_blocks > 65535) return mfail(SMEM_EINVAL, "at most 65535 blocks per call");
  if (!x || !ln_g || !ln_b || !w_qkv || !out) return mfail(SMEM_EINVAL, "x, ln_g, ln_b, w_qkv, out are required");
  const int eff = path == 2 ? 2 : 1;
  const size_t rows = (size_t)n_blocks * BT, plane = rows * d;
  if (!work && (eff == 1 || rows > 128)) return mfail(SMEM_EINVAL, "work is required for this path and size");
  const void* ptrs[] = {x, ln_g, ln_b, w_qkv, out, work};
  for (const void* p : ptrs)
    if ((uintptr_t)p & 15u) return mfail(SMEM_EINVAL, "tensors must be 16-byte aligned");
  if (n_blocks == 0) return SMEM_OK;
  uint16_t* wk = (uint16_t*)work;
  return attn_sublayer(n_blocks, d, H, (const uint16_t*)x, (const uint16_t*)ln_g, (const uint16_t*)ln_b,
                       (const uint16_t*)w_qkv, mask, eff, (uint16_t*)out, wk, wk ? wk + plane : nullptr,
                       wk ? wk + 2 * plane : nullptr, wk ? wk + 3 * plane : nullptr, s);
}

smem_status smem_linear(int32_t M, int32_t N, int32_t K, const void* x, const void* w, const void* ln_g,
                        const void* ln_b, int32_t epi, const void* res, void* y, void* ln_tmp, hipStream_t s) {
  if (M < 0 || N < 0 || K <= 0) return mfail(SMEM_EINVAL, "M, N >= 0 and K > 0 are required");
  if (K % 64) return mfail(SMEM_EINVAL, "K must be a multiple of 64");
  if (!x || !w || !y) return mfail(SMEM_EINVAL, "x, w, y are required");
  if ((ln_g == nullptr) != (ln_b == nullptr)) return mfail(SMEM_EINVAL, "ln_g and ln_b: both or neither");
  if (ln_g && K > 2048) return mfail(SMEM_EINVAL, "a fused LayerNorm needs K <= 2048");
  if (ln_g && M > 128 && !ln_tmp) return mfail(SMEM_EINVAL, "ln_tmp is required with a LayerNorm and M > 128");
  if (epi < 0 || epi > 3) return mfail(SMEM_EINVAL, "epi is 0 (store), 1 (GELU), 2 (residual) or 3 (fp32)");
  if (epi == 2 && !res) return mfail(SMEM_EINVAL, "res is required with epi = 2");
  if (epi != 3 && N % 4) return mfail(SMEM_EINVAL, "bf16 outputs need N % 4 == 0");
  const void* ptrs[] = {x, w, ln_g, ln_b, res, y, ln_tmp};
  for (const void* p : ptrs)
    if ((uintptr_t)p & 15u) return mfail(SMEM_EINVAL, "tensors must be 16-byte aligned");
  LinArgs a = lin((const uint16_t*)x, K, (const uint16_t*)w, M, N, K, (uint16_t*)y, N);
  a.lng = (const uint16_t*)ln_g;
  a.lnb = (const uint16_t*)ln_b;
  a.lnout = (uint16_t*)ln_tmp;
  hipError_t e;
  switch (epi) {
    case 0: e = linear<kLinStore>(a, s); break;
    case 1: e = linear<kLinGelu>(a, s); break;
    case 2: a.res = (const uint16_t*)res; e = linear<kLinResid>(a, s); break;
    default: a.y = nullptr; a.yf = (float*)y; e = linear<kLinF32>(a, s); break;
  }
  if (e != hipSuccess) return mfail(SMEM_EHIP, "linear map launch");
  return SMEM_OK;
}

}  // extern "C"
