// C ABI of the SMem library: argument validation, the host-authoritative
// store (block table, canonical live lists, free pages) and kernel dispatch.
//
// Store semantics follow Theorem 1 of the paper: a block index holds at most
// one block (insert into an occupied index -> SMEM_EEXIST), only a present
// block can be deleted (SMEM_ENOENT otherwise), deletion restores exactly the
// never-inserted state, and reads depend only on which blocks are present,
// taken in ascending block index.  Host metadata changes immediately; the
// device copy is updated by kernels on the caller's stream, carrying the edit
// in kernel arguments (no host buffer outlives a call).
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "common.h"
#include "smem.h"

using namespace smem;

namespace {

// Live block indices of one sequence: a bitset over 0..max_blocks-1 and a
// Fenwick tree over the words' popcounts, so an insert, a delete, the rank
// of an index (how many live blocks lie below it) and the position of the
// k-th live block each cost O(log max_blocks), whatever the table's size.
class LiveSet {
 public:
  void init(int n) {
    n_ = n;
    count_ = 0;
    w_.assign((size_t)(n + 63) / 64, 0);
    f_.assign(w_.size() + 1, 0);
  }
  int size() const { return count_; }
  bool contains(int j) const { return (w_[(size_t)j >> 6] >> (j & 63)) & 1u; }
  void insert(int j) {
    w_[(size_t)j >> 6] |= 1ull << (j & 63);
    add((int)(j >> 6), 1);
    ++count_;
  }
  void erase(int j) {
    w_[(size_t)j >> 6] &= ~(1ull << (j & 63));
    add((int)(j >> 6), -1);
    --count_;
  }
  // live indices below J
  int rank(int J) const {
    if (J <= 0) return 0;
    if (J >= n_) return count_;
    const int wi = J >> 6;
    const uint64_t below = (J & 63) ? (w_[(size_t)wi] & ((1ull << (J & 63)) - 1)) : 0ull;
    return prefix(wi) + __builtin_popcountll(below);
  }
  // index of the k-th live block (0-based), k < size()
  int select(int k) const {
    int pos = 0, step = 1;
    while (step * 2 <= (int)w_.size()) step *= 2;
    for (; step > 0; step >>= 1)               // largest word count whose prefix sum is <= k
      if (pos + step <= (int)w_.size() && f_[(size_t)(pos + step)] <= k) {
        pos += step;
        k -= f_[(size_t)pos];
      }
    uint64_t w = w_[(size_t)pos];
    for (int i = 0; i < k; ++i) w &= w - 1;    // drop the k lowest set bits
    return pos * 64 + __builtin_ctzll(w);
  }
  // live indices in ascending order
  void copy_to(int32_t* out) const {
    for (size_t wi = 0; wi < w_.size(); ++wi)
      for (uint64_t w = w_[wi]; w; w &= w - 1) *out++ = (int32_t)(wi * 64 + __builtin_ctzll(w));
  }

 private:
  void add(int wi, int d) {
    for (int i = wi + 1; i <= (int)w_.size(); i += i & -i) f_[(size_t)i] += d;
  }
  int prefix(int wi) const {                   // live blocks in words 0..wi-1
    int r = 0;
    for (int i = wi; i > 0; i -= i & -i) r += f_[(size_t)i];
    return r;
  }
  int n_ = 0, count_ = 0;
  std::vector<uint64_t> w_;
  std::vector<int32_t> f_;
};

}  // namespace

struct smem_store {
  smem_store_desc d;          // row stores: H = 1, dh = 0; the row width is rows_d
  int kind = 0;               // 0: key/value planes, 1: rows of width rows_d
  int32_t rows_d = 0;
  bool meta_only = false;
  char* pool = nullptr;
  DevLayout lay{};
  int32_t* d_table = nullptr;
  int32_t* d_live_page = nullptr;
  int32_t* d_live_blk = nullptr;
  int32_t* d_n_live = nullptr;
  float* d_ws = nullptr;
  void* d_pages = nullptr;
  std::vector<int32_t> table;              // [n_seq * max_blocks]: page or -1
  std::vector<LiveSet> live;               // per sequence, the live block indices
  std::vector<int32_t> free_pages;         // stack; back() is handed out next
};

struct smem_rope {
  smem_rope_desc d;
  float* table = nullptr;                  // [n_phases][dh/2] (cos, sin)
};

namespace {

thread_local std::string g_err;

smem_status fail(smem_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = std::string(smem_status_string(st)) + ": " + buf;
  return st;
}

}  // namespace

smem_status smem::set_error(smem_status st, const char* msg) { return fail(st, "%s", msg); }

namespace {

smem_status hip_fail(hipError_t e, const char* what) {
  return fail(SMEM_EHIP, "%s: %s", what, hipGetErrorString(e));
}

size_t esize(int dtype) { return dtype == F32 ? 4 : 2; }

bool shape_ok(int b, int H, int dh, int dtype) {
  return (b == 16 || b == 64) && (dh == 32 || dh == 64 || dh == 128) && H >= 1 && H <= 64 &&
         (dtype == F32 || dtype == BF16);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Query slots of one prefill launch: a slot is a (sequence, query block) pair,
// so one sequence may fill several (a block-parallel pass over its blocks).
int prefill_slots(const smem_store_desc* d) {
  return (int)std::min<int64_t>((int64_t)d->n_seq * d->max_blocks, std::min(kMaxSlots, kPrefillSlotChunk));
}

bool layout_of(const smem_store_desc* d, DevLayout* L) {
  if (!d) return false;
  if (d->n_seq < 1 || d->max_blocks < 1 || d->n_pages < 1) return false;
  if (!shape_ok(d->b, d->H, d->dh, d->dtype)) return false;
  const size_t nt = (size_t)d->n_seq * d->max_blocks;
  const size_t dec_rows = (size_t)d->n_seq * d->H;
  const size_t pre_rows = (size_t)prefill_slots(d) * d->b * d->H;
  L->ws_floats = std::max(dec_rows, pre_rows) * kSplitStride * (d->dh + 4);
  size_t off = 0;
  L->off_table = off;     off = align256(off + nt * 4);
  L->off_live_page = off; off = align256(off + nt * 4);
  L->off_live_blk = off;  off = align256(off + nt * 4);
  L->off_n_live = off;    off = align256(off + (size_t)d->n_seq * 4);
  L->off_ws = off;        off = align256(off + L->ws_floats * 4);
  L->off_pages = off;     off = align256(off + (size_t)d->n_pages * d->H * 2 * d->b * d->dh * esize(d->dtype));
  L->total = off;
  return true;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// ---------------------------------------------------------------- row stores

int pps_rows(int n_read) { return pages_per_split(n_read, kMinPagesRows, kRowsSplitCap); }
int splits_rows(int n_read) { return n_read > 0 ? (n_read + pps_rows(n_read) - 1) / pps_rows(n_read) : 0; }

bool rows_layout_of(const smem_rows_desc* d, DevLayout* L) {
  if (!d) return false;
  if (d->n_seq < 1 || d->max_blocks < 1 || d->n_pages < 1) return false;
  if (!(d->b == 16 || d->b == 64) || !(d->d == 512 || d->d == 768 || d->d == 1024 || d->d == 2048) || d->dtype != BF16)
    return false;
  const size_t nt = (size_t)d->n_seq * d->max_blocks;
  // splits of one read never exceed min(kRowsSplitCap, ceil(n_read / kMinPagesRows)), n_read <= max_blocks
  const int64_t per_seq = std::min(kRowsSplitCap, (d->max_blocks + kMinPagesRows - 1) / kMinPagesRows);
  // one partial per (split, head tile): a read takes at most per_seq splits of up to 4 tiles
  const int64_t cap = std::min<int64_t>(kRowsPartials, (int64_t)d->n_seq * per_seq * (kRowsMaxHeads / 16));
  L->part_cap = (int32_t)std::max<int64_t>(cap, 1);
  L->ws_floats = 0;
  size_t off = 0;
  L->off_table = off;     off = align256(off + nt * 4);
  L->off_live_page = off; off = align256(off + nt * 4);
  L->off_live_blk = off;  off = align256(off + nt * 4);
  L->off_n_live = off;    off = align256(off + (size_t)d->n_seq * 4);
  L->off_qabs = off;      off = align256(off + (size_t)kMaxSlots * kRowsMaxHeads * d->d * 2);
  L->off_intra = off;     off = align256(off + (size_t)kMaxSlots * kRowsMaxHeads * (128 + 4) * 4);
  L->off_null_kv = off;   off = align256(off + (size_t)2 * kRowsMaxHeads * 128 * 2);
  L->off_sw = off;        off = align256(off + (size_t)kMaxSlots * kRowsMaxHeads * 4);
  L->off_part = off;      off = align256(off + (size_t)L->part_cap * (16 * (size_t)d->d + 32) * 4);
  L->off_ws = L->off_part;
  L->off_pages = off;     off = align256(off + (size_t)d->n_pages * d->b * d->d * 2);
  L->total = off;
  return true;
}

size_t page_bytes(const smem_store* st) {
  return st->kind == 1 ? (size_t)st->d.b * st->rows_d * 2 : (size_t)st->d.H * 2 * st->d.b * st->d.dh * esize(st->d.dtype);
}

size_t rope_bytes_of(const smem_rope_desc* d) {
  if (!d || !(d->dh == 32 || d->dh == 64 || d->dh == 128) || d->n_phases < 1 || d->n_phases > (1 << 20) ||
      d->max_offset < 0 || d->reserved != 0 || !(d->base > 1.0) || !std::isfinite(d->base))
    return 0;
  return align256((size_t)d->n_phases * d->dh * sizeof(float));
}

// Check a rotary configuration against a call: head width, and that the
// table holds every phase used (in-block offsets < b, block turns <= max_turn).
smem_status rope_check(const smem_rope* rope, int dh, int b, int max_turn) {
  if (rope->d.dh != dh) return fail(SMEM_EINVAL, "rotary table is for dh=%d, the call has dh=%d", rope->d.dh, dh);
  const int need = std::max(b - 1, max_turn);
  if (need >= rope->d.n_phases)
    return fail(SMEM_EINVAL, "phase %d needed, the rotary table holds 0..%d", need, rope->d.n_phases - 1);
  return SMEM_OK;
}

// Largest block turn of a read from query block J: min(J, W), or J.
int rope_turn_of(const smem_rope* rope, int J) {
  return rope->d.max_offset > 0 ? std::min(J, rope->d.max_offset) : J;
}

void rope_args(ReaderArgs& a, const smem_store* st, const smem_rope* rope) {
  if (!rope) return;
  a.rope = rope->table;
  a.live_blk = st->d_live_blk;
  a.rope_clip = rope->d.max_offset > 0 ? rope->d.max_offset : INT32_MAX;
}

int n_read_of(const smem_store* st, int seq, int J) { return st->live[seq].rank(J); }

// Apply edits (seq, blk, page or -1) on the device: table entries, then the
// affected part of each edited sequence's dense live list.  Called before the
// host metadata takes the edits, so the list positions after them are the
// host's current ranks plus the edits' own shifts.  Only the table chunks
// from the first edited one up to the sequence's last live block are
// rewritten, each by its own workgroup, so an edit's cost does not grow with
// the table.
smem_status push_edits(smem_store* st, const std::vector<int32_t>& es, const std::vector<int32_t>& eb,
                       const std::vector<int32_t>& ep, hipStream_t s) {
  const int mb = st->d.max_blocks;
  const int n_chunks = (mb + kMetaChunk - 1) / kMetaChunk;
  for (size_t i0 = 0; i0 < es.size(); i0 += kMaxEdits) {
    const size_t i1 = std::min(es.size(), i0 + (size_t)kMaxEdits);
    MetaArgs a;
    memset(&a, 0, sizeof a);
    a.table = st->d_table;
    a.live_page = st->d_live_page;
    a.live_blk = st->d_live_blk;
    a.n_live = st->d_n_live;
    a.max_blocks = mb;
    a.n_edits = (int32_t)(i1 - i0);
    std::set<int32_t> seqs;
    for (size_t i = i0; i < i1; ++i) {
      a.e_seq[i - i0] = es[i];
      a.e_blk[i - i0] = eb[i];
      a.e_page[i - i0] = ep[i];
      seqs.insert(es[i]);
    }
    auto flush = [&]() -> smem_status {
      hipError_t e = launch_meta(a, s);
      if (e != hipSuccess) return hip_fail(e, "metadata update");
      a.n_items = 0;
      return SMEM_OK;
    };
    for (int32_t q : seqs) {
      const LiveSet& lv = st->live[q];
      // chunks from the first edited one to the last that can hold a live block
      int c0 = n_chunks, c1 = lv.size() > 0 ? lv.select(lv.size() - 1) / kMetaChunk : 0;
      for (size_t i = i0; i < i1; ++i)
        if (es[i] == q) c0 = std::min(c0, eb[i] / kMetaChunk);
      for (size_t i = 0; i < i1; ++i)
        if (es[i] == q) c1 = std::max(c1, eb[i] / kMetaChunk);
      for (int c = c0; c <= c1; ++c) {
        // list position of the chunk's first live block once edits 0 .. i1 - 1 are in
        int base = lv.rank(c * kMetaChunk);
        for (size_t i = 0; i < i1; ++i)
          if (es[i] == q && eb[i] < c * kMetaChunk) base += ep[i] >= 0 ? 1 : -1;
        a.i_seq[a.n_items] = q;
        a.i_chunk[a.n_items] = c;
        a.i_base[a.n_items] = base;
        a.i_last[a.n_items] = c == c1;
        if (++a.n_items == kMaxMetaItems) {
          const smem_status r = flush();
          if (r != SMEM_OK) return r;
        }
      }
    }
    if (a.n_items > 0) {
      const smem_status r = flush();
      if (r != SMEM_OK) return r;
    }
  }
  return SMEM_OK;
}

}  // namespace

extern "C" {

const char* smem_status_string(smem_status st) {
  switch (st) {
    case SMEM_OK: return "SMEM_OK";
    case SMEM_EINVAL: return "SMEM_EINVAL";
    case SMEM_ENOMEM: return "SMEM_ENOMEM";
    case SMEM_ENOENT: return "SMEM_ENOENT";
    case SMEM_EEXIST: return "SMEM_EEXIST";
    case SMEM_EHIP: return "SMEM_EHIP";
  }
  return "SMEM_UNKNOWN";
}

const char* smem_last_error(void) { return g_err.c_str(); }

size_t smem_store_bytes(const smem_store_desc* desc) {
  DevLayout L;
  if (!layout_of(desc, &L)) return 0;
  return L.total;
}

smem_status smem_store_create(const smem_store_desc* desc, void* dev_pool, size_t pool_bytes, hipStream_t s,
                              smem_store** out) {
  if (!out) return fail(SMEM_EINVAL, "out is NULL");
  *out = nullptr;
  DevLayout L;
  if (!layout_of(desc, &L))
    return fail(SMEM_EINVAL, "invalid store descriptor (need n_seq, max_blocks, n_pages >= 1, b in {16,64}, "
                             "dh in {32,64,128}, 1 <= H <= 64, dtype F32/BF16)");
  if ((size_t)desc->n_pages * desc->H * 2 * desc->b * desc->dh > ((size_t)1 << 40))
    return fail(SMEM_EINVAL, "page pool too large");
  if (dev_pool) {
    if (pool_bytes < L.total) return fail(SMEM_ENOMEM, "pool has %zu bytes, store needs %zu", pool_bytes, L.total);
    if (((uintptr_t)dev_pool & 255u) != 0) return fail(SMEM_EINVAL, "dev_pool must be 256-byte aligned");
  }
  smem_store* st = new (std::nothrow) smem_store();
  if (!st) return fail(SMEM_ENOMEM, "host allocation failed");
  st->d = *desc;
  st->lay = L;
  st->meta_only = dev_pool == nullptr;
  st->table.assign((size_t)desc->n_seq * desc->max_blocks, -1);
  st->live.assign(desc->n_seq, LiveSet());
  for (auto& lv : st->live) lv.init(desc->max_blocks);
  st->free_pages.resize(desc->n_pages);
  for (int i = 0; i < desc->n_pages; ++i) st->free_pages[i] = desc->n_pages - 1 - i;
  if (!st->meta_only) {
    st->pool = (char*)dev_pool;
    st->d_table = (int32_t*)(st->pool + L.off_table);
    st->d_live_page = (int32_t*)(st->pool + L.off_live_page);
    st->d_live_blk = (int32_t*)(st->pool + L.off_live_blk);
    st->d_n_live = (int32_t*)(st->pool + L.off_n_live);
    st->d_ws = (float*)(st->pool + L.off_ws);
    st->d_pages = st->pool + L.off_pages;
    hipError_t e = launch_init_meta(st->d_table, st->d_n_live, st->table.size(), desc->n_seq, s);
    if (e != hipSuccess) {
      delete st;
      return hip_fail(e, "store init");
    }
  }
  *out = st;
  return SMEM_OK;
}

smem_status smem_store_destroy(smem_store* st) {
  delete st;
  return SMEM_OK;
}

smem_status smem_device_copy(void* dst, const void* src, size_t bytes, int32_t via_lds, hipStream_t s) {
  if (!dst || !src) return fail(SMEM_EINVAL, "dst and src are required");
  if (!aligned16(dst) || !aligned16(src)) return fail(SMEM_EINVAL, "dst and src must be 16-byte aligned");
  if (via_lds != 0 && via_lds != 1) return fail(SMEM_EINVAL, "via_lds is 0 or 1");
  const size_t unit = via_lds ? 16384 : 16;
  if (bytes % unit) return fail(SMEM_EINVAL, "bytes must be a multiple of %zu", unit);
  const hipError_t e = via_lds ? launch_copy_dma(dst, src, bytes, s) : launch_copy16(dst, src, bytes, s);
  if (e != hipSuccess) return hip_fail(e, "device copy");
  return SMEM_OK;
}

smem_status smem_store_stats(const smem_store* st, int32_t* pages_used, int32_t* pages_free) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (pages_free) *pages_free = (int32_t)st->free_pages.size();
  if (pages_used) *pages_used = st->d.n_pages - (int32_t)st->free_pages.size();
  return SMEM_OK;
}

smem_status smem_store_put_block(smem_store* st, int32_t seq, int32_t block_idx, const void* k_rows,
                                 const void* v_rows, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->kind != 0) return fail(SMEM_EINVAL, "a row store takes smem_rows_put_block");
  const auto& d = st->d;
  if (seq < 0 || seq >= d.n_seq) return fail(SMEM_EINVAL, "seq %d out of range [0, %d)", seq, d.n_seq);
  if (block_idx < 0 || block_idx >= d.max_blocks)
    return fail(SMEM_EINVAL, "block index %d out of range [0, %d)", block_idx, d.max_blocks);
  if (st->meta_only) {
    if (k_rows || v_rows) return fail(SMEM_EINVAL, "metadata-only store takes NULL rows");
  } else {
    if (!k_rows || !v_rows) return fail(SMEM_EINVAL, "k_rows and v_rows are required");
    if (!aligned16(k_rows) || !aligned16(v_rows)) return fail(SMEM_EINVAL, "rows must be 16-byte aligned");
  }
  const size_t ti = (size_t)seq * d.max_blocks + block_idx;
  if (st->table[ti] >= 0) return fail(SMEM_EEXIST, "block %d of sequence %d is occupied", block_idx, seq);
  if (st->free_pages.empty()) return fail(SMEM_ENOMEM, "no free page (%d pages)", d.n_pages);
  const int32_t page = st->free_pages.back();
  if (!st->meta_only) {
    hipError_t e = launch_put_rows(d.dtype, st->d_pages, page, d.H, d.b, d.dh, k_rows, v_rows, s);
    if (e != hipSuccess) return hip_fail(e, "row insert");
    smem_status r = push_edits(st, {seq}, {block_idx}, {page}, s);
    if (r != SMEM_OK) return r;
  }
  st->free_pages.pop_back();
  st->table[ti] = page;
  st->live[seq].insert(block_idx);
  return SMEM_OK;
}

smem_status smem_store_put_blocks(smem_store* st, int32_t n_blocks, const int32_t* seq_ids, const int32_t* block_idx,
                                  const void* k_rows, const void* v_rows, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->kind != 0) return fail(SMEM_EINVAL, "a row store takes smem_rows_put_block");
  if (st->meta_only) return fail(SMEM_EINVAL, "metadata-only store");
  const auto& d = st->d;
  if (n_blocks < 0) return fail(SMEM_EINVAL, "n_blocks < 0");
  if (n_blocks == 0) return SMEM_OK;
  if (!seq_ids || !block_idx || !k_rows || !v_rows) return fail(SMEM_EINVAL, "seq_ids, block_idx, k_rows, v_rows are required");
  if (!aligned16(k_rows) || !aligned16(v_rows)) return fail(SMEM_EINVAL, "rows must be 16-byte aligned");
  std::set<std::pair<int32_t, int32_t>> seen;
  for (int i = 0; i < n_blocks; ++i) {
    const int32_t sq = seq_ids[i], j = block_idx[i];
    if (sq < 0 || sq >= d.n_seq) return fail(SMEM_EINVAL, "seq_ids[%d] = %d out of range", i, sq);
    if (j < 0 || j >= d.max_blocks) return fail(SMEM_EINVAL, "block_idx[%d] = %d out of range", i, j);
    if (st->table[(size_t)sq * d.max_blocks + j] >= 0) return fail(SMEM_EEXIST, "block %d of sequence %d is occupied", j, sq);
    if (!seen.insert({sq, j}).second) return fail(SMEM_EEXIST, "block %d of sequence %d given twice", j, sq);
  }
  if ((size_t)n_blocks > st->free_pages.size())
    return fail(SMEM_ENOMEM, "%d blocks to insert, %zu free pages", n_blocks, st->free_pages.size());
  std::vector<int32_t> pages(n_blocks), es_(n_blocks), eb_(n_blocks);
  for (int i = 0; i < n_blocks; ++i) {
    pages[i] = st->free_pages[st->free_pages.size() - 1 - i];
    es_[i] = seq_ids[i];
    eb_[i] = block_idx[i];
  }
  const size_t blk_bytes = (size_t)d.b * d.H * d.dh * esize(d.dtype);
  for (int i0 = 0; i0 < n_blocks; i0 += kMaxSlots) {
    const int n = std::min(kMaxSlots, n_blocks - i0);
    PutArgs a;
    memset(&a, 0, sizeof a);
    a.pages = st->d_pages;
    a.k_rows = (const char*)k_rows + i0 * blk_bytes;
    a.v_rows = (const char*)v_rows + i0 * blk_bytes;
    a.H = d.H; a.b = d.b; a.dh = d.dh;
    for (int i = 0; i < n; ++i) a.page[i] = pages[i0 + i];
    hipError_t e = launch_put_blocks(d.dtype, a, n, s);
    if (e != hipSuccess) return hip_fail(e, "row insert");
  }
  smem_status r = push_edits(st, es_, eb_, pages, s);
  if (r != SMEM_OK) return r;
  st->free_pages.resize(st->free_pages.size() - n_blocks);
  for (int i = 0; i < n_blocks; ++i) {
    st->table[(size_t)seq_ids[i] * d.max_blocks + block_idx[i]] = pages[i];
    st->live[seq_ids[i]].insert(block_idx[i]);
  }
  return SMEM_OK;
}

smem_status smem_delete_block(smem_store* st, int32_t seq, int32_t block_idx, int32_t scrub, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  const auto& d = st->d;
  if (seq < 0 || seq >= d.n_seq) return fail(SMEM_EINVAL, "seq %d out of range [0, %d)", seq, d.n_seq);
  if (block_idx < 0 || block_idx >= d.max_blocks)
    return fail(SMEM_EINVAL, "block index %d out of range [0, %d)", block_idx, d.max_blocks);
  const size_t ti = (size_t)seq * d.max_blocks + block_idx;
  const int32_t page = st->table[ti];
  if (page < 0) return fail(SMEM_ENOENT, "block %d of sequence %d is absent", block_idx, seq);
  if (!st->meta_only) {
    smem_status r = push_edits(st, {seq}, {block_idx}, {-1}, s);
    if (r != SMEM_OK) return r;
    if (scrub) {
      hipError_t e = launch_scrub((char*)st->d_pages + (size_t)page * page_bytes(st), page_bytes(st), s);
      if (e != hipSuccess) return hip_fail(e, "page scrub");
    }
  }
  st->table[ti] = -1;
  st->live[seq].erase(block_idx);
  st->free_pages.push_back(page);
  return SMEM_OK;
}

smem_status smem_store_export(smem_store* st, int32_t seq, int32_t* live_idx, int32_t* n_live, void* k_out,
                              void* v_out, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->kind != 0) return fail(SMEM_EINVAL, "a row store takes smem_rows_export");
  const auto& d = st->d;
  if (seq < 0 || seq >= d.n_seq) return fail(SMEM_EINVAL, "seq %d out of range [0, %d)", seq, d.n_seq);
  if ((k_out == nullptr) != (v_out == nullptr)) return fail(SMEM_EINVAL, "k_out and v_out: both or neither");
  if (!aligned16(k_out) || !aligned16(v_out)) return fail(SMEM_EINVAL, "k_out, v_out must be 16-byte aligned");
  if (k_out && st->meta_only) return fail(SMEM_EINVAL, "metadata-only store has no rows to export");
  const auto& lv = st->live[seq];
  if (n_live) *n_live = (int32_t)lv.size();
  if (live_idx) lv.copy_to(live_idx);
  if (k_out) {
    hipError_t e = launch_export(d.dtype, st->d_pages, st->d_live_page + (size_t)seq * d.max_blocks,
                                 (int)lv.size(), d.H, d.b, d.dh, k_out, v_out, s);
    if (e != hipSuccess) return hip_fail(e, "export");
  }
  return SMEM_OK;
}

static smem_status encode_impl(smem_store* st, const smem_attn_desc* shape, int32_t n_blocks,
                               const int32_t* seq_ids, const int32_t* block_idx, const void* q, const void* k,
                               const void* v, void* out, int32_t mask, bool replace, const smem_rope* rope,
                               hipStream_t s) {
  if (!shape) return fail(SMEM_EINVAL, "shape is NULL");
  const int b = shape->b, H = shape->H, dh = shape->dh, dtype = shape->dtype;
  if (!shape_ok(b, H, dh, dtype)) return fail(SMEM_EINVAL, "unsupported shape b=%d H=%d dh=%d dtype=%d", b, H, dh, dtype);
  if (rope) {
    const smem_status r = rope_check(rope, dh, b, 0);
    if (r != SMEM_OK) return r;
  }
  if (n_blocks < 0) return fail(SMEM_EINVAL, "n_blocks < 0");
  if (mask != SMEM_MASK_BIDIR && mask != SMEM_MASK_CAUSAL) return fail(SMEM_EINVAL, "mask %d", mask);
  if (st) {
    if (st->meta_only) return fail(SMEM_EINVAL, "metadata-only store");
    if (st->kind != 0) return fail(SMEM_EINVAL, "the encoder inserts into key/value stores only");
    if (st->d.b != b || st->d.H != H || st->d.dh != dh || st->d.dtype != dtype)
      return fail(SMEM_EINVAL, "shape differs from the store's");
  } else if (!out) {
    return fail(SMEM_EINVAL, "out is NULL and there is no store");
  }
  if (n_blocks == 0) return SMEM_OK;
  if (!q || !k || !v) return fail(SMEM_EINVAL, "q, k, v are required");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || (out && !aligned16(out)))
    return fail(SMEM_EINVAL, "tensors must be 16-byte aligned");
  std::vector<int32_t> pages;
  if (st) {
    if (!seq_ids || !block_idx) return fail(SMEM_EINVAL, "seq_ids and block_idx are required with a store");
    std::set<std::pair<int32_t, int32_t>> seen;
    for (int i = 0; i < n_blocks; ++i) {
      const int32_t sq = seq_ids[i], j = block_idx[i];
      if (sq < 0 || sq >= st->d.n_seq) return fail(SMEM_EINVAL, "seq_ids[%d] = %d out of range", i, sq);
      if (j < 0 || j >= st->d.max_blocks) return fail(SMEM_EINVAL, "block_idx[%d] = %d out of range", i, j);
      const int32_t page = st->table[(size_t)sq * st->d.max_blocks + j];
      if (replace) {
        if (page < 0) return fail(SMEM_ENOENT, "block %d of sequence %d is absent", j, sq);
        if (!seen.insert({sq, j}).second) return fail(SMEM_EINVAL, "block %d of sequence %d given twice", j, sq);
      } else {
        if (page >= 0) return fail(SMEM_EEXIST, "block %d of sequence %d is occupied", j, sq);
        if (!seen.insert({sq, j}).second) return fail(SMEM_EEXIST, "block %d of sequence %d given twice", j, sq);
      }
    }
    pages.resize(n_blocks);
    if (replace) {
      for (int i = 0; i < n_blocks; ++i) pages[i] = st->table[(size_t)seq_ids[i] * st->d.max_blocks + block_idx[i]];
    } else {
      if ((size_t)n_blocks > st->free_pages.size())
        return fail(SMEM_ENOMEM, "%d blocks to insert, %zu free pages", n_blocks, st->free_pages.size());
      for (int i = 0; i < n_blocks; ++i) pages[i] = st->free_pages[st->free_pages.size() - 1 - i];
    }
  } else if (replace) {
    return fail(SMEM_EINVAL, "re-encoding needs a store");
  }
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)dh));
  const size_t es = esize(dtype);
  const size_t blk_elems = (size_t)b * H * dh;
  for (int i0 = 0; i0 < n_blocks; i0 += kMaxSlots) {
    const int n = std::min(kMaxSlots, n_blocks - i0);
    const char* qb = (const char*)q + (size_t)i0 * blk_elems * es;
    const char* kb = (const char*)k + (size_t)i0 * blk_elems * es;
    const char* vb = (const char*)v + (size_t)i0 * blk_elems * es;
    char* ob = out ? (char*)out + (size_t)i0 * blk_elems * es : nullptr;
    hipError_t e;
    if (dtype == BF16 && b == 64) {
      int32_t sink[kMaxSlots];
      for (int i = 0; i < n; ++i) sink[i] = st ? pages[i0 + i] : -1;
      e = launch_encoder_mfma(b, dh, qb, kb, vb, ob, st ? st->d_pages : nullptr, sink, n, H, mask, scale_log2,
                              rope ? rope->table : nullptr, s);
    } else {
      if (!ob) return fail(SMEM_EINVAL, "this encoder shape needs an out tensor");
      ReaderArgs a;
      memset(&a, 0, sizeof a);
      a.q = qb; a.k_in = kb; a.v_in = vb; a.out = ob;
      a.page_sink = st ? st->d_pages : nullptr;
      a.H = H; a.b = b; a.nq = b; a.intra_mode = mask == SMEM_MASK_CAUSAL ? 1 : 0;
      a.n_slots = n; a.scale_log2 = scale_log2;
      a.rope = rope ? rope->table : nullptr;
      for (int i = 0; i < n; ++i) {
        a.seq[i] = 0; a.n_read[i] = 0; a.pps[i] = 1;
        a.aux[i] = st ? pages[i0 + i] : -1;
      }
      e = launch_reader_valu(dtype, b, dh, a, s);
    }
    if (e != hipSuccess) return hip_fail(e, "encoder launch");
  }
  if (st && !replace) {
    std::vector<int32_t> es_, eb_, ep_;
    for (int i = 0; i < n_blocks; ++i) {
      es_.push_back(seq_ids[i]);
      eb_.push_back(block_idx[i]);
      ep_.push_back(pages[i]);
    }
    smem_status r = push_edits(st, es_, eb_, ep_, s);
    if (r != SMEM_OK) return r;
    st->free_pages.resize(st->free_pages.size() - n_blocks);
    for (int i = 0; i < n_blocks; ++i) {
      st->table[(size_t)seq_ids[i] * st->d.max_blocks + block_idx[i]] = pages[i];
      st->live[seq_ids[i]].insert(block_idx[i]);
    }
  }
  return SMEM_OK;
}

smem_status smem_encode_blocks(smem_store* st, const smem_attn_desc* shape, int32_t n_blocks,
                               const int32_t* seq_ids, const int32_t* block_idx, const void* q, const void* k,
                               const void* v, void* out, int32_t mask, hipStream_t s) {
  return encode_impl(st, shape, n_blocks, seq_ids, block_idx, q, k, v, out, mask, false, nullptr, s);
}

smem_status smem_encode_blocks_rope(smem_store* st, const smem_attn_desc* shape, const smem_rope* rope,
                                    int32_t n_blocks, const int32_t* seq_ids, const int32_t* block_idx,
                                    const void* q, const void* k, const void* v, void* out, int32_t mask,
                                    hipStream_t s) {
  if (!rope) return fail(SMEM_EINVAL, "rope is NULL");
  return encode_impl(st, shape, n_blocks, seq_ids, block_idx, q, k, v, out, mask, false, rope, s);
}

smem_status smem_reencode_blocks(smem_store* st, const smem_attn_desc* shape, int32_t n_blocks,
                                 const int32_t* seq_ids, const int32_t* block_idx, const void* q, const void* k,
                                 const void* v, void* out, int32_t mask, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  return encode_impl(st, shape, n_blocks, seq_ids, block_idx, q, k, v, out, mask, true, nullptr, s);
}

// Launch order of a folding prefill: the slots that read the most pages
// first, so no long pair is left for the tail.
static void longest_first(ReaderArgs& a) {
  int idx[kMaxSlots];
  for (int i = 0; i < a.n_slots; ++i) idx[i] = i;
  std::stable_sort(idx, idx + a.n_slots, [&](int x, int y) { return a.n_read[x] > a.n_read[y]; });
  for (int i = 0; i < a.n_slots; ++i) a.order[i] = (int16_t)idx[i];
}

static smem_status prefill_impl(smem_store* st, const smem_rope* rope, int32_t n_seq, const int32_t* seq_ids,
                                const int32_t* query_block, const void* q, const void* k_intra,
                                const void* v_intra, const void* null_kv, void* out, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->meta_only) return fail(SMEM_EINVAL, "metadata-only store");
  if (st->kind != 0) return fail(SMEM_EINVAL, "a row store is read by smem_reader_decode_rows");
  const auto& d = st->d;
  if (n_seq < 0) return fail(SMEM_EINVAL, "n_seq < 0");
  if (n_seq == 0) return SMEM_OK;
  if (!seq_ids || !query_block || !q || !out) return fail(SMEM_EINVAL, "seq_ids, query_block, q, out are required");
  if ((k_intra == nullptr) != (v_intra == nullptr)) return fail(SMEM_EINVAL, "k_intra and v_intra: both or neither");
  if (!aligned16(q) || !aligned16(out) || !aligned16(k_intra) || !aligned16(v_intra) || !aligned16(null_kv))
    return fail(SMEM_EINVAL, "tensors must be 16-byte aligned");
  for (int i = 0; i < n_seq; ++i) {
    if (seq_ids[i] < 0 || seq_ids[i] >= d.n_seq) return fail(SMEM_EINVAL, "seq_ids[%d] = %d out of range", i, seq_ids[i]);
    if (query_block[i] < 0 || query_block[i] > d.max_blocks)
      return fail(SMEM_EINVAL, "query_block[%d] = %d out of range [0, %d]", i, query_block[i], d.max_blocks);
    if (rope) {
      const smem_status r = rope_check(rope, d.dh, d.b, rope_turn_of(rope, query_block[i]));
      if (r != SMEM_OK) return r;
    }
  }
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.dh));
  const size_t es = esize(d.dtype);
  const size_t blk_elems = (size_t)d.b * d.H * d.dh;
  // bf16 blocks of 64 tokens run on the MFMA kernel, other shapes on the VALU reader
  const bool mfma = d.dtype == BF16 && d.b == 64;
  std::vector<int> nr(n_seq);
  for (int i = 0; i < n_seq; ++i) nr[i] = n_read_of(st, seq_ids[i], query_block[i]);
  // One workgroup per (query block, head) folding its own splits (the MFMA
  // kernel; no rotary variant), when the launch has enough pairs or short reads
  auto fold_launch = [&](int i0, int n) {
    if (!mfma || rope != nullptr) return false;
    return fold_in_workgroup((long)n * d.H, *std::max_element(nr.begin() + i0, nr.begin() + i0 + n), d.dh);
  };
  for (int i0 = 0, n = 0; i0 < n_seq; i0 += n) {
    n = std::min(kMaxSlots, n_seq - i0);
    const bool fuse = fold_launch(i0, n);
    if (!fuse) n = std::min(n, prefill_slots(&d));      // the split partials of n slots fit the workspace
    ReaderArgs a;
    memset(&a, 0, sizeof a);
    a.q = (const char*)q + i0 * blk_elems * es;
    a.k_in = k_intra ? (const char*)k_intra + i0 * blk_elems * es : nullptr;
    a.v_in = v_intra ? (const char*)v_intra + i0 * blk_elems * es : nullptr;
    a.out = (char*)out + i0 * blk_elems * es;
    a.null_kv = null_kv;
    a.pages = st->d_pages;
    a.live_page = st->d_live_page;
    a.ws = st->d_ws;
    a.ws_stride = kSplitStride;
    a.max_blocks = d.max_blocks;
    a.H = d.H; a.b = d.b; a.nq = d.b; a.intra_mode = 1;
    a.n_slots = n; a.scale_log2 = scale_log2;
    rope_args(a, st, rope);
    for (int i = 0; i < n; ++i) {
      const int sq = seq_ids[i0 + i];
      a.seq[i] = sq;
      a.qblk[i] = query_block[i0 + i];
      a.n_read[i] = nr[i0 + i];
      a.pps[i] = mfma ? pages_per_split(a.n_read[i], kMinPagesPrefill, prefill_split_cap(d.H))
                      : pages_per_split(a.n_read[i], min_pages_decode(d.dh));
      a.aux[i] = -1;
    }
    a.fuse = fuse;
    if (fuse && d.dh <= 64 && (long)n * d.H <= kParPairs) {
      bool few = true;
      for (int i = 0; i < n; ++i) few = few && total_splits(a.n_read[i], a.pps[i]) - 1 <= kParSplits;
      if (few) a.fuse = 2;
    }
    if (a.fuse) longest_first(a);
    hipError_t e = mfma ? launch_prefill_mfma(d.b, d.dh, a, s) : launch_reader_valu(d.dtype, d.b, d.dh, a, s);
    if (e != hipSuccess) return hip_fail(e, "prefill launch");
  }
  return SMEM_OK;
}

}  // extern "C"

// ws_ext == NULL: split partials in the store's workspace (kSplitStride records
// per (query, head)).  Otherwise in ws_ext (ws_ext_floats floats), each launch
// packing its partials at a stride of its own largest split count; a call that
// would not fit is rejected before anything is enqueued.
smem_status smem::decode_impl(smem_store* st, const smem_rope* rope, int32_t n_seq, const int32_t* seq_ids,
                              const int32_t* query_block, const int32_t* pos, const void* q, const void* k_new,
                              const void* v_new, void* k_cache, void* v_cache, const void* null_kv, void* out,
                              float* ws_ext, size_t ws_ext_floats, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->meta_only) return fail(SMEM_EINVAL, "metadata-only store");
  if (st->kind != 0) return fail(SMEM_EINVAL, "a row store is read by smem_reader_decode_rows");
  const auto& d = st->d;
  if (n_seq < 0) return fail(SMEM_EINVAL, "n_seq < 0");
  if (n_seq == 0) return SMEM_OK;
  if (!seq_ids || !query_block || !q || !out) return fail(SMEM_EINVAL, "seq_ids, query_block, q, out are required");
  const int n_given = (k_new != nullptr) + (v_new != nullptr) + (k_cache != nullptr) + (v_cache != nullptr);
  if (n_given != 0 && n_given != 4) return fail(SMEM_EINVAL, "k_new, v_new, k_cache, v_cache: all or none");
  if (n_given == 4 && !pos) return fail(SMEM_EINVAL, "pos is required with in-block keys");
  if (!aligned16(q) || !aligned16(out) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) ||
      !aligned16(v_cache) || !aligned16(null_kv))
    return fail(SMEM_EINVAL, "tensors must be 16-byte aligned");
  std::set<int32_t> seen;
  for (int i = 0; i < n_seq; ++i) {
    if (seq_ids[i] < 0 || seq_ids[i] >= d.n_seq) return fail(SMEM_EINVAL, "seq_ids[%d] = %d out of range", i, seq_ids[i]);
    if (query_block[i] < 0 || query_block[i] > d.max_blocks)
      return fail(SMEM_EINVAL, "query_block[%d] = %d out of range [0, %d]", i, query_block[i], d.max_blocks);
    if (n_given == 4 && (pos[i] < 0 || pos[i] >= d.b)) return fail(SMEM_EINVAL, "pos[%d] = %d out of range [0, %d)", i, pos[i], d.b);
    if (!seen.insert(seq_ids[i]).second) return fail(SMEM_EINVAL, "sequence %d appears twice", seq_ids[i]);
    if (rope) {
      const smem_status r = rope_check(rope, d.dh, d.b, rope_turn_of(rope, query_block[i]));
      if (r != SMEM_OK) return r;
    }
  }
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.dh));
  const size_t es = esize(d.dtype);
  const size_t tok = (size_t)d.H * d.dh;
  // splits of each launch's slots (one launch per kMaxSlots sequences)
  std::vector<int32_t> nr(n_seq), pp(n_seq);
  std::vector<int32_t> stride((n_seq + kMaxSlots - 1) / kMaxSlots, 1);
  for (int i = 0; i < n_seq; ++i) {
    nr[i] = n_read_of(st, seq_ids[i], query_block[i]);
    pp[i] = pages_per_split(nr[i], min_pages_decode(d.dh));
    int32_t& w = stride[i / kMaxSlots];
    w = std::max(w, (int32_t)total_splits(nr[i], pp[i]));
  }
  if (ws_ext) {
    for (size_t c = 0; c < stride.size(); ++c) {
      const size_t n = std::min(kMaxSlots, n_seq - (int)c * kMaxSlots);
      const size_t need = n * d.H * (size_t)stride[c] * (d.dh + 4);
      if (need > ws_ext_floats)
        return fail(SMEM_EINVAL, "split partials of %zu sequences x %d heads x %d splits need %zu floats; the "
                                 "scratch holds %zu", n, d.H, stride[c], need, ws_ext_floats);
    }
  }
  for (int i0 = 0; i0 < n_seq; i0 += kMaxSlots) {
    const int n = std::min(kMaxSlots, n_seq - i0);
    ReaderArgs a;
    memset(&a, 0, sizeof a);
    a.q = (const char*)q + i0 * tok * es;
    a.out = (char*)out + i0 * tok * es;
    if (n_given == 4) {
      a.k_new = (const char*)k_new + i0 * tok * es;
      a.v_new = (const char*)v_new + i0 * tok * es;
      a.k_in = (const char*)k_cache + (size_t)i0 * d.b * tok * es;
      a.v_in = (const char*)v_cache + (size_t)i0 * d.b * tok * es;
      a.k_cache_w = (char*)k_cache + (size_t)i0 * d.b * tok * es;
      a.v_cache_w = (char*)v_cache + (size_t)i0 * d.b * tok * es;
    }
    a.null_kv = null_kv;
    a.pages = st->d_pages;
    a.live_page = st->d_live_page;
    a.ws = ws_ext ? ws_ext : st->d_ws;
    a.ws_stride = ws_ext ? stride[i0 / kMaxSlots] : kSplitStride;
    a.max_blocks = d.max_blocks;
    a.H = d.H; a.b = d.b; a.nq = 1; a.intra_mode = 2;
    a.n_slots = n; a.scale_log2 = scale_log2;
    rope_args(a, st, rope);
    for (int i = 0; i < n; ++i) {
      const int sq = seq_ids[i0 + i];
      a.seq[i] = sq;
      a.qblk[i] = query_block[i0 + i];
      a.n_read[i] = nr[i0 + i];
      a.pps[i] = pp[i0 + i];
      a.aux[i] = n_given == 4 ? pos[i0 + i] : 0;
    }
    hipError_t e = launch_reader_valu(d.dtype, d.b, d.dh, a, s);
    if (e != hipSuccess) return hip_fail(e, "decode launch");
  }
  return SMEM_OK;
}

extern "C" {

smem_status smem_reader_prefill_block(smem_store* st, int32_t n_seq, const int32_t* seq_ids,
                                      const int32_t* query_block, const void* q, const void* k_intra,
                                      const void* v_intra, const void* null_kv, void* out, hipStream_t s) {
  return prefill_impl(st, nullptr, n_seq, seq_ids, query_block, q, k_intra, v_intra, null_kv, out, s);
}

smem_status smem_reader_prefill_block_rope(smem_store* st, const smem_rope* rope, int32_t n_seq,
                                           const int32_t* seq_ids, const int32_t* query_block, const void* q,
                                           const void* k_intra, const void* v_intra, const void* null_kv,
                                           void* out, hipStream_t s) {
  if (!rope) return fail(SMEM_EINVAL, "rope is NULL");
  return prefill_impl(st, rope, n_seq, seq_ids, query_block, q, k_intra, v_intra, null_kv, out, s);
}

smem_status smem_reader_decode(smem_store* st, int32_t n_seq, const int32_t* seq_ids, const int32_t* query_block,
                               const int32_t* pos, const void* q, const void* k_new, const void* v_new,
                               void* k_cache, void* v_cache, const void* null_kv, void* out, hipStream_t s) {
  return decode_impl(st, nullptr, n_seq, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv,
                     out, nullptr, 0, s);
}

smem_status smem_reader_decode_rope(smem_store* st, const smem_rope* rope, int32_t n_seq, const int32_t* seq_ids,
                                    const int32_t* query_block, const int32_t* pos, const void* q,
                                    const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                                    const void* null_kv, void* out, hipStream_t s) {
  if (!rope) return fail(SMEM_EINVAL, "rope is NULL");
  return decode_impl(st, rope, n_seq, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv,
                     out, nullptr, 0, s);
}

size_t smem_rows_bytes(const smem_rows_desc* desc) {
  DevLayout L;
  if (!rows_layout_of(desc, &L)) return 0;
  return L.total;
}

smem_status smem_rows_create(const smem_rows_desc* desc, void* dev_pool, size_t pool_bytes, hipStream_t s,
                             smem_store** out) {
  if (!out) return fail(SMEM_EINVAL, "out is NULL");
  *out = nullptr;
  DevLayout L;
  if (!rows_layout_of(desc, &L))
    return fail(SMEM_EINVAL, "invalid row store descriptor (need n_seq, max_blocks, n_pages >= 1, b in {16,64}, "
                             "d in {512,1024,2048}, dtype BF16)");
  if (!dev_pool) return fail(SMEM_EINVAL, "dev_pool is NULL");
  if (pool_bytes < L.total) return fail(SMEM_ENOMEM, "pool has %zu bytes, row store needs %zu", pool_bytes, L.total);
  if (((uintptr_t)dev_pool & 255u) != 0) return fail(SMEM_EINVAL, "dev_pool must be 256-byte aligned");
  smem_store* st = new (std::nothrow) smem_store();
  if (!st) return fail(SMEM_ENOMEM, "host allocation failed");
  st->d = smem_store_desc{desc->n_seq, desc->max_blocks, desc->n_pages, desc->b, 1, 0, BF16};
  st->kind = 1;
  st->rows_d = desc->d;
  st->lay = L;
  st->table.assign((size_t)desc->n_seq * desc->max_blocks, -1);
  st->live.assign(desc->n_seq, LiveSet());
  for (auto& lv : st->live) lv.init(desc->max_blocks);
  st->free_pages.resize(desc->n_pages);
  for (int i = 0; i < desc->n_pages; ++i) st->free_pages[i] = desc->n_pages - 1 - i;
  st->pool = (char*)dev_pool;
  st->d_table = (int32_t*)(st->pool + L.off_table);
  st->d_live_page = (int32_t*)(st->pool + L.off_live_page);
  st->d_live_blk = (int32_t*)(st->pool + L.off_live_blk);
  st->d_n_live = (int32_t*)(st->pool + L.off_n_live);
  st->d_ws = (float*)(st->pool + L.off_ws);
  st->d_pages = st->pool + L.off_pages;
  hipError_t e = launch_init_meta(st->d_table, st->d_n_live, st->table.size(), desc->n_seq, s);
  if (e != hipSuccess) {
    delete st;
    return hip_fail(e, "row store init");
  }
  *out = st;
  return SMEM_OK;
}

smem_status smem_rows_put_block(smem_store* st, int32_t seq, int32_t block_idx, const void* rows, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->kind != 1) return fail(SMEM_EINVAL, "not a row store");
  const auto& d = st->d;
  if (seq < 0 || seq >= d.n_seq) return fail(SMEM_EINVAL, "seq %d out of range [0, %d)", seq, d.n_seq);
  if (block_idx < 0 || block_idx >= d.max_blocks)
    return fail(SMEM_EINVAL, "block index %d out of range [0, %d)", block_idx, d.max_blocks);
  if (!rows || !aligned16(rows)) return fail(SMEM_EINVAL, "rows must be a 16-byte aligned device pointer");
  const size_t ti = (size_t)seq * d.max_blocks + block_idx;
  if (st->table[ti] >= 0) return fail(SMEM_EEXIST, "block %d of sequence %d is occupied", block_idx, seq);
  if (st->free_pages.empty()) return fail(SMEM_ENOMEM, "no free page (%d pages)", d.n_pages);
  const int32_t page = st->free_pages.back();
  hipError_t e = launch_copy16((char*)st->d_pages + (size_t)page * page_bytes(st), rows, page_bytes(st), s);
  if (e != hipSuccess) return hip_fail(e, "row insert");
  smem_status r = push_edits(st, {seq}, {block_idx}, {page}, s);
  if (r != SMEM_OK) return r;
  st->free_pages.pop_back();
  st->table[ti] = page;
  st->live[seq].insert(block_idx);
  return SMEM_OK;
}

smem_status smem_rows_export(smem_store* st, int32_t seq, int32_t* live_idx, int32_t* n_live, void* rows_out,
                             hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->kind != 1) return fail(SMEM_EINVAL, "not a row store");
  if (seq < 0 || seq >= st->d.n_seq) return fail(SMEM_EINVAL, "seq %d out of range [0, %d)", seq, st->d.n_seq);
  if (!aligned16(rows_out)) return fail(SMEM_EINVAL, "rows_out must be 16-byte aligned");
  const auto& lv = st->live[seq];
  if (n_live) *n_live = (int32_t)lv.size();
  if (live_idx) lv.copy_to(live_idx);
  if (rows_out) {
    const size_t pb = page_bytes(st);
    std::vector<int32_t> idx((size_t)lv.size());
    lv.copy_to(idx.data());
    for (size_t i = 0; i < idx.size(); ++i) {
      const int32_t page = st->table[(size_t)seq * st->d.max_blocks + idx[i]];
      hipError_t e = launch_copy16((char*)rows_out + i * pb, (const char*)st->d_pages + (size_t)page * pb, pb, s);
      if (e != hipSuccess) return hip_fail(e, "row export");
    }
  }
  return SMEM_OK;
}

smem_status smem_reader_decode_rows(smem_store* st, const smem_rows_layer* layer, int32_t n_seq,
                                    const int32_t* seq_ids, const int32_t* query_block, const int32_t* pos,
                                    const void* q, const void* k_new, const void* v_new, void* k_cache,
                                    void* v_cache, void* out, hipStream_t s) {
  if (!st) return fail(SMEM_EINVAL, "store is NULL");
  if (st->kind != 1) return fail(SMEM_EINVAL, "not a row store");
  if (!layer) return fail(SMEM_EINVAL, "layer is NULL");
  const int H = layer->H, dh = layer->dh, D = st->rows_d, b = st->d.b;
  if (H < 1 || H > kRowsMaxHeads || !(dh == 32 || dh == 64 || dh == 128))
    return fail(SMEM_EINVAL, "layer shape H=%d dh=%d (need 1 <= H <= %d, dh in {32,64,128})", H, dh, kRowsMaxHeads);
  const int ht = (H + 15) / 16;
  if (!layer->w_k || !layer->w_v) return fail(SMEM_EINVAL, "w_k and w_v are required");
  if (n_seq < 0) return fail(SMEM_EINVAL, "n_seq < 0");
  if (n_seq == 0) return SMEM_OK;
  if (!seq_ids || !query_block || !q || !out) return fail(SMEM_EINVAL, "seq_ids, query_block, q, out are required");
  const int n_given = (k_new != nullptr) + (v_new != nullptr) + (k_cache != nullptr) + (v_cache != nullptr);
  if (n_given != 0 && n_given != 4) return fail(SMEM_EINVAL, "k_new, v_new, k_cache, v_cache: all or none");
  if (n_given == 4 && !pos) return fail(SMEM_EINVAL, "pos is required with in-block keys");
  if (!aligned16(q) || !aligned16(out) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) ||
      !aligned16(v_cache) || !aligned16(layer->w_k) || !aligned16(layer->w_v) || !aligned16(layer->null_row) ||
      !aligned16(layer->null_kv))
    return fail(SMEM_EINVAL, "tensors must be 16-byte aligned");
  std::set<int32_t> seen;
  for (int i = 0; i < n_seq; ++i) {
    if (seq_ids[i] < 0 || seq_ids[i] >= st->d.n_seq) return fail(SMEM_EINVAL, "seq_ids[%d] = %d out of range", i, seq_ids[i]);
    if (query_block[i] < 0 || query_block[i] > st->d.max_blocks)
      return fail(SMEM_EINVAL, "query_block[%d] = %d out of range [0, %d]", i, query_block[i], st->d.max_blocks);
    if (n_given == 4 && (pos[i] < 0 || pos[i] >= b)) return fail(SMEM_EINVAL, "pos[%d] = %d out of range [0, %d)", i, pos[i], b);
    if (!seen.insert(seq_ids[i]).second) return fail(SMEM_EINVAL, "sequence %d appears twice", seq_ids[i]);
  }
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)dh));
  const size_t tok = (size_t)H * dh;
  const auto& L = st->lay;
  uint16_t* qabs = (uint16_t*)(st->pool + L.off_qabs);
  float* intra = (float*)(st->pool + L.off_intra);
  uint16_t* null_kv = (uint16_t*)(st->pool + L.off_null_kv);
  float* part = (float*)(st->pool + L.off_part);
  // the null row through the layer's maps: given, or mapped by the first launch
  bool null_done = layer->null_kv != nullptr;
  int i0 = 0;
  while (i0 < n_seq) {
    // a launch: at most kMaxSlots sequences whose split partials fit the workspace
    int n = 0, used = 0;
    int32_t nread[kMaxSlots];
    while (i0 + n < n_seq && n < kMaxSlots) {
      const int nr = n_read_of(st, seq_ids[i0 + n], query_block[i0 + n]);
      const int sp = splits_rows(nr) * ht;
      if (n > 0 && used + sp > L.part_cap) break;
      nread[n] = nr;
      used += sp;
      ++n;
    }
    RowsPrepArgs pa;
    memset(&pa, 0, sizeof pa);
    pa.q = (const uint16_t*)q + i0 * tok;
    pa.w_k = (const uint16_t*)layer->w_k;
    pa.w_v = (const uint16_t*)layer->w_v;
    pa.null_row = null_done ? nullptr : (const uint16_t*)layer->null_row;
    pa.qabs = qabs;
    pa.null_kv = null_kv;
    pa.d = D; pa.H = H; pa.ht = ht; pa.n_slots = n; pa.scale_log2 = scale_log2;
    RowsArgs ra;
    memset(&ra, 0, sizeof ra);
    ra.pages = (const uint16_t*)st->d_pages;
    ra.live_page = st->d_live_page;
    ra.qabs = qabs;
    ra.part = part;
    ra.intra = intra;
    ra.w_v = (const uint16_t*)layer->w_v;
    ra.ubuf = qabs;     // the absorbed queries are spent once the row reader has run
    ra.sw = (float*)(st->pool + L.off_sw);
    ra.out = (uint16_t*)out + i0 * tok;
    ra.max_blocks = st->d.max_blocks; ra.b = b; ra.H = H; ra.ht = ht; ra.n_slots = n;
    int base = 0;
    for (int i = 0; i < n; ++i) {
      ra.seq[i] = seq_ids[i0 + i];
      ra.n_read[i] = nread[i];
      ra.pps[i] = pps_rows(nread[i]);
      ra.pbase[i] = base;
      base += splits_rows(nread[i]) * ht;
    }
    hipError_t e = launch_rows(D, dh, ra, pa, 0, s);
    if (e != hipSuccess) return hip_fail(e, "absorbed queries");
    null_done = true;
    // in-block keys and the mapped null row: the reader's extra split
    ra.q = (const uint16_t*)q + i0 * tok;
    if (n_given == 4) {
      ra.k_new = (const uint16_t*)k_new + i0 * tok;
      ra.v_new = (const uint16_t*)v_new + i0 * tok;
      ra.k_cache = (uint16_t*)k_cache + (size_t)i0 * b * tok;
      ra.v_cache = (uint16_t*)v_cache + (size_t)i0 * b * tok;
    }
    ra.null_kv = layer->null_kv ? (const uint16_t*)layer->null_kv : layer->null_row ? null_kv : nullptr;
    ra.intra_w = intra;
    ra.scale_log2 = scale_log2;
    for (int i = 0; i < n; ++i) ra.pos[i] = n_given == 4 ? pos[i0 + i] : 0;
    e = launch_rows(D, dh, ra, pa, 1, s);
    if (e != hipSuccess) return hip_fail(e, "row reader");
    i0 += n;
  }
  return SMEM_OK;
}

size_t smem_rope_bytes(const smem_rope_desc* desc) { return rope_bytes_of(desc); }

smem_status smem_rope_create(const smem_rope_desc* desc, void* dev_buf, size_t bytes, hipStream_t s,
                             smem_rope** out) {
  if (!out) return fail(SMEM_EINVAL, "out is NULL");
  *out = nullptr;
  const size_t need = rope_bytes_of(desc);
  if (need == 0) return fail(SMEM_EINVAL, "invalid rotary descriptor");
  if (!dev_buf) return fail(SMEM_EINVAL, "dev_buf is NULL");
  if (((uintptr_t)dev_buf & 255u) != 0) return fail(SMEM_EINVAL, "dev_buf must be 256-byte aligned");
  if (bytes < need) return fail(SMEM_ENOMEM, "rotary table needs %zu bytes, %zu given", need, bytes);
  smem_rope* r = new (std::nothrow) smem_rope;
  if (!r) return fail(SMEM_ENOMEM, "host allocation failed");
  r->d = *desc;
  r->table = (float*)dev_buf;
  hipError_t e = launch_rope_table(r->table, desc->dh, desc->n_phases, desc->base, s);
  if (e != hipSuccess) {
    delete r;
    return hip_fail(e, "rotary table");
  }
  *out = r;
  return SMEM_OK;
}

smem_status smem_rope_destroy(smem_rope* rope) {
  delete rope;
  return SMEM_OK;
}

}  // extern "C"
