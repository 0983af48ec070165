/*
 * smem.h -- C ABI of the MI355X (gfx950) SMem attention hot path.
 *
 * SMem ("Memory as a Cache: Exact Context Reuse and Deletion by
 * Construction") splits a sequence into blocks of b tokens.  An encoder
 * attends only inside each block, so every block's memory rows are a function
 * of that block and its index alone (Section 2, "Model"; Proposition 1).  The
 * memory is the multiset of all blocks' rows, listed canonically by block
 * index (Section 2, "Model").  Deleting a present block gives exactly the
 * memory in which it was never encoded (Theorem 1).  A reader query at
 * in-block position t of block J attends to its own block's keys 0..t and to
 * the memory rows of strictly earlier blocks j < J (Section 2, "Model";
 * Appendix A, "Reader").  Here the two key sets, plus an optional null row,
 * are read under one softmax.
 *
 * Conventions shared by every call
 *  - Tensors are caller-owned DEVICE pointers, row-major, with no padding:
 *      token tensors   [rows, H, dh]    (rows = n_blocks*b, n_seq*b or n_seq)
 *      null_kv         [2, H, dh]       (key vector per head, then value)
 *    Their element type is the store's dtype: fp32, or bf16 computed with
 *    fp32 accumulation.
 *  - Index arrays (seq_ids, block_idx, query_block, pos, live_idx, n_live)
 *    are HOST pointers.  They are read, or written, before the call returns.
 *  - Every device operation is enqueued on the caller's stream `s`.  Store
 *    metadata changes take effect on the host immediately.  Their device copy
 *    is updated by kernels enqueued on `s`, so stream order decides which
 *    memory state a later read sees.  Calls on one store from different
 *    streams must be ordered by the caller.
 *  - Errors: every argument and store-state check runs before anything is
 *    enqueued.  A call that returns an error has changed nothing (no partial
 *    edits).  SMEM_EHIP means a HIP launch or copy failed.
 *    smem_last_error() gives a message for the calling thread's last error.
 *  - No call allocates device memory.  The store lives in a caller-provided
 *    device buffer of smem_store_bytes() bytes.
 *  - Softmax scale is 1/sqrt(dh) (Lemma 1's 1/sqrt(d) for the head width).
 *  - Supported shapes: b in {16, 64}, dh in {32, 64, 128}, 1 <= H <= 64.
 */
#ifndef SMEM_H
#define SMEM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SMEM_OK = 0,
  SMEM_EINVAL = 1,  /* bad argument, shape or dtype */
  SMEM_ENOMEM = 2,  /* page pool full, or pool buffer too small */
  SMEM_ENOENT = 3,  /* delete/export of an absent block (Theorem 1: only a present block can be deleted) */
  SMEM_EEXIST = 4,  /* insert into an occupied block index */
  SMEM_EHIP = 5     /* a HIP runtime call failed */
} smem_status;

typedef enum { SMEM_F32 = 0, SMEM_BF16 = 1 } smem_dtype;

/* In-block mask of the encoder.  The paper's encoder is bidirectional inside
 * a block (Section 2, "Model"; Appendix A, "Encoder").  The causal mode
 * includes the query's own key. */
typedef enum { SMEM_MASK_BIDIR = 0, SMEM_MASK_CAUSAL = 1 } smem_mask;

/* Shape of one store.  A store holds n_pages blocks at once across
 * n_seq sequences.  Each sequence has block indices 0..max_blocks-1. */
typedef struct {
  int32_t n_seq;
  int32_t max_blocks;
  int32_t n_pages;
  int32_t b;
  int32_t H;
  int32_t dh;
  int32_t dtype;    /* smem_dtype */
} smem_store_desc;

/* Attention shape of an encoder call: block size, heads, head width, dtype. */
typedef struct {
  int32_t b;
  int32_t H;
  int32_t dh;
  int32_t dtype;    /* smem_dtype */
} smem_attn_desc;

typedef struct smem_store smem_store;  /* opaque; host metadata + device layout */

/* Device bytes the caller must provide for a store of this shape.
 * Covers the page pool, the device block table and live lists, and the
 * split-K workspace.  Returns 0 for an invalid descriptor. */
size_t smem_store_bytes(const smem_store_desc* desc);

/* Create a store over a caller-owned device buffer.
 * The buffer needs pool_bytes >= smem_store_bytes(desc) and 256-byte
 * alignment; it stays owned by the caller and must outlive the store.
 * Device metadata is initialised on stream s.
 * dev_pool == NULL creates a metadata-only store: the edit calls
 * (put/delete/export with NULL tensors) validate and update host metadata
 * only, and every call that needs device memory returns SMEM_EINVAL. */
smem_status smem_store_create(const smem_store_desc* desc, void* dev_pool, size_t pool_bytes,
                              hipStream_t s, smem_store** out);

/* Free the host metadata.  The device buffer is untouched.  NULL is a no-op. */
smem_status smem_store_destroy(smem_store* st);

/* Insert precomputed memory rows of block `block_idx` of sequence `seq`
 * (the append of Section 2: m <- m (+) mu_j, O(b) work).
 * k_rows, v_rows: device [b, H, dh].  SMEM_EEXIST if the index is occupied;
 * SMEM_ENOMEM if no page is free.  On a metadata-only store, pass NULL rows. */
smem_status smem_store_put_block(smem_store* st, int32_t seq, int32_t block_idx,
                                 const void* k_rows, const void* v_rows, hipStream_t s);

/* Insert precomputed rows of n_blocks blocks at once: block i's rows are
 * rows i*b .. i*b+b-1 of k_rows, v_rows (device [n_blocks*b, H, dh]) and go to
 * block block_idx[i] of sequence seq_ids[i].  All-or-nothing, errors as
 * smem_store_put_block (duplicates are SMEM_EEXIST). */
smem_status smem_store_put_blocks(smem_store* st, int32_t n_blocks, const int32_t* seq_ids,
                                  const int32_t* block_idx, const void* k_rows, const void* v_rows,
                                  hipStream_t s);

/* Block-local encoder attention (Section 2, "Model"; Appendix A, "Encoder").
 * Each (block, head) pair is computed on its own:
 *   O = softmax_mask(Q K^T / sqrt(dh)) V,  the mask limited to the block.
 * q, k, v: device [n_blocks*b, H, dh] (block-major, then token, head, dim).
 * out: device, same shape, or NULL when the rows only go into the store.
 * st == NULL: attention only; seq_ids/block_idx are ignored.
 * st != NULL: block i's output is inserted as memory block block_idx[i] of
 *   sequence seq_ids[i].  Its key plane and value plane both equal O (identity
 *   projections).  Every target index is checked first (SMEM_EEXIST,
 *   duplicates included), so the insert is all-or-nothing.  `shape` must
 *   equal the store's. */
smem_status smem_encode_blocks(smem_store* st, const smem_attn_desc* shape, int32_t n_blocks,
                               const int32_t* seq_ids, const int32_t* block_idx,
                               const void* q, const void* k, const void* v, void* out,
                               int32_t mask, hipStream_t s);

/* Re-encode present blocks in place (Section 2, the slot scheme; Appendix A,
 * "Length extension"): beyond the trained block count an append moves the
 * most recent blocks to new slots, and each such block is encoded again from
 * its new inputs at O(b) cost.  Arguments are those of smem_encode_blocks;
 * st is required.  Every (seq_ids[i], block_idx[i]) must hold a block
 * (SMEM_ENOENT otherwise, duplicates are SMEM_EINVAL), all checked before
 * anything is enqueued.  The new rows overwrite the block's own page on
 * stream s: the table and the live lists do not change, and the result is
 * the store obtained by deleting the blocks and encoding them anew.  Reads
 * enqueued earlier on s see the old rows, later ones the new rows. */
smem_status smem_reencode_blocks(smem_store* st, const smem_attn_desc* shape, int32_t n_blocks,
                                 const int32_t* seq_ids, const int32_t* block_idx,
                                 const void* q, const void* k, const void* v, void* out,
                                 int32_t mask, hipStream_t s);

/* Reader attention for whole query blocks: block-skip serving (Section 3.1).
 * Row i of q/k_intra/v_intra/out, of shape [b, H, dh] each, is block
 * query_block[i] of sequence seq_ids[i].  Query t of head h reads, under
 * one softmax, this key list in canonical order:
 *   [null row] ++ rows of every live block j < query_block[i], ascending j
 *   ++ in-block keys 0..t.
 * k_intra = v_intra = NULL: no in-block keys (the paper's cross-attention
 * sub-layer alone).  query_block[i] = 0 with null_kv = NULL: in-block causal
 * attention alone (the paper's self-attention sub-layer).  An empty key set
 * gives a zero output.
 * q, k_intra, v_intra, out: device [n_seq*b, H, dh].  null_kv: device
 * [2, H, dh] or NULL.  A sequence may appear more than once (with several
 * query blocks: a block-parallel pass over one sequence). */
smem_status smem_reader_prefill_block(smem_store* st, int32_t n_seq, const int32_t* seq_ids,
                                      const int32_t* query_block, const void* q,
                                      const void* k_intra, const void* v_intra,
                                      const void* null_kv, void* out, hipStream_t s);

/* Reader attention for one new token per sequence: KV-cached decode
 * (Section 3.1; Appendix K, "Decode").
 * The new key/value pair is first written into the in-block cache at pos[i]
 * (0 <= pos[i] < b).  The query then reads
 *   [null row] ++ memory rows of live blocks j < query_block[i] ++ cache rows 0..pos[i].
 * q, k_new, v_new, out: device [n_seq, H, dh].  k_cache, v_cache: device
 * [n_seq*b, H, dh], updated in place at row pos[i] only.
 * k_new = v_new = k_cache = v_cache = NULL: memory-only read.
 * Each seq_ids entry may appear only once. */
smem_status smem_reader_decode(smem_store* st, int32_t n_seq, const int32_t* seq_ids,
                               const int32_t* query_block, const int32_t* pos, const void* q,
                               const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                               const void* null_kv, void* out, hipStream_t s);

/* smem_reader_decode for callers that cannot allocate device memory or touch
 * a workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): same arguments, layouts, results (bit for bit) and
 * errors, but the split partials go to a 16 MiB device array that the library
 * holds on each GPU it runs on, instead of the store's workspace.  It calls no
 * allocator.  The partials of one launch (up to 128 sequences) take
 * n_seq x H x splits x (dh + 4) floats, splits = ceil(memory pages read /
 * max(8, ceil(pages / 64))) + 1 for the longest read of the launch; a call
 * that needs more than 4 Mi floats returns SMEM_EINVAL before anything is
 * enqueued.  Every call on one GPU shares that GPU's array: calls that overlap
 * on one GPU (unordered streams or threads) race; calls ordered on one stream
 * do not.  No rotary variant. */
smem_status smem_reader_decode_static(smem_store* st, int32_t n_seq, const int32_t* seq_ids,
                                      const int32_t* query_block, const int32_t* pos, const void* q,
                                      const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                                      const void* null_kv, void* out, hipStream_t s);

/* Exact deletion (Theorem 1): remove block `block_idx` of sequence `seq`.
 * The remaining blocks keep their indices, and every later read equals a
 * read of the memory in which the block was never inserted.  Cost is O(1)
 * page bookkeeping plus a rebuild of the sequence's dense live list
 * (indices only, no rows move).  SMEM_ENOENT if the block is absent.
 * scrub != 0 also zeroes the freed page on stream s. */
smem_status smem_delete_block(smem_store* st, int32_t seq, int32_t block_idx, int32_t scrub,
                              hipStream_t s);

/* Canonical export of one sequence's memory: blocks in ascending index, each
 * block's b rows in order (Section 2, "Model"; Appendix B, gate G8).
 * live_idx: host int32[max_blocks] or NULL; receives the live block indices.
 * n_live: host, receives their count.  k_out, v_out: device
 * [n_live*b, H, dh], or both NULL to list indices only. */
smem_status smem_store_export(smem_store* st, int32_t seq, int32_t* live_idx, int32_t* n_live,
                              void* k_out, void* v_out, hipStream_t s);

/* ------------------------------------------------------------------------
 * SMem+RoPE composite (Section 3, "SMem composes with RoPE"; the composite's
 * appendix, variant v2; saturating reading in the needle appendix).
 * Memory rows carry no position.  Rotary phases turn queries and keys, never
 * values: adjacent dimensions (2k, 2k+1) form pair k, turned by the angle
 * phase * base^(-2k/dh).  Inside a block the phase is the in-block offset
 * (queries and keys of the encoder and of the reader's in-block keys).
 * Across blocks it is the block index: the query of block J has phase J, a
 * memory row of block j has phase max(j, J - W) when max_offset = W > 0 (the
 * saturating reading) and j when max_offset = 0, and the null row is a row of
 * index 0 (phase max(0, J - W), or 0).  Under the joint softmax the query
 * takes phase t (its in-block offset) against its in-block keys and phase J
 * against the null row and the memory.
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t dh;          /* head width served: 32, 64 or 128 */
  int32_t n_phases;    /* phases 0..n_phases-1 are tabulated */
  int32_t max_offset;  /* W > 0: saturating block phases; 0: none */
  int32_t reserved;    /* must be 0 */
  double base;         /* frequency base (10^4 in the paper), > 1 */
} smem_rope_desc;

typedef struct smem_rope smem_rope;   /* opaque; a rotary table in device memory */

/* Device bytes of the rotary table: n_phases * dh fp32 (cos, sin pairs),
 * rounded up to 256.  0 for an invalid descriptor. */
size_t smem_rope_bytes(const smem_rope_desc* desc);

/* Create a rotary configuration over a caller-owned device buffer (256-byte
 * aligned, >= smem_rope_bytes); the table is computed on stream s in fp64 and
 * stored as fp32.  The buffer stays owned by the caller. */
smem_status smem_rope_create(const smem_rope_desc* desc, void* dev_buf, size_t bytes, hipStream_t s,
                             smem_rope** out);
smem_status smem_rope_destroy(smem_rope* rope);

/* smem_encode_blocks with rotary phases on queries and keys (in-block
 * offsets 0..b-1; needs n_phases >= b and rope dh == shape dh).  The rows put
 * into the store are the attention outputs, unturned, as in the base call. */
smem_status smem_encode_blocks_rope(smem_store* st, const smem_attn_desc* shape, const smem_rope* rope,
                                    int32_t n_blocks, const int32_t* seq_ids, const int32_t* block_idx,
                                    const void* q, const void* k, const void* v, void* out,
                                    int32_t mask, hipStream_t s);

/* smem_reader_prefill_block with rotary phases as above.  The table must hold
 * every phase the call uses: n_phases > max(b - 1, P) with P = min(J, W)
 * (saturating) or J (none) over the calls' query blocks J; SMEM_EINVAL
 * otherwise. */
smem_status smem_reader_prefill_block_rope(smem_store* st, const smem_rope* rope, int32_t n_seq,
                                           const int32_t* seq_ids, const int32_t* query_block,
                                           const void* q, const void* k_intra, const void* v_intra,
                                           const void* null_kv, void* out, hipStream_t s);

/* smem_reader_decode with rotary phases as above (the query's in-block
 * offset is pos[i]; the cache holds unturned keys).  Same table bound. */
smem_status smem_reader_decode_rope(smem_store* st, const smem_rope* rope, int32_t n_seq,
                                    const int32_t* seq_ids, const int32_t* query_block, const int32_t* pos,
                                    const void* q, const void* k_new, const void* v_new, void* k_cache,
                                    void* v_cache, const void* null_kv, void* out, hipStream_t s);

/* ------------------------------------------------------------------------
 * Row stores: decode from the memory rows (Appendix K, recomputing K/V from
 * the memory rows instead of storing it; Appendix A, "Positions and memory":
 * one row plane is shared by all D reader layers, and each layer applies its
 * own key and value maps, the null row included).
 * A row store is an smem_store whose pages hold one block's b rows of width
 * d (bf16), no key/value planes.  smem_store_destroy, smem_store_stats and
 * smem_delete_block apply to it; the key/value calls (put_block, export,
 * encode into it, prefill, decode) return SMEM_EINVAL, and the row calls
 * return SMEM_EINVAL on a key/value store.
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_seq;
  int32_t max_blocks;
  int32_t n_pages;
  int32_t b;          /* 16 or 64 */
  int32_t d;          /* row width: 512, 768, 1024 or 2048 */
  int32_t dtype;      /* SMEM_BF16 */
} smem_rows_desc;

/* One reader layer's maps, device bf16: w_k, w_v [H*dh, d] (a linear
 * layer's out x in layout: the key of row r is w_k r, head h taking outputs
 * h*dh .. h*dh+dh-1), null_row [d] or NULL.  null_kv: NULL, or the null
 * row already through the maps, [2, H, dh] (keys then values; null_row is
 * then ignored), for callers that map it once rather than on every call.
 * 1 <= H <= 64, dh in {32, 64, 128}. */
typedef struct {
  int32_t H;
  int32_t dh;
  const void* w_k;
  const void* w_v;
  const void* null_row;
  const void* null_kv;
} smem_rows_layer;

/* Device bytes of a row store: pages, block table, live lists and the
 * decode workspace.  0 for an invalid descriptor. */
size_t smem_rows_bytes(const smem_rows_desc* desc);

/* Create a row store over a caller-owned device buffer (256-byte aligned,
 * >= smem_rows_bytes); metadata initialised on stream s. */
smem_status smem_rows_create(const smem_rows_desc* desc, void* dev_pool, size_t pool_bytes, hipStream_t s,
                             smem_store** out);

/* Insert the rows [b, d] of block block_idx of sequence seq (device, copied
 * into a free page).  Errors as smem_store_put_block. */
smem_status smem_rows_put_block(smem_store* st, int32_t seq, int32_t block_idx, const void* rows, hipStream_t s);

/* Canonical export of one sequence's rows: live_idx as in smem_store_export,
 * rows_out device [n_live*b, d] or NULL. */
smem_status smem_rows_export(smem_store* st, int32_t seq, int32_t* live_idx, int32_t* n_live, void* rows_out,
                             hipStream_t s);

/* Reader decode of one layer from the row plane: the same read as
 * smem_reader_decode with every memory row's key and value given by the
 * layer's maps (k = w_k row, v = w_v row, per head slice) and the null row
 * (if any) mapped the same way.  The maps are never applied row by row: the
 * query is mapped into row space (w_k^h q), rows are weighted there, and the
 * weighted row sum is mapped back once (w_v^h), which is the same
 * arithmetic up to rounding.  q, k_new, v_new, out: [n_seq, H, dh];
 * k_cache, v_cache: [n_seq*b, H, dh] or all four NULL; pos as in
 * smem_reader_decode.  bf16. */
smem_status smem_reader_decode_rows(smem_store* st, const smem_rows_layer* layer, int32_t n_seq,
                                    const int32_t* seq_ids, const int32_t* query_block, const int32_t* pos,
                                    const void* q, const void* k_new, const void* v_new, void* k_cache,
                                    void* v_cache, void* out, hipStream_t s);

/* ------------------------------------------------------------------------
 * The whole model at given weights (Section 2, "Model"; Appendix A).
 * Encoder: E pre-LN layers of block-local bidirectional attention and a GELU
 * feed-forward (hidden 4d); a block's memory rows are the LayerNorm of the
 * encoder's final state.  Reader: D pre-LN layers, each block-local causal
 * self-attention, cross-attention into the memory of strictly earlier blocks
 * with the null row (one learned d-vector through each layer's key and value
 * maps), and the feed-forward; then a final LayerNorm and the output head.
 * Input: token embedding plus a learned position embedding indexed by
 * min(block, n_pos/b - 1) * b + in-block offset (none when n_pos = 0).
 * Linear maps are x -> x W^T, W stored [out, in], no biases; LayerNorm
 * eps 1e-5 with a scale and a shift; GELU is the exact (erf) form.  bf16
 * weights and activations, fp32 accumulation, fp32 logits.
 * Each reader layer keeps its keys and values (the memory rows through its
 * maps) in a store of its own, so encode, serve, delete and re-encode are the
 * store operations applied to every layer; or (row_plane = 1) the rows are
 * kept once and every layer reads them through its maps.
 *
 * Weights: an array of smem_model_n_weights() device pointers, in order:
 *   tok_emb [vocab, d], pos_emb [n_pos, d] (NULL when n_pos = 0),
 *   per encoder layer: ln1_g, ln1_b [d], w_qkv [3d, d], w_o [d, d],
 *                      ln2_g, ln2_b [d], w_ff1 [4d, d], w_ff2 [d, 4d],
 *   mem_ln_g, mem_ln_b [d], null_row [d],
 *   per reader layer:  ln1_g, ln1_b, w_qkv [3d, d], w_o [d, d], ln2_g, ln2_b,
 *                      w_q, w_k, w_v, w_oc [d, d], ln3_g, ln3_b,
 *                      w_ff1 [4d, d], w_ff2 [d, 4d],
 *   fin_g, fin_b [d], w_head [vocab, d].
 * The weights stay owned by the caller and must outlive the model.
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t E;            /* encoder layers (>= 0) */
  int32_t D;            /* reader layers (>= 1) */
  int32_t d, H, dh;     /* width = H * dh, a multiple of 64, <= 2048; dh in {32, 64, 128} */
  int32_t b;            /* block size: 64 */
  int32_t vocab;
  int32_t n_pos;        /* learned positions, a multiple of b; 0: none */
  int32_t n_seq, max_blocks, n_pages;   /* every reader layer's memory store */
  int32_t max_tokens;   /* tokens one launch sequence processes (a multiple of b, <= 128 b);
                           longer calls are cut into chunks of this size */
  int32_t row_plane;    /* 0: every reader layer keeps its keys and values (key/value layers);
                           1: one row store shared by all reader layers, each layer's
                           cross-attention reading it through its own key and value maps at
                           decode time (Appendix K, decode recomputing K/V from the rows;
                           Appendix A, "Positions and memory").  d in {512, 768, 1024, 2048}.
                           A row-plane model encodes, decodes and deletes; block reads
                           (smem_model_read, smem_model_prefill) return SMEM_EINVAL. */
} smem_model_desc;

typedef struct smem_model smem_model;

/* Number of weight pointers, and device bytes of the model's pool (the
 * reader layers' stores, the activation workspace, the mapped null rows, the
 * decode caches of in-block keys and values, D x 2 x n_seq x b x d bf16). */
int32_t smem_model_n_weights(const smem_model_desc* desc);
size_t smem_model_bytes(const smem_model_desc* desc);

smem_status smem_model_create(const smem_model_desc* desc, const void* const* weights, void* dev_pool,
                              size_t pool_bytes, hipStream_t s, smem_model** out);
smem_status smem_model_destroy(smem_model* m);

/* Encode n_blocks blocks of sequence seq (tokens: device int32 [n_blocks*b];
 * block_idx host) and insert their keys and values into every reader layer:
 * the append of Section 2.  All-or-nothing as smem_encode_blocks. */
smem_status smem_model_encode(smem_model* m, int32_t seq, int32_t n_blocks, const int32_t* block_idx,
                              const int32_t* tokens, hipStream_t s);

/* The same for blocks of several sequences at once: block i is block
 * block_idx[i] of sequence seq_ids[i] (host arrays), its tokens
 * tokens[i*b .. i*b + b - 1] (device int32) -- e.g. the blocks completed by a
 * batch of decoding sequences.  All-or-nothing. */
smem_status smem_model_encode_blocks(smem_model* m, int32_t n_blocks, const int32_t* seq_ids,
                                     const int32_t* block_idx, const int32_t* tokens, hipStream_t s);

/* Reader pass for n_blocks query blocks of sequence seq (tokens: device int32
 * [n_blocks*b]; query_block host): each block reads the memory of the live
 * blocks below it.  logits: device fp32 [n_blocks*b, vocab].  A fully cached
 * context is served by reading its final block alone (block-skip serving,
 * Section 3.1); the cold pass encodes every block and reads every block. */
smem_status smem_model_read(smem_model* m, int32_t seq, int32_t n_blocks, const int32_t* query_block,
                            const int32_t* tokens, float* logits, hipStream_t s);

/* Prefill of blocks first_block .. first_block + n_blocks - 1 of sequence
 * seq (tokens: device int32 [n_blocks*b]): encode and insert them into every
 * reader layer, then run the reader on each of them; logits (device fp32
 * [b, vocab]) of the final block only.  first_block = 0 is the cold prefill
 * of a context; first_block > 0 with blocks 0 .. first_block - 1 cached is
 * partial reuse: only the blocks not yet cached are encoded before the read (Section 3.1).
 * The blocks must be absent (SMEM_EEXIST otherwise; nothing is changed). */
smem_status smem_model_prefill(smem_model* m, int32_t seq, int32_t first_block, int32_t n_blocks,
                               const int32_t* tokens, float* logits, hipStream_t s);

/* One KV-cached decode step (Section 3.1, "Decode"; the serving appendix's
 * batched decode) for sequences first_seq .. first_seq + n_seq - 1: token
 * tokens[i] (device int32) at in-block position pos[i] of block
 * query_block[i] (host arrays).  In every reader layer the token's key and
 * value go into the model's in-block cache of the sequence at pos[i]; the
 * self-attention reads cached positions 0..pos[i] of the block, the
 * cross-attention the memory of the live blocks below query_block[i] with
 * the null row.  logits: device fp32 [n_seq, vocab].  Decoding a block's
 * positions 0..b-1 in order reproduces the reader pass over the block up to
 * rounding; once its last token is decoded the caller appends the block with
 * smem_model_encode (its b tokens) and moves on to block + 1, position 0.
 * Positions of one sequence are decoded in order: position p reads the
 * cache entries 0..p-1 written by earlier steps. */
smem_status smem_model_decode(smem_model* m, int32_t first_seq, int32_t n_seq, const int32_t* query_block,
                              const int32_t* pos, const int32_t* tokens, float* logits, hipStream_t s);

/* Exact deletion of block block_idx of sequence seq from every reader layer
 * (Theorem 1).  SMEM_ENOENT if absent. */
smem_status smem_model_delete_block(smem_model* m, int32_t seq, int32_t block_idx, hipStream_t s);

/* The attention part of one self-attention sub-layer of the model (Section
 * 2, "Model"; Appendix A, "Encoder" and "Reader"): per block of 64 rows and
 * per head, out = softmax(q k^T / sqrt(d_h)) v over the block's own rows
 * (all of them: mask SMEM_MASK_BIDIR, the encoder; keys up to the query's
 * row: SMEM_MASK_CAUSAL, the reader), with q | k | v = LN(x) W_qkv^T, on the
 * kernels the model uses.
 *   n_blocks: blocks of 64 rows (<= 65535); d = H d_h, d % 64 == 0,
 *     d <= 2048, d_h in {32, 64, 128};
 *   x: device bf16 [n_blocks * 64, d]; ln_g, ln_b: device bf16 [d]
 *     (LayerNorm gain and shift, eps 1e-5); w_qkv: device bf16 [3d, d]
 *     (the q, k and v maps' rows in that order, head h in rows
 *     h d_h .. h d_h + d_h - 1 of each);
 *   path: 1 the q|k|v map, then the block-local attention launch; 0 the
 *     model's choice, which is path 1 (faster at every size measured on
 *     MI355X); 2 one fused launch per call (d_h = 32 and d a multiple of 256
 *     up to 1024 only, else SMEM_EINVAL);
 *   out: device bf16 [n_blocks * 64, d], head h in columns h d_h ..;
 *   work: device bf16 [4, n_blocks * 64, d] (normalized rows, q, k, v),
 *     caller-owned; may be NULL on the fused path with n_blocks * 64 <= 128.
 * Every path gives the same bits.  Pointers 16-byte aligned. */
smem_status smem_self_attention(int32_t n_blocks, int32_t d, int32_t H, const void* x, const void* ln_g,
                                const void* ln_b, const void* w_qkv, int32_t mask, int32_t path, void* out, void* work,
                                hipStream_t s);

/* One linear map of the model's layers (Appendix A: pre-LN layers, linear
 * maps without bias, a GELU feed-forward), on the same kernels and in the
 * same reduction order the model uses: y = epi(LN(x) W^T), or epi(x W^T)
 * with ln_g = ln_b = NULL.
 *   x: device bf16 [M, K] (K % 64 == 0); w: device bf16 [N, K];
 *   ln_g, ln_b: device bf16 [K] (LayerNorm gain and shift, eps 1e-5;
 *     K <= 2048) or both NULL;
 *   epi: 0 store bf16 [M, N]; 1 GELU (erf form) then bf16; 2 add res
 *     (device bf16 [M, N], may be y) then bf16; 3 store fp32 [M, N];
 *   ln_tmp: device bf16 [M, K]: receives LN(x) when ln_g is set and M > 128
 *     (those rows are normalised by a separate pass before the map; up to
 *     128 rows the map normalises them itself); else unused, may be NULL.
 * bf16 outputs need N % 4 == 0; every pointer 16-byte aligned.  Each output
 * element is computed in one order whatever M and N are, so a row's result
 * does not depend on the other rows.  SMEM_EINVAL for bad shapes. */
smem_status smem_linear(int32_t M, int32_t N, int32_t K, const void* x, const void* w, const void* ln_g,
                        const void* ln_b, int32_t epi, const void* res, void* y, void* ln_tmp, hipStream_t s);

/* Host-side facts about a store: pages in use and free. */
smem_status smem_store_stats(const smem_store* st, int32_t* pages_used, int32_t* pages_free);

/* Device copy of `bytes` from src to dst (device pointers, 16-byte aligned,
 * not overlapping) on stream s.  Not an operation of the method: a copy of
 * known size whose hardware traffic counters calibrate the counts of the
 * attention kernels.  via_lds = 0: through registers (16-byte loads and
 * stores; bytes a multiple of 16); via_lds = 1: through LDS by DMA, the way
 * the MFMA kernels bring pages in (bytes a multiple of 16384).  SMEM_EINVAL
 * for other sizes or flags. */
smem_status smem_device_copy(void* dst, const void* src, size_t bytes, int32_t via_lds, hipStream_t s);

const char* smem_status_string(smem_status st);

/* Message of the calling thread's last failed call ("" if none). */
const char* smem_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SMEM_H */
