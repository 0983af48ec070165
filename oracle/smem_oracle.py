"""fp64 CPU oracle of the SMem attention hot path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and it
imports nothing from the product path.

Everything here is the plain definition from the paper ("Memory as a Cache:
Exact Context Reuse and Deletion by Construction"), written with numpy in
float64, with no blocking, tiling, online softmax or split reduction:

* Encoder attention (Section 2, paragraph "Model"; Appendix A, "Encoder"):
  every block of b tokens is encoded independently; inside a block, each head
  computes softmax(Q K^T / sqrt(d_h)) V with the attention mask restricted to
  the block.  The paper's encoder is bidirectional inside the block; a causal
  in-block mask is the other supported mode.
* Memory (Section 2, "Model"; Theorem 1): the multiset of every block's b
  rows, listed canonically by block index; a block index holds at most one
  block, inserting into an occupied index and deleting an absent block are
  errors, and deleting a present block gives exactly the memory in which it
  was never inserted.
* Reader attention (Section 2, "Model"; Appendix A, "Reader"): a query at
  in-block position t of block J attends to its own block's keys 0..t and to
  the memory rows of strictly earlier blocks j < J, plus an optional null row
  that is always visible.  The hot path joins the two key sets under ONE
  softmax; the paper's separate self-attention and cross-attention sub-layers
  are the special cases with no memory rows or with no in-block keys.
* Decode: the same read for one query at position p, after the new key/value
  pair is written into the in-block cache at p.  Streamed decode appends each
  block to the memory once its last token is decoded.
* Decode from the row plane (Appendix K; Appendix A, "Positions and
  memory"): keys and values recomputed from the shared rows by the layer's
  maps, then the same read.
* SMem+RoPE composite (Section 3; the composite's appendix, variant v2):
  rotary phases on queries and keys only -- in-block offsets inside the
  block, block indices (0 for the null row) across blocks, key phases
  optionally clipped to max(j, i - W).  Readings: adjacent dimensions form a
  rotary pair; under the joint softmax the query takes phase t against its
  in-block keys and phase i against the null row and memory rows.
* Slot scheme (Section 2; Appendix A, "Length extension"): beyond B blocks
  the most recent B blocks take slots 1..B and older ones slot 1, so an
  append re-encodes the B-1 blocks whose slot moved.

Readings of the paper used here (silent or ambiguous passages):
* softmax scale 1/sqrt(d_h) with d_h the head dimension (the scale Lemma 1
  writes as 1/sqrt(d));
* causal in-block masks include the query's own position;
* the null row, when given, is a per-head (k, v) pair placed first in
  canonical key order;
* an empty key set yields a zero output;
* a block inserted by the encoder stores its attention output as both its
  key plane and its value plane (identity projections), since the paper's
  per-layer K/V maps lie outside the attention path.
"""
from __future__ import annotations

import math

import numpy as np

MASK_BIDIR = 0
MASK_CAUSAL = 1

EEXIST = "EEXIST"
ENOENT = "ENOENT"
EINVAL = "EINVAL"


class StoreError(Exception):
    def __init__(self, code: str, msg: str = ""):
        super().__init__(f"{code}: {msg}")
        self.code = code


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def softmax_read(q, keys, values, scale):
    """One query against a key list: two-pass softmax, then the weighted sum.

    q [dh], keys [n, dh], values [n, dh] -> [dh].  Definition of attention
    (Section 2 "Model"): weights a_i = exp(s_i - max s) / sum_k exp(s_k - max s)
    with s_i = scale * <q, k_i>; output sum_i a_i v_i.  Empty key set -> 0."""
    q = _f64(q)
    keys = _f64(keys)
    values = _f64(values)
    if keys.shape[0] == 0:
        return np.zeros(values.shape[1], np.float64)
    s = (keys @ q) * scale
    m = np.max(s)
    e = np.exp(s - m)
    a = e / np.sum(e)
    return a @ values


def encode_blocks(q, k, v, mask=MASK_BIDIR):
    """Block-local encoder attention (Section 2 "Model"; Appendix A "Encoder").

    q, k, v: [n_blocks, b, H, dh].  Returns O [n_blocks, b, H, dh] (float64),
    each (block, head) computed on its own from that block's tokens only."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    nb, b, H, dh = q.shape
    scale = 1.0 / math.sqrt(dh)
    out = np.zeros_like(q)
    for blk in range(nb):
        for h in range(H):
            Q = q[blk, :, h, :]
            K = k[blk, :, h, :]
            V = v[blk, :, h, :]
            S = (Q @ K.T) * scale                       # [b, b]
            if mask == MASK_CAUSAL:
                allowed = np.tril(np.ones((b, b), dtype=bool))
            elif mask == MASK_BIDIR:
                allowed = np.ones((b, b), dtype=bool)
            else:
                raise StoreError(EINVAL, f"mask {mask}")
            S = np.where(allowed, S, -np.inf)
            S = S - S.max(axis=1, keepdims=True)
            E = np.exp(S)
            A = E / E.sum(axis=1, keepdims=True)
            out[blk, :, h, :] = A @ V
    return out


class Store:
    """The memory m: a map (sequence, block index) -> that block's rows.

    Theorem 1: a block index holds at most one block; deletion of a present
    block is well defined and restores the never-inserted state; the memory
    read by the reader depends only on which blocks are present, listed in
    ascending block index (the canonical order), each block's b rows in
    in-block order.  Rows are kept exactly as given (no rounding)."""

    def __init__(self, n_seq: int, max_blocks: int, b: int, H: int, dh: int):
        self.n_seq, self.max_blocks, self.b, self.H, self.dh = n_seq, max_blocks, b, H, dh
        self.rows = {}

    def _check(self, seq, j):
        if not (0 <= seq < self.n_seq and 0 <= j < self.max_blocks):
            raise StoreError(EINVAL, f"(seq {seq}, block {j}) out of range")

    def put(self, seq, j, K, V):
        self._check(seq, j)
        if (seq, j) in self.rows:
            raise StoreError(EEXIST, f"(seq {seq}, block {j}) is occupied")
        K = np.array(K, copy=True)
        V = np.array(V, copy=True)
        if K.shape != (self.b, self.H, self.dh) or V.shape != K.shape:
            raise StoreError(EINVAL, "row shape")
        self.rows[(seq, j)] = (K, V)

    def delete(self, seq, j):
        self._check(seq, j)
        if (seq, j) not in self.rows:
            raise StoreError(ENOENT, f"(seq {seq}, block {j}) is absent")
        del self.rows[(seq, j)]

    def live(self, seq):
        """Canonical list of present block indices of one sequence."""
        return sorted(j for (s, j) in self.rows if s == seq)

    def export(self, seq, below=None):
        """Canonical memory of one sequence: (block indices, K [n*b,H,dh], V [n*b,H,dh]).

        With ``below`` given, only blocks with index < below (the rows a query
        in block ``below`` may read: strictly earlier blocks)."""
        idx = [j for j in self.live(seq) if below is None or j < below]
        if not idx:
            e = np.zeros((0, self.H, self.dh))
            return idx, e, e.copy()
        K = np.concatenate([self.rows[(seq, j)][0] for j in idx], axis=0)
        V = np.concatenate([self.rows[(seq, j)][1] for j in idx], axis=0)
        return idx, K, V

    def copy(self):
        s = Store(self.n_seq, self.max_blocks, self.b, self.H, self.dh)
        s.rows = {key: (K.copy(), V.copy()) for key, (K, V) in self.rows.items()}
        return s


def encode_into_store(store: Store, seq_ids, block_idx, q, k, v, mask=MASK_BIDIR):
    """Encode blocks and insert each block's output as its memory rows.

    All-or-nothing: every target index is checked before any insert.  The
    stored key and value planes are both the encoder output (identity
    projections).  Returns the encoder output."""
    for s, j in zip(seq_ids, block_idx):
        store._check(int(s), int(j))
        if (int(s), int(j)) in store.rows:
            raise StoreError(EEXIST, f"(seq {s}, block {j}) is occupied")
    pairs = list(zip((int(s) for s in seq_ids), (int(j) for j in block_idx)))
    if len(set(pairs)) != len(pairs):
        raise StoreError(EEXIST, "duplicate target index")
    out = encode_blocks(q, k, v, mask)
    for i, (s, j) in enumerate(pairs):
        store.put(s, j, out[i], out[i])
    return out


def _memory_below(store, seq, J):
    """Memory rows a query in block J of ``seq`` may read: live blocks j < J,
    canonical order, as float64 (K, V) of shape [N, H, dh]."""
    if store is None or J <= 0:
        return None, None
    _, Km, Vm = store.export(seq, below=J)
    if Km.shape[0] == 0:
        return None, None
    return _f64(Km), _f64(Vm)


def _reader_keys(mem_k, mem_v, h, null_kv, k_in, v_in, n_in, dh):
    """Canonical key/value list for head h of one query:
    [null row] ++ memory rows (blocks j < J) ++ in-block keys 0..n_in-1."""
    ks, vs = [], []
    if null_kv is not None:
        nkv = _f64(null_kv)
        ks.append(nkv[0, h][None, :])
        vs.append(nkv[1, h][None, :])
    if mem_k is not None:
        ks.append(mem_k[:, h, :])
        vs.append(mem_v[:, h, :])
    if k_in is not None and n_in > 0:
        ks.append(_f64(k_in[:n_in, h, :]))
        vs.append(_f64(v_in[:n_in, h, :]))
    if not ks:
        return np.zeros((0, dh)), np.zeros((0, dh))
    return np.concatenate(ks, 0), np.concatenate(vs, 0)


def reader_prefill_block(store, seq_ids, query_block, q, k_intra=None, v_intra=None, null_kv=None):
    """Reader attention for whole query blocks (block-skip serving, Section 3.1).

    q, k_intra, v_intra: [n, b, H, dh]; row i is block query_block[i] of
    sequence seq_ids[i].  k_intra/v_intra None -> no in-block keys (the
    paper's cross-attention alone).  Returns [n, b, H, dh] float64."""
    q = _f64(q)
    n, b, H, dh = q.shape
    scale = 1.0 / math.sqrt(dh)
    out = np.zeros_like(q)
    for i in range(n):
        s, J = int(seq_ids[i]), int(query_block[i])
        mem_k, mem_v = _memory_below(store, s, J)
        kin = None if k_intra is None else _f64(k_intra[i])
        vin = None if v_intra is None else _f64(v_intra[i])
        for h in range(H):
            for t in range(b):
                K, V = _reader_keys(mem_k, mem_v, h, null_kv, kin, vin, t + 1, dh)
                out[i, t, h] = softmax_read(q[i, t, h], K, V, scale)
    return out


def reader_decode(store, seq_ids, query_block, pos, q, k_new=None, v_new=None,
                  k_cache=None, v_cache=None, null_kv=None):
    """Reader attention for one new token per sequence (KV-cached decode, Appendix K).

    q, k_new, v_new: [n, H, dh]; k_cache, v_cache: [n, b, H, dh] in-block
    caches; pos[i] in [0, b) is the new token's in-block position.  The new
    key/value are written at pos, then the query reads
    [null] ++ memory of blocks < query_block[i] ++ cache rows 0..pos.
    k_new None -> memory-only read.  Returns (out [n,H,dh] float64,
    updated k_cache, updated v_cache) -- the caches as copies."""
    q = _f64(q)
    n, H, dh = q.shape
    scale = 1.0 / math.sqrt(dh)
    out = np.zeros_like(q)
    kc = None if k_cache is None else np.array(k_cache, copy=True)
    vc = None if v_cache is None else np.array(v_cache, copy=True)
    for i in range(n):
        s, J, p = int(seq_ids[i]), int(query_block[i]), int(pos[i])
        if kc is not None:
            kc[i, p] = k_new[i]
            vc[i, p] = v_new[i]
        mem_k, mem_v = _memory_below(store, s, J)
        kin = None if kc is None else _f64(kc[i])
        vin = None if vc is None else _f64(vc[i])
        for h in range(H):
            K, V = _reader_keys(mem_k, mem_v, h, null_kv, kin, vin, p + 1, dh)
            out[i, h] = softmax_read(q[i, h], K, V, scale)
    return out, kc, vc


def stream_decode(store, seq_ids, start_block, q, k_new, v_new, q_enc, k_enc, v_enc,
                  null_kv=None, mask=MASK_BIDIR):
    """Token-by-token decode that appends each block as it completes
    (Section 3.1 "Decode"; Appendix K "Decode", read across block boundaries).

    Every sequence starts at in-block position 0 of block start_block[i] with
    an empty in-block cache.  Token t of sequence i sits in block
    start_block[i] + t // b at position t % b; it is decoded by reader_decode
    against the memory of the blocks below its own.  After the token at
    position b-1 the block's b encoder inputs (q_enc, k_enc, v_enc rows of
    that block) are encoded and inserted at that block's index, so the next
    token, the first of the following block, reads it.

    q, k_new, v_new: reader inputs [n, T, H, dh]; q_enc, k_enc, v_enc:
    encoder inputs [n, T, H, dh].  Mutates ``store``.  Returns [n, T, H, dh]."""
    q = _f64(q)
    n, T, H, dh = q.shape
    b = store.b
    out = np.zeros_like(q)
    kc = np.zeros((n, b, H, dh))
    vc = np.zeros((n, b, H, dh))
    for t in range(T):
        p = t % b
        J = [int(start_block[i]) + t // b for i in range(n)]
        o, kc, vc = reader_decode(store, seq_ids, J, [p] * n, q[:, t], k_new[:, t], v_new[:, t],
                                  kc, vc, null_kv)
        out[:, t] = o
        if p == b - 1:
            lo = t - b + 1
            encode_into_store(store, seq_ids, J, q_enc[:, lo:t + 1], k_enc[:, lo:t + 1],
                              v_enc[:, lo:t + 1], mask)
            kc[:] = 0.0
            vc[:] = 0.0
    return out


def reencode_into_store(store: Store, seq_ids, block_idx, q, k, v, mask=MASK_BIDIR):
    """Encode present blocks again from new inputs (Section 2, slot scheme;
    Appendix A, "Length extension").  Defined as deleting every listed block
    and encoding it anew at the same index; every block must be present
    (ENOENT otherwise) and listed once (EINVAL), checked before any change.
    Returns the encoder output."""
    pairs = [(int(s), int(j)) for s, j in zip(seq_ids, block_idx)]
    for s, j in pairs:
        store._check(s, j)
        if (s, j) not in store.rows:
            raise StoreError(ENOENT, f"(seq {s}, block {j}) is absent")
    if len(set(pairs)) != len(pairs):
        raise StoreError(EINVAL, "duplicate target index")
    for s, j in pairs:
        store.delete(s, j)
    return encode_into_store(store, [s for s, _ in pairs], [j for _, j in pairs], q, k, v, mask)


def slot_indices(n_blocks: int, B: int):
    """Slot of every block under the saturating slot scheme (Section 2): with
    at most B blocks, block j (0-based) has slot j + 1; beyond that the most
    recent B blocks have slots 1..B in order and every older block slot 1."""
    return [max(1, j - n_blocks + B + 1) if n_blocks > B else j + 1 for j in range(n_blocks)]


# ---------------------------------------------------------------- decode from the row plane
# Appendix K (the decode arm that derives keys and values from the rows at
# read time rather than keeping them) and
# Appendix A ("Positions and memory"): one plane of rows per block, shared by
# all reader layers; a layer's keys and values are the rows through that
# layer's key and value maps, the null row a d-vector mapped the same way.


def reader_decode_rows(rows_store: Store, w_k, w_v, null_row, seq_ids, query_block, pos, q,
                       k_new=None, v_new=None, k_cache=None, v_cache=None):
    """Recompute the keys and values from the rows, then read as reader_decode.

    rows_store: a Store of shape (b, 1, d) whose entries hold the rows as
    the key element of each pair; w_k, w_v: [H*dh, d] (the key of row r is
    w_k r); null_row [d] or None; q etc. as in reader_decode.  Returns
    (out, k_cache, v_cache)."""
    q = _f64(q)
    n, H, dh = q.shape
    w_k, w_v = _f64(w_k), _f64(w_v)
    kv = Store(rows_store.n_seq, rows_store.max_blocks, rows_store.b, H, dh)
    for (s, j), (R, _) in rows_store.rows.items():
        R = _f64(R).reshape(rows_store.b, rows_store.dh)
        kv.put(s, j, (R @ w_k.T).reshape(R.shape[0], H, dh), (R @ w_v.T).reshape(R.shape[0], H, dh))
    nkv = None
    if null_row is not None:
        nr = _f64(null_row)
        nkv = np.stack([(w_k @ nr).reshape(H, dh), (w_v @ nr).reshape(H, dh)])
    return reader_decode(kv, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, nkv)


# ---------------------------------------------------------------- SMem+RoPE composite
# Section 3 ("SMem composes with RoPE") and the appendix on the composite
# (variant v2): no position enters the rows; rotary phases are applied to
# queries and keys, never to values.  Self-attention inside a block uses the
# in-block offsets of query and key; cross-attention uses block indices: the
# query's block i, the memory row's block j, index 0 for the null row.  The
# saturating reading (the needle appendix) clips every key phase to
# max(j, i - W) with W = B - 1, the query phase staying i.


class Rope:
    """Rotary configuration: frequency base and the saturation window W
    (None: block phases are used as they are)."""

    def __init__(self, base: float = 10000.0, max_offset=None):
        self.base = float(base)
        self.max_offset = max_offset

    def key_phase(self, j, i):
        """Cross-attention phase of a key of block j (0 for the null row) read
        from query block i."""
        return j if self.max_offset is None else max(j, i - self.max_offset)


def rope_rotate(x, phase, base):
    """Rotate the last axis of x by the rotary phase(s): dimensions (2k, 2k+1)
    form pair k, turned by the angle phase * base^(-2k/d_h) (the rotary
    embedding's frequencies; pairs are adjacent dimensions).  ``phase`` is a
    scalar or broadcasts against x[..., 0]."""
    x = _f64(x)
    dh = x.shape[-1]
    theta = base ** (-2.0 * np.arange(dh // 2) / dh)
    ang = np.asarray(phase, np.float64)[..., None] * theta
    c, s = np.cos(ang), np.sin(ang)
    x0, x1 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


def encode_blocks_rope(q, k, v, rope: Rope, mask=MASK_BIDIR):
    """Encoder attention of the composite: queries and keys of token t carry
    rotary phase t (its in-block offset); values are not rotated."""
    q, k = _f64(q), _f64(k)
    t = np.arange(q.shape[1])[None, :, None]
    return encode_blocks(rope_rotate(q, t, rope.base), rope_rotate(k, t, rope.base), v, mask)


def _softmax_scores(s, values):
    """Two-pass softmax of scores s [n] and the weighted sum of values [n, dh]."""
    if s.shape[0] == 0:
        return np.zeros(values.shape[1], np.float64)
    e = np.exp(s - np.max(s))
    return (e / np.sum(e)) @ values


def _rope_read(store, seq, i, t, q, h, null_kv, k_in, v_in, n_in, rope: Rope, scale):
    """One query of the composite's reader: query q [dh] at in-block offset t
    of block i, head h.  Keys in canonical order, each scored against the
    query rotated for its key set: the null row and the memory rows with the
    query at phase i and the key at rope.key_phase(block, i); the in-block
    keys 0..n_in-1 with the query at phase t and key t' at phase t'."""
    base = rope.base
    qs, ks, vs = [], [], []
    if null_kv is not None:
        nkv = _f64(null_kv)
        qs.append(rope_rotate(q, i, base)[None])
        ks.append(rope_rotate(nkv[0, h], rope.key_phase(0, i), base)[None])
        vs.append(nkv[1, h][None])
    if store is not None and i > 0:
        idx, Km, Vm = store.export(seq, below=i)
        if idx:
            blk = np.repeat(np.array(idx), store.b)
            phases = np.array([rope.key_phase(int(j), i) for j in blk], np.float64)
            ks.append(rope_rotate(_f64(Km)[:, h], phases, base))
            vs.append(_f64(Vm)[:, h])
            qs.append(np.repeat(rope_rotate(q, i, base)[None], len(blk), 0))
    if k_in is not None and n_in > 0:
        ks.append(rope_rotate(_f64(k_in)[:n_in, h], np.arange(n_in), base))
        vs.append(_f64(v_in)[:n_in, h])
        qs.append(np.repeat(rope_rotate(q, t, base)[None], n_in, 0))
    if not ks:
        return np.zeros(q.shape[-1])
    Q, K, V = np.concatenate(qs), np.concatenate(ks), np.concatenate(vs)
    return _softmax_scores(np.sum(Q * K, axis=1) * scale, V)


def reader_prefill_block_rope(store, seq_ids, query_block, q, k_intra, v_intra, null_kv, rope: Rope):
    """reader_prefill_block for the composite (phases as in _rope_read)."""
    q = _f64(q)
    n, b, H, dh = q.shape
    scale = 1.0 / math.sqrt(dh)
    out = np.zeros_like(q)
    for r in range(n):
        s, J = int(seq_ids[r]), int(query_block[r])
        kin = None if k_intra is None else _f64(k_intra[r])
        vin = None if v_intra is None else _f64(v_intra[r])
        for h in range(H):
            for t in range(b):
                out[r, t, h] = _rope_read(store, s, J, t, q[r, t, h], h, null_kv, kin, vin, t + 1, rope, scale)
    return out


def reader_decode_rope(store, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv,
                       rope: Rope):
    """reader_decode for the composite: the new pair is written unrotated at
    pos, then the query at offset pos reads as in _rope_read.  Returns
    (out, updated k_cache, updated v_cache)."""
    q = _f64(q)
    n, H, dh = q.shape
    scale = 1.0 / math.sqrt(dh)
    out = np.zeros_like(q)
    kc = None if k_cache is None else np.array(k_cache, copy=True)
    vc = None if v_cache is None else np.array(v_cache, copy=True)
    for r in range(n):
        s, J, p = int(seq_ids[r]), int(query_block[r]), int(pos[r])
        if kc is not None:
            kc[r, p] = k_new[r]
            vc[r, p] = v_new[r]
        kin = None if kc is None else kc[r]
        vin = None if vc is None else vc[r]
        for h in range(H):
            out[r, h] = _rope_read(store, s, J, p, q[r, h], h, null_kv, kin, vin, p + 1, rope, scale)
    return out, kc, vc


def rel_err(y, ref):
    """max |y - ref| / rms(ref) over the whole output of a call."""
    y = _f64(y)
    ref = _f64(ref)
    rms = math.sqrt(float(np.mean(ref * ref))) if ref.size else 0.0
    if rms == 0.0:
        return float(np.max(np.abs(y - ref))) if ref.size else 0.0
    return float(np.max(np.abs(y - ref))) / rms
