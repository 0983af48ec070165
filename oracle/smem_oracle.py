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


def rel_err(y, ref):
    """max |y - ref| / rms(ref) over the whole output of a call."""
    y = _f64(y)
    ref = _f64(ref)
    rms = math.sqrt(float(np.mean(ref * ref))) if ref.size else 0.0
    if rms == 0.0:
        return float(np.max(np.abs(y - ref))) if ref.size else 0.0
    return float(np.max(np.abs(y - ref))) / rms
