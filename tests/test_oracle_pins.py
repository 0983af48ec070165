"""Pins of the fp64 oracle against things other than itself.

* hand-derived closed forms (tests/golden/hand_cases.json, each case citing
  the passage it follows);
* torch's CPU float64 scaled_dot_product_attention, an independent library
  routine, for the encoder and for the reader over concatenated keys with an
  explicit mask;
* the paper's structural guarantees: exact composition (Proposition 1),
  exact editing and path independence (Theorem 1; gates G5-G8 of Appendix B),
  the leak test (Appendix E) and decode/prefill agreement (Appendix K);
* special cases with closed forms.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import smem_oracle as O
from paper_2609_32395_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")


def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _golden_reader_store(case):
    st = O.Store(1, 8, case["b"], case["H"], case["dh"])
    for j, kv in case["memory"].items():
        st.put(0, int(j), np.array(kv["k"]), np.array(kv["v"]))
    return st


def check_golden(tol=1e-12):
    """Raise AssertionError if the oracle disagrees with any hand case."""
    g = golden()
    c = g["encoder_mask"]
    out = O.encode_blocks(c["q"], c["k"], c["v"], O.MASK_BIDIR)
    np.testing.assert_allclose(out, c["expected_bidir"], atol=tol, rtol=0)
    out = O.encode_blocks(c["q"], c["k"], c["v"], O.MASK_CAUSAL)
    np.testing.assert_allclose(out, c["expected_causal"], atol=tol, rtol=0)
    c = g["encoder_scale_and_orientation"]
    out = O.encode_blocks(c["q"], c["k"], c["v"], O.MASK_BIDIR)
    np.testing.assert_allclose(out, c["expected_bidir"], atol=tol, rtol=0)
    c = g["reader"]
    st = _golden_reader_store(c)
    J = c["query_block"]
    out = O.reader_prefill_block(st, [0], [J], c["q"], c["k_intra"], c["v_intra"], c["null_kv"])
    np.testing.assert_allclose(out, c["expected_with_null"], atol=tol, rtol=0)
    out = O.reader_prefill_block(st, [0], [J], c["q"], c["k_intra"], c["v_intra"], None)
    np.testing.assert_allclose(out, c["expected_without_null"], atol=tol, rtol=0)
    p = c["decode"]["pos"]
    kc = np.zeros((1, c["b"], 1, 1))
    vc = np.zeros((1, c["b"], 1, 1))
    kc[0, :p] = np.array(c["k_intra"])[0, :p]
    vc[0, :p] = np.array(c["v_intra"])[0, :p]
    qd = np.array(c["q"])[:, p]
    kn = np.array(c["k_intra"])[:, p]
    vn = np.array(c["v_intra"])[:, p]
    out, kc2, vc2 = O.reader_decode(st, [0], [J], [p], qd, kn, vn, kc, vc, c["null_kv"])
    np.testing.assert_allclose(out, c["decode"]["expected_with_null"], atol=tol, rtol=0)
    assert kc2[0, p, 0, 0] == kn[0, 0, 0] and vc2[0, p, 0, 0] == vn[0, 0, 0]
    st.delete(0, 0)
    out = O.reader_prefill_block(st, [0], [J], c["q"], c["k_intra"], c["v_intra"], c["null_kv"])
    np.testing.assert_allclose(out, c["expected_after_delete_0_with_null"], atol=tol, rtol=0)


def test_golden_hand_cases():
    check_golden()


# ---------------------------------------------------------------- library routine

def _sdpa(q, k, v, mask=None, causal=False):
    # q [Lq, dh], k/v [Lk, dh] float64 -> [Lq, dh]; default scale 1/sqrt(dh)
    qt = torch.from_numpy(np.ascontiguousarray(q))[None, None]
    kt = torch.from_numpy(np.ascontiguousarray(k))[None, None]
    vt = torch.from_numpy(np.ascontiguousarray(v))[None, None]
    m = None if mask is None else torch.from_numpy(mask)[None, None]
    return F.scaled_dot_product_attention(qt, kt, vt, attn_mask=m, is_causal=causal)[0, 0].numpy()


@pytest.mark.parametrize("b,H,dh", [(16, 4, 32), (64, 2, 64), (8, 3, 128), (1, 2, 32)])
@pytest.mark.parametrize("mask", [O.MASK_BIDIR, O.MASK_CAUSAL])
def test_encoder_matches_sdpa(b, H, dh, mask):
    g = np.random.default_rng(b * 1000 + H * 10 + dh + mask)
    nb = 3
    q, k, v = (g.standard_normal((nb, b, H, dh)) for _ in range(3))
    out = O.encode_blocks(q, k, v, mask)
    for blk in range(nb):
        for h in range(H):
            ref = _sdpa(q[blk, :, h], k[blk, :, h], v[blk, :, h], causal=(mask == O.MASK_CAUSAL))
            np.testing.assert_allclose(out[blk, :, h], ref, atol=1e-12, rtol=0)


def _random_store(g, n_seq, max_blocks, b, H, dh, live_frac=0.6):
    st = O.Store(n_seq, max_blocks, b, H, dh)
    for s in range(n_seq):
        for j in range(max_blocks):
            if g.random() < live_frac:
                st.put(s, j, g.standard_normal((b, H, dh)), g.standard_normal((b, H, dh)))
    return st


@pytest.mark.parametrize("with_null", [False, True])
@pytest.mark.parametrize("with_intra", [False, True])
def test_reader_matches_sdpa_over_concatenated_keys(with_null, with_intra):
    g = np.random.default_rng(7 + 2 * with_null + with_intra)
    b, H, dh, n_seq, max_blocks = 8, 2, 32, 2, 6
    st = _random_store(g, n_seq, max_blocks, b, H, dh)
    seq_ids, qblk = [0, 1], [5, 3]
    for s, J in zip(seq_ids, qblk):   # the query's own index is occupied: it must not be read
        if (s, J) not in st.rows:
            st.put(s, J, g.standard_normal((b, H, dh)), g.standard_normal((b, H, dh)))
    q = g.standard_normal((2, b, H, dh))
    ki = g.standard_normal((2, b, H, dh)) if with_intra else None
    vi = g.standard_normal((2, b, H, dh)) if with_intra else None
    nkv = g.standard_normal((2, H, dh)) if with_null else None
    out = O.reader_prefill_block(st, seq_ids, qblk, q, ki, vi, nkv)
    for i, (s, J) in enumerate(zip(seq_ids, qblk)):
        # all rows of the sequence (every present block, any index) + intra;
        # the mask decides visibility: blocks < J, intra keys <= t, null always.
        live = st.live(s)
        Kall = [st.rows[(s, j)][0] for j in live]
        Vall = [st.rows[(s, j)][1] for j in live]
        blk_of = np.concatenate([np.full(b, j) for j in live]) if live else np.zeros(0)
        for h in range(H):
            ks = [Kk[:, h] for Kk in Kall]
            vs = [Vv[:, h] for Vv in Vall]
            vis_cols = [np.ones((b, 0), bool)]
            if nkv is not None:
                ks.insert(0, nkv[0, h][None])
                vs.insert(0, nkv[1, h][None])
                vis_cols.append(np.ones((b, 1), bool))
            vis_cols.append(np.broadcast_to(blk_of[None, :] < J, (b, blk_of.size)))
            if ki is not None:
                ks.append(ki[i, :, h])
                vs.append(vi[i, :, h])
                vis_cols.append(np.tril(np.ones((b, b), bool)))
            K = np.concatenate(ks, 0)
            V = np.concatenate(vs, 0)
            mask = np.concatenate(vis_cols, 1)
            if not mask.any(axis=1).all():
                # rows with an empty key set are defined as zero
                assert np.all(out[i, :, h][~mask.any(axis=1)] == 0)
                continue
            ref = _sdpa(q[i, :, h], K, V, mask=mask)
            np.testing.assert_allclose(out[i, :, h], ref, atol=1e-12, rtol=0)


# ---------------------------------------------------------------- structural guarantees

def test_exact_composition_joint_vs_per_block():
    """Proposition 1 / gate G5: block-masked joint attention over the whole
    sequence equals per-block encoding (< 1e-12 in fp64)."""
    g = np.random.default_rng(11)
    nb, b, H, dh = 4, 16, 2, 32
    q, k, v = (g.standard_normal((nb, b, H, dh)) for _ in range(3))
    per_block = O.encode_blocks(q, k, v, O.MASK_BIDIR)
    n = nb * b
    blk = np.arange(n) // b
    mask = blk[:, None] == blk[None, :]
    for h in range(H):
        joint = _sdpa(q[:, :, h].reshape(n, dh), k[:, :, h].reshape(n, dh), v[:, :, h].reshape(n, dh), mask=mask)
        np.testing.assert_allclose(per_block[:, :, h].reshape(n, dh), joint, atol=1e-12, rtol=0)


def test_block_rows_independent_of_batch_bitwise():
    """A block's rows are identical whether encoded alone or among others."""
    g = np.random.default_rng(12)
    q, k, v = (g.standard_normal((5, 16, 4, 32)) for _ in range(3))
    allb = O.encode_blocks(q, k, v, O.MASK_CAUSAL)
    for i in range(5):
        one = O.encode_blocks(q[i:i + 1], k[i:i + 1], v[i:i + 1], O.MASK_CAUSAL)
        assert np.array_equal(one[0], allb[i])


def test_reader_invariant_to_memory_construction():
    """Gate G6: reads are the same whether memory comes from one joint encode
    or from per-block encodes (inserted in any order)."""
    g = np.random.default_rng(13)
    nb, b, H, dh = 5, 8, 2, 32
    q, k, v = (g.standard_normal((nb, b, H, dh)) for _ in range(3))
    st1 = O.Store(1, 8, b, H, dh)
    O.encode_into_store(st1, [0] * nb, list(range(nb)), q, k, v)
    st2 = O.Store(1, 8, b, H, dh)
    for i in [3, 0, 4, 2, 1]:
        O.encode_into_store(st2, [0], [i], q[i:i + 1], k[i:i + 1], v[i:i + 1])
    qq = g.standard_normal((1, b, H, dh))
    r1 = O.reader_prefill_block(st1, [0], [nb], qq, qq, qq)
    r2 = O.reader_prefill_block(st2, [0], [nb], qq, qq, qq)
    assert np.array_equal(r1, r2)


def test_delete_equals_never_inserted_bitwise():
    """Theorem 1 / gate G7: add-then-remove returns the identical memory and reads."""
    g = np.random.default_rng(14)
    b, H, dh = 8, 2, 16
    st = _random_store(g, 1, 10, b, H, dh, live_frac=1.0)
    before = st.copy()
    st.delete(0, 3)
    never = O.Store(1, 10, b, H, dh)
    for j in before.live(0):
        if j != 3:
            never.put(0, j, *before.rows[(0, j)])
    for a, c in zip(st.export(0), never.export(0)):
        assert np.array_equal(np.asarray(a), np.asarray(c))
    qq = g.standard_normal((1, b, H, dh))
    assert np.array_equal(O.reader_prefill_block(st, [0], [10], qq, qq, qq),
                          O.reader_prefill_block(never, [0], [10], qq, qq, qq))
    # add then remove
    st.put(0, 3, *before.rows[(0, 3)])
    for a, c in zip(st.export(0), before.export(0)):
        assert np.array_equal(np.asarray(a), np.asarray(c))


def test_edit_path_independence_100_orders():
    """Gate G8: 100 random edit sequences ending at the same multiset give
    bit-identical canonical memories and reads."""
    g = np.random.default_rng(15)
    b, H, dh, nb = 4, 2, 8, 12
    rows = {j: (g.standard_normal((b, H, dh)), g.standard_normal((b, H, dh))) for j in range(nb)}
    final = set(g.choice(nb, size=7, replace=False).tolist())
    qq = g.standard_normal((1, b, H, dh))
    ref_exp, ref_read = None, None
    for trial in range(100):
        r = np.random.default_rng(1000 + trial)
        st = O.Store(1, nb, b, H, dh)
        present = set()
        for _ in range(r.integers(5, 40)):
            j = int(r.integers(0, nb))
            if j in present:
                st.delete(0, j)
                present.discard(j)
            else:
                st.put(0, j, *rows[j])
                present.add(j)
        for j in sorted(present - final):
            st.delete(0, j)
        for j in sorted(final - present, reverse=bool(trial % 2)):
            st.put(0, j, *rows[j])
        exp = st.export(0)
        read = O.reader_prefill_block(st, [0], [nb], qq, qq, qq)
        if ref_exp is None:
            ref_exp, ref_read = exp, read
        assert exp[0] == ref_exp[0]
        assert np.array_equal(exp[1], ref_exp[1]) and np.array_equal(exp[2], ref_exp[2])
        assert np.array_equal(read, ref_read)


def test_read_permutation_invariant():
    """Theorem 1: the read is invariant to the order of memory rows (up to rounding)."""
    g = np.random.default_rng(16)
    K = g.standard_normal((300, 32))
    V = g.standard_normal((300, 32))
    q = g.standard_normal(32)
    a = O.softmax_read(q, K, V, 0.2)
    perm = g.permutation(300)
    c = O.softmax_read(q, K[perm], V[perm], 0.2)
    np.testing.assert_allclose(a, c, rtol=1e-13, atol=1e-14)


def test_leak_masked_data_changes_nothing():
    """Appendix E leak test: perturbing everything a query must not see leaves
    its output bitwise unchanged (later in-block keys, blocks >= J, other
    blocks of the encoder)."""
    g = np.random.default_rng(17)
    b, H, dh = 8, 2, 16
    st = _random_store(g, 1, 8, b, H, dh, live_frac=1.0)
    q, ki, vi = (g.standard_normal((1, b, H, dh)) for _ in range(3))
    base = O.reader_prefill_block(st, [0], [4], q, ki, vi)
    st2 = st.copy()
    for j in range(4, 8):
        st2.delete(0, j)
        st2.put(0, j, g.standard_normal((b, H, dh)) * 100, g.standard_normal((b, H, dh)) * 100)
    t = 5
    ki2, vi2 = ki.copy(), vi.copy()
    ki2[0, t + 1:] += 50.0
    vi2[0, t + 1:] -= 50.0
    pert = O.reader_prefill_block(st2, [0], [4], q, ki2, vi2)
    assert np.array_equal(pert[0, :t + 1], base[0, :t + 1])
    # encoder: perturbing other blocks leaves a block's output unchanged
    qe, ke, ve = (g.standard_normal((3, b, H, dh)) for _ in range(3))
    e1 = O.encode_blocks(qe, ke, ve, O.MASK_CAUSAL)
    ke2 = ke.copy()
    ke2[[0, 2]] *= -3.0
    ke2[1, t + 1:] += 9.0  # later keys of block 1 under the causal mask
    e2 = O.encode_blocks(qe, ke2, ve, O.MASK_CAUSAL)
    assert np.array_equal(e1[1, :t + 1], e2[1, :t + 1])


def test_decode_equals_prefill_row():
    """Appendix K exactness idea: decode at position p equals prefill row p."""
    g = np.random.default_rng(18)
    b, H, dh = 8, 2, 16
    st = _random_store(g, 2, 6, b, H, dh)
    nkv = g.standard_normal((2, H, dh))
    q, ki, vi = (g.standard_normal((2, b, H, dh)) for _ in range(3))
    pre = O.reader_prefill_block(st, [0, 1], [6, 4], q, ki, vi, nkv)
    for p in [0, 3, b - 1]:
        kc = np.zeros((2, b, H, dh))
        vc = np.zeros((2, b, H, dh))
        kc[:, :p] = ki[:, :p]
        vc[:, :p] = vi[:, :p]
        kc[:, p + 1:] = 1e3  # garbage after p must be ignored
        out, kc2, vc2 = O.reader_decode(st, [0, 1], [6, 4], [p, p], q[:, p], ki[:, p], vi[:, p], kc, vc, nkv)
        np.testing.assert_allclose(out, pre[:, p], atol=1e-13, rtol=0)
        assert np.array_equal(kc2[:, :p + 1], ki[:, :p + 1])


# ---------------------------------------------------------------- closed forms

def test_closed_forms():
    g = np.random.default_rng(19)
    H, dh = 3, 16
    # b = 1: a token attends only to itself -> O = V exactly
    q, k, v = (g.standard_normal((4, 1, H, dh)) for _ in range(3))
    assert np.array_equal(O.encode_blocks(q, k, v), v)
    # identical keys -> mean of the visible values (causal: prefix means)
    b = 8
    q = g.standard_normal((1, b, H, dh))
    k = np.broadcast_to(g.standard_normal((1, 1, H, dh)), (1, b, H, dh))
    v = g.standard_normal((1, b, H, dh))
    out = O.encode_blocks(q, k, v, O.MASK_CAUSAL)
    for t in range(b):
        np.testing.assert_allclose(out[0, t], v[0, :t + 1].mean(0), atol=1e-14)
    out = O.encode_blocks(q, k, v, O.MASK_BIDIR)
    np.testing.assert_allclose(out[0], np.broadcast_to(v[0].mean(0), (b, H, dh)), atol=1e-14)
    # one dominant key (score margin ~1e3) -> exactly its value
    K = np.zeros((5, dh))
    K[2, 0] = 1e3
    V = g.standard_normal((5, dh))
    qv = np.zeros(dh)
    qv[0] = 4.0
    assert np.array_equal(O.softmax_read(qv, K, V, 1.0), V[2])
    # empty memory, no null: reader == causal in-block attention
    st = O.Store(1, 4, b, H, dh)
    q, ki, vi = (g.standard_normal((1, b, H, dh)) for _ in range(3))
    r = O.reader_prefill_block(st, [0], [3], q, ki, vi)
    e = O.encode_blocks(q, ki, vi, O.MASK_CAUSAL)
    np.testing.assert_allclose(r, e, atol=1e-14)
    # intra length 1 and no memory: the first query returns its own value
    assert np.array_equal(r[0, 0], vi[0, 0])
    # empty key set -> zero output, never NaN
    r = O.reader_prefill_block(st, [0], [3], q, None, None)
    assert np.array_equal(r, np.zeros_like(r))


# ---------------------------------------------------------------- store semantics

def test_store_errors_and_canonical_order():
    b, H, dh = 2, 1, 2
    st = O.Store(2, 6, b, H, dh)
    blk = lambda x: np.full((b, H, dh), float(x))
    for j in [4, 1, 5, 0]:
        st.put(1, j, blk(j), blk(-j))
    with pytest.raises(O.StoreError) as e:
        st.put(1, 4, blk(0), blk(0))
    assert e.value.code == O.EEXIST
    with pytest.raises(O.StoreError) as e:
        st.delete(1, 2)
    assert e.value.code == O.ENOENT
    with pytest.raises(O.StoreError) as e:
        st.delete(0, 6)
    assert e.value.code == O.EINVAL
    idx, K, V = st.export(1)
    assert idx == [0, 1, 4, 5]
    assert K[:, 0, 0].tolist() == [0, 0, 1, 1, 4, 4, 5, 5]
    assert st.export(1, below=4)[0] == [0, 1]
    assert st.live(0) == []


def test_encode_into_store_all_or_nothing():
    g = np.random.default_rng(20)
    b, H, dh = 4, 2, 8
    st = O.Store(2, 4, b, H, dh)
    q, k, v = (g.standard_normal((3, b, H, dh)) for _ in range(3))
    O.encode_into_store(st, [0], [2], q[:1], k[:1], v[:1])
    with pytest.raises(O.StoreError) as e:
        O.encode_into_store(st, [1, 0, 1], [0, 2, 1], q, k, v)
    assert e.value.code == O.EEXIST
    assert st.live(1) == []  # nothing inserted
    out = O.encode_into_store(st, [1, 1], [3, 0], q[1:], k[1:], v[1:])
    assert st.live(1) == [0, 3]
    assert np.array_equal(st.rows[(1, 3)][0], out[0]) and np.array_equal(st.rows[(1, 3)][1], out[0])


# ---------------------------------------------------------------- the input generator

def test_synth_bf16_rounding_and_keys():
    x = np.array([1.0, 1.00390625, 1.005859375, -2.5e-3, 3.0e5], np.float32)
    r = synth.bf16_round(x)
    assert np.array_equal(torch.from_numpy(x).to(torch.bfloat16).float().numpy(), r)
    w = synth.TINY_F32
    a = synth.block_tokens(w, 0, synth.ROLE_Q, 0, 3)
    c = synth.block_tokens(w, 0, synth.ROLE_Q, 0, 3)
    d = synth.block_tokens(w, 0, synth.ROLE_Q, 0, 4)
    assert np.array_equal(a, c) and not np.array_equal(a, d)
    w2 = synth.ENC_160M
    kb = synth.block_tokens(w2, 0, synth.ROLE_K, 1, 2)
    assert np.array_equal(synth.bf16_round(kb), kb)
    K, V = synth.memory_blocks(w2, 0, [0, 1], [5, 6], threads=2)
    k1, v1 = synth.memory_block(w2, 0, 1, 6)
    assert np.array_equal(K[1, 1], k1) and np.array_equal(V[1, 1], v1)


# ---------------------------------------------------------------- streaming append, re-encode, slots

def _stream_case(seed=31, b=4, H=2, dh=8, T=10):
    g = np.random.default_rng(seed)
    st = O.Store(2, 12, b, H, dh)
    for s, blocks in ((0, (0, 1, 2)), (1, (0, 3, 4))):
        for j in blocks:
            st.put(s, j, g.standard_normal((b, H, dh)), g.standard_normal((b, H, dh)))
    start = [3, 5]
    dec = [g.standard_normal((2, T, H, dh)) for _ in range(3)]
    enc = [g.standard_normal((2, T, H, dh)) for _ in range(3)]
    nkv = g.standard_normal((2, H, dh))
    return st, start, dec, enc, nkv


def test_stream_decode_equals_prefill_of_each_block():
    """Decode across block boundaries (Appendix K) reads, for every token,
    exactly what the block-skip reader reads for that token's block: the
    memory of the blocks below it (streamed blocks included) and the block's
    own tokens up to the token.  A block appended before its last token is
    decoded, or at the wrong index, changes some row."""
    st, start, (q, kn, vn), (qe, ke, ve), nkv = _stream_case()
    b, T = st.b, q.shape[1]
    run = st.copy()
    out = O.stream_decode(run, [0, 1], start, q, kn, vn, qe, ke, ve, nkv)
    for blk in range(-(-T // b)):
        lo, hi = blk * b, min(T, blk * b + b)
        J = [start[0] + blk, start[1] + blk]
        pad = lambda x: np.concatenate([x[:, lo:hi], np.zeros((2, b - (hi - lo)) + x.shape[2:])], 1)
        pre = O.reader_prefill_block(run, [0, 1], J, pad(q), pad(kn), pad(vn), nkv)
        np.testing.assert_allclose(out[:, lo:hi], pre[:, :hi - lo], atol=1e-13, rtol=0)
    # the two complete blocks went in at start, start+1; the partial third did not
    assert run.live(0) == [0, 1, 2, 3, 4] and run.live(1) == [0, 3, 4, 5, 6]


def test_stream_appended_rows_equal_joint_encode():
    """Proposition 1: the blocks appended one by one during decode equal the
    joint encode of the same blocks (block-diagonal mask), bitwise."""
    st, start, (q, kn, vn), (qe, ke, ve), nkv = _stream_case()
    b = st.b
    run = st.copy()
    O.stream_decode(run, [0, 1], start, q, kn, vn, qe, ke, ve, nkv)
    for s in (0, 1):
        for blk in range(2):
            lo = blk * b
            # joint encode of both complete blocks of this sequence at once
            both = O.encode_blocks(qe[s, :2 * b].reshape(2, b, *qe.shape[2:]),
                                   ke[s, :2 * b].reshape(2, b, *ke.shape[2:]),
                                   ve[s, :2 * b].reshape(2, b, *ve.shape[2:]))
            K, V = run.rows[(s, start[s] + blk)]
            assert np.array_equal(K, both[blk]) and np.array_equal(V, both[blk])
            mask = np.kron(np.eye(2, dtype=bool), np.ones((b, b), bool))
            qq, kk, vv = (torch.from_numpy(x[s, :2 * b].transpose(1, 0, 2).copy()) for x in (qe, ke, ve))
            ref = F.scaled_dot_product_attention(qq, kk, vv, attn_mask=torch.from_numpy(mask)).numpy()
            np.testing.assert_allclose(K, ref.transpose(1, 0, 2)[lo:lo + b], atol=1e-12, rtol=0)


def test_reencode_matches_fresh_insert_and_errors_change_nothing():
    """Re-encoding present blocks equals a store where those blocks were
    encoded from the new inputs in the first place (Theorem 1: a delete is
    exact, so the old rows leave no trace); re-encoding with the original
    inputs is the identity; an absent or repeated block changes nothing."""
    g = np.random.default_rng(44)
    b, H, dh = 4, 2, 8
    x1 = [g.standard_normal((3, b, H, dh)) for _ in range(3)]
    x2 = [g.standard_normal((2, b, H, dh)) for _ in range(3)]
    st = O.Store(1, 6, b, H, dh)
    O.encode_into_store(st, [0, 0, 0], [1, 2, 4], *x1)
    same = st.copy()
    O.reencode_into_store(same, [0, 0, 0], [1, 2, 4], *x1)
    for j in (1, 2, 4):
        assert all(np.array_equal(a, c) for a, c in zip(same.rows[(0, j)], st.rows[(0, j)]))
    O.reencode_into_store(st, [0, 0], [4, 1], *x2)
    fresh = O.Store(1, 6, b, H, dh)
    O.encode_into_store(fresh, [0], [2], x1[0][1:2], x1[1][1:2], x1[2][1:2])
    O.encode_into_store(fresh, [0, 0], [4, 1], *x2)
    assert st.live(0) == fresh.live(0) == [1, 2, 4]
    for a, c in zip(st.export(0), fresh.export(0)):
        assert np.array_equal(a, c)
    q = g.standard_normal((1, b, H, dh))
    assert np.array_equal(O.reader_prefill_block(st, [0], [5], q, q, q),
                          O.reader_prefill_block(fresh, [0], [5], q, q, q))
    before = st.copy()
    for seqs, idx, code in (([0, 0], [1, 3], O.ENOENT), ([0, 0], [2, 2], O.EINVAL)):
        with pytest.raises(O.StoreError) as e:
            O.reencode_into_store(st, seqs, idx, *x2)
        assert e.value.code == code
        assert st.live(0) == before.live(0)
        for a, c in zip(st.export(0), before.export(0)):
            assert np.array_equal(a, c)


def test_slot_scheme():
    """Section 2 / Appendix A: up to B blocks every block keeps its own slot;
    beyond, the newest B blocks hold slots 1..B and older blocks share slot 1,
    so each append past B moves exactly the B-1 most recent earlier blocks."""
    B = 4
    assert O.slot_indices(3, B) == [1, 2, 3]
    assert O.slot_indices(4, B) == [1, 2, 3, 4]
    assert O.slot_indices(6, B) == [1, 1, 1, 2, 3, 4]
    for n in range(1, 12):
        sl = O.slot_indices(n, B)
        assert len(sl) == n and sl[-1] == min(n, B) and min(sl) == 1 and max(sl) == min(n, B)
        moved = [j for j, (a, c) in enumerate(zip(sl, O.slot_indices(n + 1, B))) if a != c]
        assert moved == (list(range(n - B + 1, n)) if n >= B else [])


# ---------------------------------------------------------------- SMem+RoPE composite

def test_rope_rotation_closed_forms():
    """Rotary pairs are adjacent dimensions turned by phase * base^(-2k/d_h):
    textbook values cos 1, sin 1 and exact identities of plane rotations."""
    c1, s1 = 0.5403023058681398, 0.8414709848078965          # cos(1), sin(1)
    np.testing.assert_allclose(O.rope_rotate([1.0, 0.0], 1.0, 1e4), [c1, s1], atol=1e-15)
    np.testing.assert_allclose(O.rope_rotate([0.0, 1.0], 1.0, 1e4), [-s1, c1], atol=1e-15)
    # d_h = 4, base 100: pair 1 turns at 100^(-1/2) = 0.1 rad per unit of phase
    np.testing.assert_allclose(O.rope_rotate([0.0, 0.0, 1.0, 0.0], 10.0, 100.0), [0, 0, c1, s1], atol=1e-14)
    np.testing.assert_allclose(O.rope_rotate([1.0, 0.0, 0.0, 0.0], 1.0, 100.0), [c1, s1, 0, 0], atol=1e-15)
    g = np.random.default_rng(5)
    x, y = g.standard_normal((2, 7, 64))
    a, b_, c = 13.0, 5.0, 1000.0
    R = lambda z, ph: O.rope_rotate(z, ph, 1e4)
    np.testing.assert_allclose(np.linalg.norm(R(x, a), axis=1), np.linalg.norm(x, axis=1), rtol=1e-14)
    np.testing.assert_allclose(R(R(x, a), b_), R(x, a + b_), atol=1e-12)
    np.testing.assert_allclose(R(R(x, a), -a), x, atol=1e-13)
    # scores depend on the phase difference only
    np.testing.assert_allclose(np.sum(R(x, a) * R(y, b_), 1), np.sum(R(x, a + c) * R(y, b_ + c), 1), atol=1e-11)


def _complex_rotate(x, phase, base):
    """Independent rotary map: adjacent pairs as complex numbers times e^{i angle}."""
    x = torch.as_tensor(np.asarray(x, np.float64))
    dh = x.shape[-1]
    z = torch.view_as_complex(x.reshape(*x.shape[:-1], dh // 2, 2).contiguous())
    theta = torch.tensor(base ** (-2.0 * np.arange(dh // 2) / dh))
    ang = torch.as_tensor(np.asarray(phase, np.float64))[..., None] * theta
    return torch.view_as_real(z * torch.polar(torch.ones_like(ang), ang)).reshape(x.shape)


@pytest.mark.parametrize("mask", [O.MASK_BIDIR, O.MASK_CAUSAL])
def test_rope_encoder_matches_complex_sdpa(mask):
    g = np.random.default_rng(23)
    nb, b, H, dh = 3, 8, 2, 16
    q, k, v = (g.standard_normal((nb, b, H, dh)) for _ in range(3))
    rope = O.Rope(base=1e4)
    out = O.encode_blocks_rope(q, k, v, rope, mask)
    t = np.arange(b)[None, :, None]
    qr, kr = _complex_rotate(q, t, 1e4), _complex_rotate(k, t, 1e4)
    ref = F.scaled_dot_product_attention(qr.permute(0, 2, 1, 3), kr.permute(0, 2, 1, 3),
                                         torch.as_tensor(v).permute(0, 2, 1, 3),
                                         is_causal=mask == O.MASK_CAUSAL).permute(0, 2, 1, 3).numpy()
    np.testing.assert_allclose(out, ref, atol=1e-12, rtol=0)


@pytest.mark.parametrize("max_offset", [None, 3])
@pytest.mark.parametrize("with_null", [False, True])
def test_rope_reader_matches_complex_sdpa(max_offset, with_null):
    """The composite's reader against SDPA over concatenated keys, with the
    rotary phases applied as relative turns of the keys by complex products:
    memory and null keys by (key phase - i), in-block keys by (t' - t)."""
    g = np.random.default_rng(29 + with_null)
    b, H, dh, J = 4, 2, 8, 7
    st = _random_store(g, 1, J + 2, b, H, dh, live_frac=0.7)
    rope = O.Rope(base=100.0, max_offset=max_offset)
    nkv = g.standard_normal((2, H, dh)) if with_null else None
    q, ki, vi = (g.standard_normal((1, b, H, dh)) for _ in range(3))
    out = O.reader_prefill_block_rope(st, [0], [J], q, ki, vi, nkv, rope)
    idx, Km, Vm = st.export(0, below=J)
    blk = np.repeat(np.array(idx, int), b)
    for t in range(b):
        for h in range(H):
            ks, vs = [], []
            # relative turn of a block-j key: j - J, or -min(J - j, W) when clipped
            turn = (lambda j: j - J) if max_offset is None else (lambda j: -min(J - j, max_offset))
            if with_null:
                ks.append(_complex_rotate(nkv[0, h][None], turn(0), 100.0))
                vs.append(torch.as_tensor(nkv[1, h][None]))
            if len(blk):
                ph = np.array([turn(int(j)) for j in blk], np.float64)
                ks.append(_complex_rotate(Km[:, h], ph, 100.0))
                vs.append(torch.as_tensor(Vm[:, h]))
            ks.append(_complex_rotate(ki[0, :t + 1, h], np.arange(t + 1) - t, 100.0))
            vs.append(torch.as_tensor(vi[0, :t + 1, h]))
            K, V = torch.cat(ks), torch.cat(vs)
            ref = F.scaled_dot_product_attention(torch.as_tensor(q[0, t, h])[None, None], K[None], V[None])
            np.testing.assert_allclose(out[0, t, h], ref[0, 0].numpy(), atol=1e-12, rtol=0)


def test_rope_saturation():
    """Saturated block phases (the needle appendix): identity while the query
    block is within W of block 0; beyond, all blocks at distance >= W share
    one phase, so their rows are interchangeable, and nearer ones are not."""
    g = np.random.default_rng(37)
    b, H, dh, W = 2, 1, 8, 3
    mk = lambda: (g.standard_normal((b, H, dh)), g.standard_normal((b, H, dh)))
    blocks = {j: mk() for j in range(9)}

    def store(perm):
        st = O.Store(1, 10, b, H, dh)
        for j in range(9):
            st.put(0, j, *blocks[perm.get(j, j)])
        return st
    q, ki, vi = (g.standard_normal((1, b, H, dh)) for _ in range(3))
    clip, free = O.Rope(100.0, W), O.Rope(100.0, None)
    a = O.reader_prefill_block_rope(store({}), [0], [3], q, ki, vi, None, clip)
    assert np.array_equal(a, O.reader_prefill_block_rope(store({}), [0], [3], q, ki, vi, None, free))
    base = O.reader_prefill_block_rope(store({}), [0], [9], q, ki, vi, None, clip)
    far = O.reader_prefill_block_rope(store({0: 5, 5: 0}), [0], [9], q, ki, vi, None, clip)  # both j <= 9 - W
    np.testing.assert_allclose(far, base, atol=1e-13, rtol=0)
    near = O.reader_prefill_block_rope(store({0: 7, 7: 0}), [0], [9], q, ki, vi, None, clip)
    assert np.max(np.abs(near - base)) > 1e-3
    unclipped = O.reader_prefill_block_rope(store({0: 5, 5: 0}), [0], [9], q, ki, vi, None, free)
    assert np.max(np.abs(unclipped - O.reader_prefill_block_rope(store({}), [0], [9], q, ki, vi, None, free))) > 1e-3


@pytest.mark.parametrize("max_offset", [None, 2])
def test_rope_null_row_has_block_zero_phase(max_offset):
    """The null row carries index 0: with one-row blocks, a null row equal to
    block 0's row reads exactly like block 0 itself (both clipped alike)."""
    g = np.random.default_rng(41)
    b, H, dh, J = 1, 2, 8, 6
    rows = [(g.standard_normal((1, H, dh)), g.standard_normal((1, H, dh))) for _ in range(J)]
    with_block0, without = O.Store(1, J, b, H, dh), O.Store(1, J, b, H, dh)
    for j in range(J):
        with_block0.put(0, j, *rows[j])
        if j:
            without.put(0, j, *rows[j])
    nkv = np.stack([rows[0][0][0], rows[0][1][0]])            # [2, H, dh]
    q, ki, vi = (g.standard_normal((1, b, H, dh)) for _ in range(3))
    rope = O.Rope(100.0, max_offset)
    a = O.reader_prefill_block_rope(with_block0, [0], [J], q, ki, vi, None, rope)
    c = O.reader_prefill_block_rope(without, [0], [J], q, ki, vi, nkv, rope)
    np.testing.assert_allclose(c, a, atol=1e-13, rtol=0)


def test_rope_values_not_rotated_and_decode_equals_prefill():
    g = np.random.default_rng(43)
    b, H, dh, J = 4, 2, 8, 5
    st = _random_store(g, 1, J, b, H, dh, live_frac=1.0)
    rope = O.Rope(1e4, 2)
    zero = np.zeros((1, b, H, dh))
    ki, vi = g.standard_normal((2, 1, b, H, dh))
    out = O.reader_prefill_block_rope(st, [0], [J], zero, ki, vi, None, rope)
    _, _, Vm = st.export(0, below=J)
    for t in range(b):   # all scores 0: the plain mean of the visible values
        np.testing.assert_allclose(out[0, t], np.concatenate([Vm, vi[0, :t + 1]]).mean(0), atol=1e-14)
    q = g.standard_normal((1, b, H, dh))
    nkv = g.standard_normal((2, H, dh))
    pre = O.reader_prefill_block_rope(st, [0], [J], q, ki, vi, nkv, rope)
    for p in (0, 2, b - 1):
        kc = np.full((1, b, H, dh), 7.0)
        vc = np.full((1, b, H, dh), 7.0)
        kc[:, :p], vc[:, :p] = ki[:, :p], vi[:, :p]
        dec, _, _ = O.reader_decode_rope(st, [0], [J], [p], q[:, p], ki[:, p], vi[:, p], kc, vc, nkv, rope)
        np.testing.assert_allclose(dec, pre[:, p], atol=1e-13, rtol=0)


# ---------------------------------------------------------------- decode from the row plane

def test_rows_decode_with_identity_maps_is_the_plain_read():
    """With d = H*dh and identity key/value maps, the recomputed read is the
    plain read of a store whose keys and values are the rows themselves."""
    g = np.random.default_rng(51)
    b, H, dh, J = 4, 2, 8, 5
    d = H * dh
    rows = O.Store(2, J + 1, b, 1, d)
    kv = O.Store(2, J + 1, b, H, dh)
    for s in range(2):
        for j in range(J):
            if (s + j) % 3:
                R = g.standard_normal((b, d))
                rows.put(s, j, R[:, None], R[:, None])
                kv.put(s, j, R.reshape(b, H, dh), R.reshape(b, H, dh))
    nr = g.standard_normal(d)
    q, kn, vn = (g.standard_normal((2, H, dh)) for _ in range(3))
    kc, vc = g.standard_normal((2, 2, b, H, dh))
    eye = np.eye(d)
    a, _, _ = O.reader_decode_rows(rows, eye, eye, nr, [0, 1], [J, 3], [1, 3], q, kn, vn, kc, vc)
    c, _, _ = O.reader_decode(kv, [0, 1], [J, 3], [1, 3], q, kn, vn, kc, vc, nr.reshape(1, H, dh).repeat(2, 0))
    assert np.array_equal(a, c)


def test_rows_decode_matches_sdpa_on_mapped_rows():
    """Against torch: rows mapped by matmul, SDPA over [null] ++ mapped rows ++ in-block keys."""
    g = np.random.default_rng(53)
    b, H, dh, d, J = 4, 3, 8, 20, 4
    rows = O.Store(1, J, b, 1, d)
    for j in (0, 2, 3):
        R = g.standard_normal((b, d))
        rows.put(0, j, R[:, None], R[:, None])
    wk, wv = g.standard_normal((2, H * dh, d)) / np.sqrt(d)
    nr = g.standard_normal(d)
    q, kn, vn = (g.standard_normal((1, H, dh)) for _ in range(3))
    kc, vc = g.standard_normal((2, 1, b, H, dh))
    p = 2
    out, kc2, _ = O.reader_decode_rows(rows, wk, wv, nr, [0], [J], [p], q, kn, vn, kc, vc)
    _, R, _ = rows.export(0)
    T = lambda x: torch.as_tensor(np.asarray(x, np.float64))
    lin = lambda x, w: torch.nn.functional.linear(T(x), T(w))      # x w^T, the linear layer
    K = torch.cat([lin(nr[None], wk), lin(R[:, 0], wk)]).reshape(-1, H, dh)
    V = torch.cat([lin(nr[None], wv), lin(R[:, 0], wv)]).reshape(-1, H, dh)
    K = torch.cat([K, T(kc2[0, :p + 1])])
    V = torch.cat([V, T(vc[0, :p]), T(vn[0])[None]])
    for h in range(H):
        ref = F.scaled_dot_product_attention(T(q[0, h])[None, None], K[:, h][None], V[:, h][None])
        np.testing.assert_allclose(out[0, h], ref[0, 0].numpy(), atol=1e-12, rtol=0)


def _brute_attention(qv, keys, vals):
    """One query over an explicit key list, in pure Python: scores by loops,
    the maximum subtracted, exponentials, and every sum by math.fsum."""
    dh = len(qv)
    sc = [math.fsum(qv[i] * k[i] for i in range(dh)) / math.sqrt(dh) for k in keys]
    if not sc:
        return [0.0] * len(qv)
    mx = max(sc)
    w = [math.exp(x - mx) for x in sc]
    z = math.fsum(w)
    return [math.fsum(w[j] * vals[j][i] for j in range(len(keys))) / z for i in range(len(vals[0]))]


@pytest.mark.parametrize("b,dh,mask", [(1, 2, O.MASK_BIDIR), (3, 2, O.MASK_CAUSAL), (4, 3, O.MASK_BIDIR),
                                       (4, 4, O.MASK_CAUSAL)])
def test_brute_force_tiny(b, dh, mask):
    """Tiny shapes (H = 1) against a pure-Python brute force of the
    definitions: the encoder (Section 2, "Model") block by block, and the
    reader (Section 3.1) over [null] ++ memory of live blocks below J ++
    in-block keys 0..t, with a deleted block and a block at J present."""
    g = np.random.default_rng(1000 + b * 10 + dh)
    nb = 3
    q, k, v = (g.standard_normal((nb, b, 1, dh)) for _ in range(3))
    enc = O.encode_blocks(q, k, v, mask)
    for blk, t in itertools.product(range(nb), range(b)):
        vis = range(b) if mask == O.MASK_BIDIR else range(t + 1)
        ref = _brute_attention(list(q[blk, t, 0]), [list(k[blk, j, 0]) for j in vis], [list(v[blk, j, 0]) for j in vis])
        assert np.allclose(enc[blk, t, 0], ref, rtol=0, atol=1e-13)
    st = O.Store(1, 6, b, 1, dh)
    mem = {j: (g.standard_normal((b, 1, dh)), g.standard_normal((b, 1, dh))) for j in (0, 1, 2, 4)}
    for j, (K, V) in mem.items():
        st.put(0, j, K, V)
    st.delete(0, 1)
    J = 4                                          # reads blocks 0 and 2; block 4 is present and ignored
    qr, ki, vi = (g.standard_normal((1, b, 1, dh)) for _ in range(3))
    nkv = g.standard_normal((2, 1, dh))
    out = O.reader_prefill_block(st, [0], [J], qr, ki, vi, nkv)
    for t in range(b):
        keys = [list(nkv[0, 0])] + [list(mem[j][0][r, 0]) for j in (0, 2) for r in range(b)] + \
               [list(ki[0, r, 0]) for r in range(t + 1)]
        vals = [list(nkv[1, 0])] + [list(mem[j][1][r, 0]) for j in (0, 2) for r in range(b)] + \
               [list(vi[0, r, 0]) for r in range(t + 1)]
        assert np.allclose(out[0, t, 0], _brute_attention(list(qr[0, t, 0]), keys, vals), rtol=0, atol=1e-13)
