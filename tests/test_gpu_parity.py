"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Store, index and deletion work must be bit-exact; attention outputs must be
within max|y - y_ref| / rms(y_ref) <= 1e-5 (fp32) or 2e-2 (bf16 inputs,
fp32 accumulation).  GPU-vs-GPU invariants (delete equals never inserted,
edit-path independence, batch invariance) are bitwise.
"""
import numpy as np
import pytest
import torch

from oracle import smem_oracle as O
from paper_2609_32395_amd import smem, synth
from tests.gpu_util import DT, TOL, check, dev, host, require_gpu, rows, say

pytestmark = pytest.mark.gpu

SHAPES = [("f32", 16, 4, 32), ("f32", 64, 2, 64), ("bf16", 64, 4, 64), ("bf16", 64, 2, 128),
          ("bf16", 16, 3, 32), ("f32", 16, 2, 128), ("bf16", 16, 2, 64), ("f32", 64, 2, 32),
          ("bf16", 64, 3, 32)]


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _fill(g, st, ref, seq, blocks, dtype, scale=1.0):
    for j in blocks:
        K = rows(g, st.row_shape, dtype, scale)
        V = rows(g, st.row_shape, dtype, scale)
        smem.smem_store_put_block(st, seq, j, dev(K, dtype), dev(V, dtype))
        ref.put(seq, j, K, V)


def _assert_export_equal(st, ref, seq):
    idx, K, V = smem.smem_store_export(st, seq)
    ridx, RK, RV = ref.export(seq)
    assert idx == ridx
    if idx:
        assert np.array_equal(host(K), RK) and np.array_equal(host(V), RV)


# ------------------------------------------------------------------ store

@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
def test_put_delete_export_bitwise(dt, b, H, dh):
    say("store bitwise", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(1)
    st = smem.Store(2, 10, 12, b, H, dh, dtype)
    ref = O.Store(2, 10, b, H, dh)
    _fill(g, st, ref, 0, [7, 2, 9, 0], dtype)
    _fill(g, st, ref, 1, [1, 3], dtype)
    for s in (0, 1):
        _assert_export_equal(st, ref, s)
    smem.smem_delete_block(st, 0, 2, scrub=True)
    ref.delete(0, 2)
    _fill(g, st, ref, 1, [2, 8], dtype)   # reuses the scrubbed page
    smem.smem_delete_block(st, 0, 9)
    ref.delete(0, 9)
    for s in (0, 1):
        _assert_export_equal(st, ref, s)
    with pytest.raises(smem.SmemError) as e:
        smem.smem_delete_block(st, 0, 9)
    assert e.value.code == smem.SMEM_ENOENT
    x = dev(rows(g, st.row_shape, dtype), dtype)
    with pytest.raises(smem.SmemError) as e:
        smem.smem_store_put_block(st, 1, 8, x, x)
    assert e.value.code == smem.SMEM_EEXIST
    for s in (0, 1):
        _assert_export_equal(st, ref, s)


def test_pool_exhaustion_and_reuse():
    say("pool exhaustion")
    g = np.random.default_rng(2)
    st = smem.Store(1, 8, 3, 16, 2, 32, torch.float32)
    ref = O.Store(1, 8, 16, 2, 32)
    _fill(g, st, ref, 0, [0, 1, 2], torch.float32)
    x = dev(rows(g, st.row_shape, torch.float32), torch.float32)
    with pytest.raises(smem.SmemError) as e:
        smem.smem_store_put_block(st, 0, 5, x, x)
    assert e.value.code == smem.SMEM_ENOMEM
    smem.smem_delete_block(st, 0, 1)
    ref.delete(0, 1)
    _fill(g, st, ref, 0, [5], torch.float32)
    _assert_export_equal(st, ref, 0)


# ------------------------------------------------------------------ encoder

@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
@pytest.mark.parametrize("mask", [smem.MASK_BIDIR, smem.MASK_CAUSAL])
def test_encoder_parity(dt, b, H, dh, mask):
    say("encoder parity", dt, b, H, dh, mask)
    dtype = DT[dt]
    g = np.random.default_rng(3)
    nb = 5
    q, k, v = (rows(g, (nb, b, H, dh), dtype) for _ in range(3))
    out = smem.smem_encode_blocks(None, dev(q.reshape(nb * b, H, dh), dtype), dev(k.reshape(nb * b, H, dh), dtype),
                                  dev(v.reshape(nb * b, H, dh), dtype), mask=mask, b=b)
    ref = O.encode_blocks(q, k, v, mask).reshape(nb * b, H, dh)
    check(out, ref, dtype, "encoder")


@pytest.mark.parametrize("dt,b,H,dh", [("f32", 16, 4, 32), ("bf16", 64, 4, 64), ("bf16", 64, 2, 128)])
def test_encoder_inserts_rows_and_is_batch_invariant(dt, b, H, dh):
    say("encoder insert", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(4)
    nb = 6
    q, k, v = (dev(rows(g, (nb * b, H, dh), dtype), dtype) for _ in range(3))
    st = smem.Store(2, 8, 8, b, H, dh, dtype)
    seqs, blks = [0, 1, 0, 1, 0, 0], [3, 0, 1, 5, 6, 0]
    out = smem.smem_encode_blocks(st, q, k, v, seq_ids=seqs, block_idx=blks, mask=smem.MASK_BIDIR)
    O_ = host(out).reshape(nb, b, H, dh)
    for s in (0, 1):
        idx, K, V = smem.smem_store_export(st, s)
        order = sorted((j, i) for i, (ss, j) in enumerate(zip(seqs, blks)) if ss == s)
        assert idx == [j for j, _ in order]
        exp = np.concatenate([O_[i] for _, i in order], 0)
        assert np.array_equal(host(K), exp) and np.array_equal(host(V), exp)
    # a block encoded alone gives the same bits as inside the batch
    for i in range(nb):
        one = smem.smem_encode_blocks(None, q[i * b:(i + 1) * b], k[i * b:(i + 1) * b], v[i * b:(i + 1) * b],
                                      mask=smem.MASK_BIDIR, b=b)
        assert torch.equal(one, out[i * b:(i + 1) * b])
    # all-or-nothing: one occupied target rejects the whole call and changes nothing
    before = [smem.smem_store_export(st, s) for s in (0, 1)]
    with pytest.raises(smem.SmemError) as e:
        smem.smem_encode_blocks(st, q[:2 * b], k[:2 * b], v[:2 * b], seq_ids=[1, 0], block_idx=[7, 3])
    assert e.value.code == smem.SMEM_EEXIST
    after = [smem.smem_store_export(st, s) for s in (0, 1)]
    for (i0, k0, v0), (i1, k1, v1) in zip(before, after):
        assert i0 == i1 and torch.equal(k0, k1) and torch.equal(v0, v1)
    assert st.stats()[0] == nb


# ------------------------------------------------------------------ reader prefill

def _prefill_case(dt, b, H, dh, with_null, with_intra, seed=5, n_seq=3, max_blocks=12):
    dtype = DT[dt]
    g = np.random.default_rng(seed)
    st = smem.Store(n_seq, max_blocks, n_seq * max_blocks, b, H, dh, dtype)
    ref = O.Store(n_seq, max_blocks, b, H, dh)
    for s in range(n_seq):
        blocks = [j for j in range(max_blocks) if g.random() < 0.7]
        _fill(g, st, ref, s, blocks, dtype)
    seq_ids = [0, 2, 1, 0][: n_seq + 1]
    qblk = [max_blocks, 5, 0, 9][: n_seq + 1]
    n = len(seq_ids)
    q = rows(g, (n, b, H, dh), dtype)
    ki = rows(g, (n, b, H, dh), dtype) if with_intra else None
    vi = rows(g, (n, b, H, dh), dtype) if with_intra else None
    nkv = rows(g, (2, H, dh), dtype) if with_null else None
    out = smem.smem_reader_prefill_block(
        st, seq_ids, qblk, dev(q.reshape(n * b, H, dh), dtype),
        None if ki is None else dev(ki.reshape(n * b, H, dh), dtype),
        None if vi is None else dev(vi.reshape(n * b, H, dh), dtype),
        None if nkv is None else dev(nkv, dtype))
    exp = O.reader_prefill_block(ref, seq_ids, qblk, q, ki, vi, nkv).reshape(n * b, H, dh)
    return out, exp, dtype


@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
@pytest.mark.parametrize("with_null,with_intra", [(False, True), (True, True), (True, False)])
def test_prefill_parity(dt, b, H, dh, with_null, with_intra):
    say("prefill parity", dt, b, H, dh, with_null, with_intra)
    out, exp, dtype = _prefill_case(dt, b, H, dh, with_null, with_intra)
    check(out, exp, dtype, "prefill")



@pytest.mark.parametrize("dh", [32, 64, 128])
@pytest.mark.parametrize("with_null,with_intra", [(True, True), (False, False)])
def test_prefill_one_workgroup_mode_bitwise(dh, with_null, with_intra):
    """A prefill launch of at least 512 (query block, head) pairs reads every
    split of a pair in one workgroup and folds them itself; the same block
    served alone (16 pairs) does so only if its read is short (at most 16
    pages, 8 at d_h 128), else it runs one workgroup per split and the
    merge.  Both must agree bitwise for every block, and each block must match the
    oracle.  Query blocks 0..32 of a sequence of 32 blocks (blocks 5 and 17
    deleted: 0 to 30 memory pages, 1 to 9 splits) and blocks 48, 3 and 20 of
    a sequence of 48 (up to 48 pages, 13 splits): 36 x 16 = 576 pairs."""
    say("prefill one-workgroup mode", dh, with_null, with_intra)
    dtype = torch.bfloat16
    b, H, J0, J1 = 64, 16, 32, 48
    g = np.random.default_rng(31 + dh)
    st = smem.Store(2, J1 + 1, J0 + J1, b, H, dh, dtype)
    ref = O.Store(2, J1 + 1, b, H, dh)
    _fill(g, st, ref, 0, range(J0), dtype)
    _fill(g, st, ref, 1, range(J1), dtype)
    for j in (5, 17):
        smem.smem_delete_block(st, 0, j)
        ref.delete(0, j)
    seq_ids = [0] * (J0 + 1) + [1, 1, 1]
    qblk = list(range(J0 + 1)) + [J1, 3, 20]
    n = len(seq_ids)
    assert n * H >= 512
    q = rows(g, (n, b, H, dh), dtype)
    ki = rows(g, (n, b, H, dh), dtype) if with_intra else None
    vi = rows(g, (n, b, H, dh), dtype) if with_intra else None
    nkv = rows(g, (2, H, dh), dtype) if with_null else None
    d = lambda x: None if x is None else dev(x.reshape(-1, H, dh), dtype)
    dn = None if nkv is None else dev(nkv, dtype)
    out = smem.smem_reader_prefill_block(st, seq_ids, qblk, d(q), d(ki), d(vi), dn)
    for i in range(n):
        one = smem.smem_reader_prefill_block(st, [seq_ids[i]], [qblk[i]], d(q[i]),
                                             None if ki is None else d(ki[i]), None if vi is None else d(vi[i]), dn)
        assert torch.equal(one, out[i * b:(i + 1) * b]), f"slot {i} (block {qblk[i]} of sequence {seq_ids[i]})"
    exp = O.reader_prefill_block(ref, seq_ids, qblk, q, ki, vi, nkv).reshape(n * b, H, dh)
    if not with_null and not with_intra:
        # query block 0 of sequence 0 reads nothing: its output is zero
        assert not torch.any(out[:b])
    # each query block is its own attention problem, checked at its own RMS: a
    # block with few keys has outputs of the values' size, one with a thousand
    # keys outputs about thirty times smaller
    for i in range(n):
        check(out[i * b:(i + 1) * b], exp[i * b:(i + 1) * b], dtype, f"slot {i} (block {qblk[i]})")



def test_prefill_fold_with_odd_split_sizes_bitwise():
    """32 heads of 32 (the model's heads): splits of max(4, ceil(n/16)) pages,
    so reads of 65-79 pages take splits of 5 pages.  Query blocks 60..80 of one
    sequence in one launch (672 pairs: one workgroup per pair folds its
    splits) equal each block served alone (32 pairs over more than 16 pages:
    split launch and merge), bitwise; a sample matches the oracle."""
    say("prefill fold, odd split sizes")
    dtype = torch.bfloat16
    b, H, dh, J = 64, 32, 32, 80
    g = np.random.default_rng(61)
    st = smem.Store(1, J + 1, J, b, H, dh, dtype)
    ref = O.Store(1, J + 1, b, H, dh)
    _fill(g, st, ref, 0, range(J), dtype)
    qblk = list(range(60, J + 1))
    n = len(qblk)
    q, ki, vi = (rows(g, (n, b, H, dh), dtype) for _ in range(3))
    nkv = rows(g, (2, H, dh), dtype)
    d = lambda x: dev(x.reshape(-1, H, dh), dtype)
    dn = dev(nkv, dtype)
    out = smem.smem_reader_prefill_block(st, [0] * n, qblk, d(q), d(ki), d(vi), dn)
    for i in range(n):
        one = smem.smem_reader_prefill_block(st, [0], [qblk[i]], d(q[i]), d(ki[i]), d(vi[i]), dn)
        assert torch.equal(one, out[i * b:(i + 1) * b]), f"block {qblk[i]}"
    sample = [0, 5, 12, 20]
    exp = O.reader_prefill_block(ref, [0] * len(sample), [qblk[i] for i in sample], q[sample], ki[sample],
                                 vi[sample], nkv)
    for k, i in enumerate(sample):
        check(out[i * b:(i + 1) * b], exp[k].reshape(b, H, dh), dtype, f"block {qblk[i]}")

def test_prefill_empty_key_set_is_zero():
    say("prefill empty")
    st = smem.Store(1, 4, 4, 16, 2, 32, torch.float32)
    q = torch.randn(16, 2, 32, device="cuda")
    out = smem.smem_reader_prefill_block(st, [0], [3], q)
    assert torch.count_nonzero(out) == 0


# ------------------------------------------------------------------ reader decode

@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
@pytest.mark.parametrize("with_null,with_intra", [(False, True), (True, True), (False, False)])
def test_decode_parity(dt, b, H, dh, with_null, with_intra):
    say("decode parity", dt, b, H, dh, with_null, with_intra)
    dtype = DT[dt]
    g = np.random.default_rng(6)
    n_seq, max_blocks = 5, 20
    st = smem.Store(n_seq, max_blocks, n_seq * max_blocks, b, H, dh, dtype)
    ref = O.Store(n_seq, max_blocks, b, H, dh)
    for s in range(n_seq):
        _fill(g, st, ref, s, [j for j in range(max_blocks) if g.random() < 0.8], dtype)
    seq_ids = [3, 0, 4, 1]
    qblk = [20, 13, 1, 0]
    pos = [0, b - 1, 5 % b, 7 % b]
    n = len(seq_ids)
    q = rows(g, (n, H, dh), dtype)
    nkv = rows(g, (2, H, dh), dtype) if with_null else None
    if with_intra:
        kn, vn = rows(g, (n, H, dh), dtype), rows(g, (n, H, dh), dtype)
        kc, vc = rows(g, (n, b, H, dh), dtype), rows(g, (n, b, H, dh), dtype)
        dkc, dvc = dev(kc.reshape(n * b, H, dh), dtype), dev(vc.reshape(n * b, H, dh), dtype)
        out = smem.smem_reader_decode(st, seq_ids, qblk, pos, dev(q, dtype), dev(kn, dtype), dev(vn, dtype),
                                      dkc, dvc, None if nkv is None else dev(nkv, dtype))
        exp, ekc, evc = O.reader_decode(ref, seq_ids, qblk, pos, q, kn, vn, kc, vc, nkv)
        assert np.array_equal(host(dkc).reshape(n, b, H, dh), ekc)
        assert np.array_equal(host(dvc).reshape(n, b, H, dh), evc)
    else:
        out = smem.smem_reader_decode(st, seq_ids, qblk, None, dev(q, dtype),
                                      null_kv=None if nkv is None else dev(nkv, dtype))
        exp, _, _ = O.reader_decode(ref, seq_ids, qblk, [0] * n, q, null_kv=nkv)
    if not with_null and not with_intra:
        # sequence row 3 reads block 0 of nothing: an empty key set gives zero
        assert torch.count_nonzero(out[3]) == 0
    check(out, exp, dtype, "decode")


@pytest.mark.parametrize("dt,b,H,dh", [("f32", 16, 4, 32), ("bf16", 64, 4, 64), ("bf16", 64, 2, 128)])
def test_decode_equals_prefill_row(dt, b, H, dh):
    """Decode at position p reads the same keys as prefill row p (Appendix K)."""
    say("decode vs prefill", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(7)
    st = smem.Store(2, 9, 18, b, H, dh, dtype)
    ref = O.Store(2, 9, b, H, dh)
    for s in range(2):
        _fill(g, st, ref, s, [0, 1, 3, 4, 6, 7, 8], dtype)
    q, ki, vi = (rows(g, (2, b, H, dh), dtype) for _ in range(3))
    nkv = dev(rows(g, (2, H, dh), dtype), dtype)
    pre = smem.smem_reader_prefill_block(st, [0, 1], [9, 5], dev(q.reshape(2 * b, H, dh), dtype),
                                         dev(ki.reshape(2 * b, H, dh), dtype), dev(vi.reshape(2 * b, H, dh), dtype),
                                         nkv).reshape(2, b, H, dh)
    for p in sorted({0, 1, b // 2, b - 1}):
        kc = dev(ki.reshape(2 * b, H, dh), dtype)
        vc = dev(vi.reshape(2 * b, H, dh), dtype)
        dec = smem.smem_reader_decode(st, [0, 1], [9, 5], [p, p], dev(q[:, p], dtype), dev(ki[:, p], dtype),
                                      dev(vi[:, p], dtype), kc, vc, nkv)
        check(dec, host(pre[:, p]), dtype, f"decode vs prefill row {p}", roundings=2)


# ------------------------------------------------------------------ exact editing on the GPU

@pytest.mark.parametrize("dt,b,H,dh", [("f32", 16, 4, 32), ("bf16", 64, 4, 64), ("bf16", 64, 2, 128)])
def test_delete_equals_never_inserted_bitwise(dt, b, H, dh):
    """Theorem 1 / gate G7 on the GPU: after deleting a block, reads are
    bit-identical to a store where it was never inserted."""
    say("delete == never inserted", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(8)
    nb = 12
    blocks = {j: (dev(rows(g, (b, H, dh), dtype), dtype), dev(rows(g, (b, H, dh), dtype), dtype)) for j in range(nb)}
    a = smem.Store(1, nb, nb, b, H, dh, dtype)
    c = smem.Store(1, nb, nb, b, H, dh, dtype)
    for j in range(nb):
        smem.smem_store_put_block(a, 0, j, *blocks[j])
    for j in reversed(range(nb)):
        if j != 3:
            smem.smem_store_put_block(c, 0, j, *blocks[j])
    smem.smem_delete_block(a, 0, 3, scrub=True)
    q = dev(rows(g, (b, H, dh), dtype), dtype)
    ki = dev(rows(g, (b, H, dh), dtype), dtype)
    nkv = dev(rows(g, (2, H, dh), dtype), dtype)
    ra = smem.smem_reader_prefill_block(a, [0], [nb], q, ki, ki, nkv)
    rc = smem.smem_reader_prefill_block(c, [0], [nb], q, ki, ki, nkv)
    assert torch.equal(ra, rc)
    kc = ki.clone()
    da = smem.smem_reader_decode(a, [0], [nb], [5], q[:1], ki[:1], ki[:1], kc.clone(), kc.clone(), nkv)
    dc = smem.smem_reader_decode(c, [0], [nb], [5], q[:1], ki[:1], ki[:1], kc.clone(), kc.clone(), nkv)
    assert torch.equal(da, dc)
    ia, Ka, Va = smem.smem_store_export(a, 0)
    ic, Kc, Vc = smem.smem_store_export(c, 0)
    assert ia == ic and torch.equal(Ka, Kc) and torch.equal(Va, Vc)
    # add then remove returns the identical memory and reads
    smem.smem_store_put_block(a, 0, 3, *blocks[3])
    smem.smem_delete_block(a, 0, 3)
    assert torch.equal(smem.smem_reader_prefill_block(a, [0], [nb], q, ki, ki, nkv), rc)


def test_store_edits_at_65536_blocks_bitwise():
    """The deletion-latency sweep's largest table (65,536 block indices of one
    sequence, half of them present, a tiny page shape so the oracle can hold
    every row): single deletions and re-insertions anywhere (the first live
    block among them, which shifts the whole live list), then a batch of
    more than 128 edits; the live list and the exported rows equal the oracle
    store's bit for bit after each round, and reads over all 32,768 blocks
    match the oracle."""
    dtype = torch.float32
    b, H, dh, NB = 16, 1, 32, 65536
    say("store edits at", NB, "blocks")
    g = np.random.default_rng(65536)
    st = smem.Store(1, NB, NB, b, H, dh, dtype)
    ref = O.Store(1, NB, b, H, dh)
    present = sorted(int(j) for j in g.choice(NB, NB // 2, replace=False))
    K = g.standard_normal((len(present), b, H, dh)).astype(np.float32)
    V = g.standard_normal((len(present), b, H, dh)).astype(np.float32)
    rows_of = {j: i for i, j in enumerate(present)}
    for i0 in range(0, len(present), 4096):
        blk = present[i0:i0 + 4096]
        smem.smem_store_put_blocks(st, [0] * len(blk), blk, dev(K[i0:i0 + len(blk)].reshape(-1, H, dh), dtype),
                                   dev(V[i0:i0 + len(blk)].reshape(-1, H, dh), dtype))
    for j in present:
        ref.put(0, j, K[rows_of[j]], V[rows_of[j]])

    def same():
        idx, Kx, Vx = smem.smem_store_export(st, 0)
        ridx, RK, RV = ref.export(0)
        assert idx == ridx
        assert np.array_equal(host(Kx), RK) and np.array_equal(host(Vx), RV)

    same()
    live = list(present)
    for r in range(3):
        gone = [live[0]] + [int(j) for j in g.choice(live, 40, replace=False) if j != live[0]]
        for j in gone:
            smem.smem_delete_block(st, 0, j, scrub=(j % 2 == 0))
            ref.delete(0, j)
        back = gone[: len(gone) // 2]
        for j in back:
            smem.smem_store_put_block(st, 0, j, dev(K[rows_of[j]], dtype), dev(V[rows_of[j]], dtype))
            ref.put(0, j, K[rows_of[j]], V[rows_of[j]])
        live = sorted(set(live) - set(gone) | set(back))
        same()
    # a batch of 300 inserts (three groups of edits) of absent blocks, with new rows
    absent = sorted(set(range(NB)) - set(live))
    new = sorted(int(j) for j in g.choice(absent, 300, replace=False))
    Kn = g.standard_normal((len(new), b, H, dh)).astype(np.float32)
    Vn = g.standard_normal((len(new), b, H, dh)).astype(np.float32)
    smem.smem_store_put_blocks(st, [0] * len(new), new, dev(Kn.reshape(-1, H, dh), dtype),
                               dev(Vn.reshape(-1, H, dh), dtype))
    for i, j in enumerate(new):
        ref.put(0, j, Kn[i], Vn[i])
    same()
    # reads over every present block
    q = g.standard_normal((1, b, H, dh)).astype(np.float32)
    out = smem.smem_reader_prefill_block(st, [0], [NB], dev(q.reshape(b, H, dh), dtype))
    check(out, O.reader_prefill_block(ref, [0], [NB], q).reshape(b, H, dh), dtype, "prefill over 65536 blocks")
    qd = q[:, 3]
    dec = smem.smem_reader_decode(st, [0], [NB], None, dev(qd, dtype))
    check(dec, O.reader_decode(ref, [0], [NB], [0], qd)[0], dtype, "decode over 65536 blocks")
    st.close()


@pytest.mark.parametrize("dt,b,H,dh", [("f32", 16, 2, 32), ("bf16", 64, 2, 64)])
def test_edit_path_independence_bitwise(dt, b, H, dh):
    """Gate G8 on the GPU: random edit sequences reaching one multiset give
    bit-identical exports and reads."""
    say("edit path independence", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(9)
    nb = 16
    blocks = {j: (dev(rows(g, (b, H, dh), dtype), dtype), dev(rows(g, (b, H, dh), dtype), dtype)) for j in range(nb)}
    final = set(g.choice(nb, size=9, replace=False).tolist())
    q = dev(rows(g, (b, H, dh), dtype), dtype)
    ref_read = ref_dec = ref_exp = None
    for trial in range(8):
        r = np.random.default_rng(100 + trial)
        st = smem.Store(1, nb, nb, b, H, dh, dtype)
        present = set()
        for _ in range(int(r.integers(10, 40))):
            j = int(r.integers(0, nb))
            if j in present:
                smem.smem_delete_block(st, 0, j, scrub=bool(r.integers(0, 2)))
                present.discard(j)
            else:
                smem.smem_store_put_block(st, 0, j, *blocks[j])
                present.add(j)
        for j in sorted(present - final):
            smem.smem_delete_block(st, 0, j)
        for j in sorted(final - present, reverse=bool(trial % 2)):
            smem.smem_store_put_block(st, 0, j, *blocks[j])
        read = smem.smem_reader_prefill_block(st, [0], [nb], q, q, q)
        dec = smem.smem_reader_decode(st, [0], [nb - 2], None, q[:1])
        exp = smem.smem_store_export(st, 0)
        if ref_read is None:
            ref_read, ref_dec, ref_exp = read, dec, exp
        assert torch.equal(read, ref_read) and torch.equal(dec, ref_dec)
        assert exp[0] == ref_exp[0] and torch.equal(exp[1], ref_exp[1]) and torch.equal(exp[2], ref_exp[2])


# ------------------------------------------------------------------ the tiny fp32 workload end to end

def test_tiny_workload_end_to_end():
    """fp32, 4 heads x dh 32, b = 16: encode 8 blocks (block-local causal) into
    the store, prefill block 8 over blocks 0-7, delete block 3, read again."""
    w = synth.TINY_F32
    say("tiny workload", w.name)
    dtype = torch.float32
    b, H, dh = w.b, w.H, w.dh
    qs = np.stack([synth.block_tokens(w, 0, synth.ROLE_Q, 0, j) for j in range(9)])
    ks = np.stack([synth.block_tokens(w, 0, synth.ROLE_K, 0, j) for j in range(9)])
    vs = np.stack([synth.block_tokens(w, 0, synth.ROLE_V, 0, j) for j in range(9)])
    st = smem.Store(1, 16, 16, b, H, dh, dtype)
    ref = O.Store(1, 16, b, H, dh)
    enc = smem.smem_encode_blocks(st, dev(qs[:8].reshape(-1, H, dh), dtype), dev(ks[:8].reshape(-1, H, dh), dtype),
                                  dev(vs[:8].reshape(-1, H, dh), dtype), seq_ids=[0] * 8, block_idx=list(range(8)),
                                  mask=smem.MASK_CAUSAL)
    renc = O.encode_into_store(ref, [0] * 8, list(range(8)), qs[:8], ks[:8], vs[:8], O.MASK_CAUSAL)
    check(enc, renc.reshape(-1, H, dh), dtype, "encode")
    q8, k8, v8 = (dev(x[8], dtype) for x in (qs, ks, vs))
    out = smem.smem_reader_prefill_block(st, [0], [8], q8, k8, v8)
    check(out, O.reader_prefill_block(ref, [0], [8], qs[8:9], ks[8:9], vs[8:9])[0], dtype, "prefill")
    smem.smem_delete_block(st, 0, 3)
    ref.delete(0, 3)
    out2 = smem.smem_reader_prefill_block(st, [0], [8], q8, k8, v8)
    check(out2, O.reader_prefill_block(ref, [0], [8], qs[8:9], ks[8:9], vs[8:9])[0], dtype, "re-read")
    assert smem.smem_store_export(st, 0, rows=False)[0] == [0, 1, 2, 4, 5, 6, 7]


# ------------------------------------------------------------------ launch chunking

def test_large_batches_span_several_launches():
    """More sequences, slots, blocks and edits than one launch carries: decode of
    130 sequences (128 per launch), prefill of 20 query blocks (16 per launch),
    encode of 130 blocks into a store (128 per launch, 128 edits per metadata
    launch)."""
    say("large batches")
    dtype = torch.bfloat16
    b, H, dh = 64, 1, 32       # bf16 blocks of 64: the MFMA encoder and prefill
    g = np.random.default_rng(21)
    n = 130
    st = smem.Store(n, 3, 3 * n, b, H, dh, dtype)
    ref = O.Store(n, 3, b, H, dh)
    q, k, v = (rows(g, (n, b, H, dh), dtype) for _ in range(3))
    enc = smem.smem_encode_blocks(st, dev(q.reshape(-1, H, dh), dtype), dev(k.reshape(-1, H, dh), dtype),
                                  dev(v.reshape(-1, H, dh), dtype), seq_ids=list(range(n)), block_idx=[0] * n)
    renc = O.encode_into_store(ref, list(range(n)), [0] * n, q, k, v)
    check(enc, renc.reshape(-1, H, dh), dtype, "encode 130 blocks")
    hb = host(enc).reshape(n, b, H, dh)
    for s in (0, 64, 127, 128, 129):
        idx, K, V = smem.smem_store_export(st, s)
        assert idx == [0] and np.array_equal(host(K), hb[s]) and np.array_equal(host(V), hb[s])
        ref.delete(s, 0)
        ref.put(s, 0, hb[s], hb[s])   # the oracle reads the stored rows from here on
    for s in range(n):
        if s not in (0, 64, 127, 128, 129):
            ref.delete(s, 0)
            ref.put(s, 0, hb[s], hb[s])
    _fill(g, st, ref, 7, [1], dtype)
    qd = rows(g, (n, H, dh), dtype)
    out = smem.smem_reader_decode(st, list(range(n)), [2] * n, None, dev(qd, dtype))
    exp, _, _ = O.reader_decode(ref, list(range(n)), [2] * n, [0] * n, qd)
    check(out, exp, dtype, "decode 130 sequences")
    seqs = list(range(20))
    qp = rows(g, (20, b, H, dh), dtype)
    out = smem.smem_reader_prefill_block(st, seqs, [3] * 20, dev(qp.reshape(-1, H, dh), dtype),
                                         dev(qp.reshape(-1, H, dh), dtype), dev(qp.reshape(-1, H, dh), dtype))
    exp = O.reader_prefill_block(ref, seqs, [3] * 20, qp, qp, qp)
    check(out, exp.reshape(-1, H, dh), dtype, "prefill 20 query blocks")


def test_device_copy_both_paths():
    """The calibration copies (registers, LDS by DMA) reproduce their source
    bit for bit; sizes off their unit are rejected before anything runs."""
    say("device copy")
    src = torch.arange(3 * 4096 * 2, dtype=torch.int32, device="cuda").view(torch.float32)   # 96 KiB
    for via in (False, True):
        dst = torch.zeros_like(src)
        smem.smem_device_copy(dst, src, via_lds=via)
        torch.cuda.synchronize()
        assert torch.equal(dst.view(torch.int32), src.view(torch.int32))
    with pytest.raises(smem.SmemError):
        smem.smem_device_copy(torch.zeros(1000, device="cuda"), torch.zeros(1000, device="cuda"), via_lds=True)
