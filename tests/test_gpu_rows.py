"""GPU parity of decode from the row plane (Appendix K: K/V recomputed from
the memory rows; Appendix A: one row plane shared by all reader layers)
against the fp64 oracle, through the C ABI.  The kernels fold the key and
value maps into the query and the output; the oracle recomputes K and V row
by row.  Tolerance: max|y - y_ref| / rms(y_ref) <= 2e-2 (bf16 rows, maps and
queries, fp32 accumulation); GPU-vs-GPU identities are bitwise."""
import numpy as np
import pytest
import torch

from oracle import smem_oracle as O
from paper_2609_32395_amd import smem
from tests.gpu_util import check, dev, host, require_gpu, rows, say

pytestmark = pytest.mark.gpu
BF = torch.bfloat16


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _row_store(g, b, d, n_seq=3, max_blocks=40, live=0.8, blocks=None):
    st = smem.RowStore(n_seq, max_blocks, n_seq * max_blocks, b, d)
    ref = O.Store(n_seq, max_blocks, b, 1, d)
    for s in range(n_seq):
        for j in (blocks if blocks is not None else range(max_blocks)):
            if g.random() < live:
                R = rows(g, (b, d), BF)
                smem.smem_rows_put_block(st, s, j, dev(R, BF))
                ref.put(s, j, R[:, None], R[:, None])
    return st, ref


# (b, d, H, dh); more than 16 heads run in tiles of 16 (the last one padded):
# the model's reader layers at 160M (768 wide, 24 x 32), 410M (1024, 32 x 32)
# and 1.5B (2048, 64 x 32), and a ragged 20-head case
CASES = [(64, 1024, 16, 64), (64, 512, 8, 64), (64, 2048, 16, 128), (16, 512, 3, 32), (64, 1024, 4, 128),
         (64, 768, 24, 32), (64, 1024, 32, 32), (64, 2048, 64, 32), (16, 1024, 20, 64)]


@pytest.mark.parametrize("b,d,H,dh", CASES)
@pytest.mark.parametrize("with_null", [False, True])
@pytest.mark.parametrize("with_intra", [False, True])
def test_rows_decode_parity(b, d, H, dh, with_null, with_intra):
    say("rows decode", b, d, H, dh, with_null, with_intra)
    g = np.random.default_rng(500 + d + H + dh + 2 * with_null + with_intra)
    st, ref = _row_store(g, b, d)
    wk = rows(g, (H * dh, d), BF, 1.0 / np.sqrt(d))
    wv = rows(g, (H * dh, d), BF, 1.0 / np.sqrt(d))
    nr = rows(g, (d,), BF) if with_null else None
    seqs, J = [2, 0, 1], [40, 17, 0]
    pos = [b - 1, 0, b // 3]
    q = rows(g, (3, H, dh), BF)
    kn, vn = rows(g, (3, H, dh), BF), rows(g, (3, H, dh), BF)
    kc, vc = rows(g, (3 * b, H, dh), BF), rows(g, (3 * b, H, dh), BF)
    dkc, dvc = dev(kc, BF), dev(vc, BF)
    args = dict(k_new=dev(kn, BF), v_new=dev(vn, BF), k_cache=dkc, v_cache=dvc) if with_intra else {}
    out = smem.smem_reader_decode_rows(st, dev(wk, BF), dev(wv, BF), seqs, J, pos if with_intra else None,
                                       dev(q, BF), null_row=dev(nr, BF) if with_null else None, **args)
    if with_intra:
        expect, ekc, evc = O.reader_decode_rows(ref, wk, wv, nr, seqs, J, pos, q, kn, vn,
                                                kc.reshape(3, b, H, dh), vc.reshape(3, b, H, dh))
        assert np.array_equal(host(dkc), ekc.reshape(3 * b, H, dh))
    else:
        expect, _, _ = O.reader_decode_rows(ref, wk, wv, nr, seqs, J, [0, 0, 0], q)
    check(out, expect, BF, f"rows decode b{b} d{d} H{H} dh{dh}")
    # batch invariance: each sequence alone gives the same bits
    for i in range(3):
        sl = slice(i, i + 1)
        a1 = dict(k_new=dev(kn[sl], BF), v_new=dev(vn[sl], BF), k_cache=dev(kc[i * b:(i + 1) * b], BF),
                  v_cache=dev(vc[i * b:(i + 1) * b], BF)) if with_intra else {}
        alone = smem.smem_reader_decode_rows(st, dev(wk, BF), dev(wv, BF), [seqs[i]], [J[i]],
                                             [pos[i]] if with_intra else None, dev(q[sl], BF),
                                             null_row=dev(nr, BF) if with_null else None, **a1)
        assert torch.equal(alone, out[sl])


def test_rows_decode_premapped_null_row():
    """The null row given already through the maps ([2, H, dh]) reads as the
    oracle's null row does; 48 heads (three tiles)."""
    say("rows decode, premapped null row")
    g = np.random.default_rng(91)
    b, d, H, dh = 64, 1024, 48, 32
    st, ref = _row_store(g, b, d)
    wk = rows(g, (H * dh, d), BF, 1.0 / np.sqrt(d))
    wv = rows(g, (H * dh, d), BF, 1.0 / np.sqrt(d))
    nr = rows(g, (d,), BF)
    nkv = np.stack([(wk.astype(np.float64) @ nr).reshape(H, dh), (wv.astype(np.float64) @ nr).reshape(H, dh)])
    seqs, J = [2, 0, 1], [40, 17, 0]
    q = rows(g, (3, H, dh), BF)
    out = smem.smem_reader_decode_rows(st, dev(wk, BF), dev(wv, BF), seqs, J, None, dev(q, BF),
                                       null_kv=dev(nkv.astype(np.float32), BF))
    expect, _, _ = O.reader_decode_rows(ref, wk, wv, nr, seqs, J, [0, 0, 0], q)
    check(out, expect, BF, "rows decode premapped null row")


def test_rows_many_sequences_span_launches():
    """130 sequences (two launches of at most 128) with long memories."""
    say("rows decode, 130 sequences")
    g = np.random.default_rng(77)
    b, d, H, dh = 16, 512, 2, 32
    n = 130
    st = smem.RowStore(n, 70, n * 8, b, d)
    ref = O.Store(n, 70, b, 1, d)
    for s in range(n):
        for j in g.choice(70, size=8, replace=False):
            R = rows(g, (b, d), BF)
            smem.smem_rows_put_block(st, s, int(j), dev(R, BF))
            ref.put(s, int(j), R[:, None], R[:, None])
    wk, wv = rows(g, (H * dh, d), BF, 0.05), rows(g, (H * dh, d), BF, 0.05)
    q = rows(g, (n, H, dh), BF)
    J = [int(x) for x in g.integers(0, 71, size=n)]
    out = smem.smem_reader_decode_rows(st, dev(wk, BF), dev(wv, BF), list(range(n)), J, None, dev(q, BF))
    expect, _, _ = O.reader_decode_rows(ref, wk, wv, None, list(range(n)), J, [0] * n, q)
    check(out, expect, BF, "rows decode 130 sequences")


def test_rows_delete_equals_never_inserted_and_export():
    say("rows delete/export")
    g = np.random.default_rng(78)
    b, d, H, dh = 64, 1024, 16, 64
    R = {j: rows(g, (b, d), BF) for j in range(6)}
    a = smem.RowStore(1, 8, 8, b, d)
    c = smem.RowStore(1, 8, 8, b, d)
    for j in range(6):
        smem.smem_rows_put_block(a, 0, j, dev(R[j], BF))
        if j != 2:
            smem.smem_rows_put_block(c, 0, j, dev(R[j], BF))
    smem.smem_delete_block(a, 0, 2, scrub=True)
    ia, Ra = smem.smem_rows_export(a, 0)
    ic, Rc = smem.smem_rows_export(c, 0)
    assert ia == ic == [0, 1, 3, 4, 5] and torch.equal(Ra, Rc)
    assert np.array_equal(host(Ra), np.concatenate([R[j] for j in ia]))
    wk, wv = rows(g, (H * dh, d), BF, 0.03), rows(g, (H * dh, d), BF, 0.03)
    q = dev(rows(g, (1, H, dh), BF), BF)
    oa = smem.smem_reader_decode_rows(a, dev(wk, BF), dev(wv, BF), [0], [7], None, q)
    oc = smem.smem_reader_decode_rows(c, dev(wk, BF), dev(wv, BF), [0], [7], None, q)
    assert torch.equal(oa, oc)


def test_rows_kind_errors():
    say("rows kind errors")
    import ctypes
    g = np.random.default_rng(79)
    rs = smem.RowStore(1, 4, 4, 64, 512)
    kv = smem.Store(1, 4, 4, 64, 2, 64, BF)
    x = dev(rows(g, (64, 2, 64), BF), BF)
    P = ctypes.c_void_p(x.data_ptr())
    one = smem._i32([0])
    # key/value reader on a row store (the binding's shape checks bypassed)
    assert smem.lib().smem_reader_prefill_block(rs.handle, 1, one, smem._i32([1]), P, P, P, None, P,
                                                None) == smem.SMEM_EINVAL
    r = dev(rows(g, (64, 512), BF), BF)
    assert smem.lib().smem_rows_put_block(kv.handle, 0, 0, ctypes.c_void_p(r.data_ptr()), None) == smem.SMEM_EINVAL
    wk = dev(rows(g, (65 * 8, 512), BF), BF)
    with pytest.raises(smem.SmemError) as e:          # more than 64 heads
        smem.smem_reader_decode_rows(rs, wk, wk, [0], [1], None, dev(rows(g, (1, 65, 8), BF), BF))
    assert e.value.code == smem.SMEM_EINVAL
