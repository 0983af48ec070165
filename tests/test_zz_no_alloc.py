"""The allocation-free reader decode (smem_reader_decode_static) against the
workspace decode (smem_reader_decode) through the C ABI: the two run the same
kernels with the same split boundaries and the same fold order, so their
outputs and in-block cache writes are compared bit for bit, over two calls in
a row (the second with a smaller batch and shorter reads, so the library's
device array still holds the first call's partials), and the first call is
also checked against the fp64 oracle.  A call whose partials exceed the array
is rejected before anything runs."""
import numpy as np
import pytest
import torch

from oracle import smem_oracle as O
from paper_2609_32395_amd import smem
from tests.gpu_util import DT, check, dev, host, require_gpu, rows, say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _store(g, n_seq, max_blocks, b, H, dh, dtype, fill, scale=1.0):
    st = smem.Store(n_seq, max_blocks, n_seq * max_blocks, b, H, dh, dtype)
    ref = O.Store(n_seq, max_blocks, b, H, dh)
    for s in range(n_seq):
        for j in range(max_blocks):
            if g.random() < fill:
                K = rows(g, st.row_shape, dtype, scale)
                V = rows(g, st.row_shape, dtype, scale)
                smem.smem_store_put_block(st, s, j, dev(K, dtype), dev(V, dtype))
                ref.put(s, j, K, V)
    return st, ref


def _both(st, seq_ids, qblk, pos, q, kn, vn, kc, vc, nkv):
    """Run the workspace decode and the static decode on separate cache copies."""
    kc1, vc1, kc2, vc2 = kc.clone(), vc.clone(), kc.clone(), vc.clone()
    a = smem.smem_reader_decode(st, seq_ids, qblk, pos, q, kn, vn, kc1, vc1, nkv)
    b = smem.smem_reader_decode_static(st, seq_ids, qblk, pos, q, kn, vn, kc2, vc2, nkv)
    torch.cuda.synchronize()
    assert torch.equal(a, b), "static decode differs from the workspace decode"
    assert torch.equal(kc1, kc2) and torch.equal(vc1, vc2), "in-block cache writes differ"
    return b, kc2, vc2


@pytest.mark.parametrize("dt,b,H,dh", [("bf16", 64, 16, 64), ("bf16", 64, 4, 128), ("f32", 16, 4, 32)])
def test_static_decode_equals_workspace_decode(dt, b, H, dh):
    dtype = DT[dt]
    g = np.random.default_rng(31)
    n_seq, max_blocks = 12, 40
    say("static decode", dt, b, H, dh, "store", n_seq, "x", max_blocks)
    st, ref = _store(g, n_seq, max_blocks, b, H, dh, dtype, 0.85, 0.125 if dtype == torch.bfloat16 else 1.0)
    # call 1: every sequence, long reads (several splits each), with null row and in-block keys
    seq_ids = list(range(n_seq))
    qblk = [max_blocks - (s % 3) for s in seq_ids]
    pos = [int(x) for x in g.integers(0, b, n_seq)]
    n = n_seq
    q = rows(g, (n, H, dh), dtype)
    kn, vn = rows(g, (n, H, dh), dtype), rows(g, (n, H, dh), dtype)
    kc, vc = rows(g, (n, b, H, dh), dtype), rows(g, (n, b, H, dh), dtype)
    nkv = rows(g, (2, H, dh), dtype)
    say("static decode call 1", n, "sequences")
    out, dkc, dvc = _both(st, seq_ids, qblk, pos, dev(q, dtype), dev(kn, dtype), dev(vn, dtype),
                          dev(kc.reshape(n * b, H, dh), dtype), dev(vc.reshape(n * b, H, dh), dtype), dev(nkv, dtype))
    exp, ekc, evc = O.reader_decode(ref, seq_ids, qblk, pos, q, kn, vn, kc, vc, nkv)
    assert np.array_equal(host(dkc).reshape(n, b, H, dh), ekc)
    assert np.array_equal(host(dvc).reshape(n, b, H, dh), evc)
    check(out, exp, dtype, "static decode vs oracle")
    # call 2: fewer sequences, shorter reads, memory only (no in-block keys)
    seq_ids2 = [7, 2, 5]
    qblk2 = [9, 17, 1]
    n2 = len(seq_ids2)
    q2 = rows(g, (n2, H, dh), dtype)
    say("static decode call 2", n2, "sequences")
    a = smem.smem_reader_decode(st, seq_ids2, qblk2, None, dev(q2, dtype))
    b2 = smem.smem_reader_decode_static(st, seq_ids2, qblk2, None, dev(q2, dtype))
    torch.cuda.synchronize()
    assert torch.equal(a, b2)
    exp2, _, _ = O.reader_decode(ref, seq_ids2, qblk2, [0] * n2, q2)
    check(b2, exp2, dtype, "static decode (second call) vs oracle")
    st.close()


def test_static_decode_rejects_oversized_call():
    """Partials beyond the 4 Mi-float array: SMEM_EINVAL, nothing enqueued,
    the outputs untouched; a smaller call on the same store still works."""
    dtype = torch.bfloat16
    b, H, dh = 16, 64, 128
    n_seq, n_blocks = 128, 24          # 128 x 64 heads x 4 splits x 132 floats > 4 Mi floats
    say("static decode size limit", n_seq, "x", n_blocks, "blocks, H", H, "dh", dh)
    st = smem.Store(n_seq, n_blocks, n_seq * n_blocks, b, H, dh, dtype)
    blk = torch.zeros((32 * b, H, dh), dtype=dtype, device="cuda")
    for s in range(n_seq):
        for j0 in range(0, n_blocks, 32):
            m = min(32, n_blocks - j0)
            smem.smem_store_put_blocks(st, [s] * m, list(range(j0, j0 + m)), blk[: m * b], blk[: m * b])
    q = torch.ones((n_seq, H, dh), dtype=dtype, device="cuda")
    out = torch.full((n_seq, H, dh), 7.0, dtype=dtype, device="cuda")
    with pytest.raises(smem.SmemError) as e:
        smem.smem_reader_decode_static(st, list(range(n_seq)), [n_blocks] * n_seq, None, q, out=out)
    assert e.value.code == smem.SMEM_EINVAL and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
    # 16 sequences fit (16 x 64 x 4 x 132 floats); all rows are zero, so the output is zero
    o2 = smem.smem_reader_decode_static(st, list(range(16)), [n_blocks] * 16, None, q[:16])
    torch.cuda.synchronize()
    assert torch.count_nonzero(o2) == 0
    st.close()
