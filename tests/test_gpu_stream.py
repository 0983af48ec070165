"""GPU parity of the serving loop around the store, through the C ABI:

* decode that streams across block boundaries, appending each block to the
  memory as its last token is decoded (Section 3.1 "Decode"; Appendix K,
  decode read across a block boundary);
* partial reuse: the reader runs from the first uncached block (Section 3.1),
  bitwise equal to a cold encode of every block and to full reuse;
* in-place re-encode under the slot scheme beyond the trained block count
  (Section 2; Appendix A, "Length extension").

Attention outputs are held to the oracle within max|y - y_ref| / rms(y_ref)
<= 1e-5 (fp32) or 2e-2 (bf16); GPU-vs-GPU identities are bitwise.
"""
import numpy as np
import pytest
import torch

from oracle import smem_oracle as O
from paper_2609_32395_amd import smem
from tests.gpu_util import DT, check, dev, host, require_gpu, rows, say

pytestmark = pytest.mark.gpu

SHAPES = [("f32", 16, 2, 32), ("bf16", 64, 2, 64), ("bf16", 64, 2, 128), ("bf16", 16, 3, 64)]


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _blocks(x, b):
    """[n, T, H, dh] -> [n*T, H, dh] rows (block-major when T is a multiple of b)."""
    return x.reshape(-1, *x.shape[2:])


@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
@pytest.mark.parametrize("with_null", [False, True])
def test_stream_decode_appends_at_block_boundaries(dt, b, H, dh, with_null):
    say("stream decode", dt, b, H, dh, with_null)
    dtype = DT[dt]
    g = np.random.default_rng(61 + b + dh)
    n, T = 3, 2 * b + b // 2 + 1            # two boundaries, then part of a third block
    seqs, start = [0, 2, 1], [2, 5, 0]
    st = smem.Store(3, 12, 24, b, H, dh, dtype)
    ref = O.Store(3, 12, b, H, dh)
    for s, blocks in ((0, (0, 1)), (2, (0, 2, 4)), (1, ())):
        for j in blocks:
            K, V = rows(g, st.row_shape, dtype), rows(g, st.row_shape, dtype)
            smem.smem_store_put_block(st, s, j, dev(K, dtype), dev(V, dtype))
            ref.put(s, j, K, V)
    q, kn, vn, qe, ke, ve = (rows(g, (n, T, H, dh), dtype) for _ in range(6))
    nkv = rows(g, (2, H, dh), dtype) if with_null else None
    expect = O.stream_decode(ref, seqs, start, q, kn, vn, qe, ke, ve, nkv)

    dq, dkn, dvn, dqe, dke, dve = (dev(x, dtype) for x in (q, kn, vn, qe, ke, ve))
    dnkv = dev(nkv, dtype) if with_null else None
    kc = torch.zeros((n * b, H, dh), dtype=dtype, device="cuda")
    vc = torch.zeros_like(kc)
    steps = []
    for t in range(T):
        p = t % b
        J = [start[i] + t // b for i in range(n)]
        steps.append(smem.smem_reader_decode(st, seqs, J, [p] * n, dq[:, t].contiguous(), dkn[:, t].contiguous(),
                                             dvn[:, t].contiguous(), kc, vc, dnkv))
        if p == b - 1:
            lo = t - b + 1
            cut = lambda x: _blocks(x[:, lo:t + 1].contiguous(), b)
            smem.smem_encode_blocks(st, cut(dqe), cut(dke), cut(dve), seq_ids=seqs, block_idx=J)
    out = torch.stack(steps, 1)
    # later blocks read appended rows, themselves rounded encoder outputs
    check(out, expect, dtype, f"stream decode {dt} b{b} H{H} dh{dh}", roundings=2)
    for s in range(3):
        idx, K, V = smem.smem_store_export(st, s)
        ridx, RK, _ = ref.export(s)
        assert idx == ridx
        check(K, RK, dtype, f"memory rows seq {s}")
    # the appended blocks are the bytes a one-shot encode of the same blocks gives
    whole = smem.smem_encode_blocks(None, _blocks(dqe[:, :2 * b].contiguous(), b),
                                    _blocks(dke[:, :2 * b].contiguous(), b),
                                    _blocks(dve[:, :2 * b].contiguous(), b), b=b).reshape(n, 2 * b, H, dh)
    for i, s in enumerate(seqs):
        idx, K, V = smem.smem_store_export(st, s)
        for blk in range(2):
            r = idx.index(start[i] + blk)
            assert torch.equal(K[r * b:(r + 1) * b], whole[i, blk * b:(blk + 1) * b])
            assert torch.equal(V[r * b:(r + 1) * b], whole[i, blk * b:(blk + 1) * b])


@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
def test_partial_reuse_equals_cold_and_full_reuse(dt, b, H, dh):
    """Serve block J of a context whose first c blocks are cached: encode the
    rest, then read.  Cold (nothing cached), partial and full reuse give the
    same bytes; all three match the oracle."""
    say("partial reuse", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(71 + b + dh)
    J, c = 6, 4
    qe, ke, ve = (rows(g, (J * b, H, dh), dtype) for _ in range(3))
    q, ki, vi = (rows(g, (b, H, dh), dtype) for _ in range(3))
    dqe, dke, dve, dq, dki, dvi = (dev(x, dtype) for x in (qe, ke, ve, q, ki, vi))
    outs = []
    for cached in (0, c, J):
        st = smem.Store(1, 8, 8, b, H, dh, dtype)
        if cached:        # an earlier request left blocks 0..cached-1 in the store
            smem.smem_encode_blocks(st, dqe[:cached * b], dke[:cached * b], dve[:cached * b],
                                    seq_ids=[0] * cached, block_idx=list(range(cached)))
        if cached < J:    # this request encodes only its uncached blocks
            smem.smem_encode_blocks(st, dqe[cached * b:], dke[cached * b:], dve[cached * b:],
                                    seq_ids=[0] * (J - cached), block_idx=list(range(cached, J)))
        outs.append(smem.smem_reader_prefill_block(st, [0], [J], dq, dki, dvi))
        st.close()
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])
    ref = O.Store(1, 8, b, H, dh)
    O.encode_into_store(ref, [0] * J, list(range(J)), qe.reshape(J, b, H, dh), ke.reshape(J, b, H, dh),
                        ve.reshape(J, b, H, dh))
    expect = O.reader_prefill_block(ref, [0], [J], q[None], ki[None], vi[None])
    # the memory rows are themselves rounded outputs of the encoder
    check(outs[0], expect[0], dtype, f"partial reuse {dt}", roundings=2)


@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
def test_reencode_in_place(dt, b, H, dh):
    say("re-encode", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(81 + b + dh)
    x1 = [rows(g, (3 * b, H, dh), dtype) for _ in range(3)]
    x2 = [rows(g, (2 * b, H, dh), dtype) for _ in range(3)]
    d1 = [dev(x, dtype) for x in x1]
    d2 = [dev(x, dtype) for x in x2]
    st = smem.Store(1, 6, 6, b, H, dh, dtype)
    smem.smem_encode_blocks(st, *d1, seq_ids=[0, 0, 0], block_idx=[1, 2, 4])
    _, K0, _ = smem.smem_store_export(st, 0)
    smem.smem_reencode_blocks(st, *d1, seq_ids=[0, 0, 0], block_idx=[1, 2, 4])
    _, K1, _ = smem.smem_store_export(st, 0)
    assert torch.equal(K0, K1)                      # same inputs: identity
    used0 = st.stats()
    smem.smem_reencode_blocks(st, *d2, seq_ids=[0, 0], block_idx=[4, 1])
    assert st.stats() == used0                      # in place: no page taken or freed
    fresh = smem.Store(1, 6, 6, b, H, dh, dtype)
    smem.smem_encode_blocks(fresh, *(x[b:2 * b] for x in d1), seq_ids=[0], block_idx=[2])
    smem.smem_encode_blocks(fresh, *d2, seq_ids=[0, 0], block_idx=[4, 1])
    a, b_ = smem.smem_store_export(st, 0), smem.smem_store_export(fresh, 0)
    assert a[0] == b_[0] == [1, 2, 4]
    assert torch.equal(a[1], b_[1]) and torch.equal(a[2], b_[2])
    q = dev(rows(g, (b, H, dh), dtype), dtype)
    assert torch.equal(smem.smem_reader_prefill_block(st, [0], [5], q, q, q),
                       smem.smem_reader_prefill_block(fresh, [0], [5], q, q, q))
    ref = O.Store(1, 6, b, H, dh)
    O.encode_into_store(ref, [0, 0, 0], [1, 2, 4], *(x.reshape(3, b, H, dh) for x in x1))
    O.reencode_into_store(ref, [0, 0], [4, 1], *(x.reshape(2, b, H, dh) for x in x2))
    check(a[1], ref.export(0)[1], dtype, "re-encoded rows")
    for seqs, idx, code in (([0, 0], [1, 3], smem.SMEM_ENOENT), ([0, 0], [2, 2], smem.SMEM_EINVAL)):
        with pytest.raises(smem.SmemError) as e:
            smem.smem_reencode_blocks(st, *d2, seq_ids=seqs, block_idx=idx)
        assert e.value.code == code
        c = smem.smem_store_export(st, 0)
        assert c[0] == a[0] and torch.equal(c[1], a[1])


@pytest.mark.parametrize("dt,b,H,dh", [("bf16", 64, 2, 64), ("f32", 16, 2, 32)])
def test_slot_scheme_append_beyond_trained_blocks(dt, b, H, dh):
    """Grow a context past B = 4 blocks one append at a time.  A block's
    encoder input depends on its slot (inputs drawn per (block, slot), the
    stand-in for a slot position added to the tokens), so each append past B
    re-encodes the B-1 blocks whose slot moved.  The final store equals a
    fresh encode of every block at its final slot, bitwise."""
    say("slot scheme", dt, b, H, dh)
    dtype = DT[dt]
    B, n_final = 4, 7
    g = np.random.default_rng(91)
    draws = {}

    def inputs(j, slot):
        if (j, slot) not in draws:
            draws[(j, slot)] = [rows(g, (b, H, dh), dtype) for _ in range(3)]
        return draws[(j, slot)]

    st = smem.Store(1, 8, 8, b, H, dh, dtype)
    for n in range(1, n_final + 1):
        slots = O.slot_indices(n, B)
        moved = [j for j in range(n - 1) if slots[j] != O.slot_indices(n - 1, B)[j]] if n > 1 else []
        if moved:
            xs = [np.concatenate([inputs(j, slots[j])[r] for j in moved]) for r in range(3)]
            smem.smem_reencode_blocks(st, *(dev(x, dtype) for x in xs), seq_ids=[0] * len(moved),
                                      block_idx=moved)
        assert len(moved) == (B - 1 if n > B else 0)
        smem.smem_encode_blocks(st, *(dev(x, dtype) for x in inputs(n - 1, slots[n - 1])), seq_ids=[0],
                                block_idx=[n - 1])
    slots = O.slot_indices(n_final, B)
    xs = [np.concatenate([inputs(j, slots[j])[r] for j in range(n_final)]) for r in range(3)]
    fresh = smem.Store(1, 8, 8, b, H, dh, dtype)
    smem.smem_encode_blocks(fresh, *(dev(x, dtype) for x in xs), seq_ids=[0] * n_final,
                            block_idx=list(range(n_final)))
    a, c = smem.smem_store_export(st, 0), smem.smem_store_export(fresh, 0)
    assert a[0] == c[0] == list(range(n_final))
    assert torch.equal(a[1], c[1]) and torch.equal(a[2], c[2])
    ref = O.Store(1, 8, b, H, dh)
    O.encode_into_store(ref, [0] * n_final, list(range(n_final)), *(x.reshape(n_final, b, H, dh) for x in xs))
    check(a[1], ref.export(0)[1], dtype, "slot-scheme rows")
