"""GPU parity of the SMem+RoPE composite (Section 3, "SMem composes with
RoPE"; the composite's appendix; saturating block phases of the needle
appendix) against the fp64 oracle, through the C ABI: rotary encoder,
reader prefill and decode, with and without the null row, with saturating
(W = 15 or 3) and unclipped block phases.

Tolerance: max|y - y_ref| / rms(y_ref) <= 1e-5 (fp32) or 2e-2 (bf16), as for
the base path; GPU-vs-GPU identities are bitwise.
"""
import numpy as np
import pytest
import torch

from oracle import smem_oracle as O
from paper_2609_32395_amd import smem
from tests.gpu_util import DT, check, dev, host, require_gpu, rows, say

pytestmark = pytest.mark.gpu

SHAPES = [("f32", 16, 2, 32), ("bf16", 64, 2, 64), ("bf16", 64, 2, 128), ("bf16", 16, 3, 64),
          ("f32", 64, 2, 128), ("bf16", 64, 3, 32)]
BASE = 10000.0


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _store(g, dtype, b, H, dh, n_seq=2, max_blocks=24, live=0.75):
    st = smem.Store(n_seq, max_blocks, n_seq * max_blocks, b, H, dh, dtype)
    ref = O.Store(n_seq, max_blocks, b, H, dh)
    for s in range(n_seq):
        for j in range(max_blocks):
            if g.random() < live:
                K, V = rows(g, (b, H, dh), dtype), rows(g, (b, H, dh), dtype)
                smem.smem_store_put_block(st, s, j, dev(K, dtype), dev(V, dtype))
                ref.put(s, j, K, V)
    return st, ref


@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
@pytest.mark.parametrize("mask", [O.MASK_BIDIR, O.MASK_CAUSAL])
def test_rope_encoder(dt, b, H, dh, mask):
    say("rope encoder", dt, b, H, dh, mask)
    dtype = DT[dt]
    g = np.random.default_rng(100 + b + dh + mask)
    nb = 5
    q, k, v = (rows(g, (nb * b, H, dh), dtype) for _ in range(3))
    rope = smem.Rope(dh, b, BASE)
    st = smem.Store(1, 8, 8, b, H, dh, dtype)
    out = smem.smem_encode_blocks_rope(st, rope, dev(q, dtype), dev(k, dtype), dev(v, dtype),
                                       seq_ids=[0] * nb, block_idx=list(range(nb)), mask=mask)
    ref = O.encode_blocks_rope(*(x.reshape(nb, b, H, dh) for x in (q, k, v)), O.Rope(BASE), mask)
    check(out, ref.reshape(nb * b, H, dh), dtype, f"rope encoder {dt} b{b} dh{dh} mask{mask}")
    _, K, V = smem.smem_store_export(st, 0)
    assert torch.equal(K, out) and torch.equal(V, out)     # rows stored unturned, as computed
    alone = smem.smem_encode_blocks_rope(None, rope, dev(q[b:2 * b], dtype), dev(k[b:2 * b], dtype),
                                         dev(v[b:2 * b], dtype), mask=mask, b=b)
    assert torch.equal(alone, out[b:2 * b])


@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
@pytest.mark.parametrize("with_null", [False, True])
@pytest.mark.parametrize("max_offset", [0, 3, 15])
def test_rope_prefill(dt, b, H, dh, with_null, max_offset):
    say("rope prefill", dt, b, H, dh, with_null, max_offset)
    dtype = DT[dt]
    g = np.random.default_rng(200 + b + dh + with_null + max_offset)
    st, ref = _store(g, dtype, b, H, dh)
    seqs, J = [1, 0], [21, 9]
    q, ki, vi = (rows(g, (2 * b, H, dh), dtype) for _ in range(3))
    nkv = rows(g, (2, H, dh), dtype) if with_null else None
    rope = smem.Rope(dh, max(b, 22), BASE, max_offset)
    out = smem.smem_reader_prefill_block_rope(st, rope, seqs, J, dev(q, dtype), dev(ki, dtype), dev(vi, dtype),
                                              dev(nkv, dtype) if with_null else None)
    expect = O.reader_prefill_block_rope(ref, seqs, J, *(x.reshape(2, b, H, dh) for x in (q, ki, vi)), nkv,
                                         O.Rope(BASE, max_offset or None))
    check(out, expect.reshape(2 * b, H, dh), dtype, f"rope prefill {dt} b{b} dh{dh}")
    # batch invariance: each sequence alone gives the same bits
    for i in range(2):
        alone = smem.smem_reader_prefill_block_rope(
            st, rope, [seqs[i]], [J[i]], dev(q[i * b:(i + 1) * b], dtype), dev(ki[i * b:(i + 1) * b], dtype),
            dev(vi[i * b:(i + 1) * b], dtype), dev(nkv, dtype) if with_null else None)
        assert torch.equal(alone, out[i * b:(i + 1) * b])


@pytest.mark.parametrize("dt,b,H,dh", SHAPES)
@pytest.mark.parametrize("with_null", [False, True])
@pytest.mark.parametrize("max_offset", [0, 15])
def test_rope_decode(dt, b, H, dh, with_null, max_offset):
    say("rope decode", dt, b, H, dh, with_null, max_offset)
    dtype = DT[dt]
    g = np.random.default_rng(300 + b + dh + with_null + max_offset)
    st, ref = _store(g, dtype, b, H, dh, n_seq=3)
    seqs, J = [2, 0, 1], [23, 17, 1]
    pos = [b - 1, 0, b // 2]
    q, kn, vn = (rows(g, (3, H, dh), dtype) for _ in range(3))
    kc, vc = rows(g, (3 * b, H, dh), dtype), rows(g, (3 * b, H, dh), dtype)
    nkv = rows(g, (2, H, dh), dtype) if with_null else None
    rope = smem.Rope(dh, max(b, 24), BASE, max_offset)
    dkc, dvc = dev(kc, dtype), dev(vc, dtype)
    out = smem.smem_reader_decode_rope(st, rope, seqs, J, pos, dev(q, dtype), dev(kn, dtype), dev(vn, dtype),
                                       dkc, dvc, dev(nkv, dtype) if with_null else None)
    expect, ekc, evc = O.reader_decode_rope(ref, seqs, J, pos, q, kn, vn, kc.reshape(3, b, H, dh),
                                            vc.reshape(3, b, H, dh), nkv, O.Rope(BASE, max_offset or None))
    check(out, expect, dtype, f"rope decode {dt} b{b} dh{dh}")
    assert np.array_equal(host(dkc), ekc.reshape(3 * b, H, dh)) and np.array_equal(host(dvc), evc.reshape(3 * b, H, dh))


@pytest.mark.parametrize("dt,b,H,dh", [("bf16", 64, 2, 64), ("f32", 16, 2, 32)])
def test_rope_delete_equals_never_inserted_and_shift(dt, b, H, dh):
    """Theorem 1 under rotary phases (bitwise), and the composite's relative
    phases: with unclipped block phases, moving every block and the query
    block up by the same amount reads the same, bitwise (the oracle pins the
    same fact in exact arithmetic)."""
    say("rope delete/shift", dt, b, H, dh)
    dtype = DT[dt]
    g = np.random.default_rng(400 + b)
    blocks = {j: (rows(g, (b, H, dh), dtype), rows(g, (b, H, dh), dtype)) for j in (0, 2, 3, 5, 6)}
    q, ki, vi = (dev(rows(g, (b, H, dh), dtype), dtype) for _ in range(3))
    rope = smem.Rope(dh, max(b, 40), BASE, 0)

    def build(skip=(), shift=0, extra=None):
        st = smem.Store(1, 40, 8, b, H, dh, dtype)
        if extra is not None:
            smem.smem_store_put_block(st, 0, extra, *(dev(x, dtype) for x in blocks[3]))
        for j, (K, V) in blocks.items():
            if j not in skip:
                smem.smem_store_put_block(st, 0, j + shift, dev(K, dtype), dev(V, dtype))
        return st

    edited = build(skip=(3,), extra=3)
    smem.smem_delete_block(edited, 0, 3)
    never = build(skip=(3,))
    a = smem.smem_reader_prefill_block_rope(edited, rope, [0], [7], q, ki, vi)
    c = smem.smem_reader_prefill_block_rope(never, rope, [0], [7], q, ki, vi)
    assert torch.equal(a, c)
    base = smem.smem_reader_prefill_block_rope(build(), rope, [0], [7], q, ki, vi)
    shifted = smem.smem_reader_prefill_block_rope(build(shift=30), rope, [0], [37], q, ki, vi)
    assert torch.equal(shifted, base)      # the kernels turn by J - j, identical after the shift


def test_rope_errors():
    say("rope errors")
    g = np.random.default_rng(5)
    st, _ = _store(g, torch.bfloat16, 64, 2, 64, n_seq=1, max_blocks=70, live=0.2)
    q = dev(rows(g, (64, 2, 64), torch.bfloat16), torch.bfloat16)
    short = smem.Rope(64, 64, BASE, 0)             # phases 0..63, block phases unclipped
    smem.smem_reader_prefill_block_rope(st, short, [0], [63], q, q, q)
    with pytest.raises(smem.SmemError) as e:       # block turn 64 is not tabulated
        smem.smem_reader_prefill_block_rope(st, short, [0], [64], q, q, q)
    assert e.value.code == smem.SMEM_EINVAL
    clipped = smem.Rope(64, 64, BASE, 15)          # saturating: turns <= 15 at any length
    smem.smem_reader_prefill_block_rope(st, clipped, [0], [70], q, q, q)
    wrong_dh = smem.Rope(128, 64, BASE, 15)
    with pytest.raises(smem.SmemError) as e:
        smem.smem_reader_prefill_block_rope(st, wrong_dh, [0], [10], q, q, q)
    assert e.value.code == smem.SMEM_EINVAL
    too_few = smem.Rope(64, 20, BASE, 15)          # in-block phases 0..63 are needed
    with pytest.raises(smem.SmemError) as e:
        smem.smem_encode_blocks_rope(None, too_few, q, q, q, b=64)
    assert e.value.code == smem.SMEM_EINVAL
