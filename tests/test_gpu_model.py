"""GPU parity of the whole model at random weights (Section 2, "Model";
Appendix A) through the C ABI, against the fp64 model oracle.

* logits of a served block against the oracle (bf16 weights and activations,
  fp32 accumulation; tolerance below);
* block-skip serving equals the cold full pass on the served block, bitwise
  (Section 3.1: the reader state of a block depends only on its tokens and
  the cached memory; every kernel here is row- and batch-invariant);
* deleting a block equals never encoding it, bitwise (Theorem 1);
* error codes of the store operations.

Tolerance.  Every activation is rounded to bf16 once per producing step
(unit roundoff u = 2^-8, the same u the attention checks use; RMS relative
error u/sqrt 3 per rounding).  Along
the longest path a logit sees R roundings: the embedding, 7 per encoder
layer (LayerNorm, q|k|v, attention, residual, LayerNorm, FFN hidden,
residual), the memory LayerNorm and the key/value maps, 11 per reader layer
(the encoder's 7 plus the cross-attention's query, output and residual and a
third LayerNorm) and the final LayerNorm.  Independent roundings add as a
random walk, so the logits' relative RMS error is about sqrt(R) u / sqrt 3,
and the largest of n logits lies within sqrt(2 ln n) of that; the bound
allows twice this: max |y - y_ref| / rms(y_ref) <= tol(R, n).  The RMS
relative error itself must stay within twice its random-walk size,
rms(y - y_ref) / rms(y_ref) <= 2 sqrt(R) u / sqrt 3, which a systematic
error of a few percent in one op would exceed, and the predicted tokens
(argmax over the vocabulary) must agree with the oracle's for at least 90%
of the positions.
"""
import math

import numpy as np
import pytest
import torch

from oracle import smem_model as MO
from paper_2609_32395_amd import smem, synth
from tests.gpu_util import host, require_gpu, say

pytestmark = pytest.mark.gpu



def roundings(E, D):
    return 1 + 7 * E + 2 + 11 * D + 1


U_BF16 = 2.0 ** -8


def tol(E, D, n):
    return 2.0 * math.sqrt(2.0 * math.log(n)) * math.sqrt(roundings(E, D)) * U_BF16 / math.sqrt(3.0)


def tol_rms(E, D):
    return 2.0 * math.sqrt(roundings(E, D)) * U_BF16 / math.sqrt(3.0)


def model_check(y, expect, E, D, what, full=False, argmax=True):
    """Logits against the oracle: the max bound, the RMS bound and (for a
    vocabulary row) the argmax agreement; the numbers are recorded for the
    session summary."""
    from tests import gpu_util
    y = np.asarray(y, np.float64)
    expect = np.asarray(expect, np.float64)
    rms = float(np.sqrt(np.mean(expect ** 2)))
    err = float(np.max(np.abs(y - expect))) / rms
    err_rms = float(np.sqrt(np.mean((y - expect) ** 2))) / rms
    agree = float(np.mean(y.reshape(-1, y.shape[-1]).argmax(-1) == expect.reshape(-1, y.shape[-1]).argmax(-1)))
    t, tr = tol(E, D, y.size), tol_rms(E, D)
    gpu_util.RECORDS.append((f"{what} (max)", "bf16", err, err, t, full))
    gpu_util.RECORDS.append((f"{what} (rms)", "bf16", err_rms, err_rms, tr, full))
    say(f"check {what}: max {err:.3e} (limit {t:.3e}), rms {err_rms:.3e} (limit {tr:.3e}), argmax agreement {agree:.3f}")
    assert np.all(np.isfinite(y)), what
    assert err <= t, (what, err, t)
    assert err_rms <= tr, (what, err_rms, tr)
    if argmax:
        assert agree >= 0.9, (what, agree)
    return err
SHAPE = dict(E=1, D=2, d=128, H=4, b=64, vocab=256, n_pos=256)


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def build(seed=5, n_pages=16, max_blocks=12, max_tokens=256, row_plane=False, n_seq=1, **over):
    s = dict(SHAPE, **over)
    W = synth.model_weights(smem.model_weight_shapes(s["E"], s["D"], s["d"], s["vocab"], s["n_pos"]), seed)
    dW = {k: torch.from_numpy(v).to("cuda").to(torch.bfloat16).contiguous() for k, v in W.items()}
    m = smem.Model(dW, s["E"], s["D"], s["d"], s["H"], s["b"], s["vocab"], s["n_pos"], n_seq, max_blocks, n_pages,
                   max_tokens, row_plane=row_plane)
    ref = MO.Model(W, s["E"], s["D"], s["d"], s["H"], s["b"], s["vocab"], s["n_pos"], 1, max_blocks)
    return m, ref, dW


def tok(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32).reshape(-1)).to("cuda")


# (E, D, d, H, vocab, n_pos): heads of 32 (the paper's), 64 and 128; a ragged
# head tile (vocab 1000 = 15 * 64 + 40); no encoder layer; no position table
SHAPES = [dict(), dict(E=2, D=1, d=256, H=4, vocab=1000, n_pos=0), dict(E=0, D=2, d=128, H=1, vocab=77, n_pos=128)]


@pytest.mark.parametrize("over", SHAPES, ids=["d128h4", "d256h4-nopos", "d128h1-E0"])
def test_served_block_matches_oracle(over):
    say("model: served block vs oracle", over)
    m, ref, _ = build(**over)
    s = dict(SHAPE, **over)
    g = np.random.default_rng(11)
    B = 7                                    # 6 cached blocks, two launches of 4 + 2; block 6 is past the position table
    tokens = g.integers(0, s["vocab"], size=(B, s["b"]))
    smem.smem_model_encode(m, 0, list(range(B - 1)), tok(tokens[:B - 1]))
    logits = smem.smem_model_read(m, 0, [B - 1], tok(tokens[B - 1:]))
    ref.encode(0, tokens[:B - 1], list(range(B - 1)))
    expect = ref.read(0, tokens[B - 1:], [B - 1])[0]
    y = host(logits)
    model_check(y, expect, s["E"], s["D"], f"model served block {over}")
    # the first block reads the null row alone
    first = host(smem.smem_model_read(m, 0, [0], tok(tokens[:1])))
    e0 = ref.read(0, tokens[:1], [0])[0]
    model_check(first, e0, s["E"], s["D"], f"model first block (null row only) {over}")


def test_prefill_cold_and_partial_reuse_bitwise():
    """Cold prefill's final-block logits equal block-skip serving over the
    cached context and the cold pass's last rows; partial reuse (reader from
    the first uncached block) equals the cold prefill."""
    say("model: cold prefill / partial reuse")
    g = np.random.default_rng(14)
    B = 9                                    # three read launches of 4 + 4 + 1 blocks
    tokens = g.integers(0, SHAPE["vocab"], size=(B, SHAPE["b"]))
    m, _, _ = build()
    cold = smem.smem_model_prefill(m, 0, 0, B, tok(tokens))
    skip = smem.smem_model_read(m, 0, [B - 1], tok(tokens[B - 1:]))
    assert torch.equal(cold, skip)
    full = smem.smem_model_read(m, 0, list(range(B)), tok(tokens))
    assert torch.equal(cold, full[(B - 1) * SHAPE["b"]:])
    p, _, _ = build()
    smem.smem_model_encode(p, 0, [0, 1, 2], tok(tokens[:3]))
    part = smem.smem_model_prefill(p, 0, 3, B - 3, tok(tokens[3:]))
    assert torch.equal(part, cold)
    with pytest.raises(smem.SmemError) as e:            # blocks already cached: nothing changes
        smem.smem_model_prefill(p, 0, 2, 2, tok(tokens[2:4]))
    assert e.value.code == smem.SMEM_EEXIST
    assert torch.equal(smem.smem_model_read(p, 0, [B - 1], tok(tokens[B - 1:])), cold)


def test_block_skip_equals_cold_pass_bitwise():
    say("model: block-skip vs cold pass")
    g = np.random.default_rng(12)
    B = 6
    tokens = g.integers(0, SHAPE["vocab"], size=(B, SHAPE["b"]))
    cached, _, dW = build()
    smem.smem_model_encode(cached, 0, list(range(B - 1)), tok(tokens[:B - 1]))
    skip = smem.smem_model_read(cached, 0, [B - 1], tok(tokens[B - 1:]))
    cold, _, _ = build()
    smem.smem_model_encode(cold, 0, list(range(B)), tok(tokens))
    full = smem.smem_model_read(cold, 0, list(range(B)), tok(tokens))
    assert torch.equal(skip, full[(B - 1) * SHAPE["b"]:])


def test_delete_equals_never_encoded_bitwise_and_errors():
    say("model: delete vs never encoded")
    g = np.random.default_rng(13)
    B = 6
    tokens = g.integers(0, SHAPE["vocab"], size=(B, SHAPE["b"]))
    a, _, _ = build()
    smem.smem_model_encode(a, 0, list(range(B - 1)), tok(tokens[:B - 1]))
    smem.smem_model_delete_block(a, 0, 2)
    c, _, _ = build()
    keep = [0, 1, 3, 4]
    smem.smem_model_encode(c, 0, keep, tok(tokens[keep]))
    la = smem.smem_model_read(a, 0, [B - 1], tok(tokens[B - 1:]))
    lc = smem.smem_model_read(c, 0, [B - 1], tok(tokens[B - 1:]))
    assert torch.equal(la, lc)
    with pytest.raises(smem.SmemError) as e:
        smem.smem_model_encode(a, 0, [1], tok(tokens[1:2]))
    assert e.value.code == smem.SMEM_EEXIST
    with pytest.raises(smem.SmemError) as e:
        smem.smem_model_delete_block(a, 0, 2)
    assert e.value.code == smem.SMEM_ENOENT
    # re-encoding the deleted block restores the full read exactly
    smem.smem_model_encode(a, 0, [2], tok(tokens[2:3]))
    full, _, _ = build()
    smem.smem_model_encode(full, 0, list(range(B - 1)), tok(tokens[:B - 1]))
    assert torch.equal(smem.smem_model_read(a, 0, [B - 1], tok(tokens[B - 1:])),
                       smem.smem_model_read(full, 0, [B - 1], tok(tokens[B - 1:])))


def test_tilings_agree_bitwise():
    """Every linear map keeps one reduction order per output whatever the
    kernel: a one-block read (few-row kernel), a 4-block read (64 x 64
    tiles) and a 16-block read (the 50257-like wide head on 128 x 128 tiles)
    give the same logits bit for bit, and match the oracle."""
    say("model: tilings agree")
    over = dict(vocab=4096, n_pos=1024)
    m, ref, _ = build(max_blocks=20, n_pages=20, max_tokens=1024, **over)
    g = np.random.default_rng(15)
    B = 16
    tokens = g.integers(0, 4096, size=(B, SHAPE["b"]))
    smem.smem_model_encode(m, 0, list(range(B)), tok(tokens))
    full = smem.smem_model_read(m, 0, list(range(B)), tok(tokens))
    four = smem.smem_model_read(m, 0, [9, 10, 11, 12], tok(tokens[9:13]))
    assert torch.equal(four, full[9 * 64:13 * 64])
    for j in (0, 5, 15):
        one = smem.smem_model_read(m, 0, [j], tok(tokens[j:j + 1]))
        assert torch.equal(one, full[j * 64:(j + 1) * 64]), j
    ref.encode(0, tokens[:15], list(range(15)))
    expect = ref.read(0, tokens[15:], [15])[0]
    y = host(full[15 * 64:])
    model_check(y, expect, SHAPE["E"], SHAPE["D"], "model block 15 of a 16-block tiled read")


@pytest.mark.parametrize("d,H", [(2048, 16), (832, 26)], ids=["d2048", "d832"])
def test_fused_layernorm_widths_bitwise(d, H):
    """Block-skip serving normalizes its 64 rows inside the few-row maps (at
    d = 2048 the q|k|v and FFN-up maps take the 4-column-group tile with its
    W refill; at d = 832 the last 256-chunk of every row is 2 steps); the
    cold pass over 4 blocks runs the stand-alone LayerNorm and the tiled
    GEMM.  The final block's logits agree bit for bit and match the oracle."""
    say("model: fused LayerNorm widths", d, H)
    over = dict(E=1, D=1, d=d, H=H, vocab=300, n_pos=0)
    m, ref, _ = build(max_blocks=4, n_pages=8, max_tokens=256, **over)
    g = np.random.default_rng(16)
    B = 4
    tokens = g.integers(0, 300, size=(B, SHAPE["b"]))
    cold = smem.smem_model_prefill(m, 0, 0, B, tok(tokens))
    skip = smem.smem_model_read(m, 0, [B - 1], tok(tokens[B - 1:]))
    assert torch.equal(cold, skip)
    ref.encode(0, tokens[:B - 1], list(range(B - 1)))
    expect = ref.read(0, tokens[B - 1:], [B - 1])[0]
    y = host(skip)
    model_check(y, expect, 1, 1, f"model fused LayerNorm d={d}")


def test_160m_full_size_block_skip_matches_oracle():
    """At the bench's 160M shape (d 768, E 3, D 7, 24 heads of 32, vocabulary
    50257, 1024 positions) and its 1k context, in the bench's launch
    configuration: the block-skip logits of the final block against the fp64
    model oracle, and bitwise against the cold prefill."""
    say("model: 160M full size vs oracle")
    name, d, E, D = synth.MODEL_SCALES[0]
    H, b, vocab, T, n = d // 32, 64, synth.MODEL_VOCAB, synth.MODEL_T, 1024
    J = n // b
    W = synth.model_weights_device(smem.model_weight_shapes(E, D, d, vocab, T), 3)
    m = smem.Model(W, E, D, d, H, b, vocab, T, 1, J, J, max_tokens=J * b)
    tokens = synth.model_tokens(3, name, n).reshape(J, b)
    cold = smem.smem_model_prefill(m, 0, 0, J, tok(tokens))
    skip = smem.smem_model_read(m, 0, [J - 1], tok(tokens[J - 1:]))
    assert torch.equal(cold, skip)
    ref = MO.Model({k: v.float().cpu().numpy().astype(np.float64) for k, v in W.items()}, E, D, d, H, b, vocab, T, 1, J)
    ref.encode(0, tokens[:J - 1], list(range(J - 1)))
    expect = ref.read(0, tokens[J - 1:], [J - 1])[0]
    y = host(skip)
    model_check(y, expect, E, D, "160M model block-skip read at 1024 tokens", full=True)


def test_model_edge_cases():
    """Empty calls are no-ops; a read at query block = max_blocks reads every
    cached block; token ids outside the vocabulary read embedding row 0 (the
    oracle is given token 0 there); argument errors change nothing."""
    say("model: edge cases")
    m, ref, _ = build(max_blocks=6, n_pages=6)
    g = np.random.default_rng(16)
    tokens = g.integers(0, SHAPE["vocab"], size=(6, SHAPE["b"]))
    empty = torch.empty(0, dtype=torch.int32, device="cuda")
    smem.smem_model_encode(m, 0, [], empty)
    assert smem.smem_model_read(m, 0, [], empty).shape == (0, SHAPE["vocab"])
    smem.smem_model_encode(m, 0, list(range(6)), tok(tokens))
    ref.encode(0, tokens, list(range(6)))
    q = tokens[:1].copy()
    q[0, 3], q[0, 9] = -5, SHAPE["vocab"] + 7              # out of range -> row 0
    y = host(smem.smem_model_read(m, 0, [6], tok(q)))      # query block = max_blocks: all 6 blocks below
    q_ref = q.copy()
    q_ref[0, 3] = q_ref[0, 9] = 0
    expect = ref.read(0, q_ref, [6])[0]
    model_check(y, expect, SHAPE["E"], SHAPE["D"], "model read over every cached block")
    with pytest.raises(smem.SmemError) as e:
        smem.smem_model_read(m, 0, [7], tok(q))            # beyond max_blocks
    assert e.value.code == smem.SMEM_EINVAL
    with pytest.raises(smem.SmemError) as e:
        smem.smem_model_encode(m, 1, [0], tok(q))          # no sequence 1
    assert e.value.code == smem.SMEM_EINVAL
    with pytest.raises(smem.SmemError) as e:
        smem.smem_model_prefill(m, 0, 4, 3, tok(tokens[:3]))   # blocks 4..6: past max_blocks
    assert e.value.code == smem.SMEM_EINVAL
    # the store is unchanged by the failed calls
    assert torch.equal(smem.smem_model_read(m, 0, [6], tok(q)), torch.from_numpy(y).to("cuda"))


def test_decode_matches_reader_and_oracle_across_a_boundary():
    """KV-cached decode (Section 3.1, "Decode"): decoding block J's tokens in
    order gives, at position p, the reader pass's row p of the block (the
    oracle's, within the rounding tolerance; the GPU block read's too); the
    completed block is appended and decoding continues into block J + 1."""
    say("model: decode across a boundary")
    m, ref, _ = build(max_blocks=10, n_pages=10)
    g = np.random.default_rng(17)
    J = 5
    tokens = g.integers(0, SHAPE["vocab"], size=(J + 2, SHAPE["b"]))
    smem.smem_model_encode(m, 0, list(range(J)), tok(tokens[:J]))
    ref.encode(0, tokens[:J], list(range(J)))
    block = smem.smem_model_read(m, 0, [J], tok(tokens[J:J + 1]))
    expect = ref.read(0, tokens[J:J + 1], [J])[0]
    rows = []
    for p in range(SHAPE["b"]):
        rows.append(smem.smem_model_decode(m, 0, [J], [p], tok(tokens[J, p:p + 1])))
    y = host(torch.cat(rows))
    t = tol(SHAPE["E"], SHAPE["D"], y.size)
    model_check(y, expect, SHAPE["E"], SHAPE["D"], "model decode, 64 tokens of a block")
    assert float(np.max(np.abs(y - host(block))) / np.sqrt(np.mean(expect ** 2))) <= t
    # append the completed block, continue into block J + 1
    smem.smem_model_encode(m, 0, [J], tok(tokens[J:J + 1]))
    ref.encode(0, tokens[J:J + 1], [J])
    nxt = [host(smem.smem_model_decode(m, 0, [J + 1], [p], tok(tokens[J + 1, p:p + 1])))[0] for p in range(4)]
    e2 = ref.read(0, tokens[J + 1:J + 2], [J + 1])[0][:4]
    assert float(np.max(np.abs(np.stack(nxt) - e2)) / np.sqrt(np.mean(e2 ** 2))) <= t


def test_decode_batch_invariant_bitwise():
    """Three sequences at different blocks and positions decoded in one call
    give, bit for bit, what each gives decoded alone."""
    say("model: decode batch invariance")
    s = dict(SHAPE)
    W = synth.model_weights(smem.model_weight_shapes(s["E"], s["D"], s["d"], s["vocab"], s["n_pos"]), 5)
    dW = {k: torch.from_numpy(v).to("cuda").to(torch.bfloat16).contiguous() for k, v in W.items()}
    m = smem.Model(dW, s["E"], s["D"], s["d"], s["H"], s["b"], s["vocab"], s["n_pos"], 3, 8, 24, 256)
    g = np.random.default_rng(18)
    J, P = [2, 5, 0], [3, 7, 5]
    for q in range(3):
        if J[q]:
            smem.smem_model_encode(m, q, list(range(J[q])), tok(g.integers(0, s["vocab"], size=(J[q], s["b"]))))
    toks = g.integers(0, s["vocab"], size=(3, max(P) + 1))
    for p in range(max(P)):                      # fill each sequence's in-block cache up to its position
        for q in range(3):
            if p < P[q]:
                smem.smem_model_decode(m, q, [J[q]], [p], tok(toks[q, p:p + 1]))
    batch = smem.smem_model_decode(m, 0, J, P, tok(toks[np.arange(3), P]))
    for q in range(3):
        alone = smem.smem_model_decode(m, q, [J[q]], [P[q]], tok(toks[q, P[q]:P[q] + 1]))
        assert torch.equal(alone[0], batch[q]), q


# Row plane (Appendix K, the decode arm that derives each layer's keys and
# values from the memory rows; Appendix A, "Positions and memory"): the model
# keeps the rows once, and every reader layer's cross-attention reads them
# through its own key and value maps.  Rows of 512 (the narrowest the row
# reader takes), 16 heads of 32.
ROWS_SHAPE = dict(d=512, H=16)


def test_row_plane_decode_matches_oracle_across_a_boundary():
    """Decoding block J's 64 tokens on the row plane gives the oracle's
    reader pass over the block (the key/value model's decode too, up to
    rounding); the completed block is appended and decoding continues."""
    say("model: row-plane decode across a boundary")
    m, ref, _ = build(max_blocks=10, n_pages=10, row_plane=True, **ROWS_SHAPE)
    kv, _, _ = build(max_blocks=10, n_pages=10, **ROWS_SHAPE)
    g = np.random.default_rng(27)
    J = 5
    tokens = g.integers(0, SHAPE["vocab"], size=(J + 2, SHAPE["b"]))
    for model in (m, kv):
        smem.smem_model_encode(model, 0, list(range(J)), tok(tokens[:J]))
    ref.encode(0, tokens[:J], list(range(J)))
    expect = ref.read(0, tokens[J:J + 1], [J])[0]
    rows, kv_rows = [], []
    for p in range(SHAPE["b"]):
        rows.append(smem.smem_model_decode(m, 0, [J], [p], tok(tokens[J, p:p + 1])))
        kv_rows.append(smem.smem_model_decode(kv, 0, [J], [p], tok(tokens[J, p:p + 1])))
    y, ykv = host(torch.cat(rows)), host(torch.cat(kv_rows))
    model_check(y, expect, SHAPE["E"], SHAPE["D"], "model row-plane decode, 64 tokens of a block")
    t = tol(SHAPE["E"], SHAPE["D"], y.size)
    assert float(np.max(np.abs(y - ykv)) / np.sqrt(np.mean(expect ** 2))) <= t
    smem.smem_model_encode(m, 0, [J], tok(tokens[J:J + 1]))
    ref.encode(0, tokens[J:J + 1], [J])
    nxt = [host(smem.smem_model_decode(m, 0, [J + 1], [p], tok(tokens[J + 1, p:p + 1])))[0] for p in range(4)]
    e2 = ref.read(0, tokens[J + 1:J + 2], [J + 1])[0][:4]
    model_check(np.stack(nxt), e2, SHAPE["E"], SHAPE["D"], "model row-plane decode, next block", argmax=False)


def test_row_plane_decode_batch_invariant_and_delete_bitwise():
    """Three sequences decoded in one call equal each decoded alone, bit for
    bit; deleting a block equals never encoding it; block reads are refused."""
    say("model: row-plane batch invariance, deletion")
    m, _, _ = build(max_blocks=8, n_pages=24, row_plane=True, n_seq=3, **ROWS_SHAPE)
    c, _, _ = build(max_blocks=8, n_pages=24, row_plane=True, n_seq=3, **ROWS_SHAPE)
    g = np.random.default_rng(28)
    J, P = [2, 5, 0], [3, 7, 5]
    blocks = {q: g.integers(0, SHAPE["vocab"], size=(max(J[q], 1), SHAPE["b"])) for q in range(3)}
    for q in range(3):
        if J[q]:
            smem.smem_model_encode(m, q, list(range(J[q])), tok(blocks[q][:J[q]]))
            keep = [j for j in range(J[q]) if not (q == 1 and j == 2)]
            smem.smem_model_encode(c, q, keep, tok(blocks[q][keep]))
    smem.smem_model_delete_block(m, 1, 2)
    toks = g.integers(0, SHAPE["vocab"], size=(3, max(P) + 1))
    for p in range(max(P)):
        for q in range(3):
            if p < P[q]:
                a = smem.smem_model_decode(m, q, [J[q]], [p], tok(toks[q, p:p + 1]))
                b = smem.smem_model_decode(c, q, [J[q]], [p], tok(toks[q, p:p + 1]))
                assert torch.equal(a, b), (q, p)
    batch = smem.smem_model_decode(m, 0, J, P, tok(toks[np.arange(3), P]))
    for q in range(3):
        alone = smem.smem_model_decode(c, q, [J[q]], [P[q]], tok(toks[q, P[q]:P[q] + 1]))
        assert torch.equal(alone[0], batch[q]), q
    with pytest.raises(smem.SmemError) as e:
        smem.smem_model_read(m, 0, [2], tok(blocks[0][:1]))
    assert e.value.code == smem.SMEM_EINVAL
    with pytest.raises(smem.SmemError) as e:
        smem.smem_model_prefill(m, 2, 0, 1, tok(blocks[2][:1]))
    assert e.value.code == smem.SMEM_EINVAL
