"""Op-level parity of the model's kernels through the C ABI (smem_linear):
the few-row linear map (k_linear_skinny), the same with the LayerNorm fused
(k_linear_skinny_ln), the stand-alone LayerNorm (k_ln_rows, whose output the
call returns in ln_tmp for more than 128 rows), the tiled GEMM (k_gemm) and
the GELU / residual / fp32 epilogues, against the model oracle's fp64
layer_norm, gelu and linear on the same bf16 input bytes.

Bounds (per output element), from the arithmetic: the inputs are exact bf16
values and the accumulation is fp32, so y differs from the fp64 value by at
most the output's own rounding, u |y_ref| (u = 2^-8, bf16), plus the fp32
accumulation error, at most K 2^-24 sum_k |a_k w_k|; with a LayerNorm the
normalised row a is rounded to bf16 before the product (one more rounding,
u sum_k |a_k w_k|, plus 1e-5 of it for the fp32 statistics); GELU's erf
(Abramowitz-Stegun 7.1.26, |error| <= 1.5e-7) adds 1e-6 |acc| and scales the
accumulation error by at most 1.13.  These worst-case bounds are checked for
every element; the RMS error must also stay within twice what independent
roundings give (u / sqrt 3 of rms(y_ref), plus u / sqrt 3 of the rms of
sqrt(sum_k (a_k w_k)^2) per LayerNorm rounding, plus the fp32 accumulation's
2^-24 / sqrt 3 * sqrt(K / 2) of that rms), which a systematic error of a
percent in one op would exceed.  Shapes: the 1.5B model's maps (d 2048,
4d 8192, vocabulary 50257) at 64 rows (few-row kernels) and at 520 or 136
rows (LayerNorm pass + GEMM, ragged row tiles), the head at d 1024 and 768
with at most 64 rows (the form that keeps the rows in LDS), and a ragged
width (d 832, N 1000).  The self-attention sub-layer's fused kernel (LayerNorm, q|k|v map
and block-local attention in one launch) is held to the bits of the unfused
pair, whose pieces are checked here and against the fp64 attention."""
import math

import numpy as np
import pytest
import torch

from oracle import smem_model as MO
from oracle import smem_oracle as O
from paper_2609_32395_amd import smem, synth
from tests import gpu_util
from tests.gpu_util import require_gpu, say

pytestmark = pytest.mark.gpu
U = 2.0 ** -8


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _bf(g, shape, scale=1.0):
    return synth.bf16_round((g.standard_normal(shape) * scale).astype(np.float32))


def _d(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(torch.bfloat16)


CASES = [  # name, M, N, K, layernorm, epilogue
    ("1.5B q|k|v map, 64 rows", 64, 6144, 2048, True, smem.LIN_STORE),
    ("1.5B q|k|v map, 520 rows", 520, 6144, 2048, True, smem.LIN_STORE),
    ("1.5B FFN up + GELU, 64 rows", 64, 8192, 2048, True, smem.LIN_GELU),
    ("1.5B FFN up + GELU, 520 rows", 520, 8192, 2048, True, smem.LIN_GELU),
    ("1.5B FFN down + residual, 64 rows", 64, 2048, 8192, False, smem.LIN_RESID),
    ("1.5B FFN down + residual, 520 rows", 520, 2048, 8192, False, smem.LIN_RESID),
    ("1.5B attention out + residual, 64 rows", 64, 2048, 2048, False, smem.LIN_RESID),
    ("1.5B head (fp32), 1 row", 1, 50257, 2048, True, smem.LIN_F32),
    ("1.5B head (fp32), 64 rows", 64, 50257, 2048, True, smem.LIN_F32),
    ("1.5B head (fp32), 136 rows", 136, 50257, 2048, True, smem.LIN_F32),
    ("410M head (fp32, rows in LDS), 64 rows", 64, 50257, 1024, False, smem.LIN_F32),
    ("410M head (fp32, rows in LDS), 1 row", 1, 50257, 1024, False, smem.LIN_F32),
    ("160M head (fp32, rows in LDS), 16 rows", 16, 50257, 768, False, smem.LIN_F32),
    ("160M head (fp32, rows in LDS), 40 rows", 40, 50257, 768, False, smem.LIN_F32),
    ("1.5B head (fp32, rows in LDS), 16 rows", 16, 50257, 2048, False, smem.LIN_F32),
    ("1.5B head (fp32, rows in LDS), 32 rows", 32, 50257, 2048, False, smem.LIN_F32),
    ("ragged d 832 x N 1000, 200 rows", 200, 1000, 832, True, smem.LIN_STORE),
    ("ragged d 832 x N 1000, 16 rows", 16, 1000, 832, False, smem.LIN_GELU),
]


@pytest.mark.parametrize("name,M,N,K,ln,epi", CASES, ids=[c[0] for c in CASES])
def test_linear_map_against_fp64(name, M, N, K, ln, epi):
    say("op parity", name)
    g = np.random.default_rng(M * 7 + N + K)
    x = _bf(g, (M, K))
    w = _bf(g, (N, K), 1.0 / math.sqrt(K))
    lg = synth.bf16_round((1.0 + 0.1 * g.standard_normal(K)).astype(np.float32)) if ln else None
    lb = synth.bf16_round((0.1 * g.standard_normal(K)).astype(np.float32)) if ln else None
    res = _bf(g, (M, N)) if epi == smem.LIN_RESID else None
    tmp = torch.empty((M, K), dtype=torch.bfloat16, device="cuda") if ln and M > 128 else None
    y = smem.smem_linear(_d(x), _d(w), None if lg is None else _d(lg), None if lb is None else _d(lb), epi,
                         None if res is None else _d(res), ln_tmp=tmp)
    torch.cuda.synchronize()
    y = y.float().cpu().numpy().astype(np.float64)
    a = MO.layer_norm(x.astype(np.float64), lg, lb) if ln else x.astype(np.float64)
    acc = MO.linear(a, w.astype(np.float64))
    ref = acc
    if epi == smem.LIN_GELU:
        ref = MO.gelu(acc)
    elif epi == smem.LIN_RESID:
        ref = acc + res
    absum = np.abs(a) @ np.abs(w.astype(np.float64)).T           # sum_k |a_k w_k|
    sq = np.sqrt((a * a) @ (w.astype(np.float64) ** 2).T)        # sqrt(sum_k (a_k w_k)^2)
    u_out = 0.0 if epi == smem.LIN_F32 else U
    acc_err = K * 2.0 ** -24 * absum
    bound = u_out * np.abs(ref) + acc_err * (1.13 if epi == smem.LIN_GELU else 1.0)
    if ln:
        bound = bound + (U + 1e-5) * absum * (1.13 if epi == smem.LIN_GELU else 1.0)
    if epi == smem.LIN_GELU:
        bound = bound + 1e-6 * np.abs(acc)
    excess = np.abs(y - ref) - bound
    rms_ref = float(np.sqrt(np.mean(ref * ref)))
    err_rms = float(np.sqrt(np.mean((y - ref) ** 2)))
    # fp32 accumulation: K sums whose partial sums grow like sqrt(k) carry
    # independent roundings of at most 2^-24 relative, about
    # 2^-24 / sqrt(3) * sqrt(K / 2) * sqrt(sum_k (a_k w_k)^2) in RMS (the
    # only term left for an fp32 output of un-normalized rows)
    rms_sq = float(np.sqrt(np.mean(sq * sq)))
    rms_limit = 2.0 * (u_out / math.sqrt(3.0) * rms_ref
                       + (U / math.sqrt(3.0) * rms_sq if ln else 0.0)
                       + 2.0 ** -24 / math.sqrt(3.0) * math.sqrt(K / 2.0) * rms_sq) + 1e-9 * rms_ref
    raw = float(np.max(np.abs(y - ref))) / rms_ref
    gpu_util.RECORDS.append((f"op {name} (rms error / its limit)", "op", raw, err_rms / rms_limit, 1.0, True))
    say(f"op {name}: raw max|y-ref|/rms {raw:.3e}, rms err {err_rms / rms_ref:.3e} (limit {rms_limit / rms_ref:.3e}), "
        f"worst element {float(np.max(np.abs(y - ref) / np.maximum(bound, 1e-30))):.3f} of its bound")
    assert np.all(np.isfinite(y))
    assert np.all(excess <= 0), f"{name}: {int(np.sum(excess > 0))} elements beyond their bound"
    assert err_rms <= rms_limit, (name, err_rms, rms_limit)
    if tmp is not None:                                          # the stand-alone LayerNorm's rows
        ln_rows = tmp.float().cpu().numpy().astype(np.float64)
        assert np.all(np.abs(ln_rows - a) <= U * np.abs(a) + 1e-5 * (1.0 + np.abs(a)))


def test_linear_rows_independent_bitwise():
    """A row's output does not depend on the other rows of the call: the same
    rows at 64 (few-row kernel) and inside 520 (GEMM) give the same bits."""
    say("op parity: row independence")
    g = np.random.default_rng(3)
    K, N = 2048, 6144
    x = _bf(g, (520, K))
    w = _d(_bf(g, (N, K), 1.0 / math.sqrt(K)))
    lg = _d(synth.bf16_round((1.0 + 0.1 * g.standard_normal(K)).astype(np.float32)))
    lb = _d(synth.bf16_round((0.1 * g.standard_normal(K)).astype(np.float32)))
    big = smem.smem_linear(_d(x), w, lg, lb, smem.LIN_GELU)
    small = smem.smem_linear(_d(x[100:164]), w, lg, lb, smem.LIN_GELU)
    assert torch.equal(big[100:164], small)


def test_wide_head_rows_independent_bitwise():
    """The fp32 head's few-row form (x rows kept in LDS, one workgroup per CU
    streaming the weights) gives the bits of the tiled GEMM for the same rows:
    rows 100..163 of a 200-row call, and single rows, at d 1024 and 768;
    rows 100..131 and a single row at d 2048."""
    say("op parity: wide head row independence")
    g = np.random.default_rng(5)
    for K, rows in ((1024, 64), (768, 64), (2048, 32)):
        N = 50257
        x = _bf(g, (200, K))
        w = _d(_bf(g, (N, K), 1.0 / math.sqrt(K)))
        big = smem.smem_linear(_d(x), w, epi=smem.LIN_F32)
        small = smem.smem_linear(_d(x[100:100 + rows]), w, epi=smem.LIN_F32)
        one = smem.smem_linear(_d(x[131:132]), w, epi=smem.LIN_F32)
        torch.cuda.synchronize()
        assert torch.equal(big[100:100 + rows], small), K
        assert torch.equal(big[131:132], one), K


def test_linear_argument_errors():
    """Shapes the kernels do not take are rejected before anything runs."""
    z = lambda *shape: torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    for x, w in [(z(4, 100), z(8, 100)),        # K not a multiple of 64
                 (z(4, 64), z(6, 64))]:         # bf16 output with N % 4 != 0
        with pytest.raises(smem.SmemError) as e:
            smem.smem_linear(x, w)
        assert e.value.code == smem.SMEM_EINVAL


SA_CASES = [  # name, d, H, n_blocks, mask
    ("d 256 x 8 heads, 1 block, causal", 256, 8, 1, 1),
    ("d 256 x 8 heads, 3 blocks, bidirectional", 256, 8, 3, 0),
    ("160M d 768 x 24 heads, 1 block, causal", 768, 24, 1, 1),
    ("160M d 768 x 24 heads, 5 blocks, bidirectional", 768, 24, 5, 0),
    ("410M d 1024 x 32 heads, 1 block, causal", 1024, 32, 1, 1),
    ("410M d 1024 x 32 heads, 2 blocks, causal", 1024, 32, 2, 1),
    ("410M d 1024 x 32 heads, 3 blocks, bidirectional", 1024, 32, 3, 0),
    ("d 512 x 16 heads, 130 blocks, causal", 512, 16, 130, 1),
]


@pytest.mark.parametrize("name,d,H,nb,mask", SA_CASES, ids=[c[0] for c in SA_CASES])
def test_self_attention_fused_equals_unfused(name, d, H, nb, mask):
    """The fused q|k|v + block-local attention kernel gives the bits of the
    unfused pair (the map into q, k, v, then the attention launch), with the
    LayerNorm in the kernel (up to 128 rows) or from the LayerNorm pass (more
    rows); the unfused pair's q | k | v equal the validated map's output, and
    its attention is checked against the fp64 oracle on those q, k, v."""
    say("op parity: self-attention", name)
    g = np.random.default_rng(d * 31 + nb * 7 + mask)
    M = nb * 64
    x = _bf(g, (M, d), 1.5) + synth.bf16_round(np.full((1, d), 0.25, np.float32))
    x = synth.bf16_round(x.astype(np.float32))
    w = _bf(g, (3 * d, d), 1.0 / math.sqrt(d))
    lg = synth.bf16_round((1.0 + 0.1 * g.standard_normal(d)).astype(np.float32))
    lb = synth.bf16_round((0.1 * g.standard_normal(d)).astype(np.float32))
    xd, wd, gd, bd = _d(x), _d(w), _d(lg), _d(lb)
    work = torch.zeros((4, M, d), dtype=torch.bfloat16, device="cuda")
    ref_out = smem.smem_self_attention(xd, gd, bd, wd, H, mask, path=smem.SA_UNFUSED, work=work)
    fused = smem.smem_self_attention(xd, gd, bd, wd, H, mask, path=smem.SA_FUSED,
                                     work=torch.empty((4, M, d), dtype=torch.bfloat16, device="cuda"))
    auto = smem.smem_self_attention(xd, gd, bd, wd, H, mask)
    torch.cuda.synchronize()
    assert torch.equal(fused, ref_out), f"{name}: fused != unfused"
    assert torch.equal(auto, ref_out), f"{name}: model's choice != unfused"
    qkv = smem.smem_linear(xd, wd, gd, bd, smem.LIN_STORE,
                           ln_tmp=torch.empty((M, d), dtype=torch.bfloat16, device="cuda") if M > 128 else None)
    torch.cuda.synchronize()
    for i in range(3):
        assert torch.equal(work[1 + i], qkv[:, i * d:(i + 1) * d]), f"{name}: q|k|v plane {i}"
    q, k, v = (work[1 + i].float().cpu().numpy().astype(np.float64).reshape(nb, 64, H, d // H) for i in range(3))
    expect = O.encode_blocks(q, k, v, mask).reshape(M, d)
    gpu_util.check(fused, expect, torch.bfloat16, f"op self-attention {name}", full=d >= 768)


def test_self_attention_argument_errors():
    """The fused path rejects heads other than 32 wide and widths above 1024."""
    z = lambda *shape: torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    for d, H in [(512, 8), (2048, 64)]:
        with pytest.raises(smem.SmemError) as e:
            smem.smem_self_attention(z(64, d), z(d), z(d), z(3 * d, d), H, 1, path=smem.SA_FUSED)
        assert e.value.code == smem.SMEM_EINVAL
