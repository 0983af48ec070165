"""Helpers of the GPU parity tests: device transfer of seeded inputs and the
tolerance rule (max |y - y_ref| / rms(y_ref) over one call's output; fp32
<= 1e-5, bf16 inputs with fp32 accumulation <= 2e-2, bf16 output rounding
included)."""
import os
import sys

import numpy as np
import pytest
import torch

from oracle import smem_oracle as O

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}
DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_32395_amd import smem
    smem.lib()  # raises when the library is missing: GPU tests never run without it


def say(*a):
    """Name the case before each GPU step (flushed) so a fault can be placed."""
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def dev(x, dtype):
    """numpy float32 (bf16-representable when dtype is bf16) -> device tensor; exact."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(dtype).contiguous()


def host(t):
    return t.detach().float().cpu().numpy()


# Unit roundoff of the output store: storing an fp32 result as bf16 moves it
# by at most half an ulp, 2^-8 |y| (2^-24 |y| for fp32).
UNIT_ROUNDOFF = {torch.float32: 2.0 ** -24, torch.bfloat16: 2.0 ** -8}


# Every check's numbers, printed at the end of the session (tests/conftest.py):
# (what, dtype name, raw max|y - ref| / rms(ref), error beyond output rounding,
# tolerance, full-size workload or not).
RECORDS = []


def check(y, ref, dtype, what="", roundings=1, full=False):
    """Elementwise |y - ref| <= TOL * rms(ref) + u |ref|: the tolerance bounds the
    fp32-accumulated result; u |ref| is the exact bound of the final store in
    the output dtype (its own rounding, counted once; twice when ``ref`` is
    itself a rounded output).  The raw max|y - ref| / rms(ref) (output
    rounding included) is recorded beside it and printed with the case."""
    y = host(y) if isinstance(y, torch.Tensor) else np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    excess = np.abs(y - ref) - roundings * UNIT_ROUNDOFF[dtype] * np.abs(ref)
    e = float(np.max(excess)) / rms if ref.size and rms > 0 else float(np.max(np.abs(y - ref), initial=0.0))
    raw = O.rel_err(y, ref)
    name = "bf16" if dtype == torch.bfloat16 else "fp32"
    RECORDS.append((what, name, raw, e, TOL[dtype], full))
    say(f"check {what}: raw max|y-ref|/rms {raw:.3e}, beyond output rounding {e:.3e} (limit {TOL[dtype]:.0e})")
    assert np.all(np.isfinite(y)), f"{what}: non-finite output"
    assert e <= TOL[dtype], f"{what}: error beyond output rounding {e:.3e} > {TOL[dtype]:.1e} (raw {raw:.3e})"
    return e


def rows(g, shape, dtype, scale=1.0):
    x = (g.standard_normal(shape) * scale).astype(np.float32)
    if dtype == torch.bfloat16:
        from paper_2609_32395_amd import synth
        x = synth.bf16_round(x)
    return x
