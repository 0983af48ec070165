"""Seeded synthetic inputs for the SMem attention path.

This module only draws numbers: it holds none of the method's arithmetic.
Both the fp64 oracle (through the tests) and the HIP path consume the bytes
it produces, so a parity test compares the two implementations on exactly
the same inputs.

Every array is drawn from numpy's PCG64 generator seeded by a
``SeedSequence`` whose entropy is the tuple
``(seed, workload, role, seq, block, version)``; a block's rows therefore
depend only on that key, never on how many other blocks were drawn or in
which order, which is what the edit-path tests need (the same block re-drawn
for a re-insert gives the same bytes).

Values are standard normals scaled by the workload's scale.  bf16 data is
returned as float32 arrays whose every element is exactly representable in
bf16 (round-to-nearest-even on the float32 bit pattern), so the conversion
to a device bf16 tensor is exact and the oracle sees the same values.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor

import numpy as np

# Role tags of the seed key.
ROLE_Q = 0
ROLE_K = 1
ROLE_V = 2
ROLE_KMEM = 3
ROLE_VMEM = 4
ROLE_NULL = 5
ROLE_QDEC = 6
ROLE_KNEW = 7
ROLE_VNEW = 8
ROLE_POS = 9
ROLE_EDIT = 10


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 value (ties to even).

    Returns float32 holding bf16-representable values.  NaN/Inf never occur in
    the synthetic data (finite normals), so no special casing is needed."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(x.shape)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of bf16-representable float32 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def from_bf16_bits(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def normal(shape, key, scale: float, dtype: str) -> np.ndarray:
    """Standard normals * scale, as float32 (bf16-rounded when dtype=='bf16')."""
    g = rng(*key)
    x = (g.standard_normal(size=shape, dtype=np.float64) * scale).astype(np.float32)
    if dtype == "bf16":
        x = bf16_round(x)
    elif dtype != "f32":
        raise ValueError(dtype)
    return x


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one synthetic workload (sizes of the paper's model scales)."""
    name: str
    wid: int            # workload id, part of every seed key
    dtype: str          # "f32" or "bf16"
    H: int
    dh: int
    b: int
    n_seq: int
    n_blocks: int       # blocks per sequence (memory blocks, or encoded blocks)
    scale: float        # std of every drawn tensor

    @property
    def row_shape(self):
        return (self.b, self.H, self.dh)


# The five workloads: tiny fp32 check, 160M-, 410M- and 1.5B-shaped runs.
TINY_F32 = Workload("tiny fp32: H4 x dh32, b16, 8 blocks, batch 1", 1, "f32", 4, 32, 16, 1, 8, 1.0)
ENC_160M = Workload("160M-shaped encode+prefill: H12 x dh64, b64, 16 blocks, batch 8", 2, "bf16", 12, 64, 64, 8, 16, 1.0 / 8.0)
DEC_410M = Workload("410M-shaped batched decode: H16 x dh64, b64, 64 memory blocks, batch 64", 3, "bf16", 16, 64, 64, 64, 64, 1.0 / 8.0)
SERVE_1P5B = Workload("1.5B-shaped long-context serve: H16 x dh128, b64, 512 memory blocks, batch 1", 4, "bf16", 16, 128, 64, 1, 512, 1.0 / np.sqrt(128.0))
STRESS_1P5B = Workload("1.5B-shaped stress decode: H16 x dh128, b64, 4096 memory blocks, batch 16", 5, "bf16", 16, 128, 64, 16, 4096, 1.0 / np.sqrt(128.0))

WORKLOADS = {w.wid: w for w in (TINY_F32, ENC_160M, DEC_410M, SERVE_1P5B, STRESS_1P5B)}


def block_tokens(w: Workload, seed: int, role: int, seq: int, block: int, version: int = 0) -> np.ndarray:
    """One block's [b, H, dh] tensor for a role (Q, K, V of a block to encode)."""
    return normal(w.row_shape, (seed, w.wid, role, seq, block, version), w.scale, w.dtype)


def memory_block(w: Workload, seed: int, seq: int, block: int, version: int = 0):
    """K and V rows [b, H, dh] of a memory block put directly into the store."""
    k = normal(w.row_shape, (seed, w.wid, ROLE_KMEM, seq, block, version), w.scale, w.dtype)
    v = normal(w.row_shape, (seed, w.wid, ROLE_VMEM, seq, block, version), w.scale, w.dtype)
    return k, v


def memory_blocks(w: Workload, seed: int, seqs, blocks, threads: int = 8):
    """Many memory blocks at once: returns K, V of shape [len(seqs), len(blocks), b, H, dh].

    Drawn per block (keys independent of the batch) on a thread pool; numpy's
    generators release the GIL while filling arrays."""
    seqs = list(seqs)
    blocks = list(blocks)
    K = np.empty((len(seqs), len(blocks)) + w.row_shape, np.float32)
    V = np.empty_like(K)

    def fill(ij):
        i, j = ij
        K[i, j], V[i, j] = memory_block(w, seed, seqs[i], blocks[j])

    jobs = [(i, j) for i in range(len(seqs)) for j in range(len(blocks))]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(fill, jobs))
    return K, V


def null_row(w: Workload, seed: int) -> np.ndarray:
    """A learned-null-row stand-in: K and V vectors per head, [2, H, dh]."""
    return normal((2, w.H, w.dh), (seed, w.wid, ROLE_NULL, 0, 0, 0), w.scale, w.dtype)


def decode_positions(w: Workload, seed: int, n_seq: int) -> np.ndarray:
    """In-block positions p in [0, b) of the decode query, uniform per sequence."""
    return rng(seed, w.wid, ROLE_POS, 0, 0, 0).integers(0, w.b, size=n_seq).astype(np.int32)


# ---------------------------------------------------------------- device-side draws
# The 1.5B-shaped stress store holds 16 x 4096 blocks (32 GiB of bf16 rows):
# too much to draw on the host.  Its rows are drawn on the GPU by torch's
# seeded generator, one generator seed per block key, so any block can be
# re-drawn alone (for re-inserts and for the oracle's copy) with the same
# bytes.  Both sides consume those bytes: the HIP path from device memory,
# the oracle from a host copy of the generator's output.

def block_seed(*key: int) -> int:
    """64-bit generator seed for a block key (SeedSequence hash of the key)."""
    return int(np.random.SeedSequence([int(k) for k in key]).generate_state(1, np.uint64)[0] >> np.uint64(1))


def memory_block_device(w: Workload, seed: int, seq: int, block: int, version: int = 0, device="cuda"):
    """K and V rows [b, H, dh] of a memory block drawn on the device (bf16 or fp32)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(block_seed(seed, w.wid, ROLE_KMEM, seq, block, version))
    x = torch.randn((2,) + w.row_shape, generator=g, device=device, dtype=torch.float32) * w.scale
    x = x.to(torch.bfloat16 if w.dtype == "bf16" else torch.float32)
    return x[0], x[1]


ROLE_WEIGHT = 11


def model_weights(shapes, seed: int) -> dict:
    """Random model weights, bf16-representable float32, one array per
    (name, shape): LayerNorm scales 1 + 0.1 N, shifts 0.1 N, embedding and
    null rows N(0, 1), linear maps [out, in] N(0, 1) / sqrt(in).  Each array
    is drawn from its own key (seed, weight role, index in the list)."""
    W = {}
    for i, (name, shape) in enumerate(shapes):
        g = rng(seed, ROLE_WEIGHT, i)
        x = g.standard_normal(size=shape, dtype=np.float32)
        if name.endswith("_g"):
            x = 1.0 + 0.1 * x
        elif name.endswith("_b"):
            x = 0.1 * x
        elif len(shape) == 2 and not name.endswith("_emb"):
            x = x * np.float32(1.0 / np.sqrt(shape[1]))
        W[name] = bf16_round(x)
    return W


def model_weights_device(shapes, seed: int, device="cuda") -> dict:
    """The distribution of model_weights, drawn on the device by torch's
    seeded generator (one generator seed per weight) as bf16 tensors: for
    models too large to draw on the host."""
    import torch
    W = {}
    g = torch.Generator(device=device)
    for i, (name, shape) in enumerate(shapes):
        g.manual_seed(block_seed(seed, ROLE_WEIGHT, i))
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if name.endswith("_g"):
            x = 1.0 + 0.1 * x
        elif name.endswith("_b"):
            x = 0.1 * x
        elif len(shape) == 2 and not name.endswith("_emb"):
            x = x * (1.0 / float(np.sqrt(shape[1])))
        W[name] = x.to(torch.bfloat16).contiguous()
        del x
    return W


# Model scales of Appendix A: (name, d, E, D); heads of width 32, the GPT-2
# vocabulary, T = 1024 learned positions, b = 64.
MODEL_SCALES = [("160M", 768, 3, 7), ("410M", 1024, 4, 15), ("1.5B", 2048, 4, 15)]
MODEL_VOCAB = 50257
MODEL_T = 1024
ROLE_TOKENS = 12


def model_tokens(seed: int, scale: str, n_tokens: int, vocab: int = MODEL_VOCAB) -> np.ndarray:
    """Uniform token ids int32 [n_tokens] of one synthetic context."""
    return rng(seed, ROLE_TOKENS, sum(map(ord, scale)), n_tokens).integers(0, vocab, size=n_tokens, dtype=np.int32)
