"""HIP-graph capture of the library's calls.

Store-level reads at the serve's head shape (a prefill over many pages: the
split launch and the merge; a batched decode step: the decode reader and its
merge) and the whole model's block-skip read (embedding, the LayerNorm-fused few-row
maps, the block-local attention, the few-pair prefill into the memory, the
output head) and its batched KV-cached decode step (the decode reader over
the in-block caches and the memory, with its split merge) are captured on a
side stream and the graph is replayed several times, with eager calls of the
program and host synchronizations between the replays.  Every replay must
give the eager call's bits: the calls record no memory set and no host wait,
and a replay's writes (the decode's cache row) are the eager call's."""
import numpy as np
import pytest
import torch

from paper_2609_32395_amd import smem, synth
from tests.gpu_util import require_gpu, say
from tests.test_gpu_model import SHAPE, build, tok

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    yield
    torch.cuda.synchronize()


def _capture(fn):
    """fn run once eagerly on a side stream (warm-up), then captured there."""
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=side):
        fn()
    torch.cuda.synchronize()
    return g


def test_block_skip_read_graph_replays_bitwise():
    say("graph: model block-skip read")
    g = np.random.default_rng(41)
    B = 5
    tokens = g.integers(0, SHAPE["vocab"], size=(B, SHAPE["b"]))
    m, _, _ = build()
    smem.smem_model_encode(m, 0, list(range(B - 1)), tok(tokens[:B - 1]))
    last = tok(tokens[B - 1:])
    eager = smem.smem_model_read(m, 0, [B - 1], last)
    logits = torch.empty_like(eager)
    graph = _capture(lambda: smem.smem_model_read(m, 0, [B - 1], last, logits=logits))
    for rep in range(3):
        logits.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(logits, eager), f"replay {rep}"
        # the program's own eager work between replays: another block's read
        smem.smem_model_read(m, 0, [B - 2], tok(tokens[B - 2:B - 1]))
        torch.cuda.synchronize()


def test_decode_step_graph_replays_bitwise():
    say("graph: model decode step")
    s = dict(SHAPE)
    W = synth.model_weights(smem.model_weight_shapes(s["E"], s["D"], s["d"], s["vocab"], s["n_pos"]), 7)
    dW = {k: torch.from_numpy(v).to("cuda").to(torch.bfloat16).contiguous() for k, v in W.items()}
    m = smem.Model(dW, s["E"], s["D"], s["d"], s["H"], s["b"], s["vocab"], s["n_pos"], 3, 8, 24, 256)
    g = np.random.default_rng(42)
    J, P = [3, 1, 4], [5, 2, 7]
    for q in range(3):
        smem.smem_model_encode(m, q, list(range(J[q])), tok(g.integers(0, s["vocab"], size=(J[q], s["b"]))))
    toks = g.integers(0, s["vocab"], size=(3, max(P) + 1))
    for p in range(max(P)):                       # each sequence's in-block cache up to its position
        for q in range(3):
            if p < P[q]:
                smem.smem_model_decode(m, q, [J[q]], [p], tok(toks[q, p:p + 1]))
    step = tok(toks[np.arange(3), P])
    eager = smem.smem_model_decode(m, 0, J, P, step)
    logits = torch.empty_like(eager)
    graph = _capture(lambda: smem.smem_model_decode(m, 0, J, P, step, logits=logits))
    for rep in range(3):
        logits.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()                            # rewrites each cache row P[q] with the same values
        torch.cuda.synchronize()
        assert torch.equal(logits, eager), f"replay {rep}"
        # eager work between replays: sequence 1's next position (a cache row
        # the captured step does not read)
        smem.smem_model_decode(m, 1, [J[1]], [P[1] + 1], tok(toks[1, P[1] + 1:P[1] + 2]))
        torch.cuda.synchronize()


def test_store_reads_graph_replays_bitwise():
    """Store-level reads at the serve's head shape (16 heads of 128): a
    block's prefill over 70 memory pages (one workgroup per split, then the
    merge launch) and a 4-sequence decode step (the decode reader and its
    merge), captured and replayed against the eager calls."""
    say("graph: store prefill (split + merge) and decode")
    b, H, dh, S, J = 64, 16, 128, 4, 70
    st = smem.Store(S, J + 1, S * J, b, H, dh, torch.bfloat16)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(43)
    rnd = lambda *shape: torch.randn(*shape, generator=gen, device="cuda").to(torch.bfloat16)
    for s in range(S):
        for j in range(J):
            smem.smem_store_put_block(st, s, j, rnd(b, H, dh), rnd(b, H, dh))
    q, ki, vi, nkv = rnd(b, H, dh), rnd(b, H, dh), rnd(b, H, dh), rnd(2, H, dh)
    eager_p = smem.smem_reader_prefill_block(st, [0], [J], q, ki, vi, nkv)
    out_p = torch.empty_like(eager_p)
    qd, kn, vn = rnd(S, H, dh), rnd(S, H, dh), rnd(S, H, dh)
    kc, vc = rnd(S * b, H, dh), rnd(S * b, H, dh)
    pos = [3, 17, 40, 63]
    eager_d = smem.smem_reader_decode(st, list(range(S)), [J] * S, pos, qd, kn, vn, kc, vc, nkv)
    out_d = torch.empty_like(eager_d)

    def calls():
        smem.smem_reader_prefill_block(st, [0], [J], q, ki, vi, nkv, out=out_p)
        smem.smem_reader_decode(st, list(range(S)), [J] * S, pos, qd, kn, vn, kc, vc, nkv, out=out_d)

    graph = _capture(calls)
    for rep in range(3):
        out_p.fill_(float("nan"))
        out_d.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_p, eager_p), f"prefill, replay {rep}"
        assert torch.equal(out_d, eager_d), f"decode, replay {rep}"
        smem.smem_reader_prefill_block(st, [1], [J - 3], q, ki, vi, nkv)   # eager work between replays
        torch.cuda.synchronize()
