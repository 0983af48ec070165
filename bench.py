"""Benchmark of the SMem attention hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1]

Headline workload (the timed step): 410M-shaped batched decode -- 64
sequences, 16 heads x dh 64, b = 64, 64 cached blocks (4096 memory rows) per
sequence, bf16.  One step is one smem_reader_decode call that decodes one
token for every sequence (one reader layer's attention); the in-block
position of sequence s at step t is (p_s + t) mod 64 with p_s uniform per
sequence, so 1..64 in-block keys are read besides the memory.  `value` is
decoded tokens/s with every input already resident in HBM.

Secondary workloads, timed in the same run and reported under "secondary":
  * 160M-shaped encode + prefill: 8 sequences x 16 blocks, 12 heads x dh 64,
    b = 64: block-local encoder attention over all 128 blocks (inserted into
    the store), then reader prefill of the final block of each sequence;
  * 1.5B-shaped single-block serve: 512 cached blocks (32768 rows), 16 heads
    x dh 128, batch 1: reader prefill of one fresh block over all rows, then
    100 random single-block deletions, each followed by a re-serve;
  * 410M-shaped streaming decode: the headline shape decoding 128 tokens
    from a fresh block, appending each completed block (64 blocks per
    append, encoder attention + insert) as the stream crosses a boundary;
  * 410M-shaped decode from the row plane (rows of width 1024 shared by all
    layers; one layer's key/value maps folded into the query and output);
  * the SMem+RoPE composite (saturating block phases, W = 15) timed on the
    headline decode and on the 1.5B serve, beside the base reads;
  * 1.5B-shaped stress: 16 sequences x 4096 blocks (262144 rows each, a
    32 GiB store): batch-16 decode over all rows, and single-block delete /
    re-insert latency;
  * the whole model at random weights, 160M / 410M / 1.5B scales (d 768 /
    1024 / 2048, E:D 3:7 / 4:15 / 4:15, heads of 32, GPT-2 vocabulary, 1024
    learned positions): block-skip serving of a fully cached context against
    the cold prefill, batch 1, contexts 1k / 2k / 4k / 8k; and batched
    KV-cached decode at the paper's (scale, context, batch) cells, 128 timed
    tokens after 66 warm-up tokens, completed blocks appended in the loop;
  * on request only (--workloads selfattn): the self-attention sub-layer's
    attention part at the 160M and 410M widths, the model's map + attention
    pair against the fused LayerNorm + q|k|v + attention kernel.

Timing uses HIP events on the stream the kernels are launched on (torch's
current stream, handed to the library).  The 160M encoder and prefill calls
are shorter than the host's cost of issuing them, so they are captured in a
HIP graph (repetitions of the call, no memory sets) and the replays are
timed.  The 160M encoder/prefill and the 1.5B serve also report single
calls run right after a 512 MiB read pass and enqueued while it runs
(`*_single_flushed`): the device time of a call whose data are out of the
caches, against the back-to-back throughput above.  The CPU baseline is the fp64 numpy
oracle timed on a bounded sample of the headline workload on this host
(all threads, and one thread for reference).
Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
MFMA_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published (2.5 PFLOP/s, no sparsity)

# Memory-side bytes per call (read + written) measured with rocprofv3
# FETCH_SIZE / WRITE_SIZE, scaled by copies of known size (bench.py
# --copy-probe), keyed by a hash of the sources of the kernels the call runs:
# a changed kernel reports traffic as null until measured again.  Figures
# and commands: profiles/hbm_traffic_attention_kernels.md.
CSRC = "paper_2609_32395_amd/csrc/"
TRAFFIC = {
    # 410M decode step: k_reader_valu + k_merge
    "decode": ((CSRC + "reader_valu.hip", CSRC + "common.h"), {"77e591978f5a0ddc": 1.0890e+09}),
    # 160M encoder: k_encoder_mfma (attention only)
    "encoder": ((CSRC + "attn_mfma.hip", CSRC + "attn_ring.h", CSRC + "common.h"), {"2e5d7e7c4cc7fcae": 5.0445e+07}),
    # 160M final-block prefill: k_prefill_mfma_par
    "prefill": ((CSRC + "attn_mfma.hip", CSRC + "attn_ring.h", CSRC + "common.h"), {"2e5d7e7c4cc7fcae": 2.6971e+07}),
    # 1.5B serve: k_prefill_mfma + k_merge
    "serve": ((CSRC + "attn_mfma.hip", CSRC + "attn_ring.h", CSRC + "reader_valu.hip", CSRC + "common.h"),
              {"d0b754a9272c091a": 3.0615e+08}),
    # 410M row-plane decode step: k_rows_absorb_q, k_reader_rows, k_rows_combine (with the
    # in-block keys), k_rows_project
    "rows": ((CSRC + "rows.hip", CSRC + "reader_valu.hip", CSRC + "common.h"), {"39d68117510eaddf": 6.4302e+08}),
}


def traffic_of(name):
    srcs, table = TRAFFIC[name]
    return table.get(_sources_hash(srcs))


def _sources_hash(paths):
    import hashlib
    m = hashlib.sha1()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            m.update(f.read())
    return m.hexdigest()[:16]


def _events_time(fn, steps, stream):
    import torch
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for t in range(steps):
        fn(t)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / 1e3  # seconds


def _flushed_time(fn, reps, stream, scratch):
    """Median seconds of single calls of fn, each run right after a read pass
    over `scratch` (512 MiB, twice the 256 MiB last-level cache), so every
    call starts with its working set out of the caches.  The call is enqueued
    while the flush still runs, so the interval between the two events is the
    device's time for the call (the host's enqueue cost is not in it).  The
    flush only reads: dirty lines left by a writing flush would be written
    back during the timed call and slow it for reasons of its own."""
    import torch
    ts = []
    for r in range(reps):
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        scratch.sum()
        e0.record(stream)
        fn(r)
        e1.record(stream)
        e1.synchronize()
        ts.append(e0.elapsed_time(e1) / 1e3)
    return float(np.median(ts))


def _graph_time(fn, reps, stream, replays=8):
    """Seconds per call of fn, with `reps` calls captured in one HIP graph and
    the graph replayed: for calls shorter than the host's own cost of issuing
    them (the encoder: 12 us), timing eager calls would measure the host."""
    import torch
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        fn(0)                                   # warm the path on the capture stream
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=side):
        for t in range(reps):
            fn(t)
    g.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(side):
        start.record()
        for _ in range(replays):
            g.replay()
        end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / 1e3 / (replays * reps)


def decode_workload(args, torch, smem, synth):
    """Headline: batched decode over a 4096-row memory per sequence."""
    w = synth.DEC_410M
    S, H, dh, b, NB = w.n_seq, w.H, w.dh, w.b, w.n_blocks
    dt = torch.bfloat16
    seed = args.seed
    st = smem.Store(S, NB + 1, S * NB, b, H, dh, dt)
    # memory rows: seeded per (sequence, block), uploaded one sequence at a time
    for s in range(S):
        K, V = synth.memory_blocks(w, seed, [s], range(NB), threads=16)
        Kd = torch.from_numpy(K[0]).to("cuda").to(dt)
        Vd = torch.from_numpy(V[0]).to("cuda").to(dt)
        for j in range(NB):
            smem.smem_store_put_block(st, s, j, Kd[j], Vd[j])
    steps_total = args.warmup + args.steps
    n_draw = min(steps_total, 256)
    g = synth.rng(seed, w.wid, synth.ROLE_QDEC, 0, 0, 0)
    qs = synth.bf16_round((g.standard_normal((n_draw, S, H, dh)) * w.scale).astype(np.float32))
    kn = synth.bf16_round((g.standard_normal((n_draw, S, H, dh)) * w.scale).astype(np.float32))
    vn = synth.bf16_round((g.standard_normal((n_draw, S, H, dh)) * w.scale).astype(np.float32))
    kc0 = synth.bf16_round((g.standard_normal((S * b, H, dh)) * w.scale).astype(np.float32))
    vc0 = synth.bf16_round((g.standard_normal((S * b, H, dh)) * w.scale).astype(np.float32))
    p0 = synth.decode_positions(w, seed, S)
    Q = torch.from_numpy(qs).to("cuda").to(dt)
    KN = torch.from_numpy(kn).to("cuda").to(dt)
    VN = torch.from_numpy(vn).to("cuda").to(dt)
    kc = torch.from_numpy(kc0).to("cuda").to(dt)
    vc = torch.from_numpy(vc0).to("cuda").to(dt)
    out = torch.empty((S, H, dh), dtype=dt, device="cuda")
    seq_ids = list(range(S))
    qblk = [NB] * S
    pos_tab = [[int((p0[s] + t) % b) for s in range(S)] for t in range(steps_total)]
    stream = torch.cuda.current_stream()

    def step(t, base=0):
        i = (base + t) % n_draw
        smem.smem_reader_decode(st, seq_ids, qblk, pos_tab[base + t], Q[i], KN[i], VN[i], kc, vc, None, out)

    for t in range(args.warmup):
        step(t)
    secs = _events_time(lambda t: step(t, args.warmup), args.steps, stream)
    torch.cuda.synchronize()
    rope_res = None
    if "rope" in args.workloads.split(",") and not args.no_secondary:
        # the SMem+RoPE composite on the same store and inputs: saturating
        # block phases (W = 15), in-block phases 0..63
        rope = smem.Rope(dh, b, 10000.0, 15)

        def rstep(t, base=0):
            i = (base + t) % n_draw
            smem.smem_reader_decode_rope(st, rope, seq_ids, qblk, pos_tab[base + t], Q[i], KN[i], VN[i], kc, vc,
                                         None, out)

        for t in range(args.warmup):
            rstep(t)
        rsecs = _events_time(lambda t: rstep(t, args.warmup), args.steps, stream)
        rope_res = dict(tokens_per_s=S * args.steps / rsecs, ms_per_step=rsecs / args.steps * 1e3,
                        base_ms_per_step=secs / args.steps * 1e3, max_offset=15)
        rope.close()
    # algorithmic bytes: memory K+V rows read, in-block rows read (cache rows
    # 0..p-1 plus the new pair), the query, the output and the cache write
    esz = 2
    mem_bytes = S * H * NB * b * dh * 2 * esz
    per_step_intra = [sum(p for p in pos_tab[args.warmup + t]) * H * dh * 2 * esz for t in range(args.steps)]
    tok_bytes = S * H * dh * esz
    intra = float(np.mean(per_step_intra))
    bytes_step = mem_bytes + intra + tok_bytes * (1 + 2 + 1 + 2)  # q, k_new+v_new, out, cache row write (K, V)
    flops_step = 4.0 * S * H * dh * (NB * b + float(np.mean([np.mean(np.array(pos_tab[args.warmup + t]) + 1) for t in range(args.steps)])))
    sec_step = secs / args.steps
    res = dict(
        tokens_per_s=S / sec_step,
        ms_per_step=sec_step * 1e3,
        bytes_per_step=bytes_step,
        flops_per_step=flops_step,
        gbs=bytes_step / sec_step / 1e9,
        rope=rope_res,
        store=st, S=S, H=H, dh=dh, b=b, NB=NB, pos=pos_tab, qs=qs, kn=kn, vn=vn, kc0=kc0, vc0=vc0,
    )
    return res


def encode_prefill_workload(args, torch, smem, synth):
    """160M-shaped: encoder over 8 x 16 blocks, then prefill of the final blocks."""
    w = synth.ENC_160M
    S, H, dh, b, NB = w.n_seq, w.H, w.dh, w.b, w.n_blocks
    dt = torch.bfloat16
    seed = args.seed
    nb = S * NB
    q = np.stack([synth.block_tokens(w, seed, synth.ROLE_Q, s, j) for s in range(S) for j in range(NB)])
    k = np.stack([synth.block_tokens(w, seed, synth.ROLE_K, s, j) for s in range(S) for j in range(NB)])
    v = np.stack([synth.block_tokens(w, seed, synth.ROLE_V, s, j) for s in range(S) for j in range(NB)])
    Qd, Kd, Vd = (torch.from_numpy(x.reshape(nb * b, H, dh)).to("cuda").to(dt) for x in (q, k, v))
    out = torch.empty_like(Qd)
    seq_ids = [s for s in range(S) for j in range(NB)]
    blk = [j for s in range(S) for j in range(NB)]
    stream = torch.cuda.current_stream()
    reps = max(5, args.steps // 8)
    # encoder alone (attention only), timed
    for _ in range(3):
        smem.smem_encode_blocks(None, Qd, Kd, Vd, out=out, mask=smem.MASK_BIDIR, b=b)
    enc_s = _graph_time(lambda t: smem.smem_encode_blocks(None, Qd, Kd, Vd, out=out, mask=smem.MASK_BIDIR, b=b),
                        reps, stream)
    scratch = torch.zeros(512 << 20 >> 1, dtype=torch.bfloat16, device="cuda")
    enc_flushed_s = _flushed_time(lambda t: smem.smem_encode_blocks(None, Qd, Kd, Vd, out=out, mask=smem.MASK_BIDIR,
                                                                    b=b), 9, stream, scratch)
    # encode + insert into a store, then prefill the final block of each sequence
    st = smem.Store(S, NB, S * NB, b, H, dh, dt)
    smem.smem_encode_blocks(st, Qd, Kd, Vd, out=out, seq_ids=seq_ids, block_idx=blk, mask=smem.MASK_BIDIR)
    last = [s * NB + NB - 1 for s in range(S)]
    qp = torch.cat([Qd[i * b:(i + 1) * b] for i in last])
    kp = torch.cat([Kd[i * b:(i + 1) * b] for i in last])
    vp = torch.cat([Vd[i * b:(i + 1) * b] for i in last])
    pout = torch.empty_like(qp)
    qb = [NB - 1] * S
    for _ in range(3):
        smem.smem_reader_prefill_block(st, list(range(S)), qb, qp, kp, vp, None, pout)
    pre_s = _graph_time(lambda t: smem.smem_reader_prefill_block(st, list(range(S)), qb, qp, kp, vp, None, pout),
                        reps, stream)
    pre_flushed_s = _flushed_time(lambda t: smem.smem_reader_prefill_block(st, list(range(S)), qb, qp, kp, vp, None,
                                                                           pout), 9, stream, scratch)
    del scratch
    enc_flops = 4.0 * nb * H * b * b * dh
    enc_bytes = 4.0 * nb * b * H * dh * 2
    n_mem = (NB - 1) * b
    pre_flops = 4.0 * S * H * b * dh * (n_mem + (b + 1) / 2.0)
    pre_bytes = S * H * (n_mem * dh * 2 * 2 + 4 * b * dh * 2)
    st.close()
    return dict(encoder_ms=enc_s * 1e3, encoder_tflops=enc_flops / enc_s / 1e12, encoder_gbs=enc_bytes / enc_s / 1e9,
                encoder_flops=enc_flops, encoder_bytes=enc_bytes,
                encoder_ms_single_flushed=enc_flushed_s * 1e3, encoder_gbs_single_flushed=enc_bytes / enc_flushed_s / 1e9,
                prefill_ms=pre_s * 1e3, prefill_tflops=pre_flops / pre_s / 1e12, prefill_gbs=pre_bytes / pre_s / 1e9,
                prefill_ms_single_flushed=pre_flushed_s * 1e3, prefill_gbs_single_flushed=pre_bytes / pre_flushed_s / 1e9,
                encoder_traffic=traffic_of("encoder"), prefill_traffic=traffic_of("prefill"))


def serve_workload(args, torch, smem, synth):
    """1.5B-shaped: single-block serve over 32768 rows, then 100 delete + re-serve."""
    w = synth.SERVE_1P5B
    H, dh, b, NB = w.H, w.dh, w.b, w.n_blocks
    dt = torch.bfloat16
    seed = args.seed
    st = smem.Store(1, NB + 1, NB, b, H, dh, dt)
    for j0 in range(0, NB, 64):
        K, V = synth.memory_blocks(w, seed, [0], range(j0, min(NB, j0 + 64)), threads=16)
        Kd = torch.from_numpy(K[0]).to("cuda").to(dt)
        Vd = torch.from_numpy(V[0]).to("cuda").to(dt)
        for i in range(Kd.shape[0]):
            smem.smem_store_put_block(st, 0, j0 + i, Kd[i], Vd[i])
    q = torch.from_numpy(synth.block_tokens(w, seed, synth.ROLE_Q, 0, NB)).to("cuda").to(dt)
    k = torch.from_numpy(synth.block_tokens(w, seed, synth.ROLE_K, 0, NB)).to("cuda").to(dt)
    v = torch.from_numpy(synth.block_tokens(w, seed, synth.ROLE_V, 0, NB)).to("cuda").to(dt)
    out = torch.empty_like(q)
    stream = torch.cuda.current_stream()

    def serve(t=0):
        smem.smem_reader_prefill_block(st, [0], [NB], q, k, v, None, out)

    for _ in range(3):
        serve()
    reps = max(5, args.steps // 8)
    serve_s = _events_time(serve, reps, stream) / reps
    scratch = torch.zeros(512 << 20 >> 1, dtype=torch.bfloat16, device="cuda")
    serve_flushed_s = _flushed_time(serve, 9, stream, scratch)
    del scratch
    rope_ms = None
    if "rope" in args.workloads.split(","):
        rope = smem.Rope(dh, b, 10000.0, 15)

        def rserve(t=0):
            smem.smem_reader_prefill_block_rope(st, rope, [0], [NB], q, k, v, None, out)

        for _ in range(3):
            rserve()
        rope_ms = _events_time(rserve, reps, stream) / reps * 1e3
        rope.close()
    order = synth.rng(seed, w.wid, synth.ROLE_EDIT, 0, 0, 0).permutation(NB)[:100]
    start = torch.cuda.Event(enable_timing=True)
    mid = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    del_t, re_t = [], []
    for j in order:
        torch.cuda.synchronize()
        start.record(stream)
        smem.smem_delete_block(st, 0, int(j))
        mid.record(stream)
        serve()
        end.record(stream)
        end.synchronize()
        del_t.append(start.elapsed_time(mid))
        re_t.append(mid.elapsed_time(end))
    rows = NB * b
    flops = 4.0 * H * b * dh * (rows + (b + 1) / 2.0)
    bytes_ = H * (rows * dh * 2 * 2 + 4 * b * dh * 2)
    st.close()
    return dict(serve_ms=serve_s * 1e3, serve_tflops=flops / serve_s / 1e12, serve_gbs=bytes_ / serve_s / 1e9,
                serve_ms_single_flushed=serve_flushed_s * 1e3, serve_gbs_single_flushed=bytes_ / serve_flushed_s / 1e9,
                rope_serve_ms=rope_ms,
                delete_us_median=float(np.median(del_t)) * 1e3, reserve_ms_median=float(np.median(re_t)),
                rows_after_deletes=(NB - 100) * b, serve_bytes=bytes_, serve_traffic=traffic_of("serve"))


def stream_workload(args, torch, smem, synth):
    """410M-shaped streaming decode: 64 sequences with 64 cached blocks each
    decode 128 tokens from the start of a fresh block; after every 64th token
    the completed block of every sequence is encoded and appended (64 blocks
    per append), and the next block's tokens read it."""
    w = synth.DEC_410M
    S, H, dh, b, NB = w.n_seq, w.H, w.dh, w.b, w.n_blocks
    dt = torch.bfloat16
    T = 2 * b
    st = smem.Store(S, NB + 2, S * (NB + 2), b, H, dh, dt)
    for s in range(S):
        for j in range(NB):
            smem.smem_store_put_block(st, s, j, *synth.memory_block_device(w, args.seed, s, j))
    g = torch.Generator(device="cuda")
    g.manual_seed(synth.block_seed(args.seed, w.wid, synth.ROLE_QDEC, 1, 0, 0))
    # per token: reader q, k_new, v_new and encoder q, k, v, token-major
    X = (torch.randn((6, T, S, H, dh), generator=g, device="cuda") * w.scale).to(dt)
    enc = [[X[r, blk * b:(blk + 1) * b].transpose(0, 1).reshape(S * b, H, dh).contiguous() for r in (3, 4, 5)]
           for blk in range(2)]
    kc = torch.zeros((S * b, H, dh), dtype=dt, device="cuda")
    vc = torch.zeros_like(kc)
    out = torch.empty((S, H, dh), dtype=dt, device="cuda")
    seqs = list(range(S))
    stream = torch.cuda.current_stream()

    def run(_=0):
        for t in range(T):
            p, J = t % b, NB + t // b
            smem.smem_reader_decode(st, seqs, [J] * S, [p] * S, X[0, t], X[1, t], X[2, t], kc, vc, None, out)
            if p == b - 1:
                smem.smem_encode_blocks(st, *enc[t // b], seq_ids=seqs, block_idx=[J] * S)

    def undo():
        torch.cuda.synchronize()
        for blk in range(2):
            for s in seqs:
                smem.smem_delete_block(st, s, NB + blk)

    run()
    undo()
    secs = _events_time(run, 1, stream)
    undo()
    reps = 5
    app = []
    for _ in range(reps):
        app.append(_events_time(lambda _t: smem.smem_encode_blocks(st, *enc[0], seq_ids=seqs,
                                                                   block_idx=[NB] * S), 1, stream))
        for s in seqs:
            smem.smem_delete_block(st, s, NB)
    st.close()
    return dict(tokens=S * T, appends=2, blocks_per_append=S, tokens_per_s=S * T / secs,
                ms_per_step=secs / T * 1e3, append_ms_median=float(np.median(app)) * 1e3)


def rows_workload(args, torch, smem, synth):
    """410M-shaped decode from the row plane: 64 sequences x 64 blocks of 64
    rows of width d = 1024 (one plane shared by all layers), one layer's maps
    (16 heads x dh 64), one token per sequence per step with 1-64 in-block
    keys; timed like the headline."""
    w = synth.DEC_410M
    S, H, dh, b, NB = w.n_seq, w.H, w.dh, w.b, w.n_blocks
    d = H * dh
    dt = torch.bfloat16
    st = smem.RowStore(S, NB + 1, S * NB, b, d)
    g = torch.Generator(device="cuda")
    for s in range(S):
        g.manual_seed(synth.block_seed(args.seed, w.wid, synth.ROLE_KMEM, s, 0, 1))
        R = torch.randn((NB, b, d), generator=g, device="cuda").to(dt)
        for j in range(NB):
            smem.smem_rows_put_block(st, s, j, R[j])
    g.manual_seed(synth.block_seed(args.seed, w.wid, synth.ROLE_QDEC, 2, 0, 0))
    wk = (torch.randn((H * dh, d), generator=g, device="cuda") / d ** 0.5).to(dt)
    wv = (torch.randn((H * dh, d), generator=g, device="cuda") / d ** 0.5).to(dt)
    n_draw = 64
    X = (torch.randn((3, n_draw, S, H, dh), generator=g, device="cuda") * w.scale).to(dt)
    kc = (torch.randn((S * b, H, dh), generator=g, device="cuda") * w.scale).to(dt)
    vc = torch.empty_like(kc).copy_(kc)
    p0 = synth.decode_positions(w, args.seed, S)
    out = torch.empty((S, H, dh), dtype=dt, device="cuda")
    seqs = list(range(S))
    qblk = [NB] * S
    stream = torch.cuda.current_stream()

    def step(t):
        i = t % n_draw
        pos = [int((p0[s] + t) % b) for s in range(S)]
        smem.smem_reader_decode_rows(st, wk, wv, seqs, qblk, pos, X[0, i], X[1, i], X[2, i], kc, vc, None, out)

    for t in range(args.warmup):
        step(t)
    secs = _events_time(step, args.steps, stream)
    row_bytes = S * NB * b * d * 2
    st.close()
    return dict(tokens_per_s=S * args.steps / secs, ms_per_step=secs / args.steps * 1e3, d=d,
                row_bytes_per_step=row_bytes, row_gbs=row_bytes / (secs / args.steps) / 1e9,
                traffic=traffic_of("rows"))


def stress_workload(args, torch, smem, synth):
    """1.5B-shaped stress: 16 sequences x 4096 blocks (262144 rows, 32 GiB);
    batch-16 decode over all rows, and single-block delete / re-insert latency."""
    w = synth.STRESS_1P5B
    S, H, dh, b, NB = w.n_seq, w.H, w.dh, w.b, w.n_blocks
    dt = torch.bfloat16
    st = smem.Store(S, NB, S * NB, b, H, dh, dt)
    for s in range(S):
        for j in range(NB):
            smem.smem_store_put_block(st, s, j, *synth.memory_block_device(w, args.seed, s, j))
    g = synth.rng(args.seed, w.wid, synth.ROLE_QDEC, 0, 0, 0)
    mk = lambda shape: torch.from_numpy(synth.bf16_round((g.standard_normal(shape) * w.scale).astype(np.float32))).to("cuda").to(dt)
    q, kn, vn = mk((S, H, dh)), mk((S, H, dh)), mk((S, H, dh))
    kc, vc = mk((S * b, H, dh)), mk((S * b, H, dh))
    out = torch.empty((S, H, dh), dtype=dt, device="cuda")
    p0 = synth.decode_positions(w, args.seed, S)
    stream = torch.cuda.current_stream()
    seq_ids, qblk = list(range(S)), [NB] * S

    def step(t):
        pos = [int((p0[s] + t) % b) for s in range(S)]
        smem.smem_reader_decode(st, seq_ids, qblk, pos, q, kn, vn, kc, vc, None, out)

    for t in range(2):
        step(t)
    n = max(8, args.steps // 8)
    secs = _events_time(step, n, stream) / n
    er = synth.rng(args.seed, w.wid, synth.ROLE_EDIT, 2, 0, 0)
    start, mid, end = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    d_t, p_t, ds_t = [], [], []
    for it in range(32):
        s, j = int(er.integers(0, S)), int(er.integers(0, NB))
        kj, vj = synth.memory_block_device(w, args.seed, s, j)
        scrub = it % 2 == 1                  # every other delete also zeroes the freed page
        torch.cuda.synchronize()
        start.record(stream)
        smem.smem_delete_block(st, s, j, scrub=scrub)
        mid.record(stream)
        smem.smem_store_put_block(st, s, j, kj, vj)
        end.record(stream)
        end.synchronize()
        (ds_t if scrub else d_t).append(start.elapsed_time(mid))
        p_t.append(mid.elapsed_time(end))
    bytes_step = S * H * NB * b * dh * 2 * 2
    # canonical export of one sequence (every live page gathered in block order,
    # the value plane transposed back): 2 GiB read and 2 GiB written, into
    # preallocated outputs through the C ABI
    L = smem.lib()
    n_live = ctypes.c_int32()
    smem.check_status(L.smem_store_export(st.handle, 0, None, ctypes.byref(n_live), None, None, None))
    K_out = torch.empty((n_live.value * b, H, dh), dtype=dt, device="cuda")
    V_out = torch.empty_like(K_out)
    raw = stream.cuda_stream

    def export(_t=0):
        smem.check_status(L.smem_store_export(st.handle, 0, None, ctypes.byref(n_live), ctypes.c_void_p(K_out.data_ptr()),
                                          ctypes.c_void_p(V_out.data_ptr()), ctypes.c_void_p(raw)))

    export()
    ex_secs = _events_time(export, 4, stream) / 4
    ex_bytes = 2.0 * 2 * n_live.value * H * b * dh * 2
    del K_out, V_out
    st.close()
    return dict(decode_ms=secs * 1e3, tokens_per_s=S / secs, decode_gbs=bytes_step / secs / 1e9,
                memory_rows=NB * b, store_gib=S * NB * H * 2 * b * dh * 2 / 2 ** 30,
                delete_us_median=float(np.median(d_t)) * 1e3, reinsert_us_median=float(np.median(p_t)) * 1e3,
                delete_scrub_us_median=float(np.median(ds_t)) * 1e3, page_bytes=H * 2 * b * dh * 2,
                export_ms=ex_secs * 1e3, export_gib=ex_bytes / 2 / 2 ** 30, export_gbs=ex_bytes / ex_secs / 1e9,
                export_hbm_frac=ex_bytes / ex_secs / 1e9 / HBM_PEAK_GBS)


def delete_sweep_workload(args, torch, smem, synth):
    """Deletion latency against the number of cached blocks of one sequence
    (the paper's deletion-latency sweep, 512 to 65,536 blocks): a store of
    1.5B-shaped pages (16 heads x d_h 128, b = 64, 512 KiB a page) holding
    every block, then seeded single-block deletions at random indices (one
    at index 0, the whole live list behind it), each followed by the block's
    re-insertion.  Per size: the call as the host sees it (wall clock around
    the C call), the device time of its kernels (events around the call
    enqueued behind a running kernel), and delete with scrub (the freed page
    zeroed); a batch-1 decode over the remaining rows after a deletion is
    timed too.  Page contents do not enter deletion; every page holds the
    same seeded rows."""
    w = synth.STRESS_1P5B
    H, dh, b = w.H, w.dh, w.b
    dt = torch.bfloat16
    L = smem.lib()
    stream = torch.cuda.current_stream()
    raw = ctypes.c_void_p(stream.cuda_stream)
    g = synth.rng(args.seed, w.wid, synth.ROLE_EDIT, 5, 0, 0)
    chunk = 128
    rows = torch.from_numpy(synth.bf16_round((g.standard_normal((chunk * b, H, dh)) * w.scale).astype(np.float32)))
    rows = rows.to("cuda").to(dt)
    busy = torch.empty(64 << 20, dtype=torch.float32, device="cuda")
    out = {}
    for NB in [int(x) for x in args.delete_sizes.split(",")]:
        st = smem.Store(1, NB, NB, b, H, dh, dt)
        for j0 in range(0, NB, chunk):
            n = min(chunk, NB - j0)
            smem.smem_store_put_blocks(st, [0] * n, list(range(j0, j0 + n)), rows[: n * b], rows[: n * b])
        torch.cuda.synchronize()
        order = [0] + [int(x) for x in g.integers(0, NB, 24)]
        host_us, wall_us, dev_us, scrub_us, reins_us = [], [], [], [], []
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for it, j in enumerate(order):
            # device time: the call enqueued while a kernel still runs
            torch.cuda.synchronize()
            busy.mul_(1.0)
            e0.record(stream)
            smem.check_status(L.smem_delete_block(st.handle, 0, j, 0, raw))
            e1.record(stream)
            e1.synchronize()
            dev_us.append(e0.elapsed_time(e1) * 1e3)
            smem.check_status(L.smem_store_put_block(st.handle, 0, j, ctypes.c_void_p(rows.data_ptr()),
                                                     ctypes.c_void_p(rows.data_ptr()), raw))
            # the call on an idle GPU: host time and wall time to completion
            torch.cuda.synchronize()
            e0.record(stream)
            t0 = time.perf_counter()
            smem.check_status(L.smem_delete_block(st.handle, 0, j, 0, raw))
            t1 = time.perf_counter()
            e1.record(stream)
            e1.synchronize()
            host_us.append((t1 - t0) * 1e6)
            wall_us.append(e0.elapsed_time(e1) * 1e3)
            torch.cuda.synchronize()
            e0.record(stream)
            smem.check_status(L.smem_store_put_block(st.handle, 0, j, ctypes.c_void_p(rows.data_ptr()),
                                                     ctypes.c_void_p(rows.data_ptr()), raw))
            e1.record(stream)
            e1.synchronize()
            reins_us.append(e0.elapsed_time(e1) * 1e3)
            torch.cuda.synchronize()
            e0.record(stream)
            smem.check_status(L.smem_delete_block(st.handle, 0, j, 1, raw))
            e1.record(stream)
            e1.synchronize()
            scrub_us.append(e0.elapsed_time(e1) * 1e3)
            smem.check_status(L.smem_store_put_block(st.handle, 0, j, ctypes.c_void_p(rows.data_ptr()),
                                                     ctypes.c_void_p(rows.data_ptr()), raw))
        # a read after a deletion: batch-1 decode over the remaining rows
        smem.check_status(L.smem_delete_block(st.handle, 0, order[-1], 0, raw))
        q = rows[:1].contiguous()
        dout = torch.empty_like(q)
        for _ in range(2):
            smem.smem_reader_decode(st, [0], [NB], None, q, out=dout)
        reps = 5
        read_s = _events_time(lambda t: smem.smem_reader_decode(st, [0], [NB], None, q, out=dout), reps, stream) / reps
        st.close()
        med = lambda xs: float(np.median(xs))
        out[str(NB)] = dict(delete_device_us=round(med(dev_us), 2), delete_host_us=round(med(host_us), 2),
                            delete_idle_gpu_us=round(med(wall_us), 2), delete_front_device_us=round(dev_us[0], 2),
                            delete_scrub_idle_gpu_us=round(med(scrub_us), 2),
                            reinsert_idle_gpu_us=round(med(reins_us), 2),
                            read_after_delete_ms=round(read_s * 1e3, 4),
                            read_gbs=round((NB - 1) * H * 2 * b * dh * 2 / read_s / 1e9, 1))
    del busy
    return out


def model_workload(args, torch, smem, synth):
    """Whole model at random weights (Appendix A scales): block-skip serving
    of a fully cached context (the reader on the final block alone) against
    the model's own cold prefill (encoder over every block, reader over every
    block, final-block logits), batch 1, contexts 1k-8k."""
    stream = torch.cuda.current_stream()
    lengths = [int(x) for x in args.model_lengths.split(",")]
    scales = [sc for sc in synth.MODEL_SCALES if sc[0] in args.model_scales.split(",")]
    out = {}
    for name, d, E, D in scales:
        H, b, vocab, T = d // 32, 64, synth.MODEL_VOCAB, synth.MODEL_T
        nb_max = max(lengths) // b
        W = synth.model_weights_device(smem.model_weight_shapes(E, D, d, vocab, T), args.seed)
        m = smem.Model(W, E, D, d, H, b, vocab, T, 1, nb_max, nb_max, max_tokens=min(nb_max, 128) * b)
        cells = {}
        for n in lengths:
            J = n // b
            tokens = torch.from_numpy(synth.model_tokens(args.seed, name, n, vocab)).to("cuda")
            last = tokens[(J - 1) * b:].contiguous()
            cold_t = []
            for rep in range(args.model_reps + 1):
                for j in range(J if rep else 0):
                    smem.smem_model_delete_block(m, 0, j)
                torch.cuda.synchronize()
                t0 = torch.cuda.Event(enable_timing=True)
                t1 = torch.cuda.Event(enable_timing=True)
                t0.record(stream)
                cold = smem.smem_model_prefill(m, 0, 0, J, tokens)
                t1.record(stream)
                t1.synchronize()
                if rep:                                   # rep 0 warms the path
                    cold_t.append(t0.elapsed_time(t1))
            skip_t = []
            for rep in range(args.model_reps + 2):
                torch.cuda.synchronize()
                t0 = torch.cuda.Event(enable_timing=True)
                t1 = torch.cuda.Event(enable_timing=True)
                t0.record(stream)
                skip = smem.smem_model_read(m, 0, [J - 1], last)
                t1.record(stream)
                t1.synchronize()
                if rep >= 2:
                    skip_t.append(t0.elapsed_time(t1))
            same = bool(torch.equal(skip, cold))
            # algorithmic work: block-skip reads every reader weight once, the
            # head, and the memory keys/values of J - 1 blocks in every layer;
            # the cold pass's flops are the linear maps over all n tokens (the
            # head on the final block) plus every attention score and value product
            skip_bytes = 2.0 * (14 * D * d * d + vocab * d) + 4.0 * D * (J - 1) * b * d
            lin = 2.0 * n * (E * 12 * d * d + D * 16 * d * d) + 2.0 * b * d * vocab
            pairs = E * J * b * b + D * J * b * (b + 1) / 2 + D * sum(b * (b * j + 1) for j in range(J))
            cold_flops = lin + 4.0 * pairs * d
            graph_ms = _graph_time(lambda t: smem.smem_model_read(m, 0, [J - 1], last, logits=skip), 4, stream) * 1e3
            for j in range(J):
                smem.smem_model_delete_block(m, 0, j)
            print(f"[bench] model {name} n={n}: cold {np.median(cold_t):.3f} ms, block-skip "
                  f"{np.median(skip_t):.3f} ms (graph {graph_ms:.3f} ms)", file=sys.stderr, flush=True)
            cells[str(n)] = dict(cold_prefill_ms=round(float(np.median(cold_t)), 3),
                                 block_skip_ms=round(float(np.median(skip_t)), 3),
                                 block_skip_graph_ms=round(graph_ms, 3),
                                 ttft_reduction=round(1.0 - float(np.median(skip_t)) / float(np.median(cold_t)), 4),
                                 skip_equals_cold_bitwise=same,
                                 block_skip_gbs=round(skip_bytes / float(np.median(skip_t)) / 1e6, 1),
                                 block_skip_hbm_frac=round(skip_bytes / float(np.median(skip_t)) / 1e6 / HBM_PEAK_GBS, 4),
                                 cold_tflops=round(cold_flops / float(np.median(cold_t)) / 1e9, 1),
                                 cold_mfma_frac=round(cold_flops / float(np.median(cold_t)) / 1e9 / MFMA_BF16_TFLOPS, 4))
        oracle = None
        if name == "160M" and not args.no_cpu_baseline:
            oracle = model_oracle_time(args, torch, smem, synth, W, E, D, d, H, b, vocab, T, min(lengths))
        m.close()
        del W
        torch.cuda.empty_cache()
        out[name] = dict(d=d, E=E, D=D, H=H, cells=cells)
        if oracle:
            out[name]["cpu_oracle"] = oracle
    return out


# The paper's batched decode cells (its serving appendix): scale, context, batch
DECODE_CELLS = [("160M", 4096, 64), ("160M", 8192, 16), ("160M", 8192, 64), ("410M", 1024, 64), ("410M", 4096, 16),
                ("410M", 8192, 16), ("1.5B", 1024, 64), ("1.5B", 4096, 16)]


def model_decode_workload(args, torch, smem, synth, row_plane=False):
    """Whole-model KV-cached batched decode at the paper's cells: every
    sequence holds a context of n tokens (n / b encoded blocks) and decodes
    the next tokens one step at a time, appending each block as it completes
    (one multi-sequence encode per boundary, inside the timed steps).  Token
    ids are drawn, not sampled from the logits: the work per step is the same.
    row_plane: the memory is kept as rows, read by every layer through its
    own key and value maps (the decode arm that derives keys and values from
    the rows); otherwise every layer keeps its keys and values."""
    stream = torch.cuda.current_stream()
    out = {}
    scales = {sc[0]: sc for sc in synth.MODEL_SCALES}
    cells = [c for c in DECODE_CELLS if c[0] in args.model_scales.split(",")]
    weights = {}
    for name, n, S in cells:
        _, d, E, D = scales[name]
        H, b, vocab, T = d // 32, 64, synth.MODEL_VOCAB, synth.MODEL_T
        if name not in weights:
            weights.clear()
            torch.cuda.empty_cache()
            weights[name] = synth.model_weights_device(smem.model_weight_shapes(E, D, d, vocab, T), args.seed)
        W = weights[name]
        J0 = n // b
        steps, warm = args.decode_steps, args.decode_warmup
        nb = J0 + (steps + warm) // b + 2
        m = smem.Model(W, E, D, d, H, b, vocab, T, S, nb, S * nb, max_tokens=8192, row_plane=row_plane)
        ctx = torch.from_numpy(synth.model_tokens(args.seed, name, S * n, vocab)).to("cuda")
        per = max(1, 128 // J0)                     # sequences per encode call (128 blocks)
        for s0 in range(0, S, per):
            s1 = min(S, s0 + per)
            smem.smem_model_encode_blocks(m, [q for q in range(s0, s1) for j in range(J0)],
                                          [j for q in range(s0, s1) for j in range(J0)], ctx[s0 * n:s1 * n])
        gen = torch.from_numpy(synth.model_tokens(args.seed + 1, name, S * (steps + warm + b), vocab)).to("cuda")
        gen = gen.view(S, -1)
        logits = torch.empty((S, vocab), dtype=torch.float32, device="cuda")
        state = {"t": 0}

        def step():
            t = state["t"]
            J, p = J0 + t // b, t % b
            smem.smem_model_decode(m, 0, [J] * S, [p] * S, gen[:, t].contiguous(), logits)
            if p == b - 1:                              # the block is complete: append it
                blk = gen[:, t - b + 1:t + 1].contiguous().view(-1)
                smem.smem_model_encode_blocks(m, list(range(S)), [J] * S, blk)
            state["t"] = t + 1

        for _ in range(warm):
            step()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            step()
        e1.record(stream)
        e1.synchronize()
        ms = e0.elapsed_time(e1)
        # memory read per step (average): every layer's keys and values, or
        # the rows once per layer; the row arm also reads each layer's key
        # and value maps (the query absorption and the output projection)
        kv = S * D * (J0 + (warm + steps / 2) / b) * b * d * 2 * (1 if row_plane else 2)
        wbytes = 2.0 * ((16 if row_plane else 14) * D * d * d + vocab * d)
        key = f"{name} {n}/{S}"
        out[key] = dict(tokens_per_s=round(S * steps / (ms / 1e3), 1), ms_per_step=round(ms / steps, 4),
                        hbm_gbs=round((kv + wbytes) / (ms / steps / 1e3) / 1e9, 1),
                        appends_timed=sum(1 for t in range(warm, warm + steps) if t % b == b - 1))
        print(f"[bench] decode{' (row plane)' if row_plane else ''} {key}: {out[key]['tokens_per_s']:.0f} tok/s, "
              f"{out[key]['ms_per_step']:.3f} ms/step", file=sys.stderr, flush=True)
        m.close()
        del ctx, gen
        torch.cuda.empty_cache()
    return out


def delete_generate_workload(args, torch, smem, synth):
    """Whole-model delete-then-generate, the SMem arm (the serving appendix's
    cell grid): a context of J cached blocks (batch 1) loses block j at 25, 50
    or 75% of the context (row slice: the block leaves every reader layer's
    store), then the final block is read alone (block-skip) for the next
    token's logits.  Timed: the deletion and the read, from one event to the
    next; the block is re-encoded afterwards, untimed, for the next cell."""
    stream = torch.cuda.current_stream()
    sizes = [int(x) for x in args.delgen_blocks.split(",")]
    out = {}
    for name, d, E, D in [sc for sc in synth.MODEL_SCALES if sc[0] in args.model_scales.split(",")]:
        H, b, vocab, T = d // 32, 64, synth.MODEL_VOCAB, synth.MODEL_T
        W = synth.model_weights_device(smem.model_weight_shapes(E, D, d, vocab, T), args.seed)
        for J in sizes:
            m = smem.Model(W, E, D, d, H, b, vocab, T, 1, J, J, max_tokens=128 * b)
            ctx = torch.from_numpy(synth.model_tokens(args.seed, name, J * b, vocab)).to("cuda")
            for j0 in range(0, J - 1, 128):             # cache blocks 0 .. J-2; block J-1 is the query
                j1 = min(J - 1, j0 + 128)
                smem.smem_model_encode(m, 0, list(range(j0, j1)), ctx[j0 * b:j1 * b])
            last = ctx[(J - 1) * b:].contiguous()
            logits = torch.empty((b, vocab), dtype=torch.float32, device="cuda")
            smem.smem_model_read(m, 0, [J - 1], last, logits=logits)      # warm the path
            cells = {}
            for frac in (25, 50, 75):
                j = (J - 1) * frac // 100
                ts = []
                for rep in range(3):
                    torch.cuda.synchronize()
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    smem.smem_model_delete_block(m, 0, j)
                    smem.smem_model_read(m, 0, [J - 1], last, logits=logits)
                    e1.record(stream)
                    e1.synchronize()
                    ts.append(e0.elapsed_time(e1))
                    smem.smem_model_encode(m, 0, [j], ctx[j * b:(j + 1) * b])
                cells[f"{frac}%"] = round(float(np.median(ts)), 3)
            torch.cuda.synchronize()
            mem_bytes = 4.0 * D * (J - 2) * b * d                 # memory keys/values read after the deletion
            wbytes = 2.0 * (14 * D * d * d + vocab * d)
            ms = float(np.median(list(cells.values())))
            out[f"{name} {J} blocks"] = dict(delete_then_generate_ms=cells,
                                             hbm_gbs=round((mem_bytes + wbytes) / (ms / 1e3) / 1e9, 1))
            print(f"[bench] delete-then-generate {name} {J} blocks: {cells} ms", file=sys.stderr, flush=True)
            m.close()
            del ctx, last, logits
            torch.cuda.empty_cache()
        del W
        torch.cuda.empty_cache()
    return out


def selfattn_workload(args, torch, smem, synth):
    """The attention part of a self-attention sub-layer at the model scales'
    widths (heads of 32, causal): the q|k|v map followed by the block-local
    attention launch (the model's path) against the fused kernel that runs
    the LayerNorm, the map and the attention of a (block, head) in one
    workgroup; back-to-back calls at 1, 2, 16 and 128 blocks, synthetic
    normal rows and weights of the model's scales, the two outputs compared
    bitwise."""
    stream = torch.cuda.current_stream()
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed)
    out = {}
    for name, d in (("160M", 768), ("410M", 1024)):
        H = d // 32
        w = (torch.randn(3 * d, d, generator=g, device="cuda") / math.sqrt(d)).to(torch.bfloat16)
        lg = (1.0 + 0.1 * torch.randn(d, generator=g, device="cuda")).to(torch.bfloat16)
        lb = (0.1 * torch.randn(d, generator=g, device="cuda")).to(torch.bfloat16)
        for nb in (1, 2, 16, 128):
            M = nb * 64
            x = torch.randn(M, d, generator=g, device="cuda").to(torch.bfloat16)
            work = torch.empty((4, M, d), dtype=torch.bfloat16, device="cuda")
            ys = {p: torch.empty((M, d), dtype=torch.bfloat16, device="cuda") for p in (1, 2)}
            us = {}
            for p in (1, 2):
                call = lambda _t, p=p: smem.smem_self_attention(x, lg, lb, w, H, smem.MASK_CAUSAL, path=p,
                                                                out=ys[p], work=work)
                for t in range(5):
                    call(t)
                us[p] = _events_time(call, 50, stream) / 50 * 1e6
            out[f"{name} {nb} blocks"] = dict(unfused_us=round(us[1], 2), fused_us=round(us[2], 2),
                                              bitwise_equal=bool(torch.equal(ys[1], ys[2])))
            print(f"[bench] self-attention {name} {nb} blocks: unfused {us[1]:.1f} us, fused {us[2]:.1f} us",
                  file=sys.stderr, flush=True)
            del x, work, ys
    return out


def model_oracle_time(args, torch, smem, synth, W, E, D, d, H, b, vocab, T, n):
    """The fp64 model oracle's block-skip read of the final block of an
    n-token context (the same unit as the GPU's block_skip_ms), on this host;
    the cached blocks are encoded first, untimed."""
    from oracle import smem_model as MO
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    J = n // b
    Wh = {k: v.float().cpu().numpy().astype(np.float64) for k, v in W.items()}
    ref = MO.Model(Wh, E, D, d, H, b, vocab, T, 1, J)
    tokens = synth.model_tokens(args.seed, "160M", n, vocab).reshape(J, b)
    ref.encode(0, tokens[:J - 1], list(range(J - 1)))
    t0 = time.perf_counter()
    ref.read(0, tokens[J - 1:], [J - 1])
    dt = time.perf_counter() - t0
    return {"block_skip_ms": round(dt * 1e3, 1), "cores": int(threads), "kind": "oracle",
            "sample": f"160M, {n}-token context: one block-skip read (fp64 numpy)"}


def cpu_baseline(dec, budget_s, seed):
    """The fp64 oracle on a bounded sample of the headline decode workload.

    The oracle's store is rebuilt from the seeded generator (never from the
    GPU); only the oracle's decode calls are timed."""
    from oracle import smem_oracle as O
    from paper_2609_32395_amd import synth
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    w = synth.DEC_410M
    S, H, dh, b, NB = dec["S"], dec["H"], dec["dh"], dec["b"], dec["NB"]
    n_tok, spent, s = 0, 0.0, 0
    kc_all = dec["kc0"].reshape(S, b, H, dh)
    vc_all = dec["vc0"].reshape(S, b, H, dh)
    while spent < budget_s and s < S:
        K, V = synth.memory_blocks(w, seed, [s], range(NB), threads=8)
        ref = O.Store(S, NB + 1, b, H, dh)
        for j in range(NB):
            ref.put(s, j, K[0, j], V[0, j])
        for t in range(len(dec["qs"])):
            if spent >= budget_s:
                break
            p = dec["pos"][t][s]
            t1 = time.perf_counter()
            O.reader_decode(ref, [s], [NB], [p], dec["qs"][t, s:s + 1], dec["kn"][t, s:s + 1],
                            dec["vn"][t, s:s + 1], kc_all[s:s + 1], vc_all[s:s + 1])
            spent += time.perf_counter() - t1
            n_tok += 1
        s += 1
    single = None
    try:
        from threadpoolctl import threadpool_limits
        ref = O.Store(S, NB + 1, b, H, dh)
        K, V = synth.memory_blocks(w, seed, [0], range(NB), threads=8)
        for j in range(NB):
            ref.put(0, j, K[0, j], V[0, j])
        with threadpool_limits(limits=1):
            n1, t1s = 0, 0.0
            while t1s < budget_s / 4 and n1 < len(dec["qs"]):
                p = dec["pos"][n1][0]
                t1 = time.perf_counter()
                O.reader_decode(ref, [0], [NB], [p], dec["qs"][n1, 0:1], dec["kn"][n1, 0:1], dec["vn"][n1, 0:1],
                                kc_all[0:1], vc_all[0:1])
                t1s += time.perf_counter() - t1
                n1 += 1
        single = round(n1 / t1s, 3)
    except Exception:
        pass
    # /proc/cpuinfo's model name as the host reports it (a virtual machine may
    # report a short one), with the family / model / stepping numbers
    cpu_model = ""
    try:
        info = {}
        for l in open("/proc/cpuinfo"):
            if ":" in l:
                k, v = (x.strip() for x in l.split(":", 1))
                info.setdefault(k, v)
            elif info:
                break
        cpu_model = "%s (family %s, model %s, stepping %s, %d logical CPUs)" % (
            info.get("model name", "?"), info.get("cpu family", "?"), info.get("model", "?"),
            info.get("stepping", "?"), os.cpu_count() or 0)
    except Exception:
        pass
    return {"value": round(n_tok / spent, 3), "unit": "tokens/s", "cores": int(blas_threads), "kind": "oracle",
            "sample": f"{n_tok} decode tokens (16 heads each over 4096 memory rows + in-block keys), "
                      f"fp64 numpy, {spent:.1f} s",
            "single_thread_value": single, "affinity_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--workloads", default="encode,serve,stream,rows,stress,delete_sweep,rope,model,model_decode,"
                                           "model_decode_rows,delete_generate",
                    help="secondary workloads to run (comma list of encode, serve, stream, rows, stress, rope: "
                         "the rotary composite timed beside the headline decode and the serve; model: the whole "
                         "model's block-skip serve against its cold prefill; model_decode: the whole model's "
                         "batched KV-cached decode at the paper's cells; model_decode_rows: the same cells with "
                         "the memory kept as rows and every layer reading them through its maps; "
                         "delete_sweep: deletion latency from "
                         "512 to 65,536 cached blocks; delete_generate: the whole model's delete-then-generate "
                         "cycle at 512 and 4096 cached blocks; selfattn, not run by default: the fused "
                         "self-attention kernel against the model's map + attention pair)")
    ap.add_argument("--delete-sizes", default="512,1024,4096,16384,65536")
    ap.add_argument("--delgen-blocks", default="512,4096")
    ap.add_argument("--model-scales", default="160M,410M,1.5B")
    ap.add_argument("--model-lengths", default="1024,2048,4096,8192")
    ap.add_argument("--model-reps", type=int, default=3)
    ap.add_argument("--decode-steps", type=int, default=128)
    ap.add_argument("--decode-warmup", type=int, default=66)
    ap.add_argument("--no-headline", action="store_true",
                    help="profiling runs only: skip the decode headline (value is then null)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="after the headline, copy a MIB-MiB tensor three times (torch's copy kernel, the "
                         "library's register copy and its LDS-DMA copy: known sizes, used to scale hardware "
                         "traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (the path is single-GPU; "
              f"sharding is described, not built).", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_32395_amd import smem, synth
    smem.lib()
    torch.cuda.set_device(0)

    dec = None if args.no_headline else decode_workload(args, torch, smem, synth)
    if args.copy_probe:
        # copies of known size for scaling the traffic counters: torch's copy
        # kernel, the library's 16-byte register copy, and its LDS-DMA copy
        src = torch.ones(args.copy_probe * (1 << 20) // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        smem.smem_device_copy(dst, src, via_lds=False)
        smem.smem_device_copy(dst, src, via_lds=True)
        torch.cuda.synchronize()
        del src, dst
    secondary = {}
    if not args.no_secondary:
        wl = set(args.workloads.split(","))
        if "encode" in wl:
            secondary["encode_prefill_160M"] = encode_prefill_workload(args, torch, smem, synth)
        if "serve" in wl:
            secondary["serve_1p5B"] = serve_workload(args, torch, smem, synth)
        if "stream" in wl:
            secondary["stream_410M"] = stream_workload(args, torch, smem, synth)
        if "rows" in wl:
            secondary["rows_decode_410M"] = rows_workload(args, torch, smem, synth)
        if dec is not None and dec.get("rope"):
            secondary["rope_decode_410M"] = dec["rope"]
        if "stress" in wl:
            secondary["stress_1p5B"] = stress_workload(args, torch, smem, synth)
        if "delete_sweep" in wl:
            secondary["delete_sweep_1p5B_pages"] = delete_sweep_workload(args, torch, smem, synth)
        if "model" in wl:
            secondary["model_block_skip"] = model_workload(args, torch, smem, synth)
        if "model_decode" in wl:
            secondary["model_decode"] = model_decode_workload(args, torch, smem, synth)
        if "model_decode_rows" in wl:
            secondary["model_decode_row_plane"] = model_decode_workload(args, torch, smem, synth, row_plane=True)
        if "delete_generate" in wl:
            secondary["delete_then_generate"] = delete_generate_workload(args, torch, smem, synth)
        if "selfattn" in wl:
            secondary["self_attention_fused_vs_unfused"] = selfattn_workload(args, torch, smem, synth)
    cpu = None
    if dec is None:
        print(json.dumps({"metric": "profiling run (no headline)", "value": None, "secondary": secondary}))
        return
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(dec, args.cpu_budget, args.seed)
    achieved = dec["gbs"]
    line = {
        "metric": "reader decode tokens/s + HBM GB/s; single-block serve ms; encoder attn TFLOP/s",
        "value": round(dec["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dec["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded normals, scale 1/8; random-init, no trained weights)",
        "config": {"workload": "410M-shaped batched decode: 64 seq x 16 heads x dh 64, b=64, 4096 memory rows "
                               "per sequence, one token per sequence per step, 1-64 in-block keys",
                   "global_batch": 64, "memory_rows": 4096, "heads": 16, "head_dim": 64, "block": 64,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic_of("decode"),
                     "kernel": "smem_reader_decode (k_reader_valu + k_merge)",
                     "bytes_per_launch": dec["bytes_per_step"]},
        "hbm_gbs": round(achieved, 1),
        "secondary": secondary,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
