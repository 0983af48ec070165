"""Pins of the whole-model oracle (oracle/smem_model.py) against things
other than itself:

* the elementary maps against torch's CPU float64 routines (layer_norm,
  gelu, linear);
* an independent whole-sequence formulation written here with torch: every
  attention over the full token sequence with an explicit mask (block-diagonal
  bidirectional for the encoder, block-diagonal causal for the reader's
  self-attention, block-causal over all memory rows plus the null row for
  its cross-attention) -- the masked-dense form the paper's block-local
  operators are exactly equal to (Proposition 1);
* block-skip serving equals the full reader pass (Section 3.1), deletion
  equals never-encoded (Theorem 1), and nothing leaks from masked tokens.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import smem_model as MO

SHAPE = dict(E=1, D=2, d=32, H=2, b=4, vocab=50, n_pos=12)


def random_weights(g, E, D, d, vocab, n_pos, **_):
    W = {}
    for name, shape in MO.weight_shapes(E, D, d, vocab, n_pos):
        if name.endswith("_g"):
            W[name] = 1.0 + 0.1 * g.standard_normal(shape)
        elif name.endswith("_b"):
            W[name] = 0.1 * g.standard_normal(shape)
        elif name in ("tok_emb", "pos_emb", "null_row"):
            W[name] = g.standard_normal(shape)
        else:
            W[name] = g.standard_normal(shape) / math.sqrt(shape[1])
    return W


def make(seed=3, n_seq=1, max_blocks=8, **over):
    s = dict(SHAPE, **over)
    g = np.random.default_rng(seed)
    W = random_weights(g, **s)
    m = MO.Model(W, s["E"], s["D"], s["d"], s["H"], s["b"], s["vocab"], s["n_pos"], n_seq, max_blocks)
    return m, g


def test_elementary_maps_match_torch():
    g = np.random.default_rng(1)
    x = g.standard_normal((5, 7, 16))
    gm, bt = g.standard_normal(16), g.standard_normal(16)
    T = lambda a: torch.as_tensor(a)
    np.testing.assert_allclose(MO.layer_norm(x, gm, bt),
                               F.layer_norm(T(x), (16,), T(gm), T(bt), eps=MO.EPS).numpy(), atol=1e-12)
    np.testing.assert_allclose(MO.gelu(x), F.gelu(T(x), approximate="none").numpy(), atol=1e-14)
    w = g.standard_normal((9, 16))
    np.testing.assert_allclose(MO.linear(x, w), F.linear(T(x), T(w)).numpy(), atol=1e-12)


def _torch_full_pass(m, tokens):
    """The model over a whole sequence of B blocks with dense masked attention (torch, float64)."""
    W = {k: torch.as_tensor(v) for k, v in m.W.items()}
    B, b = tokens.shape
    n, d, H, dh = B * b, m.d, m.H, m.dh
    blk = torch.arange(n) // b
    off = torch.arange(n) % b
    x = W["tok_emb"][torch.as_tensor(tokens).reshape(-1)]
    if m.n_pos:
        x = x + W["pos_emb"][torch.clamp(blk, max=m.n_pos // b - 1) * b + off]
    ln = lambda t, p: F.layer_norm(t, (d,), W[p + "_g"], W[p + "_b"], eps=MO.EPS)
    heads = lambda t: t.reshape(n, H, dh).transpose(0, 1)          # [H, n, dh]
    same = blk[:, None] == blk[None, :]
    causal = off[:, None] >= off[None, :]

    def attend(q, k, v, mask):
        return F.scaled_dot_product_attention(heads(q), heads(k), heads(v), attn_mask=mask).transpose(0, 1).reshape(n, d)
    h = x
    for l in range(m.E):
        p = f"enc{l}."
        q, k, v = F.linear(ln(h, p + "ln1"), W[p + "w_qkv"]).split(d, dim=-1)
        h = h + F.linear(attend(q, k, v, same), W[p + "w_o"])
        h = h + F.linear(F.gelu(F.linear(ln(h, p + "ln2"), W[p + "w_ff1"])), W[p + "w_ff2"])
    mu = ln(h, "mem_ln")
    nr = W["null_row"]
    for l in range(m.D):
        p = f"dec{l}."
        q, k, v = F.linear(ln(x, p + "ln1"), W[p + "w_qkv"]).split(d, dim=-1)
        x = x + F.linear(attend(q, k, v, same & causal), W[p + "w_o"])
        qc = F.linear(ln(x, p + "ln2"), W[p + "w_q"])
        kc = torch.cat([F.linear(nr[None], W[p + "w_k"]), F.linear(mu, W[p + "w_k"])])
        vc = torch.cat([F.linear(nr[None], W[p + "w_v"]), F.linear(mu, W[p + "w_v"])])
        vis = torch.cat([torch.ones(n, 1, dtype=torch.bool), blk[None, :] < blk[:, None]], 1)   # null + earlier blocks
        oc = F.scaled_dot_product_attention(qc.reshape(n, H, dh).transpose(0, 1),
                                            kc.reshape(n + 1, H, dh).transpose(0, 1),
                                            vc.reshape(n + 1, H, dh).transpose(0, 1), attn_mask=vis)
        x = x + F.linear(oc.transpose(0, 1).reshape(n, d), W[p + "w_oc"])
        x = x + F.linear(F.gelu(F.linear(ln(x, p + "ln3"), W[p + "w_ff1"])), W[p + "w_ff2"])
    return F.linear(ln(x, "fin"), W["w_head"]).reshape(B, b, -1).numpy()


@pytest.mark.parametrize("n_pos", [12, 0])
def test_blockwise_model_equals_masked_dense_pass(n_pos):
    m, g = make(n_pos=n_pos)
    B = 5                          # one block past the position table (clamped slot)
    tokens = g.integers(0, m.vocab, size=(B, m.b))
    m.encode(0, tokens, list(range(B)))
    logits = m.read(0, tokens, list(range(B)))
    np.testing.assert_allclose(logits, _torch_full_pass(m, tokens), atol=1e-10, rtol=0)


def test_block_skip_serve_equals_full_reader_pass():
    m, g = make()
    B = 5
    tokens = g.integers(0, m.vocab, size=(B, m.b))
    m.encode(0, tokens[:B - 1], list(range(B - 1)))
    skip = m.read(0, tokens[B - 1:], [B - 1])
    full = m.read(0, tokens, list(range(B)))
    np.testing.assert_allclose(skip[0], full[B - 1], atol=1e-12, rtol=0)


def test_delete_equals_never_encoded_and_no_leak():
    m, g = make()
    B = 5
    tokens = g.integers(0, m.vocab, size=(B, m.b))
    a = m.copy()
    a.encode(0, tokens[:B - 1], list(range(B - 1)))
    a.delete(0, 2)
    c = m.copy()
    c.encode(0, tokens[[0, 1, 3]], [0, 1, 3])
    assert np.array_equal(a.read(0, tokens[B - 1:], [B - 1]), c.read(0, tokens[B - 1:], [B - 1]))
    # tokens after position t of the query block, and blocks >= the query block, change nothing up to t
    base = c.read(0, tokens[1:2], [1])
    t = 1
    tok2 = tokens.copy()
    tok2[1, t + 1:] = (tok2[1, t + 1:] + 7) % m.vocab
    alt = c.copy()
    alt.encode(0, tok2[4:5], [4])                  # a later block in memory: not read by block 1
    np.testing.assert_array_equal(alt.read(0, tok2[1:2], [1])[0, :t + 1], base[0, :t + 1])
