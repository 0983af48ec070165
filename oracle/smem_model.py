"""fp64 CPU oracle of the whole SMem model at given (random) weights.

TEST INFRASTRUCTURE ONLY: only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; it imports nothing from
the product path.

The model of Section 2 ("Model") and Appendix A, written plainly in numpy
float64 on top of the attention oracle (smem_oracle):

* input: token embedding plus a learned position embedding indexed by
  (block index) * b + in-block offset, the block index clamped to the last
  trained slot (the clamped slots the paper uses for serving beyond the
  trained length); encoder and reader consume the same embedded input;
* encoder: E pre-LN layers, block-local bidirectional self-attention and a
  GELU feed-forward (hidden 4d); the memory rows of a block are the
  LayerNorm of the encoder's final state;
* reader: D pre-LN layers, each block-local causal self-attention, then
  cross-attention into the memory of strictly earlier blocks with the null
  row (one learned d-vector mapped by each layer's key and value maps), then
  the feed-forward; a final LayerNorm and the output head give the logits.

Readings (the paper is silent): no biases in the linear maps (a linear map
is x -> x W^T with W stored [out, in]); LayerNorm with epsilon 1e-5 and a
learned scale and shift; exact (erf) GELU; heads of width dh = d / H.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import smem_oracle as O

EPS = 1e-5

# weight names in order: the same order the C ABI takes its weight pointers
ENC_NAMES = ["ln1_g", "ln1_b", "w_qkv", "w_o", "ln2_g", "ln2_b", "w_ff1", "w_ff2"]
DEC_NAMES = ["ln1_g", "ln1_b", "w_qkv", "w_o", "ln2_g", "ln2_b", "w_q", "w_k", "w_v", "w_oc",
             "ln3_g", "ln3_b", "w_ff1", "w_ff2"]


def weight_shapes(E, D, d, vocab, n_pos):
    """(name, shape) of every weight, in the C ABI's order."""
    f = 4 * d
    enc = {"ln1_g": (d,), "ln1_b": (d,), "w_qkv": (3 * d, d), "w_o": (d, d), "ln2_g": (d,), "ln2_b": (d,),
           "w_ff1": (f, d), "w_ff2": (d, f)}
    dec = {"ln1_g": (d,), "ln1_b": (d,), "w_qkv": (3 * d, d), "w_o": (d, d), "ln2_g": (d,), "ln2_b": (d,),
           "w_q": (d, d), "w_k": (d, d), "w_v": (d, d), "w_oc": (d, d), "ln3_g": (d,), "ln3_b": (d,),
           "w_ff1": (f, d), "w_ff2": (d, f)}
    out = [("tok_emb", (vocab, d)), ("pos_emb", (max(n_pos, 1), d))]
    for l in range(E):
        out += [(f"enc{l}.{n}", enc[n]) for n in ENC_NAMES]
    out += [("mem_ln_g", (d,)), ("mem_ln_b", (d,)), ("null_row", (d,))]
    for l in range(D):
        out += [(f"dec{l}.{n}", dec[n]) for n in DEC_NAMES]
    out += [("fin_g", (d,)), ("fin_b", (d,)), ("w_head", (vocab, d))]
    return out


def layer_norm(x, g, b):
    x = np.asarray(x, np.float64)
    mu = x.mean(-1, keepdims=True)
    var = ((x - mu) ** 2).mean(-1, keepdims=True)
    return (x - mu) / np.sqrt(var + EPS) * np.asarray(g, np.float64) + np.asarray(b, np.float64)


_erf = np.vectorize(math.erf)


def gelu(x):
    x = np.asarray(x, np.float64)
    return 0.5 * x * (1.0 + _erf(x / math.sqrt(2.0)))


def linear(x, w):
    return np.asarray(x, np.float64) @ np.asarray(w, np.float64).T


class Model:
    """Weights (a dict name -> array) and shape; stores one memory Store per reader layer."""

    def __init__(self, W, E, D, d, H, b, vocab, n_pos, n_seq, max_blocks):
        self.W = {k: np.asarray(v, np.float64) for k, v in W.items()}
        self.E, self.D, self.d, self.H, self.b = E, D, d, H, b
        self.dh = d // H
        self.vocab, self.n_pos = vocab, n_pos
        self.stores = [O.Store(n_seq, max_blocks, b, H, self.dh) for _ in range(D)]

    def copy(self):
        m = Model.__new__(Model)
        m.__dict__.update(self.__dict__)
        m.stores = [s.copy() for s in self.stores]
        return m

    def embed(self, tokens, blocks):
        """tokens [n, b] int, blocks [n] block indices -> [n, b, d]."""
        tokens = np.asarray(tokens)
        n, b = tokens.shape
        x = self.W["tok_emb"][tokens]
        if self.n_pos:
            slots = self.n_pos // b
            pos = np.minimum(np.asarray(blocks)[:, None], slots - 1) * b + np.arange(b)[None, :]
            x = x + self.W["pos_emb"][pos]
        return x

    def _attn_in(self, h, w_qkv):
        n, b, d = h.shape
        qkv = linear(h, w_qkv)
        return [qkv[..., i * d:(i + 1) * d].reshape(n, b, self.H, self.dh) for i in range(3)]

    def memory_rows(self, tokens, blocks):
        """Encoder stack (Section 2, "Model"; Appendix A, "Encoder") -> rows [n, b, d]."""
        x = self.embed(tokens, blocks)
        W = self.W
        for l in range(self.E):
            p = f"enc{l}."
            q, k, v = self._attn_in(layer_norm(x, W[p + "ln1_g"], W[p + "ln1_b"]), W[p + "w_qkv"])
            o = O.encode_blocks(q, k, v, O.MASK_BIDIR).reshape(x.shape)
            x = x + linear(o, W[p + "w_o"])
            h = layer_norm(x, W[p + "ln2_g"], W[p + "ln2_b"])
            x = x + linear(gelu(linear(h, W[p + "w_ff1"])), W[p + "w_ff2"])
        return layer_norm(x, W["mem_ln_g"], W["mem_ln_b"])

    def encode(self, seq, tokens, blocks):
        """Encode blocks and put each reader layer's keys and values (the rows
        through that layer's maps) into its memory."""
        mu = self.memory_rows(tokens, blocks)
        n, b, d = mu.shape
        for l in range(self.D):
            p = f"dec{l}."
            K = linear(mu, self.W[p + "w_k"]).reshape(n, b, self.H, self.dh)
            V = linear(mu, self.W[p + "w_v"]).reshape(n, b, self.H, self.dh)
            for i, j in enumerate(blocks):
                self.stores[l].put(seq, int(j), K[i], V[i])
        return mu

    def null_kv(self, l):
        p = f"dec{l}."
        nr = self.W["null_row"]
        return np.stack([(self.W[p + "w_k"] @ nr).reshape(self.H, self.dh),
                         (self.W[p + "w_v"] @ nr).reshape(self.H, self.dh)])

    def read(self, seq, tokens, blocks):
        """Reader stack (Appendix A, "Reader") for query blocks -> logits [n, b, vocab]."""
        x = self.embed(tokens, blocks)
        n = x.shape[0]
        W = self.W
        for l in range(self.D):
            p = f"dec{l}."
            q, k, v = self._attn_in(layer_norm(x, W[p + "ln1_g"], W[p + "ln1_b"]), W[p + "w_qkv"])
            o = O.encode_blocks(q, k, v, O.MASK_CAUSAL).reshape(x.shape)
            x = x + linear(o, W[p + "w_o"])
            h = layer_norm(x, W[p + "ln2_g"], W[p + "ln2_b"])
            qc = linear(h, W[p + "w_q"]).reshape(n, self.b, self.H, self.dh)
            oc = O.reader_prefill_block(self.stores[l], [seq] * n, list(blocks), qc, None, None, self.null_kv(l))
            x = x + linear(oc.reshape(x.shape), W[p + "w_oc"])
            h = layer_norm(x, W[p + "ln3_g"], W[p + "ln3_b"])
            x = x + linear(gelu(linear(h, W[p + "w_ff1"])), W[p + "w_ff2"])
        return linear(layer_norm(x, W["fin_g"], W["fin_b"]), W["w_head"])

    def delete(self, seq, j):
        for st in self.stores:
            st.delete(seq, j)
