"""Planted mistakes: each test plants one plausible error in the oracle (on the
CPU, through monkeypatching) and checks that one of the pins in
test_oracle_pins.py fails.  This shows the pins are sharp enough to catch a
dropped term, a wrong index, a transposed operand or a wrong scale."""
import math
import types

import numpy as np
import pytest

from oracle import smem_oracle as O
from tests import test_oracle_pins as P


def _fails(fn, *a, **kw):
    try:
        fn(*a, **kw)
    except (AssertionError, ValueError):
        return True
    return False


class _NumpyProxy(types.ModuleType):
    def __init__(self, **overrides):
        super().__init__("np_proxy")
        self._ov = overrides

    def __getattr__(self, name):
        if name in self.__dict__.get("_ov", {}):
            return self._ov[name]
        return getattr(np, name)


def test_wrong_scale_is_caught(monkeypatch):
    fake = types.SimpleNamespace(sqrt=lambda x: x)   # 1/d_h instead of 1/sqrt(d_h)
    monkeypatch.setattr(O, "math", fake)
    assert _fails(P.check_golden)
    assert _fails(P.test_encoder_matches_sdpa, 16, 4, 32, O.MASK_BIDIR)


def test_causal_without_diagonal_is_caught(monkeypatch):
    monkeypatch.setattr(O, "np", _NumpyProxy(tril=lambda m, k=0: np.tril(m, k - 1)))
    assert _fails(P.check_golden)


def test_reading_own_block_is_caught(monkeypatch):
    orig = O._memory_below
    monkeypatch.setattr(O, "_memory_below", lambda st, s, J: orig(st, s, J + 1))
    assert _fails(P.check_golden)
    assert _fails(P.test_reader_matches_sdpa_over_concatenated_keys, False, True)


def test_dropped_null_row_is_caught(monkeypatch):
    orig = O._reader_keys
    monkeypatch.setattr(O, "_reader_keys", lambda mk, mv, h, nkv, ki, vi, n, dh: orig(mk, mv, h, None, ki, vi, n, dh))
    assert _fails(P.check_golden)
    assert _fails(P.test_reader_matches_sdpa_over_concatenated_keys, True, True)


def test_intra_off_by_one_is_caught(monkeypatch):
    orig = O._reader_keys
    monkeypatch.setattr(O, "_reader_keys", lambda mk, mv, h, nkv, ki, vi, n, dh: orig(mk, mv, h, nkv, ki, vi, n - 1, dh))
    assert _fails(P.check_golden)
    assert _fails(P.test_decode_equals_prefill_row) or _fails(P.test_closed_forms)


def test_transposed_scores_are_caught(monkeypatch):
    def encode_transposed(q, k, v, mask=O.MASK_BIDIR):
        q, k, v = (np.asarray(x, np.float64) for x in (q, k, v))
        nb, b, H, dh = q.shape
        out = np.zeros_like(q)
        for blk in range(nb):
            for h in range(H):
                Q, K, V = q[blk, :, h], k[blk, :, h], v[blk, :, h]
                S = (K @ Q.T) / math.sqrt(dh)          # planted: K Q^T
                if mask == O.MASK_CAUSAL:
                    S = np.where(np.tril(np.ones((b, b), bool)), S, -np.inf)
                E = np.exp(S - S.max(1, keepdims=True))
                out[blk, :, h] = (E / E.sum(1, keepdims=True)) @ V
        return out
    monkeypatch.setattr(O, "encode_blocks", encode_transposed)
    assert _fails(P.check_golden)


def test_unnormalised_softmax_is_caught(monkeypatch):
    def read_bad(q, keys, values, scale):
        keys = np.asarray(keys, np.float64)
        if keys.shape[0] == 0:
            return np.zeros(np.asarray(values).shape[1])
        s = keys @ np.asarray(q, np.float64) * scale
        e = np.exp(s - s.max())
        return (e / (e.sum() + 1.0)) @ np.asarray(values, np.float64)  # planted: extra term
    monkeypatch.setattr(O, "softmax_read", read_bad)
    assert _fails(P.check_golden)


def test_unsorted_store_is_caught(monkeypatch):
    monkeypatch.setattr(O.Store, "live", lambda self, seq: [j for (s, j) in self.rows if s == seq])
    assert _fails(P.test_store_errors_and_canonical_order)
    assert _fails(P.test_edit_path_independence_100_orders)


def test_value_plane_swap_is_caught(monkeypatch):
    orig = O._memory_below

    def swapped(st, s, J):
        k, v = orig(st, s, J)
        return v, k                                    # planted: K and V planes swapped
    monkeypatch.setattr(O, "_memory_below", swapped)
    assert _fails(P.check_golden)


def test_append_before_last_token_is_caught(monkeypatch):
    def stream_early(store, seq_ids, start_block, q, k_new, v_new, q_enc, k_enc, v_enc, null_kv=None,
                     mask=O.MASK_BIDIR):
        q = np.asarray(q, np.float64)
        n, T, H, dh = q.shape
        b = store.b
        out = np.zeros_like(q)
        kc = np.zeros((n, b, H, dh))
        vc = np.zeros((n, b, H, dh))
        for t in range(T):
            p = t % b
            J = [int(start_block[i]) + t // b for i in range(n)]
            if p == b - 1:                               # planted: append before the last token's read
                lo = t - b + 1
                O.encode_into_store(store, seq_ids, J, q_enc[:, lo:t + 1], k_enc[:, lo:t + 1],
                                    v_enc[:, lo:t + 1], mask)
            o, kc, vc = O.reader_decode(store, seq_ids, [j + (p == b - 1) for j in J], [p] * n, q[:, t],
                                        k_new[:, t], v_new[:, t], kc, vc, null_kv)
            out[:, t] = o
        return out
    monkeypatch.setattr(O, "stream_decode", stream_early)
    assert _fails(P.test_stream_decode_equals_prefill_of_each_block)


def test_slot_off_by_one_is_caught(monkeypatch):
    monkeypatch.setattr(O, "slot_indices",
                        lambda n, B: [max(1, j - n + B) if n > B else j + 1 for j in range(n)])
    assert _fails(P.test_slot_scheme)


def test_rope_reversed_rotation_is_caught(monkeypatch):
    orig = O.rope_rotate
    monkeypatch.setattr(O, "rope_rotate", lambda x, phase, base: orig(x, -np.asarray(phase, np.float64), base))
    assert _fails(P.test_rope_rotation_closed_forms)
    assert _fails(P.test_rope_reader_matches_complex_sdpa, None, True)


def test_rope_half_split_pairs_are_caught(monkeypatch):
    orig = O.rope_rotate

    def half_split(x, phase, base):        # planted: pairs (k, k + d/2) instead of (2k, 2k+1)
        x = np.asarray(x, np.float64)
        dh = x.shape[-1]
        perm = np.stack([np.arange(dh // 2), np.arange(dh // 2) + dh // 2], 1).reshape(-1)
        inv = np.argsort(perm)
        return orig(x[..., perm], phase, base)[..., inv]
    monkeypatch.setattr(O, "rope_rotate", half_split)
    assert _fails(P.test_rope_rotation_closed_forms)
    assert _fails(P.test_rope_encoder_matches_complex_sdpa, O.MASK_BIDIR)


def test_rope_clip_off_by_one_is_caught(monkeypatch):
    monkeypatch.setattr(O.Rope, "key_phase",
                        lambda self, j, i: j if self.max_offset is None else max(j, i - self.max_offset - 1))
    assert _fails(P.test_rope_reader_matches_complex_sdpa, 3, True)


def test_rope_unrotated_null_row_is_caught(monkeypatch):
    # planted: the null row read at the query's own phase (no turn) instead of index 0
    monkeypatch.setattr(O, "_rope_read", _rope_read_null_at_query_phase(O._rope_read))
    assert _fails(P.test_rope_reader_matches_complex_sdpa, None, True)


def _rope_read_null_at_query_phase(orig):
    def read(store, seq, i, t, q, h, null_kv, k_in, v_in, n_in, rope, scale):
        if null_kv is None:
            return orig(store, seq, i, t, q, h, null_kv, k_in, v_in, n_in, rope, scale)
        nkv = np.array(null_kv, np.float64, copy=True)
        nkv[0, h] = O.rope_rotate(nkv[0, h], i - rope.key_phase(0, i), rope.base)
        return orig(store, seq, i, t, q, h, nkv, k_in, v_in, n_in, rope, scale)
    return read


def test_rows_swapped_maps_are_caught(monkeypatch):
    orig = O.reader_decode_rows
    monkeypatch.setattr(O, "reader_decode_rows",
                        lambda st, wk, wv, *a, **k: orig(st, wv, wk, *a, **k))   # planted: maps swapped
    assert _fails(P.test_rows_decode_matches_sdpa_on_mapped_rows)


# ---------------------------------------------------------------- whole-model oracle
from oracle import smem_model as MO  # noqa: E402
from tests import test_model_pins as MP  # noqa: E402


def test_model_bidirectional_reader_self_attention_is_caught(monkeypatch):
    orig = O.encode_blocks
    monkeypatch.setattr(O, "encode_blocks", lambda q, k, v, mask=O.MASK_BIDIR: orig(q, k, v, O.MASK_BIDIR))
    assert _fails(MP.test_blockwise_model_equals_masked_dense_pass, 12)


def test_model_memory_without_layer_norm_is_caught(monkeypatch):
    monkeypatch.setattr(MO.Model, "memory_rows", lambda self, tokens, blocks: _rows_no_ln(self, tokens, blocks))
    assert _fails(MP.test_blockwise_model_equals_masked_dense_pass, 12)


def _rows_no_ln(self, tokens, blocks):
    x = self.embed(tokens, blocks)
    W = self.W
    for l in range(self.E):
        p = f"enc{l}."
        q, k, v = self._attn_in(MO.layer_norm(x, W[p + "ln1_g"], W[p + "ln1_b"]), W[p + "w_qkv"])
        x = x + MO.linear(O.encode_blocks(q, k, v, O.MASK_BIDIR).reshape(x.shape), W[p + "w_o"])
        h = MO.layer_norm(x, W[p + "ln2_g"], W[p + "ln2_b"])
        x = x + MO.linear(MO.gelu(MO.linear(h, W[p + "w_ff1"])), W[p + "w_ff2"])
    return x                                        # planted: the memory LayerNorm dropped


def test_model_unclamped_positions_are_caught(monkeypatch):
    def embed(self, tokens, blocks):
        tokens = np.asarray(tokens)
        b = tokens.shape[1]
        pos = (np.asarray(blocks)[:, None] % (self.n_pos // b)) * b + np.arange(b)[None, :]   # planted: wraps
        return self.W["tok_emb"][tokens] + self.W["pos_emb"][pos]
    monkeypatch.setattr(MO.Model, "embed", embed)
    assert _fails(MP.test_blockwise_model_equals_masked_dense_pass, 12)
