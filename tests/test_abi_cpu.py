"""CPU checks of the C ABI: the library loads, exports every symbol the
header declares, sizes stores, and its host-side store logic (error codes,
canonical live lists, page accounting) matches the oracle's store on random
edit sequences.  Nothing here touches a GPU: the edits run on
metadata-only stores."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import smem_oracle as O
from paper_2609_32395_amd import smem

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "smem.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(smem_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["smem_encode_blocks", "smem_reader_prefill_block", "smem_reader_decode", "smem_delete_block",
                     "smem_store_create", "smem_store_destroy", "smem_store_put_block", "smem_store_export",
                     "smem_store_bytes"]:
        assert required in names


def test_library_exports_every_declared_symbol():
    L = smem.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
    assert set(declared_functions()) == set(smem.SIGNATURES), "binding signatures must mirror the header"


def test_status_strings():
    L = smem.lib()
    assert L.smem_status_string(smem.SMEM_ENOENT) == b"SMEM_ENOENT"
    assert L.smem_status_string(smem.SMEM_EEXIST) == b"SMEM_EEXIST"
    assert L.smem_status_string(99) == b"SMEM_UNKNOWN"


def test_store_bytes():
    L = smem.lib()
    d = smem.StoreDesc(2, 8, 10, 64, 16, 128, smem.BF16)
    n = L.smem_store_bytes(ctypes.byref(d))
    assert n >= 10 * 16 * 2 * 64 * 128 * 2
    d2 = smem.StoreDesc(2, 8, 20, 64, 16, 128, smem.BF16)
    assert L.smem_store_bytes(ctypes.byref(d2)) - n == 10 * 16 * 2 * 64 * 128 * 2
    for bad in [(0, 8, 10, 64, 16, 128, 1), (2, 8, 10, 32, 16, 128, 1), (2, 8, 10, 64, 16, 96, 1),
                (2, 8, 10, 64, 0, 128, 1), (2, 8, 10, 64, 16, 128, 7), (2, 0, 10, 64, 16, 128, 1)]:
        assert L.smem_store_bytes(ctypes.byref(smem.StoreDesc(*bad))) == 0


def _expect(code, fn, *a, **k):
    with pytest.raises(smem.SmemError) as e:
        fn(*a, **k)
    assert e.value.code == code, str(e.value)


def test_metadata_store_matches_oracle_on_random_edits():
    rng = np.random.default_rng(0)
    n_seq, max_blocks, n_pages = 3, 12, 20
    st = smem.Store(n_seq, max_blocks, n_pages, 16, 2, 32, meta_only=True)
    ref = O.Store(n_seq, max_blocks, 16, 2, 32)
    zeros = np.zeros((16, 2, 32))
    for step in range(2000):
        s = int(rng.integers(0, n_seq))
        j = int(rng.integers(0, max_blocks))
        op = rng.integers(0, 3)
        if op == 0:
            try:
                ref.put(s, j, zeros, zeros)
                expected = None
            except O.StoreError as e:
                expected = e.code
            if expected is None and len(ref.rows) > n_pages:
                ref.delete(s, j)
                expected = "ENOMEM"
            if expected is None:
                smem.smem_store_put_block(st, s, j)
            else:
                _expect(getattr(smem, "SMEM_" + expected), smem.smem_store_put_block, st, s, j)
        elif op == 1:
            try:
                ref.delete(s, j)
                smem.smem_delete_block(st, s, j)
            except O.StoreError as e:
                _expect(getattr(smem, "SMEM_" + e.code), smem.smem_delete_block, st, s, j)
        else:
            idx, _, _ = smem.smem_store_export(st, s, rows=False)
            assert idx == ref.live(s)
        used, free = st.stats()
        assert used == len(ref.rows) and used + free == n_pages
    for s in range(n_seq):
        assert smem.smem_store_export(st, s, rows=False)[0] == ref.live(s)
    st.close()


def test_argument_errors_without_gpu():
    st = smem.Store(2, 4, 4, 16, 2, 32, meta_only=True)
    _expect(smem.SMEM_EINVAL, smem.smem_store_put_block, st, 2, 0)
    _expect(smem.SMEM_EINVAL, smem.smem_store_put_block, st, 0, 4)
    _expect(smem.SMEM_EINVAL, smem.smem_store_put_block, st, -1, 0)
    _expect(smem.SMEM_ENOENT, smem.smem_delete_block, st, 0, 1)
    smem.smem_store_put_block(st, 1, 3)
    _expect(smem.SMEM_EEXIST, smem.smem_store_put_block, st, 1, 3)
    L = smem.lib()
    # calls that need device memory refuse a metadata-only store before touching a GPU
    desc = smem.AttnDesc(16, 2, 32, smem.F32)
    assert L.smem_encode_blocks(st.handle, ctypes.byref(desc), 1, smem._i32([0]), smem._i32([0]),
                                None, None, None, None, 0, None) == smem.SMEM_EINVAL
    assert L.smem_reader_prefill_block(st.handle, 1, smem._i32([0]), smem._i32([1]),
                                       None, None, None, None, None, None) == smem.SMEM_EINVAL
    assert L.smem_reader_decode(st.handle, 1, smem._i32([0]), smem._i32([1]), smem._i32([0]),
                                None, None, None, None, None, None, None, None) == smem.SMEM_EINVAL
    assert b"metadata-only" in L.smem_last_error()
    # bad encoder shapes are rejected before anything else
    for bad in [(32, 2, 32, 0), (16, 2, 48, 0), (16, 0, 32, 0), (16, 2, 32, 3)]:
        d = smem.AttnDesc(*bad)
        assert L.smem_encode_blocks(None, ctypes.byref(d), 1, None, None, None, None, None, None, 0,
                                    None) == smem.SMEM_EINVAL
    st.close()


def test_store_create_rejects_small_or_misaligned_pool():
    L = smem.lib()
    d = smem.StoreDesc(1, 4, 4, 16, 2, 32, smem.F32)
    need = L.smem_store_bytes(ctypes.byref(d))
    h = ctypes.c_void_p()
    # these checks return before the pool pointer is ever dereferenced
    assert L.smem_store_create(ctypes.byref(d), ctypes.c_void_p(4096), need - 1, None, ctypes.byref(h)) == smem.SMEM_ENOMEM
    assert L.smem_store_create(ctypes.byref(d), ctypes.c_void_p(4096 + 16), need, None, ctypes.byref(h)) == smem.SMEM_EINVAL


def test_rope_bytes_and_invalid_descriptors():
    L = smem.lib()
    d = smem.RopeDesc(128, 100, 15, 0, 1e4)
    assert L.smem_rope_bytes(ctypes.byref(d)) == (100 * 128 * 4 + 255) // 256 * 256
    for bad in [(96, 100, 15, 0, 1e4), (64, 0, 15, 0, 1e4), (64, 10, -1, 0, 1e4), (64, 10, 0, 1, 1e4),
                (64, 10, 0, 0, 1.0), (64, 10, 0, 0, float("nan")), (64, 10, 0, 0, float("inf"))]:
        assert L.smem_rope_bytes(ctypes.byref(smem.RopeDesc(*bad))) == 0, bad
    out = ctypes.c_void_p()
    assert L.smem_rope_create(ctypes.byref(d), None, 1 << 20, None, ctypes.byref(out)) == smem.SMEM_EINVAL
    assert not out.value


def test_model_descriptor_and_weight_list():
    """Host-side model checks: weight count, pool size, descriptor limits,
    and the binding's weight list against the oracle's (the C ABI order)."""
    from oracle import smem_model as MO
    L = smem.lib()
    E, D, d, H, b, vocab, n_pos = 3, 7, 768, 24, 64, 50257, 1024
    desc = smem.ModelDesc(E, D, d, H, d // H, b, vocab, n_pos, 1, 128, 128, 4096)
    assert L.smem_model_n_weights(ctypes.byref(desc)) == len(smem.model_weight_names(E, D)) == 2 + 8 * E + 3 + 14 * D + 3
    assert smem.model_weight_shapes(E, D, d, vocab, n_pos) == MO.weight_shapes(E, D, d, vocab, n_pos)
    sd = smem.StoreDesc(1, 128, 128, b, H, d // H, smem.BF16)
    store = (L.smem_store_bytes(ctypes.byref(sd)) + 255) // 256 * 256
    ws = 6 * 4096 * d * 2 + 4096 * 4 * d * 2 + (D * 2 * d * 2 + 255) // 256 * 256
    cache = D * 2 * 1 * b * d * 2                     # decode caches: [D][2][n_seq][b][d] bf16
    assert L.smem_model_bytes(ctypes.byref(desc)) == D * store + ws + cache
    for field, bad in (("b", 16), ("dh", 48), ("d", 700), ("n_pos", 100), ("max_tokens", 100),
                       ("max_tokens", 129 * 64), ("D", 0), ("vocab", 0)):
        bd = smem.ModelDesc.from_buffer_copy(desc)
        setattr(bd, field, bad)
        assert L.smem_model_n_weights(ctypes.byref(bd)) == 0, field
        assert L.smem_model_bytes(ctypes.byref(bd)) == 0, field
    # row plane: one row store and a one-page store instead of D key/value stores
    rd = smem.ModelDesc.from_buffer_copy(desc)
    rd.row_plane = 1
    rows = (L.smem_rows_bytes(ctypes.byref(smem.RowsDesc(1, 128, 128, b, d, smem.BF16))) + 255) // 256 * 256
    one = (L.smem_store_bytes(ctypes.byref(smem.StoreDesc(1, 1, 1, b, H, d // H, smem.BF16))) + 255) // 256 * 256
    assert rows > 0 and one > 0
    assert L.smem_model_bytes(ctypes.byref(rd)) == rows + one + ws + cache
    for field, bad in (("row_plane", 2), ("d", 1536)):
        bd = smem.ModelDesc.from_buffer_copy(rd)
        setattr(bd, field, bad)
        if field == "d":
            bd.H = bad // 32
        assert L.smem_model_bytes(ctypes.byref(bd)) == 0, field
    out = ctypes.c_void_p()
    assert L.smem_model_create(ctypes.byref(desc), None, None, 0, None, ctypes.byref(out)) == smem.SMEM_EINVAL
