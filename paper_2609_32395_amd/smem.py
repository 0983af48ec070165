"""ctypes binding of libsmem.so (the C ABI declared in include/smem.h).

Argument marshalling only: every step of the attention path runs in the HIP
library.  PyTorch provides device memory (tensors, the store's pool) and the
stream.  The binding checks tensor shapes, dtypes, devices and contiguity
before each call, because the C ABI takes bare device pointers and cannot
check buffer sizes itself.

Functions carry the C names: smem_encode_blocks, smem_reencode_blocks,
smem_reader_prefill_block, smem_reader_decode, smem_delete_block,
smem_store_put_block, smem_store_export, and the rotary variants
smem_encode_blocks_rope, smem_reader_prefill_block_rope,
smem_reader_decode_rope, and the row-plane calls smem_rows_put_block,
smem_rows_export, smem_reader_decode_rows; a store is created and destroyed
by the Store class (RowStore for a row store), a rotary table by the Rope
class.
"""
from __future__ import annotations

import ctypes
import os

import torch

F32 = 0
BF16 = 1
MASK_BIDIR = 0
MASK_CAUSAL = 1

SMEM_OK, SMEM_EINVAL, SMEM_ENOMEM, SMEM_ENOENT, SMEM_EEXIST, SMEM_EHIP = range(6)
CODE_NAMES = {0: "OK", 1: "EINVAL", 2: "ENOMEM", 3: "ENOENT", 4: "EEXIST", 5: "EHIP"}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsmem.so")

_TORCH_DTYPE = {F32: torch.float32, BF16: torch.bfloat16}


class SmemError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code
        self.name = CODE_NAMES.get(code, str(code))


class StoreDesc(ctypes.Structure):
    _fields_ = [("n_seq", ctypes.c_int32), ("max_blocks", ctypes.c_int32), ("n_pages", ctypes.c_int32),
                ("b", ctypes.c_int32), ("H", ctypes.c_int32), ("dh", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class AttnDesc(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int32), ("H", ctypes.c_int32), ("dh", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class RowsDesc(ctypes.Structure):
    _fields_ = [("n_seq", ctypes.c_int32), ("max_blocks", ctypes.c_int32), ("n_pages", ctypes.c_int32),
                ("b", ctypes.c_int32), ("d", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class RowsLayer(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int32), ("dh", ctypes.c_int32), ("w_k", ctypes.c_void_p), ("w_v", ctypes.c_void_p),
                ("null_row", ctypes.c_void_p), ("null_kv", ctypes.c_void_p)]


class ModelDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("E", "D", "d", "H", "dh", "b", "vocab", "n_pos", "n_seq", "max_blocks",
                                               "n_pages", "max_tokens", "row_plane")]


class RopeDesc(ctypes.Structure):
    _fields_ = [("dh", ctypes.c_int32), ("n_phases", ctypes.c_int32), ("max_offset", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("base", ctypes.c_double)]


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int32
_IP = ctypes.POINTER(ctypes.c_int32)

# name -> (restype, argtypes); mirrors include/smem.h
SIGNATURES = {
    "smem_store_bytes": (ctypes.c_size_t, [ctypes.POINTER(StoreDesc)]),
    "smem_store_create": (_I, [ctypes.POINTER(StoreDesc), _P, ctypes.c_size_t, _P, ctypes.POINTER(_P)]),
    "smem_store_destroy": (_I, [_P]),
    "smem_store_put_block": (_I, [_P, _I, _I, _P, _P, _P]),
    "smem_store_put_blocks": (_I, [_P, _I, _IP, _IP, _P, _P, _P]),
    "smem_encode_blocks": (_I, [_P, ctypes.POINTER(AttnDesc), _I, _IP, _IP, _P, _P, _P, _P, _I, _P]),
    "smem_reencode_blocks": (_I, [_P, ctypes.POINTER(AttnDesc), _I, _IP, _IP, _P, _P, _P, _P, _I, _P]),
    "smem_reader_prefill_block": (_I, [_P, _I, _IP, _IP, _P, _P, _P, _P, _P, _P]),
    "smem_reader_decode": (_I, [_P, _I, _IP, _IP, _IP, _P, _P, _P, _P, _P, _P, _P, _P]),
    "smem_reader_decode_static": (_I, [_P, _I, _IP, _IP, _IP, _P, _P, _P, _P, _P, _P, _P, _P]),
    "smem_delete_block": (_I, [_P, _I, _I, _I, _P]),
    "smem_store_export": (_I, [_P, _I, _IP, _IP, _P, _P, _P]),
    "smem_rope_bytes": (ctypes.c_size_t, [ctypes.POINTER(RopeDesc)]),
    "smem_rope_create": (_I, [ctypes.POINTER(RopeDesc), _P, ctypes.c_size_t, _P, ctypes.POINTER(_P)]),
    "smem_rope_destroy": (_I, [_P]),
    "smem_encode_blocks_rope": (_I, [_P, ctypes.POINTER(AttnDesc), _P, _I, _IP, _IP, _P, _P, _P, _P, _I, _P]),
    "smem_reader_prefill_block_rope": (_I, [_P, _P, _I, _IP, _IP, _P, _P, _P, _P, _P, _P]),
    "smem_reader_decode_rope": (_I, [_P, _P, _I, _IP, _IP, _IP, _P, _P, _P, _P, _P, _P, _P, _P]),
    "smem_rows_bytes": (ctypes.c_size_t, [ctypes.POINTER(RowsDesc)]),
    "smem_rows_create": (_I, [ctypes.POINTER(RowsDesc), _P, ctypes.c_size_t, _P, ctypes.POINTER(_P)]),
    "smem_rows_put_block": (_I, [_P, _I, _I, _P, _P]),
    "smem_rows_export": (_I, [_P, _I, _IP, _IP, _P, _P]),
    "smem_reader_decode_rows": (_I, [_P, ctypes.POINTER(RowsLayer), _I, _IP, _IP, _IP, _P, _P, _P, _P, _P, _P, _P]),
    "smem_model_n_weights": (_I, [ctypes.POINTER(ModelDesc)]),
    "smem_model_bytes": (ctypes.c_size_t, [ctypes.POINTER(ModelDesc)]),
    "smem_model_create": (_I, [ctypes.POINTER(ModelDesc), ctypes.POINTER(_P), _P, ctypes.c_size_t, _P,
                               ctypes.POINTER(_P)]),
    "smem_model_destroy": (_I, [_P]),
    "smem_model_encode": (_I, [_P, _I, _I, _IP, _P, _P]),
    "smem_model_encode_blocks": (_I, [_P, _I, _IP, _IP, _P, _P]),
    "smem_model_read": (_I, [_P, _I, _I, _IP, _P, _P, _P]),
    "smem_model_prefill": (_I, [_P, _I, _I, _I, _P, _P, _P]),
    "smem_model_decode": (_I, [_P, _I, _I, _IP, _IP, _P, _P, _P]),
    "smem_model_delete_block": (_I, [_P, _I, _I, _P]),
    "smem_linear": (_I, [_I, _I, _I, _P, _P, _P, _P, _I, _P, _P, _P, _P]),
    "smem_self_attention": (_I, [_I, _I, _I, _P, _P, _P, _P, _I, _I, _P, _P, _P]),
    "smem_store_stats": (_I, [_P, _IP, _IP]),
    "smem_device_copy": (_I, [_P, _P, ctypes.c_size_t, _I, _P]),
    "smem_status_string": (ctypes.c_char_p, [_I]),
    "smem_last_error": (ctypes.c_char_p, []),
}


def lib() -> ctypes.CDLL:
    """Load libsmem.so; raise if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_32395_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(code: int):
    if code != SMEM_OK:
        msg = lib().smem_last_error().decode()
        raise SmemError(code, msg)


def check_status(code: int):
    """Raise SmemError for a status returned by a direct call into lib()."""
    _check(code)


def _i32(xs):
    arr = (ctypes.c_int32 * max(1, len(xs)))(*[int(x) for x in xs])
    return arr


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return F32
    if t == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t} (float32 or bfloat16)")


def _dev(t, shape, dtype, name):
    """Check a device tensor argument; return its pointer (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


class Store:
    """A memory-row store over a device pool allocated here with torch.

    meta_only=True creates a store with host metadata only (no device
    memory): edits are validated and recorded, nothing runs on a GPU."""

    def __init__(self, n_seq, max_blocks, n_pages, b, H, dh, dtype=torch.bfloat16, device="cuda",
                 stream=None, meta_only=False):
        self.dtype = dtype
        self.b, self.H, self.dh = b, H, dh
        self.n_seq, self.max_blocks, self.n_pages = n_seq, max_blocks, n_pages
        self.desc = StoreDesc(n_seq, max_blocks, n_pages, b, H, dh, _dtype_code(dtype))
        L = lib()
        nbytes = L.smem_store_bytes(ctypes.byref(self.desc))
        if nbytes == 0:
            raise SmemError(SMEM_EINVAL, "invalid store descriptor")
        self.nbytes = nbytes
        self.pool = None
        handle = ctypes.c_void_p()
        if meta_only:
            _check(L.smem_store_create(ctypes.byref(self.desc), None, 0, None, ctypes.byref(handle)))
        else:
            self.pool = torch.empty(nbytes, dtype=torch.uint8, device=device)
            _check(L.smem_store_create(ctypes.byref(self.desc), ctypes.c_void_p(self.pool.data_ptr()), nbytes,
                                       _stream(stream), ctypes.byref(handle)))
        self.handle = handle
        self.meta_only = meta_only

    # -- lifecycle
    def close(self):
        if getattr(self, "handle", None):
            lib().smem_store_destroy(self.handle)
            self.handle = None
        self.pool = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def row_shape(self):
        return (self.b, self.H, self.dh)

    def stats(self):
        used, free = ctypes.c_int32(), ctypes.c_int32()
        _check(lib().smem_store_stats(self.handle, ctypes.byref(used), ctypes.byref(free)))
        return used.value, free.value


class RowStore(Store):
    """A row store (one plane of b rows of width d per block, bf16), read by
    smem_reader_decode_rows with each layer's key and value maps."""

    def __init__(self, n_seq, max_blocks, n_pages, b, d, device="cuda", stream=None):
        self.dtype = torch.bfloat16
        self.b, self.d = b, d
        self.H, self.dh = 1, 0
        self.n_seq, self.max_blocks, self.n_pages = n_seq, max_blocks, n_pages
        self.desc = RowsDesc(n_seq, max_blocks, n_pages, b, d, BF16)
        L = lib()
        nbytes = L.smem_rows_bytes(ctypes.byref(self.desc))
        if nbytes == 0:
            raise SmemError(SMEM_EINVAL, "invalid row store descriptor")
        self.nbytes = nbytes
        self.pool = torch.empty(nbytes, dtype=torch.uint8, device=device)
        handle = ctypes.c_void_p()
        _check(L.smem_rows_create(ctypes.byref(self.desc), ctypes.c_void_p(self.pool.data_ptr()), nbytes,
                                  _stream(stream), ctypes.byref(handle)))
        self.handle = handle
        self.meta_only = False

    @property
    def row_shape(self):
        return (self.b, self.d)


def smem_rows_put_block(st: RowStore, seq: int, block_idx: int, rows, stream=None):
    rp = _dev(rows, st.row_shape, torch.bfloat16, "rows")
    _check(lib().smem_rows_put_block(st.handle, int(seq), int(block_idx), rp, _stream(stream)))


def smem_rows_export(st: RowStore, seq: int, rows: bool = True, stream=None):
    """(live block indices, rows [n_live*b, d] or None)."""
    L = lib()
    idx = (ctypes.c_int32 * st.max_blocks)()
    n = ctypes.c_int32()
    _check(L.smem_rows_export(st.handle, int(seq), idx, ctypes.byref(n), None, None))
    if not rows:
        return list(idx[: n.value]), None
    R = torch.empty((n.value * st.b, st.d), dtype=torch.bfloat16, device=st.pool.device)
    _check(L.smem_rows_export(st.handle, int(seq), idx, ctypes.byref(n), ctypes.c_void_p(R.data_ptr()),
                              _stream(stream)))
    return list(idx[: n.value]), R


def smem_reader_decode_rows(st: RowStore, w_k, w_v, seq_ids, query_block, pos, q, k_new=None, v_new=None,
                            k_cache=None, v_cache=None, null_row=None, out=None, stream=None, null_kv=None):
    """One layer's reader decode from the row plane: w_k, w_v [H*dh, d]
    (bf16, a linear layer's out x in layout), q etc. [n, H, dh], null_row
    [d] or None; null_kv [2, H, dh]: the null row already through the maps
    (null_row is then ignored)."""
    n, H, dh = q.shape
    if len(seq_ids) != n or len(query_block) != n or (pos is not None and len(pos) != n):
        raise ValueError("seq_ids, query_block and pos need one entry per query")
    bt = torch.bfloat16
    wk = _dev(w_k, (H * dh, st.d), bt, "w_k")
    wv = _dev(w_v, (H * dh, st.d), bt, "w_v")
    nr = _dev(null_row, (st.d,), bt, "null_row")
    nkv = _dev(null_kv, (2, H, dh), bt, "null_kv")
    layer = RowsLayer(H, dh, wk.value, wv.value, nr.value if nr is not None else None,
                      nkv.value if nkv is not None else None)
    tok = (n, H, dh)
    cache = (n * st.b, H, dh)
    if out is None:
        out = torch.empty(tok, dtype=bt, device=q.device)
    args = [_dev(q, tok, bt, "q"), _dev(k_new, tok, bt, "k_new"), _dev(v_new, tok, bt, "v_new"),
            _dev(k_cache, cache, bt, "k_cache"), _dev(v_cache, cache, bt, "v_cache"), _dev(out, tok, bt, "out")]
    pa = _i32(pos) if pos is not None else None
    _check(lib().smem_reader_decode_rows(st.handle, ctypes.byref(layer), n, _i32(seq_ids), _i32(query_block), pa,
                                         *args, _stream(stream)))
    return out


MODEL_ENC = ["ln1_g", "ln1_b", "w_qkv", "w_o", "ln2_g", "ln2_b", "w_ff1", "w_ff2"]
MODEL_DEC = ["ln1_g", "ln1_b", "w_qkv", "w_o", "ln2_g", "ln2_b", "w_q", "w_k", "w_v", "w_oc", "ln3_g", "ln3_b",
             "w_ff1", "w_ff2"]


def model_weight_names(E, D):
    """Weight names in the order smem_model_create takes them."""
    names = ["tok_emb", "pos_emb"]
    for l in range(E):
        names += [f"enc{l}.{n}" for n in MODEL_ENC]
    names += ["mem_ln_g", "mem_ln_b", "null_row"]
    for l in range(D):
        names += [f"dec{l}.{n}" for n in MODEL_DEC]
    return names + ["fin_g", "fin_b", "w_head"]


def model_weight_shapes(E, D, d, vocab, n_pos):
    """(name, shape) of every weight in smem_model_create's order; linear maps
    are [out, in], the feed-forward hidden width is 4d."""
    f = 4 * d
    enc = {"ln1_g": (d,), "ln1_b": (d,), "w_qkv": (3 * d, d), "w_o": (d, d), "ln2_g": (d,), "ln2_b": (d,),
           "w_ff1": (f, d), "w_ff2": (d, f)}
    dec = dict(enc, w_q=(d, d), w_k=(d, d), w_v=(d, d), w_oc=(d, d), ln3_g=(d,), ln3_b=(d,))
    shape = {"tok_emb": (vocab, d), "pos_emb": (max(n_pos, 1), d), "mem_ln_g": (d,), "mem_ln_b": (d,),
             "null_row": (d,), "fin_g": (d,), "fin_b": (d,), "w_head": (vocab, d)}
    out = []
    for nm in model_weight_names(E, D):
        if nm.startswith("enc"):
            out.append((nm, enc[nm.split(".", 1)[1]]))
        elif nm.startswith("dec"):
            out.append((nm, dec[nm.split(".", 1)[1]]))
        else:
            out.append((nm, shape[nm]))
    return out


class Model:
    """The whole model over caller-owned bf16 weights (a dict name -> device
    tensor, names as model_weight_names; pos_emb may be absent when n_pos is
    0).  The pool (the reader layers' stores and the workspace) is allocated
    here with torch."""

    def __init__(self, weights, E, D, d, H, b, vocab, n_pos, n_seq, max_blocks, n_pages, max_tokens=4096,
                 device="cuda", stream=None, row_plane=False):
        self.E, self.D, self.d, self.H, self.b, self.vocab = E, D, d, H, b, vocab
        self.dh = d // H
        self.row_plane = bool(row_plane)
        self.desc = ModelDesc(E, D, d, H, d // H, b, vocab, n_pos, n_seq, max_blocks, n_pages, max_tokens,
                              int(self.row_plane))
        L = lib()
        n = L.smem_model_n_weights(ctypes.byref(self.desc))
        if n == 0:
            raise SmemError(SMEM_EINVAL, "invalid model descriptor")
        names = model_weight_names(E, D)
        assert len(names) == n
        self.weights = weights        # kept alive
        ptrs = (ctypes.c_void_p * n)()
        for i, nm in enumerate(names):
            t = weights.get(nm)
            if t is None:
                if nm == "pos_emb" and n_pos == 0:
                    continue
                raise KeyError(nm)
            if t.dtype != torch.bfloat16 or not t.is_contiguous() or t.device.type != "cuda":
                raise ValueError(f"{nm} must be a contiguous bf16 device tensor")
            ptrs[i] = t.data_ptr()
        nbytes = L.smem_model_bytes(ctypes.byref(self.desc))
        self.pool = torch.empty(nbytes, dtype=torch.uint8, device=device)
        handle = ctypes.c_void_p()
        _check(L.smem_model_create(ctypes.byref(self.desc), ptrs, ctypes.c_void_p(self.pool.data_ptr()), nbytes,
                                   _stream(stream), ctypes.byref(handle)))
        self.handle = handle

    def close(self):
        if getattr(self, "handle", None):
            lib().smem_model_destroy(self.handle)
            self.handle = None
        self.pool = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _tokens(tokens, n_blocks, b):
    if tokens.dtype != torch.int32 or tokens.device.type != "cuda" or not tokens.is_contiguous():
        raise ValueError("tokens must be a contiguous int32 device tensor")
    if tokens.numel() != n_blocks * b:
        raise ValueError(f"tokens has {tokens.numel()} ids, expected {n_blocks * b}")
    return ctypes.c_void_p(tokens.data_ptr())


def smem_model_encode(m: Model, seq: int, block_idx, tokens, stream=None):
    n = len(block_idx)
    _check(lib().smem_model_encode(m.handle, int(seq), n, _i32(block_idx), _tokens(tokens, n, m.b), _stream(stream)))


def smem_model_encode_blocks(m: Model, seq_ids, block_idx, tokens, stream=None):
    n = len(block_idx)
    if len(seq_ids) != n:
        raise ValueError("seq_ids and block_idx differ in length")
    _check(lib().smem_model_encode_blocks(m.handle, n, _i32(seq_ids), _i32(block_idx), _tokens(tokens, n, m.b),
                                          _stream(stream)))


def smem_model_read(m: Model, seq: int, query_block, tokens, logits=None, stream=None):
    """Logits [n*b, vocab] fp32 of the query blocks."""
    n = len(query_block)
    if logits is None:
        logits = torch.empty((n * m.b, m.vocab), dtype=torch.float32, device=tokens.device)
    lp = _dev(logits, (n * m.b, m.vocab), torch.float32, "logits")
    _check(lib().smem_model_read(m.handle, int(seq), n, _i32(query_block), _tokens(tokens, n, m.b), lp,
                                 _stream(stream)))
    return logits


def smem_model_prefill(m: Model, seq: int, first_block: int, n_blocks: int, tokens, logits=None, stream=None):
    """Encode and read blocks first_block .. first_block + n_blocks - 1; logits [b, vocab] of the last."""
    if logits is None:
        logits = torch.empty((m.b, m.vocab), dtype=torch.float32, device=tokens.device)
    lp = _dev(logits, (m.b, m.vocab), torch.float32, "logits")
    _check(lib().smem_model_prefill(m.handle, int(seq), int(first_block), int(n_blocks), _tokens(tokens, n_blocks, m.b),
                                    lp, _stream(stream)))
    return logits


def smem_model_decode(m: Model, first_seq: int, query_block, pos, tokens, logits=None, stream=None):
    """One decode step for sequences first_seq .. first_seq + n - 1; logits [n, vocab]."""
    n = len(query_block)
    if len(pos) != n:
        raise ValueError("query_block and pos differ in length")
    if logits is None:
        logits = torch.empty((n, m.vocab), dtype=torch.float32, device=tokens.device)
    lp = _dev(logits, (n, m.vocab), torch.float32, "logits")
    if tokens.dtype != torch.int32 or tokens.device.type != "cuda" or not tokens.is_contiguous() or tokens.numel() != n:
        raise ValueError("tokens must be a contiguous int32 device tensor of n ids")
    _check(lib().smem_model_decode(m.handle, int(first_seq), n, _i32(query_block), _i32(pos),
                                   ctypes.c_void_p(tokens.data_ptr()), lp, _stream(stream)))
    return logits


LIN_STORE, LIN_GELU, LIN_RESID, LIN_F32 = 0, 1, 2, 3


def smem_linear(x, w, ln_g=None, ln_b=None, epi=LIN_STORE, res=None, y=None, ln_tmp=None, stream=None):
    """One of the model's linear maps: y = epi(LN(x) W^T) (or epi(x W^T)); x [M, K]
    and w [N, K] bf16; y bf16 [M, N], fp32 for epi=LIN_F32."""
    M, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K:
        raise ValueError("w must be [N, K]")
    if y is None:
        y = torch.empty((M, N), dtype=torch.float32 if epi == LIN_F32 else torch.bfloat16, device=x.device)
    if ln_g is not None and M > 128 and ln_tmp is None:
        ln_tmp = torch.empty((M, K), dtype=torch.bfloat16, device=x.device)
    p = lambda t, shape, dt, n: _dev(t, shape, dt, n)
    _check(lib().smem_linear(M, N, K, p(x, (M, K), torch.bfloat16, "x"), p(w, (N, K), torch.bfloat16, "w"),
                             p(ln_g, (K,), torch.bfloat16, "ln_g"), p(ln_b, (K,), torch.bfloat16, "ln_b"), int(epi),
                             p(res, (M, N), torch.bfloat16, "res"),
                             p(y, (M, N), torch.float32 if epi == LIN_F32 else torch.bfloat16, "y"),
                             p(ln_tmp, (M, K), torch.bfloat16, "ln_tmp"), _stream(stream)))
    return y


SA_AUTO, SA_UNFUSED, SA_FUSED = 0, 1, 2


def smem_self_attention(x, ln_g, ln_b, w_qkv, H, mask, path=SA_AUTO, out=None, work=None, stream=None):
    """The attention part of a self-attention sub-layer on the model's kernels:
    per block of 64 rows and head, Attn(q, k, v) with q | k | v = LN(x) W_qkv^T;
    x [n_blocks * 64, d] bf16, w_qkv [3d, d] bf16; returns out [n_blocks * 64, d]."""
    M, d = x.shape
    if M % 64:
        raise ValueError("x rows must be whole blocks of 64")
    if w_qkv.shape != (3 * d, d):
        raise ValueError("w_qkv must be [3d, d]")
    if out is None:
        out = torch.empty((M, d), dtype=torch.bfloat16, device=x.device)
    if work is None:
        work = torch.empty((4, M, d), dtype=torch.bfloat16, device=x.device)
    p = lambda t, shape, n: _dev(t, shape, torch.bfloat16, n)
    _check(lib().smem_self_attention(M // 64, d, int(H), p(x, (M, d), "x"), p(ln_g, (d,), "ln_g"),
                                     p(ln_b, (d,), "ln_b"), p(w_qkv, (3 * d, d), "w_qkv"), int(mask), int(path),
                                     p(out, (M, d), "out"), p(work, (4, M, d), "work"), _stream(stream)))
    return out


def smem_model_delete_block(m: Model, seq: int, block_idx: int, stream=None):
    _check(lib().smem_model_delete_block(m.handle, int(seq), int(block_idx), _stream(stream)))


class Rope:
    """Rotary configuration of the SMem+RoPE composite: a table of
    n_phases phases for heads of width dh in a torch-allocated buffer.
    max_offset = W > 0 clips block phases to max(j, J - W); 0 does not."""

    def __init__(self, dh, n_phases, base=10000.0, max_offset=0, device="cuda", stream=None):
        self.dh, self.n_phases, self.base, self.max_offset = dh, n_phases, float(base), int(max_offset)
        self.desc = RopeDesc(dh, n_phases, int(max_offset), 0, float(base))
        L = lib()
        nbytes = L.smem_rope_bytes(ctypes.byref(self.desc))
        if nbytes == 0:
            raise SmemError(SMEM_EINVAL, "invalid rotary descriptor")
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        handle = ctypes.c_void_p()
        _check(L.smem_rope_create(ctypes.byref(self.desc), ctypes.c_void_p(self.buf.data_ptr()), nbytes,
                                  _stream(stream), ctypes.byref(handle)))
        self.handle = handle

    def close(self):
        if getattr(self, "handle", None):
            lib().smem_rope_destroy(self.handle)
            self.handle = None
        self.buf = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def smem_store_put_block(st: Store, seq: int, block_idx: int, k_rows=None, v_rows=None, stream=None):
    if st.meta_only:
        kp = vp = None
    else:
        kp = _dev(k_rows, st.row_shape, st.dtype, "k_rows")
        vp = _dev(v_rows, st.row_shape, st.dtype, "v_rows")
    _check(lib().smem_store_put_block(st.handle, int(seq), int(block_idx), kp, vp,
                                      None if st.meta_only else _stream(stream)))


def smem_store_put_blocks(st: Store, seq_ids, block_idx, k_rows, v_rows, stream=None):
    """Insert len(seq_ids) blocks at once; k_rows, v_rows [n*b, H, dh]."""
    n = len(seq_ids)
    if len(block_idx) != n:
        raise ValueError("block_idx needs one entry per block")
    shape = (n * st.b, st.H, st.dh)
    kp = _dev(k_rows, shape, st.dtype, "k_rows")
    vp = _dev(v_rows, shape, st.dtype, "v_rows")
    _check(lib().smem_store_put_blocks(st.handle, n, _i32(seq_ids), _i32(block_idx), kp, vp, _stream(stream)))


def smem_device_copy(dst, src, via_lds: bool = False, stream=None):
    """Copy src into dst (device tensors of equal byte size) through registers
    or, via_lds=True, through LDS by DMA (a copy of known size, for
    calibrating hardware traffic counters)."""
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes or not dst.is_contiguous() or not src.is_contiguous():
        raise ValueError("dst and src: contiguous, same byte size")
    _check(lib().smem_device_copy(ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()), nbytes,
                                  int(bool(via_lds)), _stream(stream)))


def smem_delete_block(st: Store, seq: int, block_idx: int, scrub: bool = False, stream=None):
    _check(lib().smem_delete_block(st.handle, int(seq), int(block_idx), int(bool(scrub)),
                                   None if st.meta_only else _stream(stream)))


def smem_store_export(st: Store, seq: int, rows: bool = True, stream=None):
    """Canonical memory of one sequence: (live block indices, K, V) with K, V of
    shape [n_live*b, H, dh] (None when rows=False)."""
    L = lib()
    idx = (ctypes.c_int32 * st.max_blocks)()
    n = ctypes.c_int32()
    if not rows or st.meta_only:
        _check(L.smem_store_export(st.handle, int(seq), idx, ctypes.byref(n), None, None, None))
        return list(idx[: n.value]), None, None
    _check(L.smem_store_export(st.handle, int(seq), None, ctypes.byref(n), None, None, None))
    K = torch.empty((n.value * st.b, st.H, st.dh), dtype=st.dtype, device=st.pool.device)
    V = torch.empty_like(K)
    _check(L.smem_store_export(st.handle, int(seq), idx, ctypes.byref(n), ctypes.c_void_p(K.data_ptr()),
                               ctypes.c_void_p(V.data_ptr()), _stream(stream)))
    return list(idx[: n.value]), K, V


def smem_encode_blocks(st, q, k, v, out=None, seq_ids=None, block_idx=None, mask=MASK_BIDIR, b=None, stream=None):
    """Block-local encoder attention over q, k, v of shape [n_blocks*b, H, dh].

    With a store, block i's output becomes memory block block_idx[i] of
    sequence seq_ids[i].  Returns out (allocated when not given)."""
    return _encode(lib().smem_encode_blocks, st, q, k, v, out, seq_ids, block_idx, mask, b, stream)


def smem_encode_blocks_rope(st, rope: Rope, q, k, v, out=None, seq_ids=None, block_idx=None, mask=MASK_BIDIR,
                            b=None, stream=None):
    """smem_encode_blocks with rotary phases (in-block offsets) on q and k."""
    fn = lib().smem_encode_blocks_rope
    return _encode(lambda h, d, *rest: fn(h, d, rope.handle, *rest), st, q, k, v, out, seq_ids, block_idx, mask,
                   b, stream)


def smem_reencode_blocks(st, q, k, v, out=None, seq_ids=None, block_idx=None, mask=MASK_BIDIR, stream=None):
    """Encode present blocks again from new inputs, overwriting their rows in
    place (the slot scheme's re-encode).  Returns out."""
    if st is None:
        raise ValueError("re-encoding needs a store")
    return _encode(lib().smem_reencode_blocks, st, q, k, v, out, seq_ids, block_idx, mask, None, stream)


def _encode(fn, st, q, k, v, out, seq_ids, block_idx, mask, b, stream):
    if st is not None:
        b = st.b
    if b is None:
        raise ValueError("b is required without a store")
    rows, H, dh = q.shape
    if rows % b:
        raise ValueError(f"q has {rows} rows, not a multiple of b={b}")
    nb = rows // b
    dt = q.dtype
    if out is None:
        out = torch.empty_like(q)
    shape = (rows, H, dh)
    ptrs = [_dev(x, shape, dt, n) for x, n in ((q, "q"), (k, "k"), (v, "v"), (out, "out"))]
    desc = AttnDesc(b, H, dh, _dtype_code(dt))
    if st is not None:
        if seq_ids is None or block_idx is None or len(seq_ids) != nb or len(block_idx) != nb:
            raise ValueError("seq_ids and block_idx need one entry per block")
        sa, ba = _i32(seq_ids), _i32(block_idx)
        h = st.handle
    else:
        sa = ba = None
        h = None
    _check(fn(h, ctypes.byref(desc), nb, sa, ba, *ptrs, int(mask), _stream(stream)))
    return out


def smem_reader_prefill_block(st: Store, seq_ids, query_block, q, k_intra=None, v_intra=None, null_kv=None,
                              out=None, stream=None):
    """Reader attention for whole query blocks; q etc. [n*b, H, dh]."""
    return _prefill(st, None, seq_ids, query_block, q, k_intra, v_intra, null_kv, out, stream)


def smem_reader_prefill_block_rope(st: Store, rope: Rope, seq_ids, query_block, q, k_intra=None, v_intra=None,
                                   null_kv=None, out=None, stream=None):
    """smem_reader_prefill_block with the composite's rotary phases."""
    return _prefill(st, rope, seq_ids, query_block, q, k_intra, v_intra, null_kv, out, stream)


def _prefill(st, rope, seq_ids, query_block, q, k_intra, v_intra, null_kv, out, stream):
    n = len(seq_ids)
    if len(query_block) != n:
        raise ValueError("query_block needs one entry per sequence")
    shape = (n * st.b, st.H, st.dh)
    if out is None:
        out = torch.empty(shape, dtype=st.dtype, device=q.device)
    qp = _dev(q, shape, st.dtype, "q")
    kp = _dev(k_intra, shape, st.dtype, "k_intra")
    vp = _dev(v_intra, shape, st.dtype, "v_intra")
    np_ = _dev(null_kv, (2, st.H, st.dh), st.dtype, "null_kv")
    op = _dev(out, shape, st.dtype, "out")
    rest = (n, _i32(seq_ids), _i32(query_block), qp, kp, vp, np_, op, _stream(stream))
    if rope is None:
        _check(lib().smem_reader_prefill_block(st.handle, *rest))
    else:
        _check(lib().smem_reader_prefill_block_rope(st.handle, rope.handle, *rest))
    return out


def smem_reader_decode(st: Store, seq_ids, query_block, pos, q, k_new=None, v_new=None, k_cache=None,
                       v_cache=None, null_kv=None, out=None, stream=None):
    """Reader attention for one new token per sequence; q etc. [n, H, dh],
    caches [n*b, H, dh] (row pos[i] of sequence row i is written)."""
    return _decode(st, None, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv, out, stream)


def smem_reader_decode_static(st: Store, seq_ids, query_block, pos, q, k_new=None, v_new=None, k_cache=None,
                              v_cache=None, null_kv=None, out=None, stream=None):
    """smem_reader_decode with the split partials in the library's own device
    array instead of the store's workspace (no allocation by the library)."""
    return _decode(st, "static", seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv, out, stream)


def smem_reader_decode_rope(st: Store, rope: Rope, seq_ids, query_block, pos, q, k_new=None, v_new=None,
                            k_cache=None, v_cache=None, null_kv=None, out=None, stream=None):
    """smem_reader_decode with the composite's rotary phases."""
    return _decode(st, rope, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv, out, stream)


def _decode(st, rope, seq_ids, query_block, pos, q, k_new, v_new, k_cache, v_cache, null_kv, out, stream):
    n = len(seq_ids)
    if len(query_block) != n or (pos is not None and len(pos) != n):
        raise ValueError("query_block and pos need one entry per sequence")
    tok = (n, st.H, st.dh)
    cache = (n * st.b, st.H, st.dh)
    if out is None:
        out = torch.empty(tok, dtype=st.dtype, device=q.device)
    args = [_dev(q, tok, st.dtype, "q"), _dev(k_new, tok, st.dtype, "k_new"), _dev(v_new, tok, st.dtype, "v_new"),
            _dev(k_cache, cache, st.dtype, "k_cache"), _dev(v_cache, cache, st.dtype, "v_cache"),
            _dev(null_kv, (2, st.H, st.dh), st.dtype, "null_kv"), _dev(out, tok, st.dtype, "out")]
    pa = _i32(pos) if pos is not None else None
    rest = (n, _i32(seq_ids), _i32(query_block), pa, *args, _stream(stream))
    if rope is None:
        _check(lib().smem_reader_decode(st.handle, *rest))
    elif rope == "static":
        _check(lib().smem_reader_decode_static(st.handle, *rest))
    else:
        _check(lib().smem_reader_decode_rope(st.handle, rope.handle, *rest))
    return out
