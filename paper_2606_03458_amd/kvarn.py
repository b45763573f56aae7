"""ctypes binding of libkvarn (the HIP library built from ``csrc/``).

Argument marshalling only: torch tensors are passed as device pointers with the current HIP
stream; every step of the hot path runs in the library's kernels.  Loading fails loudly when
the library has not been built -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvarn.so")

KVARN_F32, KVARN_BF16 = 0, 1
KVARN_KEYS, KVARN_VALUES = 0, 1
KVARN_AUX_F32, KVARN_AUX_COMPACT = 0, 1
STATUS = {0: "KVARN_OK", -1: "KVARN_EINVAL", -2: "KVARN_EUNSUPPORTED", -3: "KVARN_ECAPACITY", -4: "KVARN_EHIP",
          -5: "KVARN_EWORKSPACE"}
EXPORTS = ("kvarn_params_init", "kvarn_tile_bytes", "kvarn_cache_sizes", "kvarn_quantize_block", "kvarn_prefill",
           "kvarn_append_token", "kvarn_decode_workspace_bytes", "kvarn_decode_attention",
           "kvarn_decode_attention_noalloc", "kvarn_append_decode")
NOALLOC_SCRATCH_BYTES = 32 << 20  # KVARN_NOALLOC_SCRATCH_BYTES


class KVarNError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} returned {status} ({STATUS.get(status, '?')})")
        self.status = status


class kvarn_params(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("varn_iters", ctypes.c_int32), ("n_sink", ctypes.c_int32),
                ("var_min", ctypes.c_float), ("var_max", ctypes.c_float), ("log_lo", ctypes.c_float),
                ("log_hi", ctypes.c_float), ("aux_format", ctypes.c_int32), ("rotate", ctypes.c_int32)]


class kvarn_cache(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_kv", ctypes.c_int32), ("max_blocks", ctypes.c_int32),
                ("k_body", ctypes.c_void_p), ("v_body", ctypes.c_void_p), ("k_resid", ctypes.c_void_p),
                ("v_resid", ctypes.c_void_p), ("k_sink", ctypes.c_void_p), ("v_sink", ctypes.c_void_p),
                ("seq_len", ctypes.c_void_p), ("err_word", ctypes.c_void_p), ("block_table", ctypes.c_void_p),
                ("n_phys", ctypes.c_int32)]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def lib():
    """Load libkvarn.so (raises if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is not built; run __graft_entry__.build() "
                              "(python paper_2606_03458_amd/build.py) first")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        P, C = ctypes.POINTER(kvarn_params), ctypes.POINTER(kvarn_cache)
        L.kvarn_params_init.argtypes = [P, i32]
        L.kvarn_params_init.restype = ctypes.c_int
        L.kvarn_tile_bytes.argtypes = [P]
        L.kvarn_tile_bytes.restype = sz
        L.kvarn_cache_sizes.argtypes = [P, i32, i32, i32, ctypes.POINTER(sz)]
        L.kvarn_cache_sizes.restype = ctypes.c_int
        L.kvarn_quantize_block.argtypes = [P, i32, vp, i32, i64, i64, i64, i64, i64, vp, i64, i64, vp, vp]
        L.kvarn_quantize_block.restype = ctypes.c_int
        L.kvarn_append_token.argtypes = [P, C, vp, vp, i32, i32, vp]
        L.kvarn_prefill.argtypes = [P, C, vp, vp, i32, vp, i32, vp]
        L.kvarn_prefill.restype = ctypes.c_int
        L.kvarn_append_token.restype = ctypes.c_int
        L.kvarn_decode_workspace_bytes.argtypes = [P, C, i32, i32]
        L.kvarn_decode_workspace_bytes.restype = sz
        L.kvarn_decode_attention.argtypes = [P, C, i32, vp, i32, vp, i32, ctypes.c_float, i32, vp, sz, vp]
        L.kvarn_decode_attention.restype = ctypes.c_int
        L.kvarn_decode_attention_noalloc.argtypes = [P, C, i32, vp, i32, vp, i32, ctypes.c_float, i32, vp]
        L.kvarn_decode_attention_noalloc.restype = ctypes.c_int
        L.kvarn_append_decode.argtypes = [P, C, vp, vp, i32, i32, i32, vp, i32, vp, i32, ctypes.c_float, vp, sz, vp]
        L.kvarn_append_decode.restype = ctypes.c_int
        _lib = L
    return _lib


def _check(fn: str, st: int):
    if st != 0:
        raise KVarNError(fn, st)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    return torch.cuda.current_stream().cuda_stream


def _dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return KVARN_F32
    if t.dtype == torch.bfloat16:
        return KVARN_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


# ------------------------------------------------------------------------------------------
# The C entry points, same names
# ------------------------------------------------------------------------------------------

def kvarn_params_init(bits: int = 2, **overrides) -> kvarn_params:
    p = kvarn_params()
    _check("kvarn_params_init", lib().kvarn_params_init(ctypes.byref(p), bits))
    for k, v in overrides.items():
        setattr(p, k, v)
    return p


def kvarn_tile_bytes(p: kvarn_params) -> int:
    return int(lib().kvarn_tile_bytes(ctypes.byref(p)))


def kvarn_cache_sizes(p: kvarn_params, batch: int, n_kv: int, max_blocks: int) -> list[int]:
    arr = (ctypes.c_size_t * 7)()
    _check("kvarn_cache_sizes", lib().kvarn_cache_sizes(ctypes.byref(p), batch, n_kv, max_blocks, arr))
    return list(arr)


def kvarn_quantize_block(p: kvarn_params, kind: int, x, x_dtype: int, n_outer: int, n_inner: int,
                         x_outer_stride: int, x_inner_stride: int, x_token_stride: int, out,
                         out_outer_stride: int, out_inner_stride: int, best_iter=None, stream=None) -> None:
    st = lib().kvarn_quantize_block(ctypes.byref(p), kind, _ptr(x), x_dtype, n_outer, n_inner, x_outer_stride,
                                    x_inner_stride, x_token_stride, _ptr(out), out_outer_stride, out_inner_stride,
                                    _ptr(best_iter), _stream(stream))
    _check("kvarn_quantize_block", st)


def kvarn_prefill(p: kvarn_params, cache: "Cache", k, v, dtype: int, cu_seqlens, max_len: int, stream=None) -> None:
    d = cache.desc()
    st = lib().kvarn_prefill(ctypes.byref(p), ctypes.byref(d), _ptr(k), _ptr(v), dtype, _ptr(cu_seqlens), max_len,
                             _stream(stream))
    _check("kvarn_prefill", st)


def kvarn_append_token(p: kvarn_params, cache: "Cache", k_new, v_new, dtype: int, host_len_before: int,
                       stream=None) -> None:
    d = cache.desc()
    st = lib().kvarn_append_token(ctypes.byref(p), ctypes.byref(d), _ptr(k_new), _ptr(v_new), dtype,
                                  host_len_before, _stream(stream))
    _check("kvarn_append_token", st)


def kvarn_decode_workspace_bytes(p: kvarn_params, cache: "Cache", n_q: int, max_len_hint: int) -> int:
    d = cache.desc()
    return int(lib().kvarn_decode_workspace_bytes(ctypes.byref(p), ctypes.byref(d), n_q, max_len_hint))


def kvarn_decode_attention(p: kvarn_params, cache: "Cache", n_q: int, q, q_dtype: int, out, out_dtype: int,
                           sm_scale: float, max_len_hint: int, workspace, workspace_bytes: int,
                           stream=None) -> None:
    d = cache.desc()
    st = lib().kvarn_decode_attention(ctypes.byref(p), ctypes.byref(d), n_q, _ptr(q), q_dtype, _ptr(out), out_dtype,
                                      sm_scale, max_len_hint, _ptr(workspace), workspace_bytes, _stream(stream))
    _check("kvarn_decode_attention", st)


def kvarn_decode_attention_noalloc(p: kvarn_params, cache: "Cache", n_q: int, q, q_dtype: int, out, out_dtype: int,
                                   sm_scale: float, max_len_hint: int, stream=None) -> None:
    d = cache.desc()
    st = lib().kvarn_decode_attention_noalloc(ctypes.byref(p), ctypes.byref(d), n_q, _ptr(q), q_dtype, _ptr(out),
                                              out_dtype, sm_scale, max_len_hint, _stream(stream))
    _check("kvarn_decode_attention_noalloc", st)


def kvarn_append_decode(p: kvarn_params, cache: "Cache", k_new, v_new, kv_dtype: int, host_len_before: int, n_q: int,
                        q, q_dtype: int, out, out_dtype: int, sm_scale: float, workspace, workspace_bytes: int,
                        stream=None) -> None:
    d = cache.desc()
    st = lib().kvarn_append_decode(ctypes.byref(p), ctypes.byref(d), _ptr(k_new), _ptr(v_new), kv_dtype, host_len_before,
                                   n_q, _ptr(q), q_dtype, _ptr(out), out_dtype, sm_scale, _ptr(workspace),
                                   workspace_bytes, _stream(stream))
    _check("kvarn_append_decode", st)


# ------------------------------------------------------------------------------------------
# Device buffers of a cache (torch allocates; the library only receives pointers)
# ------------------------------------------------------------------------------------------

class Cache:
    """Caller-owned cache buffers in the layout of kvarn.h, allocated with torch."""

    def __init__(self, p: kvarn_params, batch: int, n_kv: int, max_blocks: int, device="cuda", n_phys: int = 0):
        """Dense body [batch][n_kv][max_blocks] tiles, or, with n_phys > 0, a paged pool
        [n_phys][n_kv] tiles plus a block table [batch][max_blocks] (filled with -1: the
        caller assigns pool blocks)."""
        sizes = kvarn_cache_sizes(p, batch, n_kv, max_blocks)
        self.batch, self.n_kv, self.max_blocks, self.bits, self.n_sink = batch, n_kv, max_blocks, p.bits, p.n_sink
        self.aux, self.rotate, self.n_phys = p.aux_format, p.rotate, n_phys
        tb = kvarn_tile_bytes(p)
        u8 = dict(dtype=torch.uint8, device=device)
        body_shape = (n_phys, n_kv, tb) if n_phys > 0 else (batch, n_kv, max_blocks, tb)
        self.k_body = torch.zeros(body_shape, **u8)
        self.v_body = torch.zeros(body_shape, **u8)
        self.block_table = torch.full((batch, max_blocks), -1, dtype=torch.int32, device=device) if n_phys > 0 else None
        self.k_resid = torch.zeros((batch, n_kv, 128, 128), dtype=torch.bfloat16, device=device)
        self.v_resid = torch.zeros((batch, n_kv, 128, 128), dtype=torch.bfloat16, device=device)
        ns = max(p.n_sink, 0)
        self.k_sink = torch.zeros((batch, n_kv, ns, 128), dtype=torch.bfloat16, device=device) if ns else None
        self.v_sink = torch.zeros((batch, n_kv, ns, 128), dtype=torch.bfloat16, device=device) if ns else None
        self.seq_len = torch.zeros(batch, dtype=torch.int32, device=device)
        self.err_word = torch.zeros(1, dtype=torch.int32, device=device)
        assert (n_phys > 0 or self.k_body.numel() == sizes[0]) and self.k_resid.numel() * 2 == sizes[2]

    def desc(self) -> kvarn_cache:
        return kvarn_cache(self.batch, self.n_kv, self.max_blocks, _ptr(self.k_body), _ptr(self.v_body),
                           _ptr(self.k_resid), _ptr(self.v_resid), _ptr(self.k_sink), _ptr(self.v_sink),
                           _ptr(self.seq_len), _ptr(self.err_word), _ptr(self.block_table), self.n_phys)


def quantize_into_body(p: kvarn_params, kind: int, x: torch.Tensor, body: torch.Tensor, block0: int = 0,
                       best_iter=None, stream=None) -> None:
    """Quantize x [S, T, 128] (T a multiple of 128) into body [S, max_blocks, tile_bytes]
    tiles block0 .. block0 + T/128 - 1 (a prefill).  Marshals strides only."""
    assert x.is_contiguous() and body.is_contiguous()
    S, T, D = x.shape
    assert D == 128 and T % 128 == 0 and body.shape[0] == S
    nb = T // 128
    assert block0 + nb <= body.shape[1]
    out = body[:, block0:]
    kvarn_quantize_block(p, kind, x, _dtype(x), S, nb, T * 128, 128 * 128, 128, out.data_ptr(), body.shape[1], 1,
                         best_iter, stream)
