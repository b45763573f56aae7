"""KVarN CPU oracle -- TEST INFRASTRUCTURE ONLY.

Python view of ``kvarn_oracle.c``: a plain fp64 implementation of the KVarN quantize and
decode-attention path (KVarN, arXiv 2606.03458: Sec. 2.1 Eq. 1, Sec. 2.2, Sec. 3.3, App. D,
App. H Algorithm 1).  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it.  It shares no code with the GPU library in
``paper_2606_03458_amd``; neither imports the other.

Parity status of each function (pins are in ``tests/test_oracle_*.py``):
  hadamard128      pinned (scipy.linalg.hadamard, involution, norm preservation)
  varn             pinned (closed-form half steps, K=0, equivariances, convergence, best tracking)
  rtn_group        pinned (brute-force argmin, error bound, endpoints)
  pack / unpack    pinned (hand-derived golden words, round trip)
  quantize_tile    pinned through the above plus the dequantization error bound
  decode / attend  pinned (rotation invariance, special cases, numpy softmax on tiny inputs)
  append           pinned (region bookkeeping against a direct re-quantization)
  e4m3 / fp16      pinned (all E4M3 values enumerated from the format definition, brute-force
                   nearest / upward rounding; numpy's binary16 conversion)
  compact aux      pinned through the conversions, the round trip and the error bound; the
                   tile-wide power-of-two shift between its two scales (a reading of App. D)
                   through its minimality and the bound at large magnitudes
  prefill          pinned (equals appending the same tokens one by one)
  properties       random tiles, layouts and caches (``tests/test_oracle_properties.py``)
  c_min, c_max     parity unpinned: the paper does not give their values.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvarn_oracle.c")
_LIB = os.path.join(_HERE, "libkvarn_oracle.so")

KEYS, VALUES = 0, 1
D = 128
G = 128


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
               "-shared", "-fPIC", "-Wall", "-Wextra", "-o", _LIB + ".tmp", _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class _Params(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("varn_iters", ctypes.c_int32),
                ("c_min", ctypes.c_double), ("c_max", ctypes.c_double),
                ("log_lo", ctypes.c_double), ("log_hi", ctypes.c_double),
                ("imb_floor", ctypes.c_double), ("ddof", ctypes.c_int32), ("aux", ctypes.c_int32),
                ("force_best", ctypes.c_int32), ("rotate", ctypes.c_int32)]


class _Cache(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_kv", ctypes.c_int32), ("max_blocks", ctypes.c_int32),
                ("n_sink", ctypes.c_int32), ("bits", ctypes.c_int32), ("aux", ctypes.c_int32),
                ("rotate", ctypes.c_int32),
                ("k_body", ctypes.c_void_p), ("v_body", ctypes.c_void_p),
                ("k_resid", ctypes.c_void_p), ("v_resid", ctypes.c_void_p),
                ("k_sink", ctypes.c_void_p), ("v_sink", ctypes.c_void_p),
                ("seq_len", ctypes.c_void_p), ("block_table", ctypes.c_void_p), ("n_phys", ctypes.c_int32)]


@dataclass
class Params:
    """Constants of Algorithm 1 plus the RTN bit width.

    log_lo/log_hi = -0.3/10.0 and imb_floor = 1e-8 are printed in Algorithm 1; K = 8 is the
    iteration count of the runtime experiment (Sec. 4.2); c_min/c_max are unstated (unpinned).
    aux selects the stored aux format: 0 = fp32 vectors, 1 = compact (App. D: E4M3 scales,
    binary16 offset).  force_best (test use) keeps iteration k's scales instead of Algorithm 1's
    selection: the outcome had k won a near-tie of Imb.  rotate = 0 drops the Hadamard rotation
    (with varn_iters = 0: KIVI-style RTN; with K > 0: VarN alone, the ablations of Fig. 1).
    """
    bits: int = 2
    varn_iters: int = 8
    c_min: float = 1e-8
    c_max: float = 1e8
    log_lo: float = -0.3
    log_hi: float = 10.0
    imb_floor: float = 1e-8
    ddof: int = 1
    aux: int = 0
    force_best: int = -1
    rotate: int = 1

    def c(self) -> _Params:
        return _Params(self.bits, self.varn_iters, self.c_min, self.c_max, self.log_lo, self.log_hi,
                       self.imb_floor, self.ddof, self.aux, self.force_best, self.rotate)


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        vp = ctypes.c_void_p
        L.kvo_hadamard128.argtypes = [vp]
        L.kvo_imbalance.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double]
        L.kvo_imbalance.restype = ctypes.c_double
        L.kvo_varn.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.POINTER(_Params), vp, vp, vp, vp, vp, vp, vp]
        L.kvo_rtn_group.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, vp, ctypes.c_int, vp, vp, vp,
                                    ctypes.c_int]
        L.kvo_quantize_tile.argtypes = [vp, ctypes.c_int, ctypes.POINTER(_Params), vp, vp, vp, vp, vp, vp, vp, vp,
                                        vp, vp, vp, vp]
        L.kvo_tile_bytes.argtypes = [ctypes.c_int, ctypes.c_int]
        L.kvo_set_threads.argtypes = [ctypes.c_int]
        L.kvo_tile_bytes.restype = ctypes.c_size_t
        L.kvo_pack_tile.argtypes = [vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, vp]
        L.kvo_unpack_tile.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp]
        L.kvo_dequantize_tile.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, vp]
        L.kvo_error_decomposition.argtypes = [vp, vp, ctypes.c_int32, vp, vp, vp]
        L.kvo_e4m3_to_double.argtypes = [ctypes.c_uint8]
        L.kvo_e4m3_to_double.restype = ctypes.c_double
        L.kvo_e4m3_from_double.argtypes = [ctypes.c_double, ctypes.c_int]
        L.kvo_e4m3_from_double.restype = ctypes.c_uint8
        L.kvo_fp16_to_double.argtypes = [ctypes.c_uint16]
        L.kvo_fp16_to_double.restype = ctypes.c_double
        L.kvo_fp16_from_double.argtypes = [ctypes.c_double]
        L.kvo_fp16_from_double.restype = ctypes.c_uint16
        L.kvo_quantize_pack.argtypes = [vp, ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.POINTER(_Params), vp]
        L.kvo_quantize_tiles.argtypes = [vp, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.POINTER(_Params), vp,
                                         ctypes.c_int64, ctypes.c_int64]
        L.kvo_attend.argtypes = [vp, vp, vp, ctypes.c_int32, ctypes.c_double, vp]
        L.kvo_gather_stream.argtypes = [ctypes.POINTER(_Cache), ctypes.c_int32, ctypes.c_int32, vp, vp]
        L.kvo_decode.argtypes = [ctypes.POINTER(_Cache), ctypes.c_int32, vp, ctypes.c_int, ctypes.c_double, vp]
        L.kvo_append.argtypes = [ctypes.POINTER(_Cache), vp, vp, ctypes.POINTER(_Params)]
        L.kvo_append.restype = ctypes.c_int
        L.kvo_prefill.argtypes = [ctypes.POINTER(_Cache), vp, vp, ctypes.c_int, vp, ctypes.c_int32,
                                  ctypes.POINTER(_Params)]
        L.kvo_prefill.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


# --------------------------------------------------------------------------------------------
# Elementary steps
# --------------------------------------------------------------------------------------------

def hadamard128(x) -> np.ndarray:
    """Orthonormal Sylvester Walsh-Hadamard transform of each length-128 row (Sec. 2.2)."""
    y = _f64(x).copy()
    flat = y.reshape(-1, D)
    for i in range(flat.shape[0]):
        lib().kvo_hadamard128(_p(flat[i]))
    return y


def imbalance(X, params: Params = Params()) -> float:
    """Imb(X) of Algorithm 1."""
    X = _f64(X)
    return lib().kvo_imbalance(_p(X), X.shape[0], X.shape[1], params.ddof, params.imb_floor)


@dataclass
class VarNResult:
    Sc: np.ndarray
    Sr: np.ndarray
    B: np.ndarray
    imb: np.ndarray
    Lc: np.ndarray
    Lr: np.ndarray
    best_iter: int


def varn(T, params: Params = Params()) -> VarNResult:
    """Algorithm 1 on one R x C tile (rows = tokens, columns = channels)."""
    T = _f64(T)
    R, C = T.shape
    K = params.varn_iters
    Sc, Sr, B = np.zeros(C), np.zeros(R), np.zeros((R, C))
    imb, Lc, Lr = np.zeros(K + 1), np.zeros((K + 1, C)), np.zeros((K + 1, R))
    best = ctypes.c_int(-1)
    pc = params.c()
    lib().kvo_varn(_p(T), R, C, ctypes.byref(pc), _p(Sc), _p(Sr), _p(B), _p(imb), _p(Lc), _p(Lr),
                   ctypes.cast(ctypes.byref(best), ctypes.c_void_p))
    return VarNResult(Sc, Sr, B, imb, Lc, Lr, best.value)


def rtn_group(x, bits: int):
    """Asymmetric RTN of one group (Sec. 2.1, Eq. 1).  Returns (codes, mn, s, u)."""
    x = _f64(x)
    n = x.shape[0]
    codes = np.zeros(n, dtype=np.uint8)
    u = np.zeros(n)
    mn, s = ctypes.c_double(), ctypes.c_double()
    lib().kvo_rtn_group(_p(x), n, 1, bits, _p(codes), 1, ctypes.cast(ctypes.byref(mn), ctypes.c_void_p),
                        ctypes.cast(ctypes.byref(s), ctypes.c_void_p), _p(u), 1)
    return codes, mn.value, s.value, u


@dataclass
class TileResult:
    codes: np.ndarray  # [128 tokens][128 channels] uint8
    a: np.ndarray      # fp32
    b: np.ndarray
    s2: np.ndarray
    T: np.ndarray      # rotated tile
    B: np.ndarray      # balanced tile
    u: np.ndarray      # unrounded RTN quotients
    Sc: np.ndarray
    Sr: np.ndarray
    imb: np.ndarray
    best_iter: int
    pre: np.ndarray    # [3][128]: a, b, s2 before rounding to the stored format


def quantize_tile(X, kind: int, params: Params = Params()) -> TileResult:
    """Quantize one 128 x 128 token-major tile of keys (kind 0) or values (kind 1)."""
    X = _f64(X)
    assert X.shape == (G, D)
    codes = np.zeros((G, D), dtype=np.uint8)
    a, b, s2 = (np.zeros(128, dtype=np.float32) for _ in range(3))
    T, B, u = np.zeros((G, D)), np.zeros((G, D)), np.zeros((G, D))
    Sc, Sr = np.zeros(D), np.zeros(G)
    imb = np.zeros(params.varn_iters + 1)
    pre = np.zeros((3, 128))
    best = ctypes.c_int(-1)
    pc = params.c()
    lib().kvo_quantize_tile(_p(X), kind, ctypes.byref(pc), _p(codes), _p(a), _p(b), _p(s2), _p(T), _p(B), _p(u),
                            _p(Sc), _p(Sr), _p(imb), ctypes.cast(ctypes.byref(best), ctypes.c_void_p), _p(pre))
    return TileResult(codes, a, b, s2, T, B, u, Sc, Sr, imb, best.value, pre)


def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (timing only; results do not depend on it)."""
    lib().kvo_set_threads(int(n))


def tile_bytes(bits: int, aux: int = 0) -> int:
    return int(lib().kvo_tile_bytes(bits, aux))


def pack_tile(codes, a, b, s2, kind: int, bits: int, aux: int = 0) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    a, b, s2 = (np.ascontiguousarray(v, dtype=np.float32) for v in (a, b, s2))
    out = np.zeros(tile_bytes(bits, aux), dtype=np.uint8)
    lib().kvo_pack_tile(_p(codes), _p(a), _p(b), _p(s2), kind, bits, aux, _p(out))
    return out


def unpack_tile(tile, kind: int, bits: int, aux: int = 0):
    tile = np.ascontiguousarray(tile, dtype=np.uint8)
    codes = np.zeros((G, D), dtype=np.uint8)
    a, b, s2 = (np.zeros(128, dtype=np.float32) for _ in range(3))
    lib().kvo_unpack_tile(_p(tile), kind, bits, aux, _p(codes), _p(a), _p(b), _p(s2))
    return codes, a, b, s2


def dequantize_tile(tile, kind: int, bits: int, aux: int = 0, rotate: int = 1) -> np.ndarray:
    tile = np.ascontiguousarray(tile, dtype=np.uint8)
    X = np.zeros((G, D))
    lib().kvo_dequantize_tile(_p(tile), kind, bits, aux, rotate, _p(X))
    return X


def error_decomposition(K, Kdq):
    """Per-token (E_T, E_M, E_D) of Sec. 3.1 Eq. 3 for rows of 128."""
    K, Kdq = _f64(K).reshape(-1, D), _f64(Kdq).reshape(-1, D)
    n = K.shape[0]
    ET, EM, ED = np.zeros(n), np.zeros(n), np.zeros(n)
    lib().kvo_error_decomposition(_p(K), _p(Kdq), n, _p(ET), _p(EM), _p(ED))
    return ET, EM, ED


def e4m3_decode(v: int) -> float:
    return float(lib().kvo_e4m3_to_double(int(v)))


def e4m3_encode(x: float, round_up: bool = False) -> int:
    return int(lib().kvo_e4m3_from_double(float(x), int(round_up)))


def fp16_decode(h: int) -> float:
    return float(lib().kvo_fp16_to_double(int(h)))


def fp16_encode(x: float) -> int:
    return int(lib().kvo_fp16_from_double(float(x)))


def quantize_tiles(x: np.ndarray, kind: int, params: Params = Params()) -> np.ndarray:
    """Quantize + pack every tile of x: [..., n_tiles*128, 128] (fp32 or bf16-as-uint16).

    Returns packed tiles shaped [..., n_tiles, tile_bytes].
    """
    x = np.ascontiguousarray(x)
    dtype = 0 if x.dtype == np.float32 else 1
    assert x.dtype in (np.float32, np.uint16)
    lead = x.shape[:-2]
    T = x.shape[-2]
    assert T % G == 0 and x.shape[-1] == D
    n_outer = int(np.prod(lead)) if lead else 1
    n_inner = T // G
    tb = tile_bytes(params.bits, params.aux)
    out = np.zeros(lead + (n_inner, tb), dtype=np.uint8)
    pc = params.c()
    lib().kvo_quantize_tiles(_p(x), dtype, n_outer, n_inner, T * D, G * D, D, kind, ctypes.byref(pc), _p(out),
                             n_inner, 1)
    return out


# --------------------------------------------------------------------------------------------
# Cache-level operations
# --------------------------------------------------------------------------------------------

class HostCache:
    """Host copy of the cache in the shared layout (numpy arrays; bf16 held as uint16)."""

    def __init__(self, batch, n_kv, max_blocks, bits=2, n_sink=0, aux=0, rotate=1, n_phys=0):
        """Dense body, or with n_phys > 0 a pool [n_phys][n_kv] of tiles and a block table
        [batch][max_blocks] (filled with -1)."""
        tb = tile_bytes(bits, aux)
        self.batch, self.n_kv, self.max_blocks, self.bits, self.n_sink = batch, n_kv, max_blocks, bits, n_sink
        self.aux, self.rotate, self.n_phys = aux, rotate, n_phys
        shape = (n_phys, n_kv, tb) if n_phys > 0 else (batch, n_kv, max_blocks, tb)
        self.k_body = np.zeros(shape, dtype=np.uint8)
        self.v_body = np.zeros(shape, dtype=np.uint8)
        self.block_table = np.full((batch, max_blocks), -1, dtype=np.int32) if n_phys > 0 else None
        self.k_resid = np.zeros((batch, n_kv, G, D), dtype=np.uint16)
        self.v_resid = np.zeros((batch, n_kv, G, D), dtype=np.uint16)
        self.k_sink = np.zeros((batch, n_kv, max(n_sink, 1), D), dtype=np.uint16)
        self.v_sink = np.zeros((batch, n_kv, max(n_sink, 1), D), dtype=np.uint16)
        self.seq_len = np.zeros(batch, dtype=np.int32)

    def c(self) -> _Cache:
        return _Cache(self.batch, self.n_kv, self.max_blocks, self.n_sink, self.bits, self.aux, self.rotate,
                      self.k_body.ctypes.data, self.v_body.ctypes.data, self.k_resid.ctypes.data,
                      self.v_resid.ctypes.data, self.k_sink.ctypes.data, self.v_sink.ctypes.data,
                      self.seq_len.ctypes.data,
                      self.block_table.ctypes.data if self.block_table is not None else None, self.n_phys)


def gather_stream(cache: HostCache, b: int, kh: int):
    n = int(cache.seq_len[b])
    K, V = np.zeros((max(n, 1), D)), np.zeros((max(n, 1), D))
    cc = cache.c()
    lib().kvo_gather_stream(ctypes.byref(cc), b, kh, _p(K), _p(V))
    return K[:n], V[:n]


def attend(q, K, V, scale: float) -> np.ndarray:
    q, K, V = _f64(q), _f64(K), _f64(V)
    o = np.zeros(D)
    lib().kvo_attend(_p(q), _p(K), _p(V), K.shape[0], scale, _p(o))
    return o


def decode(cache: HostCache, q: np.ndarray, scale: float) -> np.ndarray:
    """Decode attention for q [batch][n_q][128] (fp32 or bf16-as-uint16) -> fp64 output."""
    q = np.ascontiguousarray(q)
    assert q.dtype in (np.float32, np.uint16)
    n_q = q.shape[1]
    out = np.zeros(q.shape, dtype=np.float64)
    cc = cache.c()
    lib().kvo_decode(ctypes.byref(cc), n_q, _p(q), 0 if q.dtype == np.float32 else 1, scale, _p(out))
    return out


def append(cache: HostCache, k_new: np.ndarray, v_new: np.ndarray, params: Params = Params()) -> int:
    """Append one bf16 token per (sequence, kv head); flushes full residuals into the body."""
    assert params.bits == cache.bits and params.aux == cache.aux and params.rotate == cache.rotate
    k_new = np.ascontiguousarray(k_new, dtype=np.uint16)
    v_new = np.ascontiguousarray(v_new, dtype=np.uint16)
    cc = cache.c()
    pc = params.c()
    return lib().kvo_append(ctypes.byref(cc), _p(k_new), _p(v_new), ctypes.byref(pc))


def prefill(cache: HostCache, k: np.ndarray, v: np.ndarray, cu_seqlens, max_len: int,
            params: Params = Params()) -> int:
    """Write whole prompts (rows cu[b] .. cu[b+1]-1 of k, v: [total][n_kv][128] fp32 or
    bf16-as-uint16) into the cache: sink, quantized full groups, residual, seq_len."""
    assert params.bits == cache.bits and params.aux == cache.aux and params.rotate == cache.rotate
    assert k.dtype == v.dtype and k.dtype in (np.float32, np.uint16)
    k, v = np.ascontiguousarray(k), np.ascontiguousarray(v)
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    cc = cache.c()
    pc = params.c()
    return lib().kvo_prefill(ctypes.byref(cc), _p(k), _p(v), 0 if k.dtype == np.float32 else 1, _p(cu), max_len,
                             ctypes.byref(pc))


# --------------------------------------------------------------------------------------------
# bf16 helpers (storage conversions only)
# --------------------------------------------------------------------------------------------

def bf16_bits_to_f64(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round to bf16, nearest-even (through binary32)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)
