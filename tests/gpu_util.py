"""Comparison helpers for the GPU-vs-oracle parity tests.

Tolerances (fixed before any kernel was run):
  codes    bit-exact, except a mismatch of one level where the oracle's unrounded quotient is
           within 1e-4 (code units) of a rounding tie; such excused mismatches must be at most
           1e-4 of all codes (plus one, for samples smaller than 10^4 codes).
  aux      products along both axes, keys a[c]*s2[t], b[c]*s2[t] (values a[t]*s2[c], b[t]*s2[c]):
           relative error <= 1e-5; for b the error is measured against max(|b*s2|, qmax*a*s2).
  best     a tile whose kept VarN iteration differs from the oracle's must still meet the
           code and aux bars above, unless the oracle's imbalances of the two iterations agree
           to 1e-5 (a tie at fp32 resolution); then only the dequantization bound is checked
           for that tile, and at most 1 % of the tiles (at least one) may take this route.
           Where the GPU's kept iteration is not known (tiles written by a flush), the route
           is open to a tile whose oracle imbalances have such a tie with the kept one.
  output   per (sequence, query head): ||o - o_ref|| / ||o_ref|| <= 2e-3 and
           max|o - o_ref| <= 2e-3 * max|o_ref| for fp32 output; a bf16 output may add the
           rounding of the stored value, 2^-8 * |o_ref| per element.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle

TIE_WINDOW = 1e-4
TIE_FRACTION = 1e-4
AUX_RTOL = 1e-5
OUT_TOL = 2e-3


def bf16_tensor_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def tiles_to_host(x: torch.Tensor) -> np.ndarray:
    """[..., 128 tokens, 128] tile input exactly as the GPU saw it, in float64."""
    return x.detach().float().cpu().numpy().astype(np.float64)


def _tile_mismatch(codes, a, b, s2, r, qmax):
    """(hard code mismatches, excused mismatches, worst aux product error) of one tile."""
    mism = codes != r.codes
    hard = excused = 0
    if mism.any():
        d = np.abs(codes.astype(int) - r.codes.astype(int))
        tie = np.abs(r.u - np.floor(r.u) - 0.5) < TIE_WINDOW
        hard = int((mism & ~((d == 1) & tie)).sum())
        excused = int(mism.sum()) - hard
    a64, b64, s264 = (v.astype(np.float64) for v in (a, b, s2))
    ra, rb, rs2 = (v.astype(np.float64) for v in (r.a, r.b, r.s2))
    # products along both axes are independent of how a scale is split between the axes
    Pa, Pb, Ra, Rb = np.outer(a64, s264), np.outer(b64, s264), np.outer(ra, rs2), np.outer(rb, rs2)
    ea = np.abs(Pa - Ra) / np.abs(Ra)
    eb = np.abs(Pb - Rb) / np.maximum(np.abs(Rb), qmax * np.abs(Ra))
    return hard, excused, float(max(ea.max(), eb.max()))


def compare_tiles(gpu_tiles: np.ndarray, X: np.ndarray, kind: int, bits: int, gpu_best=None, params=None,
                  tie_fraction: float = TIE_FRACTION, max_best_ties=None):
    """gpu_tiles [n, tile_bytes] uint8 (GPU output); X [n, 128, 128] float64 (exact input).

    A tile whose kept VarN iteration differs from the oracle's is still compared code by
    code; only if that comparison fails and the two iterations' imbalances agree to 1e-5
    (a tie at fp32 resolution) is it checked against the dequantization bound instead.
    max_best_ties bounds such tiles (default: 1 % of the tiles, at least one); degenerate tiles
    (constant rows or columns, where clamped variances make Imb values tie systematically) may
    pass a larger bound.  Returns a stats dict; raises AssertionError on any violation."""
    params = params or oracle.Params(bits=bits)
    qmax = (1 << bits) - 1
    n = gpu_tiles.shape[0]
    stats = dict(tiles=n, codes=0, excused=0, best_differs=0, best_ties=0, max_aux_rel=0.0)
    for i in range(n):
        r = oracle.quantize_tile(X[i], kind, params)
        codes, a, b, s2 = oracle.unpack_tile(gpu_tiles[i], kind, bits)
        hard, excused, aux = _tile_mismatch(codes, a, b, s2, r, qmax)
        differs = gpu_best is not None and int(gpu_best[i]) != r.best_iter
        stats["best_differs"] += int(differs)
        if hard or aux > AUX_RTOL:
            I, k_o = r.imb, r.best_iter
            if gpu_best is not None:
                assert differs, (i, hard, aux)
                k_g = int(gpu_best[i])
                assert abs(I[k_g] - I[k_o]) <= 1e-5 * abs(I[k_o]), (i, k_g, k_o, I)
            else:
                near = [k for k in range(len(I)) if k != k_o and abs(I[k] - I[k_o]) <= 1e-5 * abs(I[k_o])]
                assert near, (i, hard, aux, k_o, I)
            stats["best_ties"] += 1
            _check_dequant_bound(gpu_tiles[i], X[i], kind, bits, params.rotate)
            continue
        stats["codes"] += codes.size
        stats["excused"] += excused
        stats["max_aux_rel"] = max(stats["max_aux_rel"], aux)
    assert stats["excused"] <= tie_fraction * max(stats["codes"], 1) + 1, stats
    assert stats["best_ties"] <= (max(1, n // 100) if max_best_ties is None else max_best_ties), stats
    return stats


def _check_dequant_bound(tile: np.ndarray, X: np.ndarray, kind: int, bits: int, rotate: int = 1):
    """Error of a tile in its stored (rotated) domain within half an RTN step times both scales."""
    codes, a, b, s2 = oracle.unpack_tile(tile, kind, bits)
    Xd = oracle.dequantize_tile(tile, kind, bits, rotate=rotate)
    a, b, s2 = (v.astype(np.float64) for v in (a, b, s2))
    step = np.outer(a, s2) if kind == 1 else np.outer(s2, a)
    Xr = oracle.hadamard128(Xd) if rotate else Xd  # back to the stored domain
    T = oracle.hadamard128(X) if rotate else X
    big = (np.abs(np.outer(b, s2)) if kind == 1 else np.abs(np.outer(s2, b))) + (1 << bits) * step
    assert np.all(np.abs(T - Xr) <= step / 2 + 1e-5 * big)


def host_cache(cache, bits=None) -> "oracle.HostCache":
    """Copy a GPU cache (paper_2606_03458_amd.kvarn.Cache) to an oracle host cache."""
    hc = oracle.HostCache(cache.batch, cache.n_kv, cache.max_blocks, bits=bits or cache.bits, n_sink=cache.n_sink,
                          aux=cache.aux, rotate=cache.rotate)
    hc.k_body[:] = cache.k_body.cpu().numpy()
    hc.v_body[:] = cache.v_body.cpu().numpy()
    hc.k_resid[:] = cache.k_resid.view(torch.int16).cpu().numpy().view(np.uint16)
    hc.v_resid[:] = cache.v_resid.view(torch.int16).cpu().numpy().view(np.uint16)
    if cache.n_sink:
        hc.k_sink[:] = cache.k_sink.view(torch.int16).cpu().numpy().view(np.uint16)
        hc.v_sink[:] = cache.v_sink.view(torch.int16).cpu().numpy().view(np.uint16)
    hc.seq_len[:] = cache.seq_len.cpu().numpy()
    return hc


def q_to_host(q: torch.Tensor) -> np.ndarray:
    if q.dtype == torch.float32:
        return q.cpu().numpy()
    return q.view(torch.int16).cpu().numpy().view(np.uint16)


def check_output(got: np.ndarray, ref: np.ndarray, bf16_out: bool, tol: float = OUT_TOL):
    """got, ref: [..., 128].  Returns the worst normwise relative error."""
    got = got.reshape(-1, 128).astype(np.float64)
    ref = ref.reshape(-1, 128)
    worst = 0.0
    for r in range(ref.shape[0]):
        nr = np.linalg.norm(ref[r])
        if nr == 0.0:
            assert np.all(got[r] == 0.0), r
            continue
        err = got[r] - ref[r]
        slack = 2.0 ** -8 * np.abs(ref[r]) if bf16_out else 0.0
        assert np.all(np.abs(err) <= tol * np.abs(ref[r]).max() + slack), (r, np.abs(err).max())
        rel = np.linalg.norm(np.maximum(np.abs(err) - slack, 0.0)) / nr
        assert rel <= tol, (r, rel)
        worst = max(worst, float(np.linalg.norm(err) / nr))
    return worst


def host_streams(cache, streams) -> "oracle.HostCache":
    """Copy the (sequence, kv head) streams listed in `streams` of a GPU cache to an oracle host
    cache with one kv head per sequence (stream i of the list becomes sequence i)."""
    hc = oracle.HostCache(len(streams), 1, cache.max_blocks, bits=cache.bits, n_sink=cache.n_sink, aux=cache.aux,
                          rotate=cache.rotate)
    lens = cache.seq_len.cpu().numpy()
    for i, (b, kh) in enumerate(streams):
        hc.k_body[i, 0] = cache.k_body[b, kh].cpu().numpy()
        hc.v_body[i, 0] = cache.v_body[b, kh].cpu().numpy()
        hc.k_resid[i, 0] = cache.k_resid[b, kh].view(torch.int16).cpu().numpy().view(np.uint16)
        hc.v_resid[i, 0] = cache.v_resid[b, kh].view(torch.int16).cpu().numpy().view(np.uint16)
        if cache.n_sink:
            hc.k_sink[i, 0] = cache.k_sink[b, kh].view(torch.int16).cpu().numpy().view(np.uint16)
            hc.v_sink[i, 0] = cache.v_sink[b, kh].view(torch.int16).cpu().numpy().view(np.uint16)
        hc.seq_len[i] = lens[b]
    return hc


# ---- compact aux (binary16 b, E4M3 a and s2) ------------------------------------------------
# The stored values are roundings of fp32 (GPU) and fp64 (oracle) quantities that agree to about
# 1e-7; they can only differ where the oracle's unrounded value lies within FORMAT_TIE (relative)
# of a rounding boundary of the narrow format.  Such an E4M3 scale tie changes the codes of a
# whole row or group, so the tile takes the dequantization-bound route (at most 1 % of tiles,
# as for VarN iteration ties); a binary16 offset tie may move b by one step, which widens the
# code tie window of that group by the shift |db| / a.  The tile-wide power of two moved into
# s2 is an integer decided by comparisons with 448; a tile near such a threshold may take the
# other value (all of s2, a and b then differ by that power of two) and takes the bound route.
FORMAT_TIE = 1e-5
_E4M3 = None


def _e4m3_values() -> np.ndarray:
    global _E4M3
    if _E4M3 is None:
        v = torch.arange(128, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
        _E4M3 = np.unique(v[np.isfinite(v)])
    return _E4M3


def _near_e4m3_boundary(x: float, upward: bool) -> bool:
    vals = _e4m3_values()
    bounds = vals if upward else (vals[1:] + vals[:-1]) / 2
    return bool(np.min(np.abs(bounds - x)) <= FORMAT_TIE * abs(x))


def _near_fp16_midpoint(x: float, slack: float = 0.0) -> bool:
    h = np.float16(x)
    up, dn = np.nextafter(h, np.float16(np.inf)), np.nextafter(h, np.float16(-np.inf))
    mids = [(float(h) + float(up)) / 2, (float(h) + float(dn)) / 2]
    return min(abs(m - x) for m in mids) <= FORMAT_TIE * abs(x) + slack


def _near_shift_tie(r, kind) -> bool:
    """The tile-wide power of two moved into s2 was decided near one of its thresholds: the
    largest step times 2^-j near 448, or the largest other-axis scale times 2^(j+1) near 448."""
    so = (r.Sr if kind == 0 else r.Sc).astype(np.float64)
    e = int(round(np.log2(r.pre[2][0] / so[0])))
    m0 = float(np.max(r.pre[0])) * 2.0 ** e
    near = lambda x: abs(x / 448.0 - 1.0) <= FORMAT_TIE
    return any(near(m0 * 2.0 ** -j) or near(so.max() * 2.0 ** (j + 1)) for j in range(e + 1))


def _compact_tile_status(codes, a, b, s2, r, kind):
    """("match", excused codes, b steps) if the tile meets the bar, ("tie", ...) if it differs
    only where a format tie allows, ("mismatch", ...) otherwise."""
    s2_bad, a_bad = np.flatnonzero(s2 != r.s2), np.flatnonzero(a != r.a)
    if s2_bad.size or a_bad.size:
        pre_s2 = np.clip(r.pre[2], 2.0 ** -6, 448.0)
        tie = all(_near_e4m3_boundary(pre_s2[k], False) for k in s2_bad) and \
            all(_near_e4m3_boundary(r.pre[0][k], True) for k in a_bad)
        tie = tie or _near_shift_tie(r, kind)
        return ("tie" if tie else "mismatch"), 0, 0
    b_bad = np.flatnonzero(b != r.b)
    # the group minimum comes out of the rotation, a sum of 128 terms: in fp32 its absolute
    # error scales with the tile's magnitude, not with the (possibly cancelled) value itself
    slack = 2.0 ** -20 * float(np.abs(r.T).max()) / float(r.s2.astype(np.float64).min()) if b_bad.size else 0.0
    for k in b_bad:
        adjacent = np.nextafter(np.float16(r.b[k]), np.float16(b[k])) == np.float16(b[k])
        if not (adjacent and _near_fp16_midpoint(r.pre[1][k], slack)):
            return "mismatch", 0, 0
    mism = codes != r.codes
    if not mism.any():
        return "match", 0, int(b_bad.size)
    win = TIE_WINDOW + np.abs(b.astype(np.float64) - r.b) / r.a.astype(np.float64)  # per group
    wmap = win[None, :] if kind == 0 else win[:, None]
    d = np.abs(codes.astype(int) - r.codes.astype(int))
    tie = np.abs(r.u - np.floor(r.u) - 0.5) < wmap
    if (mism & ~((d == 1) & tie)).any():
        return "mismatch", 0, 0
    # codes of a group whose offset took the other side of a binary16 tie moved with it (the
    # widened window above checks them); only the others count as rounding ties of the codes
    shifted = np.zeros(128, dtype=bool)
    shifted[b_bad] = True
    smap = shifted[None, :] if kind == 0 else shifted[:, None]
    return "match", int((mism & ~smap).sum()), int(b_bad.size)


def compare_tiles_compact(gpu_tiles: np.ndarray, X: np.ndarray, kind: int, bits: int, gpu_best=None,
                          varn_iters: int = 8, max_ties=None, tie_fraction: float = TIE_FRACTION):
    """compare_tiles for the compact aux format (see the comment above for the tie rules).  As
    there, a tile whose kept VarN iteration differs is still compared value by value first."""
    params = oracle.Params(bits=bits, aux=1, varn_iters=varn_iters)
    n = gpu_tiles.shape[0]
    stats = dict(tiles=n, codes=0, excused=0, best_differs=0, ties=0, b_steps=0)
    for i in range(n):
        r = oracle.quantize_tile(X[i], kind, params)
        codes, a, b, s2 = oracle.unpack_tile(gpu_tiles[i], kind, bits, aux=1)
        differs = gpu_best is not None and int(gpu_best[i]) != r.best_iter
        stats["best_differs"] += int(differs)
        status, excused, b_steps = _compact_tile_status(codes, a, b, s2, r, kind)
        if status != "match" and differs:
            # a near-tie of Imb: compare against the oracle's outcome for the GPU's iteration
            I, k_g, k_o = r.imb, int(gpu_best[i]), r.best_iter
            assert abs(I[k_g] - I[k_o]) <= 1e-5 * abs(I[k_o]), (i, k_g, k_o, I)
            r = oracle.quantize_tile(X[i], kind, oracle.Params(bits=bits, aux=1, varn_iters=varn_iters, force_best=k_g))
            status, excused, b_steps = _compact_tile_status(codes, a, b, s2, r, kind)
            differs = False
        elif status != "match" and gpu_best is None:
            # kept iteration unknown (flush output): try every iteration tied with the oracle's
            I, k_o = r.imb, r.best_iter
            for k in range(len(I)):
                if k == k_o or abs(I[k] - I[k_o]) > 1e-5 * abs(I[k_o]):
                    continue
                rk = oracle.quantize_tile(X[i], kind, oracle.Params(bits=bits, aux=1, varn_iters=varn_iters, force_best=k))
                st = _compact_tile_status(codes, a, b, s2, rk, kind)
                if st[0] == "match":
                    status, excused, b_steps = st
                    break
        if status == "match":
            stats["codes"] += codes.size
            stats["excused"] += excused
            stats["b_steps"] += b_steps
            continue
        if differs:
            I, k_g, k_o = r.imb, int(gpu_best[i]), r.best_iter
            assert abs(I[k_g] - I[k_o]) <= 1e-5 * abs(I[k_o]), (i, status, k_g, k_o, I)
        else:
            assert status == "tie", (i, status)
        stats["ties"] += 1
        _check_dequant_bound_compact(gpu_tiles[i], X[i], kind, bits)
    assert stats["excused"] <= tie_fraction * max(stats["codes"], 1) + 1, stats
    assert stats["ties"] <= (max(1, n // 100) if max_ties is None else max_ties), stats
    return stats


def _check_dequant_bound_compact(tile: np.ndarray, X: np.ndarray, kind: int, bits: int):
    """Rotated-domain error within the stored step's half plus the offset rounding, times s2."""
    codes, a, b, s2 = (v.astype(np.float64) if v.dtype != np.uint8 else v for v in
                       oracle.unpack_tile(tile, kind, bits, aux=1))
    T = oracle.hadamard128(X)
    if kind == 0:
        dq = (codes * a[None, :] + b[None, :]) * s2[:, None]
        tol = (a[None, :] / 2 + 2.0 ** -11 * np.abs(b[None, :]) + 2.0 ** -24) * s2[:, None]
    else:
        dq = (codes * a[:, None] + b[:, None]) * s2[None, :]
        tol = (a[:, None] / 2 + 2.0 ** -11 * np.abs(b[:, None]) + 2.0 ** -24) * s2[None, :]
    assert np.all(np.abs(T - dq) <= tol * (1 + 1e-5) + 1e-6 * np.abs(T)), np.max(np.abs(T - dq) - tol)
