"""Comparison helpers for the GPU-vs-oracle parity tests.

Tolerances (fixed before any kernel was run):
  codes    bit-exact, except a mismatch of one level where the oracle's unrounded quotient is
           within 1e-4 (code units) of a rounding tie.  Excused mismatches are counted per
           distinct quotient: equal inputs of a tile share one quotient and one rounding
           decision, so a tie that moves all of them is one tie.  The count must be at most
           1e-4 of all codes (plus one, for samples smaller than 10^4 codes).
  aux      products along both axes, keys a[c]*s2[t], b[c]*s2[t] (values a[t]*s2[c], b[t]*s2[c]):
           relative error <= 1e-5; for b the error is measured against max(|b*s2|, qmax*a*s2).
  best     a tile whose kept VarN iteration differs from the oracle's is compared against the
           oracle's outcome for the GPU's iteration (the oracle's force_best), to the same code
           and aux bars; this is allowed only where the oracle's imbalances of the two
           iterations agree to 1e-5 (a tie at fp32 resolution).  Where the GPU's kept
           iteration is not known (tiles written by a flush), every iteration tied with the
           oracle's is tried.  A tile that meets the bars for none of them is checked against
           the dequantization bound only; at most 1 % of the tiles (at least one) may take
           that route.
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


EXACT_MIDPOINT = 1e-9


def distinct_ties(u: np.ndarray, excused: np.ndarray) -> int:
    """Number of distinct unrounded quotients among the excused code mismatches of a tile that
    count toward the tie cap.  A quotient within 1e-9 of a half-integer (the oracle's fp64
    evaluation is good to ~1e-15 there, the kernel's fp32 one to ~1e-6) is an exact midpoint of
    the data itself -- sparse bf16 rows take few distinct values after the rotation and hit
    them at a rate the data fixes -- where both roundings are correct; such ties stay excused
    (a code one step away) but do not count."""
    if not excused.any():
        return 0
    uu = u[excused]
    return int(np.unique(uu[np.abs(uu - np.floor(uu) - 0.5) > EXACT_MIDPOINT]).size)


def _tile_mismatch(codes, a, b, s2, r, qmax):
    """(hard code mismatches, excused ties counted per distinct quotient, worst aux product
    error) of one tile against the oracle's result r."""
    mism = codes != r.codes
    hard = excused = 0
    if mism.any():
        d = np.abs(codes.astype(int) - r.codes.astype(int))
        tie = np.abs(r.u - np.floor(r.u) - 0.5) < TIE_WINDOW
        hard = int((mism & ~((d == 1) & tie)).sum())
        excused = distinct_ties(r.u, mism & (d == 1) & tie)
    a64, b64, s264 = (v.astype(np.float64) for v in (a, b, s2))
    ra, rb, rs2 = (v.astype(np.float64) for v in (r.a, r.b, r.s2))
    # products along both axes are independent of how a scale is split between the axes
    Pa, Pb, Ra, Rb = np.outer(a64, s264), np.outer(b64, s264), np.outer(ra, rs2), np.outer(rb, rs2)
    ea = np.abs(Pa - Ra) / np.abs(Ra)
    # an offset is a group minimum out of the rotation, a sum of 128 terms: in fp32 its absolute
    # error scales with the tile's magnitude, not with the (possibly cancelled) value itself, so
    # the part of the difference within 2^-20 of the tile's largest rotated value is not counted
    # (as for the compact format's binary16 offsets)
    slack = 2.0 ** -20 * float(np.abs(r.T).max())
    eb = np.maximum(np.abs(Pb - Rb) - slack, 0.0) / np.maximum(np.abs(Rb), qmax * np.abs(Ra))
    return hard, excused, float(max(ea.max(), eb.max()))


def _imb_tied(I, k, k_o) -> bool:
    return abs(I[k] - I[k_o]) <= 1e-5 * abs(I[k_o])


def compare_tiles(gpu_tiles: np.ndarray, X: np.ndarray, kind: int, bits: int, gpu_best=None, params=None,
                  tie_fraction: float = TIE_FRACTION, max_best_ties=None):
    """gpu_tiles [n, tile_bytes] uint8 (GPU output); X [n, 128, 128] float64 (exact input).

    A tile is compared code by code and aux by aux with the oracle's result.  If that fails and
    the GPU kept another VarN iteration whose imbalance ties the oracle's at fp32 resolution,
    it is compared the same way with the oracle's outcome for the GPU's iteration.  Only a tile
    that fails both takes the dequantization-bound route (max_best_ties: default 1 % of the
    tiles, at least one).  Returns a stats dict; raises AssertionError on any violation."""
    params = params or oracle.Params(bits=bits)
    qmax = (1 << bits) - 1
    n = gpu_tiles.shape[0]
    stats = dict(tiles=n, codes=0, excused=0, best_differs=0, forced=0, best_ties=0, max_aux_rel=0.0)
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
                candidates = [int(gpu_best[i])]
                assert _imb_tied(I, candidates[0], k_o), (i, candidates[0], k_o, I)
            else:
                candidates = [k for k in range(len(I)) if k != k_o and _imb_tied(I, k, k_o)]
                assert candidates, (i, hard, aux, k_o, I)
            matched = False
            for k in candidates:
                pf = oracle.Params(**{**params.__dict__, "force_best": k})
                hard, excused, aux = _tile_mismatch(codes, a, b, s2, oracle.quantize_tile(X[i], kind, pf), qmax)
                if not hard and aux <= AUX_RTOL:
                    matched = True
                    break
            if not matched:
                stats["best_ties"] += 1
                _check_dequant_bound(gpu_tiles[i], X[i], kind, bits, params.rotate)
                continue
            stats["forced"] += 1
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


def oracle_cache_from_inputs(built, inputs, appended=(), aux=None) -> "oracle.HostCache":
    """The oracle's own cache of a workload (end-to-end parity): every layer's raw K/V as kept by
    workloads.build(keep_inputs=True) written by the oracle's prefill (its own quantization of
    every body tile), then the tokens of `appended` ([(k, v)] of [batch, n_kv, 128] tensors)
    through the oracle's append path."""
    spec, cache = built.spec, built.cache
    B, n_kv, T = spec["batch"], spec["n_kv"], built.length - len(appended)
    hc = oracle.HostCache(cache.batch, n_kv, cache.max_blocks, bits=cache.bits, n_sink=cache.n_sink,
                          aux=cache.aux if aux is None else aux, rotate=cache.rotate)
    po = oracle.Params(bits=cache.bits, aux=hc.aux, rotate=cache.rotate, varn_iters=built.params.varn_iters)
    k = torch.cat(inputs["K"])  # [L*B, n_kv, T, 128]
    v = torch.cat(inputs["V"])
    conv = (lambda t: t.cpu().numpy()) if k.dtype == torch.float32 else q_to_host
    kh = np.ascontiguousarray(conv(k.permute(0, 2, 1, 3).contiguous()).reshape(-1, n_kv, 128))
    vh = np.ascontiguousarray(conv(v.permute(0, 2, 1, 3).contiguous()).reshape(-1, n_kv, 128))
    cu = np.arange(cache.batch + 1, dtype=np.int32) * T
    assert oracle.prefill(hc, kh, vh, cu, T, po) == 0
    for kt, vt in appended:
        assert oracle.append(hc, q_to_host(kt), q_to_host(vt), po) == 0
    return hc


def _body_tiles(hc, b):
    L = int(hc.seq_len[b])
    return (L - hc.n_sink) // 128 if L > hc.n_sink else 0


def resolve_ties(hc, gc, raw_tile, params=None) -> dict:
    """End-to-end tie rule.  hc is the oracle's own cache, built from the raw tokens; gc a host
    copy of the GPU's cache in the same (dense) layout; raw_tile(b, kh, blk, kind) returns the
    128 x 128 tokens (float64) that both quantized into body tile blk of (sequence b, kv head kh).
    A body tile whose codes equal the oracle's stays as the oracle wrote it (its aux included).
    A tile whose codes differ must pass the tile rules against those tokens (code ties, a VarN
    iteration tied at fp32 resolution, a rounding tie of a compact scale or offset); then, if
    only code ties separate it (same iteration, the oracle's aux kept), the GPU's codes replace
    the oracle's, and otherwise the whole GPU tile does -- so hc becomes the oracle's cache with
    the GPU's tie decisions.  Excused code ties over all compared tiles stay within the 1e-4 cap,
    and at most 1 % of the tiles (at least one) take the dequantization-bound route.  params:
    the quantizer's (default: Algorithm 1's constants with the cache's bits, aux format and
    rotation).  Returns the counts and the set of (b, kh) streams with a replaced tile."""
    bits, aux = hc.bits, hc.aux
    params = params or oracle.Params(bits=bits, aux=aux, rotate=hc.rotate)
    assert params.bits == bits and params.aux == aux and params.rotate == hc.rotate
    cb = bits * 2048
    st = dict(tiles=0, codes=0, excused=0, bound=0, codes_replaced=0, tiles_replaced=0, streams=set())
    for b in range(hc.batch):
        for kh in range(hc.n_kv):
            for blk in range(_body_tiles(hc, b)):
                for kind, ob, gb in ((0, hc.k_body, gc.k_body), (1, hc.v_body, gc.v_body)):
                    st["tiles"] += 1
                    # compact aux values are exact on both sides except at rounding ties, so a
                    # compact tile is compared whole: an s2 tie can leave every code unchanged
                    n_cmp = cb if aux == 0 else ob.shape[-1]
                    if np.array_equal(ob[b, kh, blk, :n_cmp], gb[b, kh, blk, :n_cmp]):
                        st["codes"] += 128 * 128
                        continue
                    X = raw_tile(b, kh, blk, kind)[None]
                    if aux == 0:
                        t = compare_tiles(gb[b, kh, blk][None], X, kind, bits, params=params, tie_fraction=1.0,
                                          max_best_ties=1)
                        bound, whole = t["best_ties"], t["forced"] + t["best_ties"] > 0
                    else:
                        t = compare_tiles_compact(gb[b, kh, blk][None], X, kind, bits, varn_iters=params.varn_iters,
                                                  tie_fraction=1.0, max_ties=1)
                        bound = t["ties"]
                        whole = t["forced"] + t["ties"] > 0 or not np.array_equal(ob[b, kh, blk, cb:], gb[b, kh, blk, cb:])
                    st["codes"] += t["codes"]
                    st["excused"] += t["excused"]
                    st["bound"] += bound
                    st["tiles_replaced" if whole else "codes_replaced"] += 1
                    st["streams"].add((b, kh))
                    if whole:
                        ob[b, kh, blk] = gb[b, kh, blk]
                    else:
                        ob[b, kh, blk, :cb] = gb[b, kh, blk, :cb]
    assert st["excused"] <= TIE_FRACTION * max(st["codes"], 1) + 1, st
    assert st["bound"] <= max(1, st["tiles"] // 100), st
    return st


def check_end_to_end(got: np.ndarray, hc, gc, raw_tile, qh: np.ndarray, bf16_out: bool, scale: float,
                     params=None) -> dict:
    """got [batch][n_q][128]: the GPU's output over its own cache; hc: the oracle's own cache of
    the same tokens (modified: see resolve_ties); gc: host copy of the GPU's cache; qh: the
    queries as given to the GPU.  Every stream must match the oracle's decode of its own cache
    with the GPU's tie decisions, and a stream none of whose tiles needed one must match the
    oracle's decode of its own cache as it was, both to the output bar."""
    ref_raw = oracle.decode(hc, qh, scale)
    st = resolve_ties(hc, gc, raw_tile, params)
    ref = oracle.decode(hc, qh, scale) if st["streams"] else ref_raw
    st["worst"] = check_output(got, ref, bf16_out)
    g = qh.shape[1] // hc.n_kv
    clean = [(b, kh) for b in range(hc.batch) for kh in range(hc.n_kv) if (b, kh) not in st["streams"]]
    if clean:
        sel = lambda a: np.stack([a[b, kh * g:(kh + 1) * g] for b, kh in clean])
        st["worst_untouched"] = check_output(sel(got), sel(ref_raw), bf16_out)
    print("end to end:", {k: (len(v) if k == "streams" else v) for k, v in st.items()}, flush=True)
    return st


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
        # the tile is quantized against the stored s2 (absorb, then round), so a rounding tie of
        # an s2 entry moves the steps, offsets and codes of every group it enters: with s2 ties
        # only, the group steps need no tie of their own
        tie = all(_near_e4m3_boundary(pre_s2[k], False) for k in s2_bad) and \
            (s2_bad.size > 0 or all(_near_e4m3_boundary(r.pre[0][k], True) for k in a_bad))
        tie = tie or _near_shift_tie(r, kind)
        return ("tie" if tie else "mismatch"), 0, 0
    b_bad = np.flatnonzero(b != r.b)
    # the group minimum comes out of the rotation, a sum of 128 terms: in fp32 its absolute
    # error scales with the tile's magnitude, not with the (possibly cancelled) value itself
    slack = 2.0 ** -20 * float(np.abs(r.T).max()) / float(r.s2.astype(np.float64).min()) if b_bad.size else 0.0
    for k in b_bad:
        adjacent = np.nextafter(np.float16(r.b[k]), np.float16(b[k])) == np.float16(b[k])
        # or the binary16 rounding of a minimum within the fp32 bound of the oracle's: where the
        # minimum is a cancelled sum far below the tile's magnitude, that bound spans several
        # binary16 steps
        half = 0.5 * float(np.spacing(np.abs(np.float16(b[k]))))
        within = abs(float(b[k]) - float(r.pre[1][k])) <= slack + half
        if not ((adjacent and _near_fp16_midpoint(r.pre[1][k], slack)) or within):
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
    return "match", distinct_ties(r.u, mism & ~smap), int(b_bad.size)


def compare_tiles_compact(gpu_tiles: np.ndarray, X: np.ndarray, kind: int, bits: int, gpu_best=None,
                          varn_iters: int = 8, max_ties=None, tie_fraction: float = TIE_FRACTION):
    """compare_tiles for the compact aux format (see the comment above for the tie rules).  As
    there, a tile whose kept VarN iteration differs is still compared value by value first."""
    params = oracle.Params(bits=bits, aux=1, varn_iters=varn_iters)
    n = gpu_tiles.shape[0]
    stats = dict(tiles=n, codes=0, excused=0, best_differs=0, forced=0, ties=0, b_steps=0)
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
            stats["forced"] += int(status == "match")
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
                    stats["forced"] += 1
                    break
                if st[0] == "tie":
                    # a tied iteration whose outcome differs only by a format tie: both ties are
                    # allowed, so it is a tie tile (dequantization bound, counted)
                    status = "tie"
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
