"""Property tests of the oracle (Hypothesis, derandomized): random tiles of several shapes of
structure and magnitude, both bit widths, both tile kinds, both aux formats, with and without
the rotation, and random cache layouts.  Each property follows from the definitions of Sec. 2.1
(RTN, Eq. 1), Sec. 2.2 (Hadamard), Algorithm 1 (VarN's selection rule and clamps), App. D (the
three cache regions and the stored aux) and softmax attention; the expected values are computed
here from independent routines (scipy's Hadamard matrix, numpy's softmax, torch's E4M3 and
numpy's binary16 conversions)."""
import os

import numpy as np
import pytest
import scipy.linalg
import torch
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from tiles import STRUCTURES, make_tile

H = scipy.linalg.hadamard(128).astype(np.float64) / np.sqrt(128.0)
SETTINGS = dict(derandomize=True, database=None, deadline=None, suppress_health_check=[HealthCheck.too_slow])
# KVARN_PROPERTY_SCALE multiplies every example count (a longer run of the same search)
SCALE_EXAMPLES = max(1, int(os.environ.get("KVARN_PROPERTY_SCALE", "1")))


def e4m3_grid(v: np.ndarray) -> np.ndarray:
    return torch.tensor(v, dtype=torch.float64).to(torch.float8_e4m3fn).double().numpy()


tile_cases = st.fixed_dictionaries(dict(
    structure=st.sampled_from(STRUCTURES), seed=st.integers(0, 2 ** 31 - 1),
    log_scale=st.floats(-3.0, 3.5), bits=st.sampled_from([2, 4]), kind=st.sampled_from([0, 1]),
    varn_iters=st.sampled_from([0, 1, 2, 8]), rotate=st.sampled_from([0, 1]), aux=st.sampled_from([0, 1])))


@settings(max_examples=150 * SCALE_EXAMPLES, **SETTINGS)
@given(case=tile_cases)
def test_quantize_tile_properties(case):
    c = case
    if c["aux"] == 1 and c["rotate"] == 0:
        c = dict(c, rotate=1)  # the compact format is defined for the rotated domain
    X = make_tile(c["structure"], c["seed"], c["log_scale"])
    p = oracle.Params(bits=c["bits"], varn_iters=c["varn_iters"], rotate=c["rotate"], aux=c["aux"])
    bits, kind, qmax = c["bits"], c["kind"], (1 << c["bits"]) - 1
    r = oracle.quantize_tile(X, kind, p)
    assert r.codes.max() <= qmax

    # rotation (Sec. 2.2): T = X H per token, with the matrix form of the transform
    T_ref = X @ H.T if c["rotate"] else X
    assert np.allclose(r.T, T_ref, rtol=0, atol=1e-12 * max(np.abs(X).max(), 1e-300))

    # Algorithm 1: the kept iteration has the smallest imbalance, a later one wins a tie
    I = r.imb
    assert len(I) == c["varn_iters"] + 1 and 0 <= r.best_iter <= c["varn_iters"]
    assert I[r.best_iter] == I.min() and np.all(I[r.best_iter + 1:] > I[r.best_iter])
    lo, hi = np.exp(p.log_lo), np.exp(p.log_hi)
    for S in (r.Sc, r.Sr):
        assert np.all(S >= lo * (1 - 1e-12)) and np.all(S <= hi * (1 + 1e-12))
    assert np.allclose(r.B, r.T / r.Sc[None, :] / r.Sr[:, None], rtol=1e-14, atol=0)

    a, b, s2 = (v.astype(np.float64) for v in (r.a, r.b, r.s2))
    q = r.codes.astype(np.float64)
    if kind == 0:
        dq = (q * a[None, :] + b[None, :]) * s2[:, None]
    else:
        dq = (q * a[:, None] + b[:, None]) * s2[None, :]
    if c["aux"] == 0:
        # RTN (Eq. 1) along the group axis of the balanced tile: the group's minimum gets code 0
        # and its maximum code qmax; the error is at most half a step, scaled back
        Bg = r.B.T if kind == 0 else r.B  # [group][element]
        codes_g = r.codes.T if kind == 0 else r.codes
        rng_g = Bg.max(axis=1) - Bg.min(axis=1)
        live = rng_g > 0
        idx = np.arange(128)
        assert np.all(codes_g[idx, Bg.argmin(axis=1)][live] == 0)
        assert np.all(codes_g[idx, Bg.argmax(axis=1)][live] == qmax)
        assert np.all(codes_g[~live] == 0)
        step = np.outer(s2, a) if kind == 0 else np.outer(a, s2)
        big = (np.abs(np.outer(s2, b)) if kind == 0 else np.abs(np.outer(b, s2))) + (qmax + 1) * step
        assert np.all(np.abs(r.T - dq) <= step / 2 * (1 + 1e-6) + 4e-7 * big)
        if c["structure"] == "single_outlier" and not c["rotate"]:
            # two distinct values per group: both are levels, so only fp32 rounding remains
            assert np.allclose(dq, X, rtol=0, atol=1e-6 * np.abs(X).max())
    else:
        # App. D compact aux: E4M3 scales (at most 448), binary16 offsets, codes for stored values
        assert np.array_equal(e4m3_grid(a), a) and np.array_equal(e4m3_grid(s2), s2)
        assert a.max() <= 448.0 and s2.max() <= 448.0 and s2.min() >= 2.0 ** -6
        assert np.array_equal(b.astype(np.float16).astype(np.float64), b)
        mn = r.pre[1]
        if kind == 0:
            tol = (a[None, :] / 2 + np.abs(b - mn)[None, :]) * s2[:, None]
        else:
            tol = (a[:, None] / 2 + np.abs(b - mn)[:, None]) * s2[None, :]
        if r.pre[0].max() <= 448.0:  # the tile lies inside the format's range
            assert np.all(np.abs(r.T - dq) <= tol * (1 + 1e-12) + 1e-12 * np.abs(r.T))
    if c["structure"] == "zeros":
        assert np.all(dq == 0.0)

    # the packed tile holds exactly these values; dequantizing undoes the rotation
    packed = oracle.pack_tile(r.codes, r.a, r.b, r.s2, kind, bits, aux=c["aux"])
    assert packed.size == oracle.tile_bytes(bits, c["aux"])
    c2, a2, b2, s22 = oracle.unpack_tile(packed, kind, bits, aux=c["aux"])
    assert np.array_equal(c2, r.codes) and np.array_equal(a2, r.a) and np.array_equal(b2, r.b)
    assert np.array_equal(s22, r.s2)
    Xd = oracle.dequantize_tile(packed, kind, bits, aux=c["aux"], rotate=c["rotate"])
    expect = dq @ H if c["rotate"] else dq
    assert np.allclose(Xd, expect, rtol=0, atol=1e-12 * max(np.abs(dq).max(), 1e-300))


@settings(max_examples=40 * SCALE_EXAMPLES, **SETTINGS)
@given(bits=st.sampled_from([2, 4]), kind=st.sampled_from([0, 1]), aux=st.sampled_from([0, 1]),
       seed=st.integers(0, 2 ** 31 - 1))
def test_pack_roundtrip_and_coverage(bits, kind, aux, seed):
    """Packing is a bijection of the code region: random codes and aux round-trip exactly, all-ones
    codes set every bit of the code region, and each code occupies `bits` bits of its own."""
    rng = np.random.default_rng(seed)
    qmax = (1 << bits) - 1
    codes = rng.integers(0, qmax + 1, (128, 128)).astype(np.uint8)
    if aux == 0:
        a, b, s2 = (rng.standard_normal(128).astype(np.float32) * np.float32(10.0 ** rng.uniform(-3, 3))
                    for _ in range(3))
    else:
        a = e4m3_grid(np.exp(rng.uniform(np.log(2.0 ** -9), np.log(448.0), 128))).astype(np.float32)
        s2 = e4m3_grid(np.exp(rng.uniform(np.log(2.0 ** -6), np.log(448.0), 128))).astype(np.float32)
        b = (rng.standard_normal(128) * 10.0 ** rng.uniform(-4, 4)).astype(np.float16).astype(np.float32)
    t = oracle.pack_tile(codes, a, b, s2, kind, bits, aux)
    c2, a2, b2, s22 = oracle.unpack_tile(t, kind, bits, aux)
    assert np.array_equal(c2, codes) and np.array_equal(a2, a) and np.array_equal(b2, b)
    assert np.array_equal(s22, s2)
    full = oracle.pack_tile(np.full((128, 128), qmax, np.uint8), a, b, s2, kind, bits, aux)
    assert np.all(full[:bits * 2048] == 0xFF)
    one = np.zeros((128, 128), np.uint8)
    tt, cc = rng.integers(128), rng.integers(128)
    one[tt, cc] = qmax
    bits_set = np.unpackbits(oracle.pack_tile(one, a, b, s2, kind, bits, aux)[:bits * 2048]).sum()
    assert bits_set == bits


# --------------------------------------------------------------------------------------------
# Cache level: random lengths, sink sizes, layouts
# --------------------------------------------------------------------------------------------

def _tokens(rng, total, n_kv):
    x = rng.standard_normal((total, n_kv, 128)) * np.exp(rng.standard_normal((1, n_kv, 128)))
    return oracle.f64_to_bf16_bits(x)


cache_cases = st.fixed_dictionaries(dict(
    bits=st.sampled_from([2, 4]), aux=st.sampled_from([0, 1]), n_sink=st.sampled_from([0, 1, 7, 128]),
    n_kv=st.integers(1, 2), seed=st.integers(0, 2 ** 31 - 1),
    lens=st.lists(st.integers(0, 2 * 128 + 140), min_size=1, max_size=3)))


@settings(max_examples=12 * SCALE_EXAMPLES, **SETTINGS)
@given(case=cache_cases)
def test_prefill_equals_appends_property(case):
    """Writing whole prompts equals appending the same tokens one by one (App. D's regions)."""
    lens, H_, ns = case["lens"], case["n_kv"], case["n_sink"]
    rng = np.random.default_rng(case["seed"])
    B = len(lens)
    MB = max(1, max((L - ns) // 128 for L in lens) + 1)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    K, V = _tokens(rng, int(cu[-1]), H_), _tokens(rng, int(cu[-1]), H_)
    p = oracle.Params(bits=case["bits"], aux=case["aux"])
    mk = lambda: oracle.HostCache(B, H_, MB, bits=case["bits"], n_sink=ns, aux=case["aux"])
    pre = mk()
    assert oracle.prefill(pre, K, V, cu, max(lens), p) == 0
    app = mk()
    for b, L in enumerate(lens):  # one sequence at a time through a one-sequence view
        one = oracle.HostCache(1, H_, MB, bits=case["bits"], n_sink=ns, aux=case["aux"])
        for t in range(L):
            assert oracle.append(one, K[cu[b] + t][None], V[cu[b] + t][None], p) == 0
        for f in ("k_body", "v_body", "k_resid", "v_resid", "k_sink", "v_sink"):
            getattr(app, f)[b] = getattr(one, f)[0]
        app.seq_len[b] = one.seq_len[0]
    np.testing.assert_array_equal(pre.seq_len, lens)
    np.testing.assert_array_equal(app.seq_len, lens)
    for b, L in enumerate(lens):
        nb = (L - ns) // 128 if L > ns else 0
        nr = (L - ns) % 128 if L > ns else 0
        for f in ("k_body", "v_body"):
            np.testing.assert_array_equal(getattr(pre, f)[b, :, :nb], getattr(app, f)[b, :, :nb], err_msg=f)
        for f in ("k_sink", "v_sink"):
            np.testing.assert_array_equal(getattr(pre, f)[b, :, :min(L, ns)], getattr(app, f)[b, :, :min(L, ns)])
        for f in ("k_resid", "v_resid"):
            np.testing.assert_array_equal(getattr(pre, f)[b, :, :nr], getattr(app, f)[b, :, :nr], err_msg=f)


decode_cases = st.fixed_dictionaries(dict(
    bits=st.sampled_from([2, 4]), aux=st.sampled_from([0, 1]), n_sink=st.sampled_from([0, 5, 128]),
    n_kv=st.integers(1, 3), g=st.integers(1, 16), paged=st.booleans(), q_bf16=st.booleans(),
    seed=st.integers(0, 2 ** 31 - 1), lens=st.lists(st.integers(0, 3 * 128 + 140), min_size=1, max_size=3)))


def _stream(hc: oracle.HostCache, b: int, kh: int, which: str) -> np.ndarray:
    """The K or V rows of (sequence b, kv head kh) rebuilt from the three regions: bf16 sink,
    dequantized body tiles in block order (through the block table when paged), bf16 residual."""
    L, ns = int(hc.seq_len[b]), hc.n_sink
    kind = 0 if which == "k" else 1
    parts = [oracle.bf16_bits_to_f64(getattr(hc, which + "_sink")[b, kh, :min(L, ns)])]
    body = getattr(hc, which + "_body")
    nb = (L - ns) // 128 if L > ns else 0
    for blk in range(nb):
        tile = body[hc.block_table[b, blk], kh] if hc.n_phys else body[b, kh, blk]
        parts.append(oracle.dequantize_tile(tile, kind, hc.bits, aux=hc.aux))
    nr = (L - ns) % 128 if L > ns else 0
    parts.append(oracle.bf16_bits_to_f64(getattr(hc, which + "_resid")[b, kh, :nr]))
    return np.concatenate(parts, axis=0)


@settings(max_examples=25 * SCALE_EXAMPLES, **SETTINGS)
@given(case=decode_cases)
def test_decode_is_attention_over_the_dequantized_stream(case):
    """Decode of query head h of sequence b is softmax attention over kv head h // g's stream
    (sink, dequantized body, residual), for dense and paged bodies and either query dtype."""
    lens, nkv, g, ns = case["lens"], case["n_kv"], case["g"], case["n_sink"]
    rng = np.random.default_rng(case["seed"])
    B = len(lens)
    MB = max(1, max((L - ns) // 128 for L in lens) + 1)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    K, V = _tokens(rng, int(cu[-1]), nkv), _tokens(rng, int(cu[-1]), nkv)
    n_phys = B * MB + 2 if case["paged"] else 0
    hc = oracle.HostCache(B, nkv, MB, bits=case["bits"], n_sink=ns, aux=case["aux"], n_phys=n_phys)
    if n_phys:
        hc.block_table[:] = rng.permutation(n_phys)[:B * MB].reshape(B, MB).astype(np.int32)
    assert oracle.prefill(hc, K, V, cu, max(lens), oracle.Params(bits=case["bits"], aux=case["aux"])) == 0
    qf = rng.standard_normal((B, g * nkv, 128)) * 2.0
    q = oracle.f64_to_bf16_bits(qf) if case["q_bf16"] else qf.astype(np.float32)
    qv = oracle.bf16_bits_to_f64(q) if case["q_bf16"] else q.astype(np.float64)
    scale = 1.0 / np.sqrt(128.0)
    out = oracle.decode(hc, q, scale)
    for b in range(B):
        for h in range(g * nkv):
            Ks, Vs = _stream(hc, b, h // g, "k"), _stream(hc, b, h // g, "v")
            if Ks.shape[0] == 0:
                assert np.all(out[b, h] == 0.0)
                continue
            s = scale * (Ks @ qv[b, h])
            w = np.exp(s - s.max())
            ref = (w / w.sum()) @ Vs
            np.testing.assert_allclose(out[b, h], ref, rtol=1e-9, atol=1e-12 * np.abs(Vs).max())
