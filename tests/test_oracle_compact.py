"""Pins of the compact aux format (App. D "Effective memory overhead": per group of 128 values,
both scales in an 8-bit float format and the zero point in a 16-bit one): the narrow-format
conversions against independent library implementations (torch's float8_e4m3fn for OCP E4M3,
numpy's float16 for binary16), brute force over the E4M3 value set, the code choice given the
stored aux, the stated error bound, the packed round trip and the paper's printed 2.25
bits/element."""
import os

import numpy as np
import pytest
import torch

import oracle
from tiles import tile as make_tile

E4M3_ALL = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
E4M3_POS = np.array(sorted({v for v in E4M3_ALL[:127] if np.isfinite(v) and v > 0}))


def test_e4m3_decode_matches_library():
    for v in range(256):
        ref = E4M3_ALL[v]
        got = oracle.e4m3_decode(v)
        if np.isnan(ref):
            continue  # the NaN patterns are never produced (encoding saturates)
        assert got == ref, (v, got, ref)


def test_e4m3_nearest_matches_library():
    rng = np.random.default_rng(0)
    xs = np.concatenate([np.exp(rng.uniform(np.log(1e-4), np.log(460.0), 20000)), E4M3_POS,
                         (E4M3_POS[1:] + E4M3_POS[:-1]) / 2])  # every tie between neighbours
    xs = xs[xs < 464.0]
    ref = torch.tensor(xs, dtype=torch.float64).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = np.array([oracle.e4m3_encode(x) for x in xs], dtype=np.uint8)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, [(xs[i], got[i], ref[i]) for i in bad[:5]]


def test_e4m3_upward_is_smallest_value_not_below():
    rng = np.random.default_rng(1)
    xs = np.concatenate([np.exp(rng.uniform(np.log(1e-3), np.log(440.0), 5000)), E4M3_POS[:-1]])
    for x in xs:
        v = oracle.e4m3_decode(oracle.e4m3_encode(x, round_up=True))
        brute = E4M3_POS[np.searchsorted(E4M3_POS, x, side="left")]
        assert v == brute, (x, v, brute)
    assert oracle.e4m3_decode(oracle.e4m3_encode(1e6)) == 448.0  # saturation


def test_fp16_matches_numpy():
    rng = np.random.default_rng(2)
    xs = np.concatenate([rng.standard_normal(20000) * np.exp(rng.uniform(-12, 10, 20000)),
                         [0.0, 6.1e-5, 5.96e-8, 65504.0, -65504.0, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11]])
    xs = xs[np.abs(xs) < 65504.0]
    ref = xs.astype(np.float16).view(np.uint16)
    got = np.array([oracle.fp16_encode(x) for x in xs], dtype=np.uint16)
    assert np.array_equal(got, ref)
    for h in ref[:2000]:
        assert oracle.fp16_decode(int(h)) == float(np.uint16(h).view(np.float16))


def test_compact_bits_per_element_is_the_papers():
    """2-bit codes plus 512 bytes of aux per 128 x 128 tile: the 2.25 bits/element printed in
    App. D (tests/golden/paper_constants.txt)."""
    path = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.txt")
    printed = next(float(l.split()[1]) for l in open(path) if l.startswith("paper_bits_per_element"))
    assert oracle.tile_bytes(2, aux=1) * 8 / (128 * 128) == printed
    assert oracle.tile_bytes(4, aux=1) * 8 / (128 * 128) == printed + 2


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("dist", ["tinyK", "tinyV", "stressK"])
def test_compact_quantize_properties(kind, bits, dist):
    X = make_tile(dist, seed=11 + bits)
    r = oracle.quantize_tile(X, kind, oracle.Params(bits=bits, aux=1))
    qmax = (1 << bits) - 1
    a, b, s2 = (v.astype(np.float64) for v in (r.a, r.b, r.s2))
    step, mn, So = r.pre
    # stored values sit on their grids; s2 is the nearest E4M3 of the (range-limited) scale,
    # a the E4M3 rounded upward from the step, b the nearest binary16 of the group minimum
    s2_ref = torch.tensor(np.clip(So, 2.0 ** -6, 448.0)).to(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(s2, s2_ref)
    assert np.all(a >= step) and np.all(a <= step * (1 + 2.0 ** -3) + 2.0 ** -9)
    assert np.array_equal(b, mn.astype(np.float16).astype(np.float64))
    # z = T / s2 along the other axis; per group the code is the level nearest to z given (a, b)
    T = r.T
    Z = T / s2[:, None] if kind == 0 else T / s2[None, :]
    Zg = Z if kind == 1 else Z.T  # [group][element]
    codes = r.codes if kind == 1 else r.codes.T
    levels = np.arange(qmax + 1)[None, None, :] * a[:, None, None] + b[:, None, None]
    dist_ = np.abs(Zg[:, :, None] - levels)
    best = dist_.argmin(axis=2)
    ties = np.sort(dist_, axis=2)[:, :, 1] - np.sort(dist_, axis=2)[:, :, 0] < 1e-9 * (np.abs(Zg) + a[:, None])
    assert np.all((best == codes) | ties)
    # error bound of the stored format: |z - dq| <= a / 2 + |b - mn| (clipping at the ends)
    dq = codes * a[:, None] + b[:, None]
    assert np.all(np.abs(Zg - dq) <= a[:, None] / 2 + np.abs(b - mn)[:, None] + 1e-12 * (np.abs(Zg) + 1))
    # the packed tile holds exactly these values, and dequantizes to (code * a + b) * s2 un-rotated
    packed = oracle.pack_tile(r.codes, r.a, r.b, r.s2, kind, bits, aux=1)
    c2, a2, b2, s22 = oracle.unpack_tile(packed, kind, bits, aux=1)
    assert np.array_equal(c2, r.codes) and np.array_equal(a2, r.a) and np.array_equal(b2, r.b)
    assert np.array_equal(s22, r.s2)
    Xd = oracle.dequantize_tile(packed, kind, bits, aux=1)
    rot = (r.codes * a[None, :] + b[None, :]) * s2[:, None] if kind == 0 else \
        (r.codes * a[:, None] + b[:, None]) * s2[None, :]
    assert np.allclose(oracle.hadamard128(Xd), rot, rtol=0, atol=1e-9 * np.abs(rot).max())


def test_compact_matches_fp32_format_codes_mostly():
    """Both formats quantize the same balanced tile; the compact one differs only through the
    rounding of s2 and a, so most codes agree."""
    X = make_tile("tinyK", seed=5)
    r32 = oracle.quantize_tile(X, 0, oracle.Params(bits=2))
    r8 = oracle.quantize_tile(X, 0, oracle.Params(bits=2, aux=1))
    assert r32.best_iter == r8.best_iter
    assert (r32.codes == r8.codes).mean() > 0.8


@pytest.mark.parametrize("kind,dist", [(0, "tinyK"), (0, "stressK"), (1, "tinyV")])
def test_compact_tile_shift_keeps_large_tiles_in_range(kind, dist):
    """E4M3 holds at most 448 in each of a and s2, while their product is fixed by the data.  A
    tile whose largest step exceeds 448 moves a tile-wide power of two 2^e into s2: the smallest
    such e, every dequantized value within the stored format's bound, and errors as small
    (relative to the tile) as at unit magnitude.  Unit-magnitude tiles keep e = 0."""
    bits = 2
    base = make_tile(dist, seed=29)
    errs = {}
    for mag in (1.0, 300.0, 3000.0):
        X = base * mag
        r = oracle.quantize_tile(X, kind, oracle.Params(bits=bits, aux=1))
        So = (r.Sr if kind == 0 else r.Sc).astype(np.float64)
        ratio = r.pre[2] / So
        e = int(round(np.log2(ratio[0])))
        assert np.all(ratio == 2.0 ** e)
        # largest step without the shift, from the E4M3-rounded unshifted s2 (power-of-two
        # scaling commutes with E4M3 rounding in the normal range)
        s2_0 = torch.tensor(np.clip(So, 2.0 ** -6, 448.0)).to(torch.float8_e4m3fn).double().numpy()
        Z0 = r.T / s2_0[:, None] if kind == 0 else r.T / s2_0[None, :]
        Zg0 = Z0.T if kind == 0 else Z0
        m0 = float(((Zg0.max(axis=1) - Zg0.min(axis=1)) / ((1 << bits) - 1)).max())
        if mag == 1.0:
            assert e == 0 and m0 <= 448.0
        if e > 0:  # smallest e: one less would not fit (and s2 times 2^e stays within 448)
            assert m0 * 2.0 ** -(e - 1) > 448.0 >= m0 * 2.0 ** -e
            assert np.all(So * 2.0 ** e <= 448.0)
        if mag == 3000.0 and kind == 0:
            assert e > 0 and m0 > 448.0  # without the shift, a would saturate
        a, b, s2 = (v.astype(np.float64) for v in (r.a, r.b, r.s2))
        assert a.max() <= 448.0 and s2.max() <= 448.0
        if kind == 0:
            dq = (r.codes * a[None, :] + b[None, :]) * s2[:, None]
            tol = (a[None, :] / 2 + np.abs(b - r.pre[1])[None, :]) * s2[:, None]
        else:
            dq = (r.codes * a[:, None] + b[:, None]) * s2[None, :]
            tol = (a[:, None] / 2 + np.abs(b - r.pre[1])[:, None]) * s2[None, :]
        assert np.all(np.abs(r.T - dq) <= tol * (1 + 1e-12) + 1e-12 * np.abs(r.T))
        errs[mag] = np.linalg.norm(r.T - dq) / np.linalg.norm(r.T)
    assert errs[300.0] < 1.5 * errs[1.0] and errs[3000.0] < 1.5 * errs[1.0], errs
