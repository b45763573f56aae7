"""Pins of the oracle's round-to-nearest (Sec. 2.1, Eq. 1), of the packed tile format and of
the whole quantize step (Fig. 2, Sec. 3.3, App. D)."""
import numpy as np
import pytest

from tiles import tile


@pytest.mark.parametrize("bits", [2, 4])
def test_rtn_brute_force(orc, bits):
    """Codes equal the argmin over the 2^bits reconstruction levels (brute force), except on
    exact ties; the error is at most half a step; min -> 0 and max -> top code."""
    rng = np.random.default_rng(bits)
    for trial in range(50):
        x = rng.standard_normal(128) * np.exp(rng.standard_normal()) + rng.standard_normal()
        codes, mn, s, u = orc.rtn_group(x, bits)
        levels = mn + s * np.arange(2 ** bits)
        brute = np.argmin(np.abs(x[:, None] - levels[None, :]), axis=1)
        tie = np.abs(u - np.floor(u) - 0.5) < 1e-9
        np.testing.assert_array_equal(codes[~tie], brute[~tie])
        np.testing.assert_array_less(np.abs(x - (codes * s + mn)), s / 2 * (1 + 1e-12))
        assert codes[np.argmin(x)] == 0 and codes[np.argmax(x)] == 2 ** bits - 1
        np.testing.assert_allclose(s, (x.max() - x.min()) / (2 ** bits - 1), rtol=1e-15)


def test_rtn_ties_round_half_even(orc):
    # levels 0, 1, 2, 3 (s = 1): 0.5 -> 0, 1.5 -> 2, 2.5 -> 2
    codes, mn, s, _ = orc.rtn_group(np.array([0.0, 0.5, 1.5, 2.5, 3.0]), 2)
    assert (mn, s) == (0.0, 1.0)
    np.testing.assert_array_equal(codes, [0, 0, 2, 2, 3])


def test_rtn_constant_group(orc):
    codes, mn, s, _ = orc.rtn_group(np.full(128, -0.75), 2)
    np.testing.assert_array_equal(codes, 0)
    assert mn == -0.75 and s == 1.0


def test_tile_bytes_and_bits_per_element(orc):
    # 2-bit: 4096 code bytes + 3 x 128 fp32 = 5632 bytes for 16384 elements -> 2.75 bits/elem
    # (the paper's 8-bit auxiliary format gives 2.25 bits/elem, App. D)
    assert orc.tile_bytes(2) == 5632 and orc.tile_bytes(4) == 9728
    assert orc.tile_bytes(2) * 8 / 16384 == 2.75 and orc.tile_bytes(4) * 8 / 16384 == 4.75


# Hand-derived word / bit positions from the format description, 2-bit and 4-bit tiles
# (tests/golden/format_2bit_positions.txt; the derivation rules are in its header).
def _hand_positions():
    """Rows (kind, (t, c), {bits: (word, bit)})."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "format_2bit_positions.txt")
    table = {0: [], 1: []}
    with open(path) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                k, t, c, w2, b2, w4, b4 = (int(v) for v in line.split())
                table[k].append(((t, c), {2: (w2, b2), 4: (w4, b4)}))
    return table


HAND = _hand_positions()


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("bits", [2, 4])
def test_pack_hand_positions(orc, kind, bits):
    code = 3 if bits == 2 else 13
    for (t, c), pos in HAND[kind]:
        word, bit = pos[bits]
        codes = np.zeros((128, 128), dtype=np.uint8)
        codes[t, c] = code
        packed = orc.pack_tile(codes, np.zeros(128), np.zeros(128), np.zeros(128), kind, bits)
        words = packed[:bits * 2048].view("<u4")
        nz = np.flatnonzero(words)
        assert list(nz) == [word], (t, c, nz)
        assert words[word] == code << bit, (t, c, hex(words[word]))


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("bits", [2, 4])
def test_pack_roundtrip_bijective(orc, kind, bits):
    rng = np.random.default_rng(kind * 10 + bits)
    codes = rng.integers(0, 2 ** bits, size=(128, 128), dtype=np.uint8)
    a, b, s2 = (rng.standard_normal(128).astype(np.float32) for _ in range(3))
    packed = orc.pack_tile(codes, a, b, s2, kind, bits)
    c2, a2, b2, s22 = orc.unpack_tile(packed, kind, bits)
    np.testing.assert_array_equal(c2, codes)
    np.testing.assert_array_equal(a2, a)
    np.testing.assert_array_equal(b2, b)
    np.testing.assert_array_equal(s22, s2)
    # every code bit is used exactly once: all-max codes fill the code region with ones
    full = orc.pack_tile(np.full((128, 128), 2 ** bits - 1, np.uint8), a, b, s2, kind, bits)
    assert np.all(full[:bits * 2048] == 0xFF)
    np.testing.assert_array_equal(full[bits * 2048:].view(np.float32), np.concatenate([a, b, s2]))


@pytest.mark.parametrize("kind_name,kind", [("tinyK", 0), ("tinyV", 1), ("stressK", 0)])
@pytest.mark.parametrize("bits", [2, 4])
def test_quantize_tile_dequant_bound(orc, kind_name, kind, bits):
    """End-to-end error bound of one tile: in the rotated domain every element is within half
    an RTN step (scaled back by both Sinkhorn scales) of its reconstruction
    (code * a + b) * s2, and un-rotating with H preserves the per-token error norm."""
    X = tile(kind_name, 31)
    p = orc.Params(bits=bits)
    r = orc.quantize_tile(X, kind, p)
    a, b, s2 = (v.astype(np.float64) for v in (r.a, r.b, r.s2))
    q = r.codes.astype(np.float64)
    if kind == 0:
        Xr = (q * a[None, :] + b[None, :]) * s2[:, None]
        step = a[None, :] * s2[:, None]
        big = (np.abs(b)[None, :] + (2 ** bits) * a[None, :]) * s2[:, None]
    else:
        Xr = (q * a[:, None] + b[:, None]) * s2[None, :]
        step = a[:, None] * s2[None, :]
        big = (np.abs(b)[:, None] + (2 ** bits) * a[:, None]) * s2[None, :]
    # half a step, plus fp32 rounding of the stored a, b, s2
    np.testing.assert_array_less(np.abs(r.T - Xr), step / 2 + 4e-7 * big)
    Xd = orc.dequantize_tile(orc.pack_tile(r.codes, r.a, r.b, r.s2, kind, bits), kind, bits)
    np.testing.assert_allclose(np.linalg.norm(Xd - X, axis=1), np.linalg.norm(Xr - r.T, axis=1), rtol=1e-9,
                               atol=1e-12)
    # the absorbed form equals the product of RTN step, Sinkhorn scales (P10 of the format)
    if kind == 0:
        np.testing.assert_allclose(step, (a / r.Sc)[None, :] * r.Sc[None, :] * r.Sr[:, None], rtol=1e-6)
    # dequantization is much closer than the tile's own spread
    assert np.linalg.norm(Xd - X) < 0.7 * np.linalg.norm(X - X.mean())


def test_quantize_tile_keys_group_axis(orc):
    """Keys are quantized per channel: every channel of B uses all four 2-bit levels between
    its own min and max; values per token."""
    X = tile("tinyK", 41)
    rk = orc.quantize_tile(X, 0)
    for c in range(128):
        col = rk.B[:, c]
        assert rk.codes[np.argmin(col), c] == 0 and rk.codes[np.argmax(col), c] == 3
    rv = orc.quantize_tile(X, 1)
    for t in range(128):
        row = rv.B[t]
        assert rv.codes[t, np.argmin(row)] == 0 and rv.codes[t, np.argmax(row)] == 3


def test_quantize_degenerate_tiles(orc):
    """A zero tile gives zero codes; a constant tile rotates to a single non-zero channel,
    i.e. two-level data, which every group reconstructs exactly."""
    for X in (np.zeros((128, 128)), np.full((128, 128), 0.5)):
        for kind in (0, 1):
            r = orc.quantize_tile(X, kind)
            if not X.any():
                np.testing.assert_array_equal(r.codes, 0)
            Xd = orc.dequantize_tile(orc.pack_tile(r.codes, r.a, r.b, r.s2, kind, 2), kind, 2)
            np.testing.assert_allclose(Xd, X, atol=1e-6)
