"""Pins of the oracle's decode attention over the three-region cache (App. D "Quantization",
App. A rotation layout, App. I fused dual-scale dequantization) and of its streaming append
(Fig. 4 pseudo-decode)."""
import numpy as np
import pytest
import scipy.linalg
import scipy.special

from tiles import tile

H = scipy.linalg.hadamard(128).astype(np.float64) / np.sqrt(128.0)


def test_attend_matches_scipy_softmax(orc):
    rng = np.random.default_rng(0)
    for n in (1, 2, 7, 300):
        q = rng.standard_normal(128)
        K = rng.standard_normal((n, 128)) * 2
        V = rng.standard_normal((n, 128))
        scale = 1 / np.sqrt(128)
        expect = scipy.special.softmax(scale * K @ q) @ V
        np.testing.assert_allclose(orc.attend(q, K, V, scale), expect, rtol=1e-12, atol=1e-14)


def test_attend_special_cases(orc):
    rng = np.random.default_rng(1)
    K = rng.standard_normal((50, 128))
    V = rng.standard_normal((50, 128))
    np.testing.assert_allclose(orc.attend(rng.standard_normal(128), K[:1], V[:1], 0.1), V[0], rtol=1e-15)
    np.testing.assert_allclose(orc.attend(np.zeros(128), K, V, 0.1), V.mean(axis=0), rtol=1e-12)
    # very large logits do not overflow (max subtraction): one-hot on the largest
    q = K[17] * 1e3
    np.testing.assert_allclose(orc.attend(q, K, V, 1.0), V[np.argmax(K @ q)], rtol=1e-12)


def test_rotation_invariance(orc):
    """attn(Hq, HK, HV) H = attn(q, K, V): decode may run in the rotated domain (App. A)."""
    rng = np.random.default_rng(2)
    q, K, V = rng.standard_normal(128), rng.standard_normal((64, 128)), rng.standard_normal((64, 128))
    o = orc.attend(q, K, V, 0.09)
    o_rot = orc.attend(H @ q, K @ H, V @ H, 0.09)
    np.testing.assert_allclose(o_rot @ H, o, rtol=1e-11, atol=1e-13)


def _bf16(x):
    import oracle
    return oracle.f64_to_bf16_bits(x)


def _fill_cache(orc, cache, lengths, seed, bits=2):
    """Fill a host cache directly: quantized body tiles, residual and sink in bf16."""
    rng = np.random.default_rng(seed)
    p = orc.Params(bits=bits)
    raw = {}
    for b, n in enumerate(lengths):
        for kh in range(cache.n_kv):
            Kx = _bf16(tile("tinyK", seed * 100 + b * 10 + kh)[np.arange(n) % 128] * (1 + 0.01 * np.arange(n))[:, None])
            Vx = _bf16(rng.standard_normal((n, 128)))
            raw[b, kh] = (Kx, Vx)
            ns = min(n, cache.n_sink)
            cache.k_sink[b, kh, :ns] = Kx[:ns]
            cache.v_sink[b, kh, :ns] = Vx[:ns]
            rest = n - ns
            nb, nr = rest // 128, rest % 128
            if nb:
                cache.k_body[b, kh, :nb] = orc.quantize_tiles(Kx[ns:ns + nb * 128].reshape(nb * 128, 128), 0, p)
                cache.v_body[b, kh, :nb] = orc.quantize_tiles(Vx[ns:ns + nb * 128].reshape(nb * 128, 128), 1, p)
            cache.k_resid[b, kh, :nr] = Kx[ns + nb * 128:]
            cache.v_resid[b, kh, :nr] = Vx[ns + nb * 128:]
        cache.seq_len[b] = n
    return raw


@pytest.mark.parametrize("n_sink", [0, 128])
def test_gather_regions(orc, n_sink):
    cache = orc.HostCache(batch=3, n_kv=2, max_blocks=4, n_sink=n_sink)
    lengths = [5, 128 + n_sink + 3, 2 * 128 + n_sink]
    raw = _fill_cache(orc, cache, lengths, seed=3)
    for b, n in enumerate(lengths):
        for kh in range(2):
            K, V = orc.gather_stream(cache, b, kh)
            Kx, Vx = (orc.bf16_bits_to_f64(v) for v in raw[b, kh])
            assert K.shape == (n, 128)
            ns = min(n, n_sink)
            nb = (n - ns) // 128
            # sink and residual are exact bf16; body is within the quantization error
            np.testing.assert_array_equal(K[:ns], Kx[:ns])
            np.testing.assert_array_equal(V[ns + nb * 128:], Vx[ns + nb * 128:])
            np.testing.assert_array_equal(K[ns + nb * 128:], Kx[ns + nb * 128:])
            for blk in range(nb):
                sl = slice(ns + blk * 128, ns + (blk + 1) * 128)
                np.testing.assert_allclose(K[sl], orc.dequantize_tile(cache.k_body[b, kh, blk], 0, 2), rtol=0,
                                           atol=0)
                err = np.linalg.norm(K[sl] - Kx[sl]) / np.linalg.norm(Kx[sl])
                assert err < 0.6


def test_decode_equals_attention_over_gathered(orc):
    cache = orc.HostCache(batch=2, n_kv=2, max_blocks=3)
    _fill_cache(orc, cache, [300, 129], seed=4)
    rng = np.random.default_rng(5)
    q = rng.standard_normal((2, 8, 128)).astype(np.float32)
    out = orc.decode(cache, q, 1 / np.sqrt(128))
    for b in range(2):
        for h in range(8):
            K, V = orc.gather_stream(cache, b, h // 4)
            expect = scipy.special.softmax(K @ q[b, h].astype(np.float64) / np.sqrt(128)) @ V
            np.testing.assert_allclose(out[b, h], expect, rtol=1e-11, atol=1e-13)


def test_decode_gqa_equals_duplicated_mha(orc):
    cache = orc.HostCache(batch=1, n_kv=2, max_blocks=2)
    _fill_cache(orc, cache, [200], seed=6)
    dup = orc.HostCache(batch=1, n_kv=4, max_blocks=2)
    for name in ("k_body", "v_body", "k_resid", "v_resid", "k_sink", "v_sink"):
        getattr(dup, name)[:] = np.repeat(getattr(cache, name), 2, axis=1)
    dup.seq_len[:] = cache.seq_len
    q = np.random.default_rng(7).standard_normal((1, 4, 128)).astype(np.float32)
    np.testing.assert_array_equal(orc.decode(cache, q, 0.1), orc.decode(dup, q, 0.1))


def test_decode_bf16_query(orc):
    cache = orc.HostCache(batch=1, n_kv=1, max_blocks=2)
    _fill_cache(orc, cache, [140], seed=8)
    qf = np.random.default_rng(9).standard_normal((1, 1, 128))
    qb = orc.f64_to_bf16_bits(qf)
    np.testing.assert_array_equal(orc.decode(cache, qb, 0.1), orc.decode(cache, orc.bf16_bits_to_f64(qb).astype(np.float32), 0.1))


@pytest.mark.parametrize("n_sink", [0, 128])
@pytest.mark.parametrize("bits", [2, 4])
def test_append_stream_matches_direct_layout(orc, n_sink, bits):
    """Appending tokens one by one yields the same cache as laying the sequence out directly:
    sink = first n_sink tokens, body tiles = quantized 128-token groups, residual = rest."""
    batch, n_kv, n = 2, 2, n_sink + 2 * 128 + 5
    p = orc.Params(bits=bits)
    cache = orc.HostCache(batch, n_kv, max_blocks=3, bits=bits, n_sink=n_sink)
    rng = np.random.default_rng(10)
    Ks = _bf16(rng.standard_normal((n, batch, n_kv, 128)) * np.exp(rng.standard_normal(128)))
    Vs = _bf16(rng.standard_normal((n, batch, n_kv, 128)))
    for t in range(n):
        assert orc.append(cache, Ks[t], Vs[t], p) == 0
    assert list(cache.seq_len) == [n] * batch
    for b in range(batch):
        for kh in range(n_kv):
            Kx, Vx = Ks[:, b, kh], Vs[:, b, kh]
            np.testing.assert_array_equal(cache.k_sink[b, kh, :n_sink], Kx[:n_sink])
            np.testing.assert_array_equal(cache.v_sink[b, kh, :n_sink], Vx[:n_sink])
            body_k = orc.quantize_tiles(np.ascontiguousarray(Kx[n_sink:n_sink + 256]), 0, p)
            body_v = orc.quantize_tiles(np.ascontiguousarray(Vx[n_sink:n_sink + 256]), 1, p)
            np.testing.assert_array_equal(cache.k_body[b, kh, :2], body_k)
            np.testing.assert_array_equal(cache.v_body[b, kh, :2], body_v)
            np.testing.assert_array_equal(cache.k_resid[b, kh, :5], Kx[n_sink + 256:])
            np.testing.assert_array_equal(cache.v_resid[b, kh, :5], Vx[n_sink + 256:])


def test_append_capacity(orc):
    cache = orc.HostCache(1, 1, max_blocks=1)
    tok = np.zeros((1, 1, 128), dtype=np.uint16)
    for _ in range(128 + 127):
        assert orc.append(cache, tok, tok) == 0
    assert orc.append(cache, tok, tok) == -3  # the flush would need a second body tile
    assert cache.seq_len[0] == 255
