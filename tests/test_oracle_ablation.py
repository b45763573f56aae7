"""Pins of the ablation switches (Fig. 1: KIVI-style RTN, Hadamard only, VarN only, KVarN) and of
the error decomposition of Sec. 3.1 Eq. 3."""
import numpy as np
import pytest

import oracle
from tiles import tile


def test_error_decomposition_hand_cases():
    K = np.zeros((3, 128))
    Q = np.zeros((3, 128))
    K[0, :2], Q[0, :2] = (3.0, 4.0), (6.0, 8.0)   # same direction, norm 5 -> 10
    K[1, 0], Q[1, 1] = 1.0, 1.0                   # orthogonal unit vectors
    K[2, :3] = Q[2, :3] = (1.0, -2.0, 2.0)         # identical
    ET, EM, ED = oracle.error_decomposition(K, Q)
    assert np.allclose(ET, [25.0, 2.0, 0.0]) and np.allclose(EM, [25.0, 0.0, 0.0])
    assert np.allclose(ED, [0.0, 2.0, 0.0], atol=1e-12)


def test_error_decomposition_identity_and_angle_form():
    rng = np.random.default_rng(0)
    K = rng.standard_normal((200, 128)) * np.exp(rng.standard_normal((200, 1)))
    Q = K + 0.3 * rng.standard_normal((200, 128)) * np.exp(rng.standard_normal((200, 1)))
    ET, EM, ED = oracle.error_decomposition(K, Q)
    nk, nq = np.linalg.norm(K, axis=1), np.linalg.norm(Q, axis=1)
    # Eq. 3; the right side is formed from squared norms, so rounding scales with them
    assert np.all(np.abs(ET - (EM + ED)) <= 1e-13 * (nk ** 2 + nq ** 2))
    theta = np.arccos(np.clip((K * Q).sum(1) / (nk * nq), -1, 1))
    assert np.allclose(ED, 2 * nk * nq * (1 - np.cos(theta)), rtol=1e-9)
    assert np.all(EM >= 0) and np.all(ED >= -1e-9 * ET)


@pytest.mark.parametrize("kind", [0, 1])
def test_no_rotation_no_varn_is_plain_rtn(kind):
    """rotate = 0 with K = 0: the tile is quantized as given, one RTN per group (KIVI's scheme,
    Sec. 2.1): keys per channel, values per token, unit second scale."""
    X = tile("tinyK", 3)
    r = oracle.quantize_tile(X, kind, oracle.Params(bits=2, varn_iters=0, rotate=0))
    assert np.array_equal(r.T, X) and np.all(r.s2 == 1.0)
    for g in range(128):
        x = X[:, g] if kind == 0 else X[g, :]
        codes, mn, s, u = oracle.rtn_group(x, 2)
        got = r.codes[:, g] if kind == 0 else r.codes[g, :]
        assert np.array_equal(got, codes)
        assert r.a[g] == np.float32(s) and r.b[g] == np.float32(mn)
    packed = oracle.pack_tile(r.codes, r.a, r.b, r.s2, kind, 2)
    Xd = oracle.dequantize_tile(packed, kind, 2, rotate=0)
    step = (r.a.astype(np.float64)[None, :] if kind == 0 else r.a.astype(np.float64)[:, None])
    assert np.all(np.abs(Xd - X) <= step / 2 * (1 + 1e-6))


def test_rotation_commutes_with_varn_only_through_the_tile():
    """rotate = 1 equals rotating the input by hand and quantizing it unrotated."""
    X = tile("tinyV", 8)
    r1 = oracle.quantize_tile(X, 1, oracle.Params(bits=2))
    r0 = oracle.quantize_tile(oracle.hadamard128(X), 1, oracle.Params(bits=2, rotate=0))
    assert np.array_equal(r1.codes, r0.codes) and np.array_equal(r1.a, r0.a) and np.array_equal(r1.s2, r0.s2)


def test_ablation_order_on_llama_shaped_keys():
    """The paper's mechanism on synthetic keys with per-channel and per-token scales (Fig. 1):
    among the largest 5 % errors, the share due to magnitude falls from KIVI-style RTN to
    Hadamard only or VarN only, and is smallest with both (KVarN)."""
    share, mean = {}, {}
    for name, rot, it in [("KIVI", 0, 0), ("HK", 1, 0), ("VarN", 0, 8), ("KVarN", 1, 8)]:
        ET, EM = [], []
        for s in range(16):
            X = tile("tinyK", 100 + s)
            r = oracle.quantize_tile(X, 0, oracle.Params(bits=2, varn_iters=it, rotate=rot))
            Xd = oracle.dequantize_tile(oracle.pack_tile(r.codes, r.a, r.b, r.s2, 0, 2), 0, 2, rotate=rot)
            et, em, _ = oracle.error_decomposition(X, Xd)
            ET.append(et)
            EM.append(em)
        ET, EM = np.concatenate(ET), np.concatenate(EM)
        top = np.argsort(ET)[-len(ET) // 20:]
        share[name] = EM[top].sum() / ET[top].sum()
        mean[name] = ET.mean()
    assert share["KVarN"] < min(share["HK"], share["VarN"]) and max(share["HK"], share["VarN"]) < share["KIVI"]
    assert mean["KVarN"] < mean["KIVI"]
