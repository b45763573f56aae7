"""Pins of the prefill and of the paged body layout: a prefill equals appending the same bf16
tokens one by one (App. D's three regions, Fig. 4's streaming writes), and a paged cache with
permuted pool blocks holds and decodes exactly what the dense one does."""
import numpy as np
import pytest

import oracle


def _tokens(rng, total, n_kv):
    x = rng.standard_normal((total, n_kv, 128)) * np.exp(rng.standard_normal((1, n_kv, 128)))
    return oracle.f64_to_bf16_bits(x)


@pytest.mark.parametrize("n_sink", [0, 128])
def test_prefill_equals_appends(n_sink):
    rng = np.random.default_rng(n_sink + 1)
    lens = [0, 5, n_sink + 127, n_sink + 128, n_sink + 2 * 128 + 3, n_sink // 2]
    B, H, MB = len(lens), 2, 3
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    K, V = _tokens(rng, cu[-1], H), _tokens(rng, cu[-1], H)
    p = oracle.Params(bits=2)
    pre = oracle.HostCache(B, H, MB, n_sink=n_sink)
    assert oracle.prefill(pre, K, V, cu, max(lens), p) == 0
    app = oracle.HostCache(B, H, MB, n_sink=n_sink)
    for t in range(max(lens)):  # one token per step; shorter sequences sit out (one at a time)
        for b in range(B):
            if t < lens[b]:
                one = oracle.HostCache(1, H, MB, n_sink=n_sink)
                for f in ("k_body", "v_body", "k_resid", "v_resid", "k_sink", "v_sink"):
                    getattr(one, f)[0] = getattr(app, f)[b]
                one.seq_len[0] = app.seq_len[b]
                assert oracle.append(one, K[cu[b] + t][None], V[cu[b] + t][None], p) == 0
                for f in ("k_body", "v_body", "k_resid", "v_resid", "k_sink", "v_sink"):
                    getattr(app, f)[b] = getattr(one, f)[0]
                app.seq_len[b] = one.seq_len[0]
    np.testing.assert_array_equal(pre.seq_len, lens)
    np.testing.assert_array_equal(pre.seq_len, app.seq_len)
    for f in ("k_body", "v_body", "k_sink", "v_sink"):
        np.testing.assert_array_equal(getattr(pre, f), getattr(app, f), err_msg=f)
    for b, L in enumerate(lens):  # residual rows in use
        nr = (L - n_sink) % 128 if L > n_sink else 0
        np.testing.assert_array_equal(pre.k_resid[b, :, :nr], app.k_resid[b, :, :nr])
        np.testing.assert_array_equal(pre.v_resid[b, :, :nr], app.v_resid[b, :, :nr])


def test_paged_layout_matches_dense():
    rng = np.random.default_rng(5)
    lens = [3 * 128 + 17, 128, 2 * 128 + 127]
    B, H, MB = len(lens), 2, 4
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    K, V = _tokens(rng, cu[-1], H), _tokens(rng, cu[-1], H)
    p = oracle.Params(bits=2)
    dense = oracle.HostCache(B, H, MB)
    assert oracle.prefill(dense, K, V, cu, max(lens), p) == 0
    paged = oracle.HostCache(B, H, MB, n_phys=B * MB + 3)
    paged.block_table[:] = rng.permutation(B * MB + 3)[:B * MB].reshape(B, MB).astype(np.int32)
    assert oracle.prefill(paged, K, V, cu, max(lens), p) == 0
    for b in range(B):
        for blk in range((lens[b]) // 128):
            ph = paged.block_table[b, blk]
            np.testing.assert_array_equal(paged.k_body[ph], dense.k_body[b, :, blk])
            np.testing.assert_array_equal(paged.v_body[ph], dense.v_body[b, :, blk])
    q = oracle.f64_to_bf16_bits(rng.standard_normal((B, 4 * H, 128)))
    np.testing.assert_array_equal(oracle.decode(paged, q, 0.088), oracle.decode(dense, q, 0.088))
    # appends through the table flush into the mapped pool block
    tok = _tokens(rng, 1, H * B).reshape(B, H, 128)
    for c in (dense, paged):
        for _ in range(128 - 17):
            assert oracle.append(c, tok, tok, p) == 0
    ph = paged.block_table[0, 3]
    np.testing.assert_array_equal(paged.k_body[ph], dense.k_body[0, :, 3])


def test_prefill_and_append_errors():
    rng = np.random.default_rng(9)
    lens = [300, 40]
    cu = np.array([0, 300, 340], dtype=np.int32)
    K = _tokens(rng, 340, 1)
    c = oracle.HostCache(2, 1, 2)
    assert oracle.prefill(c, K, K, cu, 299, oracle.Params()) == -3  # first prompt above max_len
    assert list(c.seq_len) == [0, 40]
    c2 = oracle.HostCache(2, 1, 1)
    assert oracle.prefill(c2, K, K, cu, 300, oracle.Params()) == -3  # 2 groups, 1 block
    paged = oracle.HostCache(2, 1, 3, n_phys=2)
    paged.block_table[:] = [[0, 5, -1], [1, -1, -1]]  # 5 is outside the pool
    assert oracle.prefill(paged, K, K, cu, 300, oracle.Params()) == -4
