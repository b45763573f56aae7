"""GPU parity of the serving layout: whole-prompt prefill of variable-length prompts and the
paged body (block table), through the C ABI against the oracle and against the dense layout."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import check_end_to_end, check_output, compare_tiles, host_cache, q_to_host

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module")
def K():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    torch.cuda.set_device(0)
    return kvarn


def _prompts(lens, H, dtype, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    total = int(sum(lens))
    sc = torch.exp(torch.randn((1, H, 128), generator=g, device="cuda"))
    k = (torch.randn((total, H, 128), generator=g, device="cuda") * sc).to(dtype)
    v = torch.randn((total, H, 128), generator=g, device="cuda").to(dtype)
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device="cuda")
    return k, v, cu


def _host(x):
    return x.cpu().numpy() if x.dtype == torch.float32 else q_to_host(x)


def _decode(K, p, cache, q, max_len):
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, q.shape[1], max_len)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    K.kvarn_decode_attention(p, cache, q.shape[1], q, K.KVARN_BF16, out, K.KVARN_F32, SCALE, max_len, ws, ws_bytes)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("bits,n_sink,dtype", [(2, 0, torch.bfloat16), (4, 128, torch.bfloat16),
                                               (2, 128, torch.float32)])
def test_prefill_matches_oracle(K, bits, n_sink, dtype):
    lens = [0, 7, n_sink + 127, n_sink + 128, n_sink + 3 * 128 + 29, n_sink // 2 + 1]
    B, H, MB = len(lens), 2, 4
    k, v, cu = _prompts(lens, H, dtype, seed=bits + n_sink)
    p = K.kvarn_params_init(bits)
    p.n_sink = n_sink
    cache = K.Cache(p, B, H, MB)
    K.kvarn_prefill(p, cache, k, v, K.KVARN_BF16 if dtype == torch.bfloat16 else K.KVARN_F32, cu, max(lens))
    torch.cuda.synchronize()
    assert int(cache.err_word[0]) == 0
    hc = oracle.HostCache(B, H, MB, bits=bits, n_sink=n_sink)
    assert oracle.prefill(hc, _host(k), _host(v), cu.cpu().numpy(), max(lens), oracle.Params(bits=bits)) == 0
    gc = host_cache(cache)
    np.testing.assert_array_equal(gc.seq_len, lens)
    if n_sink:
        for b, L in enumerate(lens):
            ns = min(L, n_sink)
            np.testing.assert_array_equal(gc.k_sink[b, :, :ns], hc.k_sink[b, :, :ns])
            np.testing.assert_array_equal(gc.v_sink[b, :, :ns], hc.v_sink[b, :, :ns])
    kk, vv, cun = _host(k), _host(v), cu.cpu().numpy()
    for b, L in enumerate(lens):
        nr = (L - n_sink) % 128 if L > n_sink else 0
        np.testing.assert_array_equal(gc.k_resid[b, :, :nr], hc.k_resid[b, :, :nr])
        np.testing.assert_array_equal(gc.v_resid[b, :, :nr], hc.v_resid[b, :, :nr])
        for blk in range((L - n_sink) // 128 if L > n_sink else 0):
            r0 = cun[b] + n_sink + blk * 128
            for kind, src, body in ((0, kk, gc.k_body), (1, vv, gc.v_body)):
                X = src[r0:r0 + 128].transpose(1, 0, 2)  # [H][128 tokens][128]
                X = X.astype(np.float64) if dtype == torch.float32 else oracle.bf16_bits_to_f64(X)
                compare_tiles(body[b, :, blk], X, kind, bits)
    q = torch.randn((B, 4 * H, 128), device="cuda").to(torch.bfloat16)
    out = _decode(K, p, cache, q, max(lens) + 1)
    check_output(out.cpu().numpy(), oracle.decode(gc, q_to_host(q), SCALE), bf16_out=False)
    # end to end: the oracle's own prefill of the same prompts

    def raw(b, h, blk, kind):
        r0 = cun[b] + n_sink + blk * 128
        X = (kk, vv)[kind][r0:r0 + 128, h]
        return X.astype(np.float64) if dtype == torch.float32 else oracle.bf16_bits_to_f64(X)

    check_end_to_end(out.cpu().numpy(), hc, gc, raw, q_to_host(q), False, SCALE)


def test_paged_equals_dense(K):
    """A permuted pool behind a block table: prefill writes the same tiles, decode gives the same
    bits, and appends flush into the mapped pool blocks."""
    lens = [5 * 128 + 61, 128, 3 * 128 + 127, 0]
    B, H, MB = len(lens), 2, 7
    k, v, cu = _prompts(lens, H, torch.bfloat16, seed=3)
    p = K.kvarn_params_init(2)
    dense = K.Cache(p, B, H, MB)
    n_phys = B * MB + 5
    paged = K.Cache(p, B, H, MB, n_phys=n_phys)
    perm = torch.randperm(n_phys, generator=torch.Generator().manual_seed(1))[:B * MB]
    paged.block_table.copy_(perm.view(B, MB).to(torch.int32))
    for c in (dense, paged):
        K.kvarn_prefill(p, c, k, v, K.KVARN_BF16, cu, max(lens))
    q = torch.randn((B, 4 * H, 128), device="cuda").to(torch.bfloat16)
    o_d, o_p = _decode(K, p, dense, q, max(lens) + 1), _decode(K, p, paged, q, max(lens) + 1)
    assert torch.equal(o_d, o_p)
    bt = paged.block_table.cpu().numpy()
    for b, L in enumerate(lens):
        for blk in range(L // 128):
            assert torch.equal(paged.k_body[bt[b, blk]], dense.k_body[b, :, blk])
            assert torch.equal(paged.v_body[bt[b, blk]], dense.v_body[b, :, blk])
    g = torch.Generator(device="cuda").manual_seed(4)
    for t in range(128 + 5):
        kt = torch.randn((B, H, 128), generator=g, device="cuda").to(torch.bfloat16)
        for c in (dense, paged):
            K.kvarn_append_token(p, c, kt, kt, K.KVARN_BF16, -1)
    torch.cuda.synchronize()
    assert torch.equal(dense.seq_len, paged.seq_len)
    assert int(dense.err_word[0]) == 0 and int(paged.err_word[0]) == 0
    for b in range(B):
        nb = int(dense.seq_len[b]) // 128
        for blk in range(nb):
            assert torch.equal(paged.k_body[bt[b, blk]], dense.k_body[b, :, blk]), (b, blk)
    o_d, o_p = _decode(K, p, dense, q, max(lens) + 200), _decode(K, p, paged, q, max(lens) + 200)
    assert torch.equal(o_d, o_p)
    check_output(o_p.cpu().numpy(), oracle.decode(host_cache(dense), q_to_host(q), SCALE), bf16_out=False)


@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("aux", [0, 1])
@pytest.mark.parametrize("g", [4, 5, 6, 12])
def test_paged_every_kernel(K, bits, aux, g):
    """Every decode kernel (code width x aux format x query-group class 1-4, 5, 6-8, 9-16) on a
    permuted pool: bit-equal to the dense layout and within the output bar of the oracle, with
    ragged lengths (a residual, an exact block boundary, a sequence shorter than one block)."""
    lens = [9 * 128 + 77, 3 * 128, 90]  # 9 body tiles: split streams, merged by the merge kernel
    B, H, MB = len(lens), 2, 10
    k, v, cu = _prompts(lens, H, torch.bfloat16, seed=11 + bits + 2 * aux + g)
    p = K.kvarn_params_init(bits, aux_format=aux)
    dense = K.Cache(p, B, H, MB)
    n_phys = B * MB + 3
    paged = K.Cache(p, B, H, MB, n_phys=n_phys)
    perm = torch.randperm(n_phys, generator=torch.Generator().manual_seed(g))[:B * MB]
    paged.block_table.copy_(perm.view(B, MB).to(torch.int32))
    for c in (dense, paged):
        K.kvarn_prefill(p, c, k, v, K.KVARN_BF16, cu, max(lens))
    q = torch.randn((B, g * H, 128), device="cuda").to(torch.bfloat16)
    o_d, o_p = _decode(K, p, dense, q, max(lens)), _decode(K, p, paged, q, max(lens))
    assert torch.equal(o_d, o_p)
    assert int(paged.err_word[0]) == 0
    check_output(o_d.cpu().numpy(), oracle.decode(host_cache(dense), q_to_host(q), SCALE), bf16_out=False)


def test_serving_error_flags(K):
    """Conditions the kernels check themselves: a prompt longer than max_len is not written
    (seq_len 0, bit 0); a pool id outside the pool sets bit 1, and decode then skips that
    sequence's body while the other sequences are unaffected."""
    lens = [300, 200]
    B, H, MB = 2, 1, 3
    k, v, cu = _prompts(lens, H, torch.bfloat16, seed=8)
    p = K.kvarn_params_init(2)
    c = K.Cache(p, B, H, MB)
    K.kvarn_prefill(p, c, k, v, K.KVARN_BF16, cu, 250)
    torch.cuda.synchronize()
    assert c.seq_len.tolist() == [0, 200] and int(c.err_word[0]) & 1
    paged = K.Cache(p, B, H, MB, n_phys=4)
    paged.block_table.copy_(torch.tensor([[0, 1, 2], [9, -1, -1]], dtype=torch.int32))
    K.kvarn_prefill(p, paged, k, v, K.KVARN_BF16, cu, 300)  # sequence 1's tile 0 has id 9
    torch.cuda.synchronize()
    assert int(paged.err_word[0]) & 2
    paged.err_word.zero_()
    paged.block_table[1, 0], paged.block_table[1, 1] = 3, 9  # tile 1 of sequence 1 outside the pool
    paged.seq_len.copy_(torch.tensor([300, 2 * 128 + 5], dtype=torch.int32))
    q = torch.randn((B, 4, 128), device="cuda").to(torch.bfloat16)
    out = _decode(K, p, paged, q, 300)
    assert int(paged.err_word[0]) & 2
    assert bool(torch.isfinite(out).all())
    dense = K.Cache(p, B, H, MB)
    K.kvarn_prefill(p, dense, k, v, K.KVARN_BF16, cu, 300)
    ref = _decode(K, p, dense, q, 300)
    assert torch.equal(out[0], ref[0])  # the sequence with valid ids is unaffected
