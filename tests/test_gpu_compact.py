"""GPU parity of the compact aux format (two E4M3 scales and a binary16 offset per group,
App. D "Effective memory overhead"): quantized tiles, decode attention and the append stream,
through the C ABI against the oracle with aux=1.  Tie rules in gpu_util.compare_tiles_compact."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import check_end_to_end, check_output, compare_tiles_compact, host_cache, q_to_host, tiles_to_host

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module")
def K():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    torch.cuda.set_device(0)
    return kvarn


def _params(K, bits, **over):
    p = K.kvarn_params_init(bits, **over)
    p.aux_format = K.KVARN_AUX_COMPACT
    return p


def _quantize(K, x, kind, bits, **over):
    n = x.shape[0]
    p = _params(K, bits, **over)
    out = torch.zeros((n, K.kvarn_tile_bytes(p)), dtype=torch.uint8, device="cuda")
    best = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    dt = K.KVARN_F32 if x.dtype == torch.float32 else K.KVARN_BF16
    K.kvarn_quantize_block(p, kind, x, dt, n, 1, 128 * 128, 0, 128, out, 1, 0, best)
    torch.cuda.synchronize()
    return out.cpu().numpy(), best.cpu().numpy()


@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("dist", ["llama", "stress"])
def test_compact_quantize_tiles(K, bits, dist):
    from paper_2606_03458_amd import datagen
    Kx, Vx = datagen.kv_tokens(21 + bits, 0, 1, 2, 32 * 64, dist, dtype=torch.bfloat16, device="cuda")
    for kind, x in ((0, Kx), (1, Vx)):
        xt = x.reshape(32, 128, 128).contiguous()
        tiles, best = _quantize(K, xt, kind, bits)
        st = compare_tiles_compact(tiles, tiles_to_host(xt), kind, bits, best)
        assert st["codes"] >= 30 * 16384, st


def test_compact_degenerate_tiles(K):
    """Zero, constant, single-outlier, huge and tiny tiles (scales at the E4M3 range ends)."""
    x = torch.zeros((5, 128, 128), dtype=torch.float32, device="cuda")
    x[1] = 0.75
    x[2, 17, 33] = 40.0
    g = torch.Generator(device="cuda").manual_seed(3)
    x[3] = torch.randn((128, 128), generator=g, device="cuda") * 1e3
    x[4] = torch.randn((128, 128), generator=g, device="cuda") * 1e-3
    for kind in (0, 1):
        tiles, best = _quantize(K, x, kind, 2)
        compare_tiles_compact(tiles, tiles_to_host(x), kind, 2, best)


def _decode(K, built, q):
    p, cache = built.params, built.cache
    max_len = built.length + 1
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, built.n_q, max_len)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    K.kvarn_decode_attention(p, cache, built.n_q, q, K.KVARN_BF16, out, K.KVARN_F32, SCALE, max_len, ws, ws_bytes)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("bits,n_sink,name", [(2, 0, "llama"), (4, 128, "llama"), (2, 0, "stress")])
def test_compact_decode(K, bits, n_sink, name):
    """Decode over compact tiles: group sizes 4 and 5, sink, ragged lengths, split plan."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build(name, bits=bits, n_sink=n_sink, context=n_sink + 20 * 128 + 77, batch=3, aux=1)
    assert K.kvarn_tile_bytes(built.params) == (4608 if bits == 2 else 8704)
    lens = [built.length, n_sink + 2 * 128 + 5, n_sink + 131]
    built.cache.seq_len.copy_(torch.tensor(lens, dtype=torch.int32))
    q = workloads.decode_queries(built, seed=9)
    out = _decode(K, built, q)
    ref = oracle.decode(host_cache(built.cache), q_to_host(q), SCALE)
    check_output(out.cpu().numpy(), ref, bf16_out=False)


def test_compact_append_stream(K):
    """Appends across two flushes on the GPU and in the oracle; flushed tiles compared."""
    B, H, steps, bits = 2, 2, 2 * 128 + 9, 2
    p = _params(K, bits)
    cache = K.Cache(p, B, H, max_blocks=3)
    hc = oracle.HostCache(B, H, 3, bits=bits, aux=1)
    po = oracle.Params(bits=bits, aux=1)
    g = torch.Generator(device="cuda").manual_seed(17)
    scales = torch.exp(torch.randn((1, H, 128), generator=g, device="cuda"))
    ks, vs = [], []
    for t in range(steps):
        kt = (torch.randn((B, H, 128), generator=g, device="cuda") * scales).to(torch.bfloat16)
        vt = torch.randn((B, H, 128), generator=g, device="cuda").to(torch.bfloat16)
        K.kvarn_append_token(p, cache, kt, vt, K.KVARN_BF16, t)
        ks.append(q_to_host(kt))
        vs.append(q_to_host(vt))
        assert oracle.append(hc, ks[-1], vs[-1], po) == 0
    torch.cuda.synchronize()
    gc = host_cache(cache)
    np.testing.assert_array_equal(gc.seq_len, hc.seq_len)
    toks = {0: np.stack(ks), 1: np.stack(vs)}
    for kind, body in ((0, gc.k_body), (1, gc.v_body)):
        for blk in range(2):
            X = np.stack([oracle.bf16_bits_to_f64(toks[kind][blk * 128:(blk + 1) * 128, b, h])
                          for b in range(B) for h in range(H)])
            tiles = np.stack([body[b, h, blk] for b in range(B) for h in range(H)])
            compare_tiles_compact(tiles, X, kind, bits)
    q = torch.randn((B, 4 * H, 128), generator=g, device="cuda").to(torch.bfloat16)
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, 4 * H, steps + 1)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    K.kvarn_decode_attention(p, cache, 4 * H, q, K.KVARN_BF16, out, K.KVARN_F32, SCALE, steps + 1, ws, ws_bytes)
    torch.cuda.synchronize()
    check_output(out.cpu().numpy(), oracle.decode(gc, q_to_host(q), SCALE), bf16_out=False)
    raw = lambda b, h, blk, kind: oracle.bf16_bits_to_f64(toks[kind][blk * 128:(blk + 1) * 128, b, h])
    check_end_to_end(out.cpu().numpy(), hc, gc, raw, q_to_host(q), False, SCALE)  # end to end
