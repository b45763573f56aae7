"""GPU parity: the HIP path through the C ABI against the CPU oracle, on the same seeded
inputs (exact bytes copied to the host).  Tolerances are defined in gpu_util."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (check_end_to_end, check_output, compare_tiles, host_cache, oracle_cache_from_inputs,
                      q_to_host, tiles_to_host)

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module")
def K():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    torch.cuda.set_device(0)
    return kvarn


def _quantize(K, x: torch.Tensor, kind: int, bits: int, **pover):
    """x [n, 128, 128] on the GPU -> (tiles uint8 [n, tile_bytes], best [n])."""
    n = x.shape[0]
    p = K.kvarn_params_init(bits, **pover)
    out = torch.zeros((n, K.kvarn_tile_bytes(p)), dtype=torch.uint8, device="cuda")
    best = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    dt = K.KVARN_F32 if x.dtype == torch.float32 else K.KVARN_BF16
    K.kvarn_quantize_block(p, kind, x, dt, n, 1, 128 * 128, 0, 128, out, 1, 0, best)
    torch.cuda.synchronize()
    return out.cpu().numpy(), best.cpu().numpy()


def _sample_tiles(dist, n, dtype, seed):
    from paper_2606_03458_amd import datagen
    Kx, Vx = datagen.kv_tokens(seed, 0, 1, 2, n * 64, dist, dtype=dtype, device="cuda")
    return Kx.reshape(n, 128, 128).contiguous(), Vx.reshape(n, 128, 128).contiguous()


# ---- quantizer --------------------------------------------------------------------------

def test_quantize_tiny_fp32(K):
    """Tiny workload: 256 tokens of fp32 K and V (2 tiles each), 2-bit, seed 0."""
    from paper_2606_03458_amd import datagen
    Kx, Vx = datagen.kv_tokens(0, 0, 1, 1, 256, "llama", dtype=torch.float32, device="cuda")
    for kind, x in ((0, Kx), (1, Vx)):
        xt = x.reshape(2, 128, 128).contiguous()
        tiles, best = _quantize(K, xt, kind, 2)
        st = compare_tiles(tiles, tiles_to_host(xt), kind, 2, best)
        assert st["codes"] == 2 * 16384


@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("dist", ["llama", "stress"])
def test_quantize_bf16_tiles(K, bits, dist):
    """32 bf16 tiles of each of K and V drawn like the llama / heavy-tailed workloads."""
    Kx, Vx = _sample_tiles(dist, 32, torch.bfloat16, seed=11 + bits)
    for kind, x in ((0, Kx), (1, Vx)):
        tiles, best = _quantize(K, x, kind, bits)
        compare_tiles(tiles, tiles_to_host(x), kind, bits, best)


def test_quantize_degenerate_tiles(K):
    """Zero, constant, single-outlier and huge-range tiles, and iteration counts 0 and 1."""
    x = torch.zeros((5, 128, 128), dtype=torch.float32, device="cuda")
    x[1] = 0.75
    x[2, 17, 33] = 40.0
    x[3] = torch.randn((128, 128), device="cuda") * 1e4
    x[4] = torch.randn((128, 128), device="cuda") * 1e-3
    for kind in (0, 1):
        for iters in (8, 0, 1):
            tiles, best = _quantize(K, x, kind, 2, varn_iters=iters)
            compare_tiles(tiles, tiles_to_host(x), kind, 2, best, params=oracle.Params(bits=2, varn_iters=iters))


def test_quantize_strided_views(K):
    """Tiles read through strides: a [T][H][128] token-major layout (token stride H*128),
    several outer/inner tiles, written to a strided output."""
    H, T, S = 3, 256, 2
    x = torch.randn((S, T, H, 128), device="cuda", dtype=torch.bfloat16) * 2
    p = K.kvarn_params_init(2)
    tb = K.kvarn_tile_bytes(K.kvarn_params_init(2))
    out = torch.zeros((S * H, 5, tb), dtype=torch.uint8, device="cuda")
    for s in range(S):
        # outer = head, inner = block; out row s*H + h, tiles at blocks 1 and 3 (stride 2)
        K.kvarn_quantize_block(p, 1, x[s], K.KVARN_BF16, H, T // 128, 128, 128 * H * 128, H * 128,
                               out[s * H:, 1:], 5, 2, None)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    for s in range(S):
        for h in range(H):
            for blk in range(2):
                X = x[s, blk * 128:(blk + 1) * 128, h].float().cpu().numpy().astype(np.float64)
                compare_tiles(o[s * H + h, 1 + 2 * blk][None], X[None], 1, 2)
            for untouched in (0, 2, 4):
                assert not o[s * H + h, untouched].any()


def test_quantize_deterministic(K):
    Kx, _ = _sample_tiles("llama", 16, torch.bfloat16, seed=5)
    t1, _ = _quantize(K, Kx, 0, 2)
    t2, _ = _quantize(K, Kx, 0, 2)
    np.testing.assert_array_equal(t1, t2)


# ---- decode attention ---------------------------------------------------------------------

def _decode(K, built, q, out_dtype=torch.float32, max_len=None):
    p, cache = built.params, built.cache
    max_len = built.length + 1 if max_len is None else max_len
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, built.n_q, max_len)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    out = torch.empty(q.shape, dtype=out_dtype, device="cuda")
    qd = K.KVARN_F32 if q.dtype == torch.float32 else K.KVARN_BF16
    od = K.KVARN_F32 if out_dtype == torch.float32 else K.KVARN_BF16
    K.kvarn_decode_attention(p, cache, built.n_q, q, qd, out, od, SCALE, max_len, ws, ws_bytes)
    torch.cuda.synchronize()
    return out


def _ref(built, q):
    return oracle.decode(host_cache(built.cache), q_to_host(q), SCALE)


def _raw_tile(inputs):
    """Raw tokens of body tile blk of (sequence b, kv head kh) of a one-layer workload."""
    return lambda b, kh, blk, kind: tiles_to_host((inputs["K"], inputs["V"])[kind][0][b, kh, blk * 128:(blk + 1) * 128])


def test_decode_tiny(K):
    """Tiny workload: decode over the GPU's cache, and end to end against the oracle's own cache
    of the same fp32 K/V (its own quantization of both tiles of K and of V)."""
    from paper_2606_03458_amd import workloads
    built, inputs = workloads.build("tiny", keep_inputs=True)
    q = workloads.decode_queries(built, seed=0)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)
    hc = oracle_cache_from_inputs(built, inputs)
    check_end_to_end(out.cpu().numpy(), hc, host_cache(built.cache), _raw_tile(inputs), q_to_host(q), False, SCALE)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_decode_llama_layer(K, out_dtype):
    """Llama-3-8B-shaped layer: 32 q / 8 kv heads, 8192-token prefill, then one appended
    token (residual = 1), bf16 q."""
    from paper_2606_03458_amd import workloads
    built, inputs = workloads.build("llama", keep_inputs=True)
    kt, vt = workloads.step_tokens(built, seed=1, step=0)
    K.kvarn_append_token(built.params, built.cache, kt, vt, K.KVARN_BF16, built.length)
    built.length += 1
    q = workloads.decode_queries(built, seed=1)
    out = _decode(K, built, q, out_dtype)
    assert int(built.cache.seq_len[0]) == 8193
    got = out.float().cpu().numpy()
    check_output(got, _ref(built, q), bf16_out=out_dtype == torch.bfloat16)
    # end to end, all 8 kv-head streams: the oracle's own cache of the same K/V and token
    hc = oracle_cache_from_inputs(built, inputs, appended=[(kt, vt)])
    check_end_to_end(got, hc, host_cache(built.cache), _raw_tile(inputs), q_to_host(q),
                     out_dtype == torch.bfloat16, SCALE)


@pytest.mark.parametrize("bits,n_sink,name", [(2, 128, "llama"), (4, 0, "llama"), (2, 0, "stress"),
                                              (4, 128, "stress"), (2, 100, "llama"), (4, 100, "stress")])
def test_decode_variants(K, bits, n_sink, name):
    """Sink region, 4-bit codes, GQA 5, ragged lengths (including 0 and sink-only) and a
    residual, on a small batch that the split-K plan divides into many splits."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build(name, bits=bits, n_sink=n_sink, context=n_sink + 20 * 128 + 77, batch=5)
    lens = [built.length, n_sink + 2 * 128, n_sink + 131, n_sink // 2 if n_sink else 0, 0]
    built.cache.seq_len.copy_(torch.tensor(lens, dtype=torch.int32))
    q = workloads.decode_queries(built, seed=3)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)


@pytest.mark.parametrize("batch,n_sink,body,n_split", [
    (2, 100, 20, 18),   # 10 body splits + one per sink / residual chunk (4 + 4)
    (31, 0, 20, 11),    # 10 body splits + one split for all chunks (one per chunk would not fit)
    (31, 0, 24, 12),    # 12 body splits sharing the chunks
])
def test_decode_residual_placement(K, batch, n_sink, body, n_split):
    """The three places the split plan gives a stream's sink and residual chunks (32 tokens
    each) when the partials go to memory (fewer than 256 streams): a split per chunk, one split
    for all chunks, or the body splits in turn.  Ragged lengths
    give every residual size class (empty, one token, a partial and full chunks, 127 tokens) and a
    sink-only sequence; the split count is checked through the workspace size."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", n_sink=n_sink, context=n_sink + body * 128 + 77, batch=batch)
    L = built.length
    base = n_sink + (body - 1) * 128
    cycle = [L, base, base + 1, base + 31, base + 32, base + 33, base + 100, base + 127, n_sink // 2]
    lens = [cycle[i % len(cycle)] for i in range(batch)]
    built.cache.seq_len.copy_(torch.tensor(lens, dtype=torch.int32))
    ws_bytes = K.kvarn_decode_workspace_bytes(built.params, built.cache, built.n_q, L + 1)
    assert ws_bytes == batch * built.n_q * n_split * 1040
    q = workloads.decode_queries(built, seed=9)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)


@pytest.mark.parametrize("bits,n_q,body,n_split", [
    (2, 16, 64, 68),   # 32 body splits + one split per sink / residual chunk (32 + 4)
    (2, 16, 3, 1),     # one wave per stream walks all 36 chunks after its 3 tiles
    (4, 40, 20, 46),   # 4 bits, group size 10 (two chunks of 5 heads: the extra-head kernel)
])
def test_decode_max_sink(K, bits, n_q, body, n_split):
    """The largest sink the library takes (1024 bf16 tokens: 32 chunks per stream) with a
    residual, ragged lengths down to sink-only and empty; the split count through the workspace
    size."""
    from paper_2606_03458_amd import workloads
    ns = 1024
    built, _ = workloads.build("llama", bits=bits, n_q=n_q, n_kv=4, batch=4, n_sink=ns, context=ns + body * 128 + 77)
    L = built.length
    lens = [L, ns + 5, ns - 1, 0]
    built.cache.seq_len.copy_(torch.tensor(lens, dtype=torch.int32))
    ws_bytes = K.kvarn_decode_workspace_bytes(built.params, built.cache, built.n_q, L + 1)
    assert ws_bytes == (4 * n_q * n_split * 1040 if n_split > 1 else 0)
    q = workloads.decode_queries(built, seed=12)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)


def test_decode_long_context(K):
    """One sequence of 262,221 tokens (2048 body tiles per kv head, 8 kv heads): 342 body splits
    of 6 tiles and 4 residual-chunk splits per stream, merged by four waves per query head over
    346 partials."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", batch=1, context=2048 * 128 + 77)
    L = built.length
    ws_bytes = K.kvarn_decode_workspace_bytes(built.params, built.cache, built.n_q, L + 1)
    assert ws_bytes == 1 * 32 * 346 * 1040
    q = workloads.decode_queries(built, seed=13)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)


@pytest.mark.parametrize("bits,n_q,batch,aux,n_sink", [
    (2, 8, 768, 0, 0),     # group 4: 1536 streams, two splits each
    (4, 8, 512, 1, 128),   # group 4 at 4 bits, compact aux, a sink for the second split
    (2, 10, 512, 0, 0),    # group 5 (the extra-head variant)
    (4, 16, 512, 0, 100),  # group 8 (two head groups) at 4 bits, partial sink chunks
])
def test_decode_pair_mode(K, bits, n_q, batch, aux, n_sink):
    """Streams of exactly two splits that share the sink/residual chunks (batch x 2 kv heads just
    below two rounds of resident waves) run as the two waves of one workgroup and merge there: no
    workspace.  Ragged lengths give a second split without body tiles, a sink-only and an empty
    sequence."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", bits=bits, n_q=n_q, n_kv=2, batch=batch, aux=aux, n_sink=n_sink,
                               context=n_sink + 4 * 128 + 77)
    L = built.length
    cycle = [L, n_sink + 2 * 128 + 5, n_sink + 128, n_sink + 3, n_sink // 2, 0, L - 64]
    lens = [cycle[i % len(cycle)] for i in range(batch)]
    built.cache.seq_len.copy_(torch.tensor(lens, dtype=torch.int32))
    # (one split per stream would leave a third of the wave slots empty: the plan is two splits)
    assert K.kvarn_decode_workspace_bytes(built.params, built.cache, n_q, L + 1) == 0
    q = workloads.decode_queries(built, seed=10)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)


@pytest.mark.parametrize("bits,n_q,batch,tiles,aux,n_sink", [
    (2, 32, 80, 8, 0, 0),     # group 4: 3 body splits + one sink/residual split (a short stream)
    (2, 32, 64, 50, 0, 0),    # group 4: 4 body splits sharing the residual chunks
    (2, 32, 96, 6, 1, 0),     # group 4, compact aux: 3 body splits + one sink/residual split
    (4, 32, 64, 12, 0, 128),  # group 4 at 4 bits with a sink: 3 body splits + one sink/residual split
    (4, 32, 64, 50, 1, 100),  # the same at 4 bits, compact aux, 4 body splits sharing the chunks
    (2, 40, 48, 6, 0, 0),     # group 5 (the extra-head variant): 3 body splits + one residual split
    (2, 64, 64, 12, 0, 0),    # group 8 (two head groups): 3 body splits + one residual split
    (2, 128, 48, 12, 0, 0),   # group 16 (two chunks of 8 heads, a workgroup per chunk): 3 body splits
])
def test_decode_group_mode(K, bits, n_q, batch, tiles, aux, n_sink):
    """Streams of three or four splits (batch x 8 kv heads, 384 to 768 streams) run as the waves
    of one workgroup and merge there: no workspace.  Ragged lengths leave later splits without body
    tiles, and give sink-only and empty sequences."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", bits=bits, n_q=n_q, n_kv=8, batch=batch, aux=aux, n_sink=n_sink,
                               context=n_sink + tiles * 128 + 77)
    L = built.length
    cycle = [L, n_sink + 5 * 128 + 1, n_sink + 2 * 128 + 100, n_sink + 40, n_sink // 2, 0, L - 100, n_sink + 128]
    lens = [cycle[i % len(cycle)] for i in range(batch)]
    built.cache.seq_len.copy_(torch.tensor(lens, dtype=torch.int32))
    assert K.kvarn_decode_workspace_bytes(built.params, built.cache, n_q, L + 1) == 0
    q = workloads.decode_queries(built, seed=11)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)
    # the same cache behind a block table over a permuted pool: bit-equal
    c = built.cache
    B, H, MB = c.batch, c.n_kv, c.max_blocks
    paged = K.Cache(built.params, B, H, MB, n_phys=B * MB)
    perm = torch.randperm(B * MB, generator=torch.Generator().manual_seed(bits + n_q)).cuda()
    paged.block_table.copy_(perm.view(B, MB).to(torch.int32))
    for src, dst in ((c.k_body, paged.k_body), (c.v_body, paged.v_body)):
        dst.index_copy_(0, perm, src.permute(0, 2, 1, 3).reshape(B * MB, H, -1))
    for f in ("k_resid", "v_resid", "k_sink", "v_sink", "seq_len"):
        if getattr(c, f) is not None:
            getattr(paged, f).copy_(getattr(c, f))
    built.cache = paged
    assert torch.equal(_decode(K, built, q), out)


@pytest.mark.parametrize("n_q,n_kv", [(2, 2), (4, 2), (6, 2), (8, 2), (10, 2), (12, 2), (32, 2)])
def test_decode_group_sizes(K, n_q, n_kv):
    """Every query-group size class (1 .. 4, 5, 6 .. 8, 9 .. 16 take different kernels), with a
    residual and enough body tiles for the plan to split every stream."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", context=12 * 128 + 45, batch=2, n_q=n_q, n_kv=n_kv)
    q = workloads.decode_queries(built, seed=6)
    out = _decode(K, built, q)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)


@pytest.mark.parametrize("mult", [4.0, 16.0])
def test_decode_peaked_softmax(K, mult):
    """Logits scaled up so that most tiles' probabilities sit near or below fp32 underflow
    relative to the running maximum: the output stays finite and matches the oracle."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", context=64 * 128 + 3, batch=2)
    q = workloads.decode_queries(built, seed=7)
    p, cache = built.params, built.cache
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    max_len = built.length + 1
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, built.n_q, max_len)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    K.kvarn_decode_attention(p, cache, built.n_q, q, K.KVARN_BF16, out, K.KVARN_F32, SCALE * mult, max_len, ws,
                             ws_bytes)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all())
    ref = oracle.decode(host_cache(cache), q_to_host(q), SCALE * mult)
    check_output(out.cpu().numpy(), ref, bf16_out=False)


def test_decode_length_above_hint(K):
    """A max_len_hint below the true length still attends every token (last split extends)."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", context=2048, batch=1)
    q = workloads.decode_queries(built, seed=4)
    out = _decode(K, built, q, max_len=300)
    check_output(out.cpu().numpy(), _ref(built, q), bf16_out=False)


def test_decode_workspace_reuse(K):
    """One workspace serves consecutive calls on caches of different shapes and split plans (more
    streams after fewer, many splits after few; every kernel family): each call rewrites what it
    reads, so every output equals that of a call with a fresh workspace."""
    from paper_2606_03458_amd import workloads
    cases = []
    for i, (batch, n_q, n_kv, ctx) in enumerate([(1, 32, 8, 64 * 128 + 40), (6, 40, 8, 24 * 128 + 5),
                                                  (2, 64, 4, 40 * 128 + 99), (1, 8, 1, 96 * 128 + 1)]):
        built, _ = workloads.build("llama", context=ctx, batch=batch, n_q=n_q, n_kv=n_kv)
        cases.append((built, workloads.decode_queries(built, seed=40 + i)))
    sizes = [K.kvarn_decode_workspace_bytes(b.params, b.cache, b.n_q, b.length) for b, _ in cases]
    assert all(n > 0 for n in sizes)
    shared = torch.zeros(max(sizes), dtype=torch.uint8, device="cuda")
    for rep in range(2):
        for (built, q), n in zip(cases, sizes):
            p, cache = built.params, built.cache
            got = torch.empty(q.shape, dtype=torch.float32, device="cuda")
            ref = torch.empty(q.shape, dtype=torch.float32, device="cuda")
            K.kvarn_decode_attention(p, cache, built.n_q, q, K.KVARN_BF16, got, K.KVARN_F32, SCALE, built.length,
                                     shared, shared.numel())
            fresh = torch.zeros(n, dtype=torch.uint8, device="cuda")
            K.kvarn_decode_attention(p, cache, built.n_q, q, K.KVARN_BF16, ref, K.KVARN_F32, SCALE, built.length,
                                     fresh, n)
            torch.cuda.synchronize()
            assert torch.equal(got, ref), (rep, n)
    check_output(got.cpu().numpy(), _ref(cases[-1][0], cases[-1][1]), bf16_out=False)


def test_decode_deterministic(K):
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", context=1024 + 5, batch=2)
    q = workloads.decode_queries(built, seed=5)
    o1 = _decode(K, built, q)
    o2 = _decode(K, built, q)
    assert torch.equal(o1, o2)


# ---- streaming append ---------------------------------------------------------------------

@pytest.mark.parametrize("bits,n_sink,hint", [(2, 0, True), (4, 128, True), (2, 128, False)])
def test_append_stream(K, bits, n_sink, hint):
    """Append tokens one by one from an empty cache (flushes included), on the GPU and in
    the oracle, from the same bf16 tokens."""
    B, H, steps = 2, 2, n_sink + 2 * 128 + 9
    p = K.kvarn_params_init(bits)
    p.n_sink = n_sink
    cache = K.Cache(p, B, H, max_blocks=3)
    hc = oracle.HostCache(B, H, 3, bits=bits, n_sink=n_sink)
    po = oracle.Params(bits=bits)
    g = torch.Generator(device="cuda").manual_seed(7)
    scales = torch.exp(torch.randn((1, H, 128), generator=g, device="cuda"))
    ks, vs = [], []
    for t in range(steps):
        kt = (torch.randn((B, H, 128), generator=g, device="cuda") * scales).to(torch.bfloat16)
        vt = torch.randn((B, H, 128), generator=g, device="cuda").to(torch.bfloat16)
        K.kvarn_append_token(p, cache, kt, vt, K.KVARN_BF16, t if hint else -1)
        ks.append(q_to_host(kt))
        vs.append(q_to_host(vt))
        assert oracle.append(hc, ks[-1], vs[-1], po) == 0
    torch.cuda.synchronize()
    gc = host_cache(cache)
    np.testing.assert_array_equal(gc.seq_len, hc.seq_len)
    np.testing.assert_array_equal(gc.k_resid, hc.k_resid)
    np.testing.assert_array_equal(gc.v_resid, hc.v_resid)
    if n_sink:
        np.testing.assert_array_equal(gc.k_sink, hc.k_sink)
        np.testing.assert_array_equal(gc.v_sink, hc.v_sink)
    # body tiles: both sides quantized the same 128 bf16 tokens of each stream
    toks = {0: np.stack(ks), 1: np.stack(vs)}  # [steps, B, H, 128]
    for kind, body in ((0, gc.k_body), (1, gc.v_body)):
        for blk in range(2):
            t0 = n_sink + blk * 128
            for b in range(B):
                for h in range(H):
                    X = oracle.bf16_bits_to_f64(toks[kind][t0:t0 + 128, b, h])
                    compare_tiles(body[b, h, blk][None], X[None], kind, bits)
    assert not gc.k_body[:, :, 2].any() and not gc.v_body[:, :, 2].any()
    assert int(cache.err_word[0]) == 0
    # decode over the GPU's cache, and end to end over the oracle's own (its own flushes)
    q = torch.randn((B, 4 * H, 128), generator=g, device="cuda").to(torch.bfloat16)
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, 4 * H, steps + 1)
    ws = torch.zeros(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    K.kvarn_decode_attention(p, cache, 4 * H, q, K.KVARN_BF16, out, K.KVARN_F32, SCALE, steps + 1, ws, ws_bytes)
    torch.cuda.synchronize()
    check_output(out.cpu().numpy(), oracle.decode(gc, q_to_host(q), SCALE), bf16_out=False)
    raw = lambda b, h, blk, kind: oracle.bf16_bits_to_f64(toks[kind][n_sink + blk * 128:n_sink + (blk + 1) * 128, b, h])
    check_end_to_end(out.cpu().numpy(), hc, gc, raw, q_to_host(q), False, SCALE)


def test_append_no_hint_many_tiles(K):
    """Without the length hint the flush runs on a resident-size grid whose workgroups check
    several tiles each (here 1536 tiles): sequences of staggered lengths, 130 appends each, must
    leave exactly the cache that a prefill of the whole final sequences writes (the same
    quantizer on the same bf16 rows), and then decode identically."""
    B, H, steps = 384, 2, 130
    g = torch.Generator(device="cuda").manual_seed(9)
    lens = torch.randint(0, 300, (B,), generator=g, device="cuda").cpu().numpy()
    final = lens + steps
    MB = int(final.max()) // 128 + 1
    total = int(final.sum())
    k = (torch.randn((total, H, 128), generator=g, device="cuda") * 3).to(torch.bfloat16)
    v = torch.randn((total, H, 128), generator=g, device="cuda").to(torch.bfloat16)
    cu_f = np.concatenate([[0], np.cumsum(final)]).astype(np.int32)
    p = K.kvarn_params_init(2)
    full = K.Cache(p, B, H, MB)
    K.kvarn_prefill(p, full, k, v, K.KVARN_BF16, torch.tensor(cu_f, device="cuda"), int(final.max()))
    # the prompts (first lens[b] rows of each sequence), then the rest one token per call
    idx = np.concatenate([np.arange(cu_f[b], cu_f[b] + lens[b]) for b in range(B)]).astype(np.int64)
    idx_t = torch.tensor(idx, device="cuda")
    cu_p = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    inc = K.Cache(p, B, H, MB)
    K.kvarn_prefill(p, inc, k[idx_t].contiguous(), v[idx_t].contiguous(), K.KVARN_BF16,
                    torch.tensor(cu_p, device="cuda"), int(lens.max()))
    starts = torch.tensor(cu_f[:-1] + lens, device="cuda", dtype=torch.int64)
    for t in range(steps):
        K.kvarn_append_token(p, inc, k[starts + t].contiguous(), v[starts + t].contiguous(), K.KVARN_BF16, -1)
    torch.cuda.synchronize()
    assert int(inc.err_word[0]) == 0 and int(full.err_word[0]) == 0
    assert torch.equal(inc.seq_len, full.seq_len)
    for b in range(B):
        nb, nr = int(final[b]) // 128, int(final[b]) % 128
        assert torch.equal(inc.k_body[b, :, :nb], full.k_body[b, :, :nb]), b
        assert torch.equal(inc.v_body[b, :, :nb], full.v_body[b, :, :nb]), b
        assert torch.equal(inc.k_resid[b, :, :nr], full.k_resid[b, :, :nr]), b
        assert torch.equal(inc.v_resid[b, :, :nr], full.v_resid[b, :, :nr]), b
    q = torch.randn((B, 4 * H, 128), generator=g, device="cuda").to(torch.bfloat16)
    outs = []
    for c in (inc, full):
        ws_bytes = K.kvarn_decode_workspace_bytes(p, c, 4 * H, int(final.max()))
        ws = torch.zeros(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
        out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
        K.kvarn_decode_attention(p, c, 4 * H, q, K.KVARN_BF16, out, K.KVARN_F32, SCALE, int(final.max()), ws, ws_bytes)
        outs.append(out)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


def test_append_overflow_flag(K):
    """With no length hint, a flush that has no body tile left is refused on the device: the
    token is dropped, err_word is set, and nothing is written out of bounds."""
    p = K.kvarn_params_init(2)
    cache = K.Cache(p, 1, 1, max_blocks=1)
    tok = torch.ones((1, 1, 128), dtype=torch.bfloat16, device="cuda")
    for t in range(128 + 127):
        K.kvarn_append_token(p, cache, tok, tok, K.KVARN_BF16, -1)
    torch.cuda.synchronize()
    assert int(cache.err_word[0]) == 0 and int(cache.seq_len[0]) == 255
    K.kvarn_append_token(p, cache, tok, tok, K.KVARN_BF16, -1)
    torch.cuda.synchronize()
    assert int(cache.err_word[0]) == 1 and int(cache.seq_len[0]) == 255
    with pytest.raises(K.KVarNError) as e:
        K.kvarn_append_token(p, cache, tok, tok, K.KVARN_BF16, 255)
    assert e.value.status == -3
