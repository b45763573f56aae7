"""Parity at the full sizes of the benchmark workloads.

The whole cache is built, extended through the append path (one flush included) and decoded
on the GPU in the launch configuration the benchmark times.  The oracle then recomputes a
seeded sample of 64 (sequence, kv head) streams one by one from the GPU's cache, re-quantizes a
sample of body tiles from inputs regenerated with the same seeds, and, end to end, builds its
own cache of a sample of streams from the same raw K/V (its own quantization of every body
tile, the appended tokens through its own append path) and decodes it.  Tolerances are those
of gpu_util."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (check_end_to_end, check_output, compare_tiles, compare_tiles_compact, host_streams, q_to_host,
                      tiles_to_host)

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module")
def K():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    torch.cuda.set_device(0)
    return kvarn


def _run(K, name, n_append, n_streams, n_tiles, out_dtype, aux=0, e2e_streams=8):
    from paper_2606_03458_amd import datagen, workloads
    spec = datagen.WORKLOADS[name]
    seed = datagen.SEEDS[name]
    built, inputs = workloads.build(name, extra_blocks=(n_append + 127) // 128 + 1, best_iter=True, aux=aux)
    compare = compare_tiles_compact if aux else compare_tiles
    p, cache = built.params, built.cache
    T0 = built.length
    appended = []
    for s in range(n_append):
        kt, vt = workloads.step_tokens(built, seed, s)
        assert K.kvarn_append_token(p, cache, kt, vt, K.KVARN_BF16, built.length) is None
        built.length += 1
        appended.append((kt, vt))
    assert int(cache.err_word.item()) == 0
    q = workloads.decode_queries(built, seed, 0)
    max_len = built.length + 1
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, built.n_q, max_len)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    out = torch.empty(q.shape, dtype=out_dtype, device="cuda")
    K.kvarn_decode_attention(p, cache, built.n_q, q, K.KVARN_BF16, out,
                             K.KVARN_BF16 if out_dtype == torch.bfloat16 else K.KVARN_F32, SCALE, max_len, ws,
                             ws_bytes)
    torch.cuda.synchronize()

    # decode: sampled streams, the first and the last included
    rng = np.random.default_rng(seed)
    n_kv, g = cache.n_kv, built.n_q // cache.n_kv
    total = cache.batch * n_kv
    pick = np.concatenate([[0, total - 1], 1 + rng.choice(total - 2, n_streams - 2, replace=False)])
    streams = [divmod(int(s), n_kv) for s in np.sort(pick)]
    hc = host_streams(cache, streams)
    qh = q_to_host(q)
    qs = np.stack([qh[b, kh * g:(kh + 1) * g] for b, kh in streams])
    ref = oracle.decode(hc, qs.reshape(len(streams), g, 128), SCALE)
    got = np.stack([out[b, kh * g:(kh + 1) * g].float().cpu().numpy() for b, kh in streams])
    worst = check_output(got, ref, bf16_out=out_dtype == torch.bfloat16)

    # quantize: body tiles of two layers from regenerated inputs, and the flushed tile; end to
    # end: the oracle's own cache of e2e_streams streams of those layers, built from the same
    # raw K/V, decoded by the oracle against the GPU's output for the same queries
    L, B = spec["layers"], spec["batch"]
    nb = T0 // 128
    stats = []
    e2e = {"streams": [], "K": [], "V": []}
    for layer in sorted({0, L - 1}):
        lseed = seed * 1000 + layer
        sig = datagen.channel_log_scales(lseed, n_kv, spec["dist"], device="cuda")
        Kx, Vx = datagen.kv_tokens(lseed, 0, B, n_kv, T0, spec["dist"], dtype=torch.bfloat16, device="cuda",
                                   sigma_c=sig)
        sel = [(int(rng.integers(B)), int(rng.integers(n_kv)), int(rng.integers(nb))) for _ in range(n_tiles)]
        for kind, X, body, best in ((K.KVARN_KEYS, Kx, cache.k_body, inputs["best_k"][layer]),
                                    (K.KVARN_VALUES, Vx, cache.v_body, inputs["best_v"][layer])):
            xs = torch.stack([X[b, kh, t * 128:(t + 1) * 128] for b, kh, t in sel])
            tiles = torch.stack([body[layer * B + b, kh, t] for b, kh, t in sel]).cpu().numpy()
            bi = np.array([int(best[(b * n_kv + kh) * nb + t]) for b, kh, t in sel])
            stats.append(compare(tiles, tiles_to_host(xs), kind, p.bits, gpu_best=bi))
        for _ in range(e2e_streams // 2 if L > 1 else e2e_streams):
            b, kh = int(rng.integers(B)), int(rng.integers(n_kv))
            e2e["streams"].append((layer * B + b, kh))
            for key, X, app in (("K", Kx, 0), ("V", Vx, 1)):
                tail = torch.stack([tok[app][layer * B + b, kh] for tok in appended])  # [n_append][128]
                e2e[key].append(torch.cat([X[b, kh], tail]).view(torch.int16).cpu().numpy().view(np.uint16))
        del Kx, Vx
    worst_e2e = _end_to_end(p, cache, e2e, out, q, g, T0, n_append, aux, out_dtype)
    if n_append >= 128:
        kst = torch.stack([k for k, _ in appended[:128]])  # [128, L*B, n_kv, 128]
        vst = torch.stack([v for _, v in appended[:128]])
        for kind, X, body in ((K.KVARN_KEYS, kst, cache.k_body), (K.KVARN_VALUES, vst, cache.v_body)):
            xs = torch.stack([X[:, b, kh] for b, kh in streams[:n_tiles]])
            tiles = torch.stack([body[b, kh, nb] for b, kh in streams[:n_tiles]]).cpu().numpy()
            stats.append(compare(tiles, tiles_to_host(xs), kind, p.bits))
    return worst, stats, worst_e2e


def _end_to_end(p, cache, e2e, out, q, g, prompt, n_append, aux, out_dtype):
    """The oracle quantizes the sampled streams' raw tokens itself (prefill of the prompt, then
    the appended tokens one by one through its append path: a flush and a residual) and
    decodes its own cache; the GPU output for the same streams must match it to the output bar
    (gpu_util.check_end_to_end: tiles where a rounding tie went the other way enter with the
    GPU's decision after passing the tile rules against the raw tokens)."""
    n = len(e2e["streams"])
    length = prompt + n_append
    assert all(k.shape == (length, 128) for k in e2e["K"] + e2e["V"])
    hc = oracle.HostCache(n, 1, (length + 127) // 128 + 1, bits=p.bits, aux=aux)
    po = oracle.Params(bits=p.bits, aux=aux)
    Ks, Vs = np.stack(e2e["K"]), np.stack(e2e["V"])  # [n][length][128] bf16 bits
    cu = np.arange(n + 1, dtype=np.int32) * prompt
    assert oracle.prefill(hc, np.ascontiguousarray(Ks[:, :prompt].reshape(-1, 1, 128)),
                          np.ascontiguousarray(Vs[:, :prompt].reshape(-1, 1, 128)), cu, prompt, po) == 0
    for t in range(prompt, length):
        assert oracle.append(hc, np.ascontiguousarray(Ks[:, t, None]), np.ascontiguousarray(Vs[:, t, None]), po) == 0
    assert np.all(hc.seq_len == length)
    qh = q_to_host(q)
    qs = np.stack([qh[b, kh * g:(kh + 1) * g] for b, kh in e2e["streams"]])
    got = np.stack([out[b, kh * g:(kh + 1) * g].float().cpu().numpy() for b, kh in e2e["streams"]])
    raw = lambda b, kh, blk, kind: oracle.bf16_bits_to_f64((Ks, Vs)[kind][b, blk * 128:(blk + 1) * 128])
    return check_end_to_end(got, hc, host_streams(cache, e2e["streams"]), raw, qs, out_dtype == torch.bfloat16,
                            SCALE)


def test_full_size_throughput(K):
    """32 layers x batch 32 (1024 sequences), 32 q / 8 kv heads, 32768-token 2-bit cache plus
    132 appended tokens (one flush), bf16 q and output, a single split per stream."""
    _run(K, "throughput", n_append=132, n_streams=64, n_tiles=12, out_dtype=torch.bfloat16)


def test_full_size_stress(K):
    """Heavy-tailed keys, 40 q / 8 kv heads (GQA 5), batch 128, 16384-token 2-bit cache."""
    _run(K, "stress", n_append=130, n_streams=64, n_tiles=12, out_dtype=torch.float32)


def test_full_size_gqa8(K):
    """Query groups of 8 (64 q / 8 kv heads, two head groups per wave), batch 128, 16384-token
    2-bit cache."""
    _run(K, "gqa8", n_append=130, n_streams=64, n_tiles=12, out_dtype=torch.bfloat16)


def test_full_size_throughput_compact(K):
    """The throughput workload with the compact aux format (2.25 bits/element)."""
    _run(K, "throughput", n_append=130, n_streams=64, n_tiles=12, out_dtype=torch.bfloat16, aux=1)


def test_full_size_stress_compact(K):
    """The stress workload with the compact aux format."""
    _run(K, "stress", n_append=130, n_streams=64, n_tiles=12, out_dtype=torch.float32, aux=1)


@pytest.mark.parametrize("bits,aux", [(2, 0), (4, 0), (2, 1)])
def test_full_size_streaming(K, bits, aux):
    """The streaming workload's shape (64 sequences x 8 kv heads, 32 q heads) from an empty
    cache: 261 tokens appended one step at a time (two flushes of 1024 tiles each), decoded at
    the steps around the flushes in the benchmark's launch configuration; sampled streams are
    recomputed by the oracle from the GPU cache, and the flushed tiles are re-quantized by the
    oracle from the appended tokens."""
    from paper_2606_03458_amd import datagen
    spec = datagen.WORKLOADS["streaming"]
    seed = datagen.SEEDS["streaming"]
    B, n_kv, n_q = spec["batch"], spec["n_kv"], spec["n_q"]
    g, T = n_q // n_kv, 2 * 128 + 5
    p = K.kvarn_params_init(bits, aux_format=aux)
    cache = K.Cache(p, B, n_kv, 3)
    sig = datagen.channel_log_scales(seed * 1000, n_kv, spec["dist"], device="cuda")
    Kx, Vx = datagen.kv_tokens(seed * 1000, 0, B, n_kv, T, spec["dist"], dtype=torch.bfloat16, device="cuda",
                               sigma_c=sig)
    rng = np.random.default_rng(seed)
    total = B * n_kv
    pick = np.unique(np.concatenate([[0, total - 1], rng.choice(total, 14, replace=False)]))
    streams = [divmod(int(s), n_kv) for s in pick]
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, n_q, T)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    for t in range(T):
        kt, vt = Kx[:, :, t].contiguous(), Vx[:, :, t].contiguous()
        assert K.kvarn_append_token(p, cache, kt, vt, K.KVARN_BF16, t) is None
        if t in (0, 126, 127, 128, 255, T - 1):
            q = datagen.queries(seed, t, B, n_q, dtype=torch.bfloat16, device="cuda")
            out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
            K.kvarn_decode_attention(p, cache, n_q, q, K.KVARN_BF16, out, K.KVARN_F32, SCALE, t + 1, ws, ws_bytes)
            torch.cuda.synchronize()
            assert np.all(cache.seq_len.cpu().numpy() == t + 1)
            hc = host_streams(cache, streams)
            qh = q_to_host(q)
            qs = np.stack([qh[b, kh * g:(kh + 1) * g] for b, kh in streams])
            ref = oracle.decode(hc, qs, SCALE)
            got = np.stack([out[b, kh * g:(kh + 1) * g].cpu().numpy() for b, kh in streams])
            check_output(got, ref, bf16_out=False)
    assert int(cache.err_word.item()) == 0
    compare = compare_tiles_compact if aux else compare_tiles
    for blk in range(2):
        for kind, X, body in ((K.KVARN_KEYS, Kx, cache.k_body), (K.KVARN_VALUES, Vx, cache.v_body)):
            xs = torch.stack([X[b, kh, 128 * blk:128 * (blk + 1)] for b, kh in streams])
            tiles = torch.stack([body[b, kh, blk] for b, kh in streams]).cpu().numpy()
            compare(tiles, tiles_to_host(xs), kind, bits)
