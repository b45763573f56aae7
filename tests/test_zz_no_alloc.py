"""The allocation-free decode entry point (kvarn_decode_attention_noalloc) through the C ABI:
its output equals kvarn_decode_attention's on the same cache and queries (the same kernels,
the split partials in the library's per-device scratch array instead of a caller workspace),
and meets the output bar against the oracle, on consecutive calls whose split plans shrink, so
that a later call finds the earlier call's partials in the shared array."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import check_output, host_cache, q_to_host

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module")
def K():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    torch.cuda.set_device(0)
    return kvarn


def _case(K, batch, n_q, n_kv, context, bits, aux, n_sink, seed):
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", bits=bits, n_sink=n_sink, context=context, batch=batch, n_q=n_q, n_kv=n_kv,
                               aux=aux)
    lens = [context - 131 * b for b in range(batch)]  # ragged: the plan still splits the longest
    built.cache.seq_len.copy_(torch.tensor(lens, dtype=torch.int32))
    q = workloads.decode_queries(built, seed=seed)
    return built, q


def _both(K, built, q):
    p, cache, n_q = built.params, built.cache, built.n_q
    max_len = built.length
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, n_q, max_len)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    ref = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    got = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    K.kvarn_decode_attention(p, cache, n_q, q, K.KVARN_BF16, ref, K.KVARN_F32, SCALE, max_len, ws, ws_bytes)
    K.kvarn_decode_attention_noalloc(p, cache, n_q, q, K.KVARN_BF16, got, K.KVARN_F32, SCALE, max_len)
    torch.cuda.synchronize()
    return ws_bytes, ref, got


def test_noalloc_equals_decode(K):
    cases = [  # (batch, n_q, n_kv, context, bits, aux, n_sink): each plan smaller than the one before
        (3, 40, 8, 40 * 128 + 77, 2, 0, 0),
        (2, 32, 8, 24 * 128 + 5, 4, 1, 128),
        (1, 8, 2, 12 * 128 + 100, 2, 0, 0),
        (2, 8, 2, 3 * 128 + 3, 2, 0, 0),  # one split per stream: no partials at all
    ]
    sizes = []
    for i, (B, nq, nkv, T, bits, aux, ns) in enumerate(cases):
        built, q = _case(K, B, nq, nkv, T, bits, aux, ns, seed=20 + i)
        ws_bytes, ref, got = _both(K, built, q)
        sizes.append(ws_bytes)
        assert ws_bytes <= K.NOALLOC_SCRATCH_BYTES
        assert bool(torch.isfinite(got).all())
        assert torch.equal(got, ref), i  # same kernels and plan: bit-identical
        check_output(got.cpu().numpy(), oracle.decode(host_cache(built.cache), q_to_host(q), SCALE), bf16_out=False)
    assert sizes[0] > sizes[1] > sizes[2] > 0 and sizes[3] == 0, sizes
