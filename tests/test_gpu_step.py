"""The fused decode step (kvarn_append_decode, Fig. 4's append-then-attend step over the App. D
cache) against its definition: kvarn_append_token followed by kvarn_decode_attention on a copy
of the same cache, bit for bit in the output and in every cache buffer, over steps that cross a
flush (the fused launch on the steps that only append to the residual, the two kernels on the
others); and the device-side check of the lock-step length."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)
FIELDS = ("k_body", "v_body", "k_resid", "v_resid", "k_sink", "v_sink", "seq_len", "err_word", "block_table")


@pytest.fixture(scope="module")
def K():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    torch.cuda.set_device(0)
    return kvarn


def _clone(K, p, c):
    d = K.Cache(p, c.batch, c.n_kv, c.max_blocks, n_phys=c.n_phys)
    for f in FIELDS:
        if getattr(c, f) is not None:
            getattr(d, f).copy_(getattr(c, f))
    return d


def _paged(K, p, c, seed):
    B, H, MB = c.batch, c.n_kv, c.max_blocks
    d = K.Cache(p, B, H, MB, n_phys=B * MB)
    perm = torch.randperm(B * MB, generator=torch.Generator().manual_seed(seed)).cuda()
    d.block_table.copy_(perm.view(B, MB).to(torch.int32))
    for src, dst in ((c.k_body, d.k_body), (c.v_body, d.v_body)):
        dst.index_copy_(0, perm, src.permute(0, 2, 1, 3).reshape(B * MB, H, -1))
    for f in ("k_resid", "v_resid", "k_sink", "v_sink", "seq_len"):
        if getattr(c, f) is not None:
            getattr(d, f).copy_(getattr(c, f))
    return d


def _same(a, b, what):
    for f in FIELDS:
        x, y = getattr(a, f), getattr(b, f)
        if x is not None:
            assert torch.equal(x, y), f"{what}: {f} differs"


# (bits, aux, n_q, n_kv, batch, n_sink, context, paged, token dtype): the plans and kernels a
# step can take
CASES = [
    (2, 0, 32, 8, 96, 0, 6 * 128 + 124, False, "bf16"),     # 768 streams: 3 body splits + a residual split, one workgroup
    (2, 0, 32, 8, 64, 0, 50 * 128 + 124, False, "bf16"),    # 512 streams: 4 body splits sharing the chunks
    (2, 0, 32, 8, 3, 100, 20 * 128 + 224, False, "bf16"),   # 24 streams: many splits, residual splits, merge kernel
    (2, 0, 32, 8, 400, 0, 3 * 128 + 124, False, "bf16"),    # 3200 streams: one split each
    (2, 0, 40, 8, 48, 0, 6 * 128 + 124, False, "bf16"),     # group size 5 (the extra-head kernel)
    (2, 0, 64, 8, 64, 0, 12 * 128 + 124, False, "bf16"),    # group size 8 (two head groups)
    (2, 0, 128, 8, 48, 0, 12 * 128 + 124, False, "bf16"),   # group size 16 (two head chunks read the new row)
    (4, 1, 32, 8, 64, 0, 12 * 128 + 124, True, "bf16"),     # 4 bits, compact aux, paged body
    (2, 1, 32, 8, 32, 128, 126, False, "bf16"),             # sink tokens, then the first residual rows
    (2, 0, 32, 8, 96, 0, 6 * 128 + 124, False, "fp32"),     # fp32 tokens: the two kernels every step
]


@pytest.mark.parametrize("bits,aux,n_q,n_kv,batch,n_sink,context,paged,tok", CASES)
def test_append_decode_equals_two_calls(K, bits, aux, n_q, n_kv, batch, n_sink, context, paged, tok):
    from paper_2606_03458_amd import workloads
    print(f"[gpu case] step bits={bits} aux={aux} n_q={n_q} batch={batch} sink={n_sink} ctx={context} "
          f"paged={paged} tok={tok}", flush=True)
    built, _ = workloads.build("llama", bits=bits, aux=aux, n_q=n_q, n_kv=n_kv, batch=batch, n_sink=n_sink,
                               context=context)
    p = built.params
    a = _paged(K, p, built.cache, seed=bits + n_q) if paged else built.cache
    b = _clone(K, p, a)
    gen = torch.Generator(device="cuda").manual_seed(batch + n_q)
    dt = torch.bfloat16 if tok == "bf16" else torch.float32
    kvdt = K.KVARN_BF16 if tok == "bf16" else K.KVARN_F32
    L = built.length
    ws_bytes = max(K.kvarn_decode_workspace_bytes(p, a, n_q, L + s + 1) for s in range(6))
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    for s in range(6):
        length = L + s
        kt = (2 * torch.randn(batch, n_kv, 128, generator=gen, device="cuda")).to(dt)
        vt = torch.randn(batch, n_kv, 128, generator=gen, device="cuda").to(dt)
        q = workloads.decode_queries(built, seed=40, step=s)
        got = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
        ref = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
        K.kvarn_append_decode(p, a, kt, vt, kvdt, length, n_q, q, K.KVARN_BF16, got, K.KVARN_F32, SCALE, ws, ws_bytes)
        K.kvarn_append_token(p, b, kt, vt, kvdt, length)
        K.kvarn_decode_attention(p, b, n_q, q, K.KVARN_BF16, ref, K.KVARN_F32, SCALE, length + 1, ws, ws_bytes)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), f"step {s} (length {length}): outputs differ"
        _same(a, b, f"step {s}")
        assert int(a.seq_len.min()) == int(a.seq_len.max()) == length + 1
        assert int(a.err_word.item()) == 0


def test_append_decode_length_check(K):
    """A sequence whose stored length is not the host's (set so from the host) is left as it is
    and flagged with bit 2 of err_word; the other sequences step as usual."""
    from paper_2606_03458_amd import workloads
    built, _ = workloads.build("llama", n_q=32, n_kv=8, batch=96, context=6 * 128 + 100)
    p, a = built.params, built.cache
    b = _clone(K, p, a)
    L, bad = built.length, 5
    a.seq_len[bad] += 3
    before = {f: getattr(a, f)[bad].clone() for f in ("k_resid", "v_resid", "seq_len")}
    gen = torch.Generator(device="cuda").manual_seed(7)
    kt = torch.randn(96, 8, 128, generator=gen, device="cuda").to(torch.bfloat16)
    vt = torch.randn(96, 8, 128, generator=gen, device="cuda").to(torch.bfloat16)
    q = workloads.decode_queries(built, seed=41)
    ws_bytes = K.kvarn_decode_workspace_bytes(p, a, 32, L + 1)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    got = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    ref = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    K.kvarn_append_decode(p, a, kt, vt, K.KVARN_BF16, L, 32, q, K.KVARN_BF16, got, K.KVARN_F32, SCALE, ws, ws_bytes)
    K.kvarn_append_token(p, b, kt, vt, K.KVARN_BF16, L)
    K.kvarn_decode_attention(p, b, 32, q, K.KVARN_BF16, ref, K.KVARN_F32, SCALE, L + 1, ws, ws_bytes)
    torch.cuda.synchronize()
    assert int(a.err_word.item()) == 4
    for f, v in before.items():
        assert torch.equal(getattr(a, f)[bad], v), f
    keep = torch.arange(96, device="cuda") != bad
    assert torch.equal(got[keep], ref[keep])
    for f in ("k_resid", "v_resid", "seq_len"):
        assert torch.equal(getattr(a, f)[keep], getattr(b, f)[keep]), f
