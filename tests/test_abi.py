"""Host-only tests of the C ABI: the library loads, exports every entry point its header
declares, and rejects bad arguments with status codes before touching the GPU."""
import ctypes
import os
import re

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def K():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    return kvarn


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "kvarn.h")).read()
    return re.findall(r"KVARN_API\s+[\w\s\*]+?\b(kvarn_\w+)\s*\(", text)


def test_exports_every_declared_symbol(K):
    names = declared_symbols()
    assert set(names) == set(K.EXPORTS)
    L = ctypes.CDLL(K.library_path())
    for n in names:
        assert hasattr(L, n), n
    text = open(os.path.join(ROOT, "include", "kvarn.h")).read()
    m = re.search(r"#define KVARN_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == K.NOALLOC_SCRATCH_BYTES


def test_params_and_sizes(K):
    p = K.kvarn_params_init(2)
    assert (p.bits, p.varn_iters, p.n_sink) == (2, 8, 0)
    assert p.log_lo == pytest.approx(-0.3) and p.log_hi == 10.0
    p2, p4 = K.kvarn_params_init(2), K.kvarn_params_init(4)
    assert K.kvarn_tile_bytes(p2) == 5632 and K.kvarn_tile_bytes(p4) == 9728
    p2.aux_format = p4.aux_format = K.KVARN_AUX_COMPACT
    assert K.kvarn_tile_bytes(p2) == 4608 and K.kvarn_tile_bytes(p4) == 8704
    p2.bits = 3
    assert K.kvarn_tile_bytes(p2) == 0
    p4.aux_format = 2
    assert K.kvarn_tile_bytes(p4) == 0
    with pytest.raises(K.KVarNError) as e:
        K.kvarn_params_init(3)
    assert e.value.status == -2
    p.n_sink = 128
    s = K.kvarn_cache_sizes(p, 3, 8, 10)
    assert s == [3 * 8 * 10 * 5632] * 2 + [3 * 8 * 128 * 128 * 2] * 2 + [3 * 8 * 128 * 128 * 2] * 2 + [12]
    with pytest.raises(K.KVarNError):
        K.kvarn_cache_sizes(p, 0, 8, 10)
    # at most 2^26 (sequence, kv head) pairs: the kernels index them in 32 bits
    assert K.kvarn_cache_sizes(p, 1 << 13, 1 << 13, 0)[6] == 4 << 13
    with pytest.raises(K.KVarNError) as e:
        K.kvarn_cache_sizes(p, (1 << 13) + 1, 1 << 13, 0)
    assert e.value.status == -1


def _fake(n, align=256):
    """A host buffer standing in for device memory: only its address is validated."""
    buf = (ctypes.c_uint8 * (n + align))()
    addr = ctypes.addressof(buf)
    return buf, addr + (-addr) % align


def test_quantize_validation(K):
    p = K.kvarn_params_init(2)
    keep, x = _fake(1 << 16)
    keep2, out = _fake(1 << 16)
    ok = dict(p=p, kind=0, x=x, x_dtype=1, n_outer=1, n_inner=1, x_outer_stride=0, x_inner_stride=0,
              x_token_stride=128, out=out, out_outer_stride=0, out_inner_stride=0)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        K.kvarn_quantize_block(**a, stream=0)

    bad = [dict(kind=2), dict(x_dtype=5), dict(x=None), dict(out=None), dict(x=x + 2), dict(out=out + 4),
           dict(x_token_stride=100), dict(x_token_stride=-128), dict(n_outer=-1), dict(x_outer_stride=3),
           dict(x_inner_stride=-8)]
    for kw in bad:
        with pytest.raises(K.KVarNError) as e:
            call(**kw)
        assert e.value.status == -1, kw
    # zero tiles: nothing to do, even with null pointers
    call(n_outer=0, x=None, out=None)
    call(n_inner=0)
    for field, val, code in [("bits", 3, -2), ("varn_iters", -1, -1), ("varn_iters", 65, -1), ("var_min", 0.0, -1),
                             ("var_min", float("nan"), -1), ("var_min", 1e-31, -1), ("var_max", 1e31, -1),
                             ("var_max", float("inf"), -1), ("log_lo", 11.0, -1), ("log_lo", -41.0, -1),
                             ("log_hi", 41.0, -1), ("log_hi", float("nan"), -1), ("n_sink", -5, -1),
                             ("aux_format", 2, -2), ("aux_format", -1, -2), ("rotate", 2, -1), ("rotate", -1, -1)]:
        q = K.kvarn_params_init(2)
        setattr(q, field, val)
        with pytest.raises(K.KVarNError) as e:
            call(p=q)
        assert e.value.status == code, field


class _HostCache:
    """kvarn_cache descriptor over host addresses (validation only)."""

    def __init__(self, K, batch=2, n_kv=2, max_blocks=1, sink=False, table=None, n_phys=0):
        self.keep = []
        self.batch, self.n_kv, self.max_blocks = batch, n_kv, max_blocks
        self.table, self.n_phys = table, n_phys
        ptrs = []
        for _ in range(7):
            b, a = _fake(1024)
            self.keep.append(b)
            ptrs.append(a)
        self.ptrs = ptrs
        self.sink = sink

    def desc(self):
        from paper_2606_03458_amd.kvarn import kvarn_cache
        p = self.ptrs
        return kvarn_cache(self.batch, self.n_kv, self.max_blocks, p[0], p[1], p[2], p[3],
                           p[4] if self.sink else None, p[5] if self.sink else None, p[6], None, self.table,
                           self.n_phys)


def test_append_validation(K):
    p = K.kvarn_params_init(2)
    c = _HostCache(K, max_blocks=1)
    keep, tok = _fake(4096)
    # capacity from the lock-step hint: length 255 means the next token fills the residual of a
    # cache whose only body tile is already used
    with pytest.raises(K.KVarNError) as e:
        K.kvarn_append_token(p, c, tok, tok, 1, 128 + 127, stream=0)
    assert e.value.status == -3
    for args, code in [((None, tok, 1, 0), -1), ((tok, tok, 7, 0), -1), ((tok + 2, tok, 1, 0), -1),
                       ((tok, tok + 8, 0, 0), -1), ((tok, tok, 1, -2), -1)]:
        with pytest.raises(K.KVarNError) as e:
            K.kvarn_append_token(p, c, *args, stream=0)
        assert e.value.status == code, args
    p.n_sink = 128
    with pytest.raises(K.KVarNError) as e:  # sink buffers required when n_sink > 0
        K.kvarn_append_token(p, c, tok, tok, 1, 0, stream=0)
    assert e.value.status == -1
    big = _HostCache(K, batch=(1 << 13) + 1, n_kv=1 << 13)
    with pytest.raises(K.KVarNError) as e:  # more (sequence, kv head) pairs than the kernels index
        K.kvarn_append_token(K.kvarn_params_init(2), big, tok, tok, 1, 0, stream=0)
    assert e.value.status == -1


def test_decode_validation(K):
    p = K.kvarn_params_init(2)
    c = _HostCache(K, batch=2, n_kv=2, max_blocks=32)
    keep, buf = _fake(1 << 20)
    need = K.kvarn_decode_workspace_bytes(p, c, 8, 4096)  # 4 streams x 32 tiles: split
    assert need > 0
    assert K.kvarn_decode_workspace_bytes(p, c, 8, 384) == 0  # 3 tiles: one split, no partials
    good = dict(n_q=8, q=buf, q_dtype=1, out=buf, out_dtype=1, sm_scale=0.088, max_len_hint=4096, workspace=buf,
                workspace_bytes=need)

    def call(**kw):
        a = dict(good)
        a.update(kw)
        K.kvarn_decode_attention(p, c, **a, stream=0)

    for kw, code in [(dict(n_q=7), -1), (dict(n_q=0), -1), (dict(n_q=2 * 17), -1), (dict(q=None), -1),
                     (dict(out_dtype=4), -1), (dict(sm_scale=float("inf")), -1), (dict(max_len_hint=-1), -1),
                     (dict(workspace_bytes=need - 1), -5), (dict(workspace=None), -5)]:
        with pytest.raises(K.KVarNError) as e:
            call(**kw)
        assert e.value.status == code, kw
    # the workspace grows with the split plan and the number of query heads
    assert K.kvarn_decode_workspace_bytes(p, c, 16, 4096) == 2 * need
    assert K.kvarn_decode_workspace_bytes(p, c, 8, -1) == 0


def test_append_decode_validation(K):
    """The fused step validates the arguments of both halves before enqueuing anything: an error in
    the decode's arguments enqueues no append either."""
    p = K.kvarn_params_init(2)
    c = _HostCache(K, batch=2, n_kv=2, max_blocks=32)
    keep, buf = _fake(1 << 20)
    need = K.kvarn_decode_workspace_bytes(p, c, 8, 4096 + 1)
    assert need > 0
    good = dict(k_new=buf, v_new=buf, kv_dtype=1, host_len_before=4096, n_q=8, q=buf, q_dtype=1, out=buf,
                out_dtype=1, sm_scale=0.088, workspace=buf, workspace_bytes=need)
    for kw, code in [(dict(host_len_before=-1), -1), (dict(host_len_before=2 ** 31 - 1), -1), (dict(k_new=None), -1),
                     (dict(v_new=buf + 2), -1), (dict(kv_dtype=5), -1), (dict(n_q=7), -1), (dict(q=None), -1),
                     (dict(out=buf + 4), -1), (dict(sm_scale=float("inf")), -1),
                     (dict(workspace_bytes=need - 1), -5), (dict(workspace=None), -5),
                     # a flush that would need body tile max_blocks
                     (dict(host_len_before=32 * 128 + 127), -3)]:
        with pytest.raises(K.KVarNError) as e:
            K.kvarn_append_decode(K.kvarn_params_init(2), c, **{**good, **kw}, stream=0)
        assert e.value.status == code, kw


def test_decode_noalloc_validation(K):
    """The allocation-free decode validates like kvarn_decode_attention, before any HIP call, and
    every split plan's partials fit its scratch array."""
    p = K.kvarn_params_init(2)
    c = _HostCache(K, batch=2, n_kv=2, max_blocks=32)
    keep, buf = _fake(1 << 20)
    good = dict(n_q=8, q=buf, q_dtype=1, out=buf, out_dtype=1, sm_scale=0.088, max_len_hint=4096)
    for kw, code in [(dict(n_q=7), -1), (dict(q=None), -1), (dict(out=buf + 2), -1), (dict(q_dtype=9), -1),
                     (dict(sm_scale=float("nan")), -1), (dict(max_len_hint=-1), -1)]:
        with pytest.raises(K.KVarNError) as e:
            K.kvarn_decode_attention_noalloc(p, c, **{**good, **kw}, stream=0)
        assert e.value.status == code, kw
    # The largest plan with partials in memory: 255 streams of 8 query heads in 9 splits, 18.2 MiB
    # (from 256 streams on, 4 splits per stream give every SIMD a wave and the plan stops there).
    # Plans of up to 4 splits whose LDS blocks fit merge inside the workgroup and need none (511
    # streams of 8 heads in 4 splits, 1023 in 3, 1023 streams of 16 heads in 2).
    mid = _HostCache(K, batch=255, n_kv=1, max_blocks=2049)
    need = K.kvarn_decode_workspace_bytes(p, mid, 8, 2048 * 128)
    assert need == 255 * 8 * 9 * 1040 <= K.NOALLOC_SCRATCH_BYTES
    assert K.kvarn_decode_workspace_bytes(p, _HostCache(K, batch=511, n_kv=1, max_blocks=2049), 8, 2048 * 128) == 0
    big = _HostCache(K, batch=1023, n_kv=1, max_blocks=2049)
    assert K.kvarn_decode_workspace_bytes(p, big, 8, 2048 * 128) == 0
    assert K.kvarn_decode_workspace_bytes(p, big, 16, 2048 * 128) == 0


def test_no_cpu_fallback(K, monkeypatch, tmp_path):
    """The binding refuses to run without the built library."""
    import importlib
    mod = importlib.import_module("paper_2606_03458_amd.kvarn")
    monkeypatch.setattr(mod, "_LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(mod, "_lib", None)
    with pytest.raises(ImportError):
        mod.lib()


def test_prefill_validation(K):
    p = K.kvarn_params_init(2)
    c = _HostCache(K)
    keep, buf = _fake(4096)
    for args, code in [((None, buf, 1, buf, 10), -1), ((buf, None, 1, buf, 10), -1), ((buf, buf, 3, buf, 10), -1),
                       ((buf, buf, 1, None, 10), -1), ((buf, buf, 1, buf, -1), -1), ((buf + 8, buf, 1, buf, 10), -1),
                       ((buf, buf, 1, buf + 2, 10), -1)]:
        with pytest.raises(K.KVarNError) as e:
            K.kvarn_prefill(p, c, *args, stream=0)
        assert e.value.status == code, args


def test_paged_cache_validation(K):
    """A block table needs a positive pool size and 4-byte alignment (checked before launch)."""
    p = K.kvarn_params_init(2)
    keep, tok = _fake(4096)
    for table, n_phys in [(tok, 0), (tok + 2, 4)]:
        c = _HostCache(K, table=table, n_phys=n_phys)
        with pytest.raises(K.KVarNError) as e:
            K.kvarn_append_token(p, c, tok, tok, 1, 0, stream=0)
        assert e.value.status == -1, (table, n_phys)
