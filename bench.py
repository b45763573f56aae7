#!/usr/bin/env python
"""KVarN decode-step benchmark on one MI355X.

Workload (N=1): 32 layers x batch 32 folded into 1024 sequences, 32 query / 8 kv heads,
head_dim 128, 32768-token context held as a 2-bit KVarN body plus a bf16 residual; bf16 q.
One step = the whole hot path for one new token of every sequence in every layer:
kvarn_append_token (copy into the residual, and the VarN quantization of full residuals into
the body when due) followed by kvarn_decode_attention over all 32 layers' heads.  The residual
is pre-filled so that one flush (16384 tiles quantized) falls inside the timed steps.

Prints one JSON line.  value = decode tokens/s = 32 sequences x steps / wall time.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn tokens/s + quantize GB/s over 2-bit KVarN cache; % of HBM roofline"
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="throughput")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target wall time of the oracle sample")
    ap.add_argument("--calib-copy-gib", type=float, default=0.0,
                    help="after the run, copy this many GiB device-to-device (a known-size reference for "
                         "hardware byte counters)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2606_03458_amd import datagen, workloads
    from paper_2606_03458_amd import kvarn as K

    torch.cuda.set_device(0)
    dev = "cuda:0"
    name = args.workload
    spec = datagen.WORKLOADS[name]
    seed = datagen.SEEDS[name]
    W, S = args.warmup, args.steps
    # residual fill so that one flush lands in the middle of the timed steps
    r0 = (128 - W - max(S // 2, 1)) % 128
    total_tokens = spec["context"] + r0 + W + S
    extra = (total_tokens - spec["context"] + 127) // 128 + 1
    print(f"[bench] building {name}: {spec}", file=sys.stderr, flush=True)
    t0 = time.time()
    built, _ = workloads.build(name, device=dev, extra_blocks=extra)
    p, cache = built.params, built.cache
    n_seq = cache.batch
    B_logical = spec["batch"]
    length = built.length
    for t in range(r0):  # pre-fill the residual through the append path
        kt, vt = workloads.step_tokens(built, seed, -1 - t)
        K.kvarn_append_token(p, cache, kt, vt, K.KVARN_BF16, length)
        length += 1
    torch.cuda.synchronize()
    print(f"[bench] built in {time.time() - t0:.1f}s; length {length}, max_blocks {cache.max_blocks}",
          file=sys.stderr, flush=True)

    # inputs of every step drawn before timing
    toks = [workloads.step_tokens(built, seed, s) for s in range(W + S)]
    qs = [workloads.decode_queries(built, seed, s) for s in range(W + S)]
    scale = 1.0 / np.sqrt(128.0)
    max_len = total_tokens + 1
    ws_bytes = K.kvarn_decode_workspace_bytes(p, cache, built.n_q, max_len)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty_like(qs[0])
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(S)]
    tb = K.kvarn_tile_bytes(p.bits)

    def decode_bytes(L):
        nb = L // 128
        nr = L % 128
        per_stream = nb * 2 * tb + nr * 2 * 128 * 2
        return n_seq * spec["n_kv"] * per_stream + 2 * n_seq * built.n_q * 128 * 2

    alg_bytes = []
    for s in range(W + S):
        kt, vt = toks[s]
        K.kvarn_append_token(p, cache, kt, vt, K.KVARN_BF16, length)
        length += 1
        if s == W:
            torch.cuda.synchronize()
            t_start = time.perf_counter()
        if s >= W:
            ev[s - W][0].record(stream)
        K.kvarn_decode_attention(p, cache, built.n_q, qs[s], K.KVARN_BF16, out, K.KVARN_BF16, scale, max_len, ws,
                                 ws_bytes)
        if s >= W:
            ev[s - W][1].record(stream)
            alg_bytes.append(decode_bytes(length))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    if not bool(torch.isfinite(out).all()):
        raise RuntimeError("decode output has non-finite values")
    dec_ms = [a.elapsed_time(b) for a, b in ev]
    dec_avg_s = sum(dec_ms) / len(dec_ms) / 1e3
    bytes_avg = sum(alg_bytes) / len(alg_bytes)
    achieved = bytes_avg / dec_avg_s / 1e9
    tokens_per_s = B_logical * S / elapsed
    print(f"[bench] {S} steps in {elapsed * 1e3:.2f} ms; decode avg {dec_avg_s * 1e3:.3f} ms, "
          f"{achieved:.0f} GB/s", file=sys.stderr, flush=True)

    # ---- quantize throughput: one layer's keys (8 kv heads x 32 sequences x 256 tiles) --------
    q_res = None
    try:
        sig = datagen.channel_log_scales(seed * 1000, spec["n_kv"], spec["dist"], device=dev)
        Kx, _ = datagen.kv_tokens(seed * 1000 + 999, 0, spec["batch"], spec["n_kv"], spec["context"], spec["dist"],
                                  dtype=torch.bfloat16, device=dev, sigma_c=sig)
        x = Kx.view(-1, spec["context"], 128)
        n_tiles = x.shape[0] * (spec["context"] // 128)
        body = torch.empty((x.shape[0], spec["context"] // 128, tb), dtype=torch.uint8, device=dev)
        K.quantize_into_body(p, K.KVARN_KEYS, x, body)  # warm-up
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 3
        e0.record(stream)
        for _ in range(reps):
            K.quantize_into_body(p, K.KVARN_KEYS, x, body)
        e1.record(stream)
        torch.cuda.synchronize()
        qt = e0.elapsed_time(e1) / reps / 1e3
        qbytes = n_tiles * (128 * 128 * 2 + tb)
        q_res = {"value": round(qbytes / qt / 1e9, 2), "unit": "GB/s", "tiles_per_s": round(n_tiles / qt),
                 "tiles": n_tiles, "bytes_per_tile": 128 * 128 * 2 + tb, "frac_hbm": round(qbytes / qt / 1e9 /
                                                                                            HBM_PEAK_GBS, 4)}
        del Kx, x, body
    except Exception as e:  # report, do not hide
        q_res = {"error": repr(e)}

    # ---- CPU baseline: the oracle on a sample of the same streams ------------------------
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(built, qs[-1], length, scale, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": round(tokens_per_s, 2), "unit": "tokens/s", "n_gpus": 1, "steps": S,
        "warmup": W, "ms_per_step": round(elapsed / S * 1e3, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp32", "data": "synthetic",
        "config": {"workload": f"{name}: {spec['layers']} layers x batch {spec['batch']} = {n_seq} sequences, "
                               f"{spec['n_q']} q / {spec['n_kv']} kv heads, head_dim 128, "
                               f"{spec['context']}-token context, {p.bits}-bit KVarN body + bf16 residual, "
                               f"append + decode per step",
                   "layers": spec["layers"], "batch": spec["batch"], "context": spec["context"], "bits": p.bits},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(name),
                     "kernel": "kvarn_decode_attention", "alg_bytes_per_launch": int(bytes_avg),
                     "avg_launch_ms": round(dec_avg_s * 1e3, 4)},
        "cpu_baseline": cpu,
        "quantize": q_res,
    }
    print(json.dumps(line), flush=True)

    if args.calib_copy_gib > 0:
        nbytes = int(args.calib_copy_gib * (1 << 30))
        src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy: {nbytes} bytes read + {nbytes} bytes written", file=sys.stderr, flush=True)


COUNTER_SUMMARY = os.path.join(ROOT, "profiles", "k_decode4_throughput_hbm_counters.md")
DECODE_SOURCES = [os.path.join(ROOT, "paper_2606_03458_amd", "csrc", f) for f in ("decode.hip", "common.hpp")]


def decode_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per decode launch (FETCH_SIZE + WRITE_SIZE, calibrated) from the committed
    rocprofv3 counter summary; None unless it covers this workload and was taken on the
    current decode sources."""
    try:
        with open(COUNTER_SUMMARY) as fh:
            text = fh.read()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        line = line.strip().strip("`")
        if ":" in line and line.split(":", 1)[0] in ("workload", "source_sha256", "hbm_bytes_per_launch"):
            k, v = line.split(":", 1)
            fields[k] = v.strip()
    if fields.get("workload") != workload or fields.get("source_sha256") != decode_source_hash():
        return None
    try:
        return int(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(built, q, length, scale, target_s):
    """Time the oracle's decode on a sample of (sequence, kv head) streams of the same cache,
    scaled to the metric's unit (tokens/s of the whole 1024-sequence step)."""
    import numpy as np

    import oracle

    cache = built.cache
    n_kv = cache.n_kv
    g = built.n_q // n_kv
    total_streams = cache.batch * n_kv
    rng = np.random.default_rng(0)

    def sample(n):
        idx = rng.choice(total_streams, size=n, replace=False)
        hc = oracle.HostCache(n, 1, cache.max_blocks, bits=cache.bits)
        qh = np.zeros((n, g, 128), dtype=np.uint16)
        for i, s in enumerate(idx):
            b, kh = divmod(int(s), n_kv)
            hc.k_body[i, 0] = cache.k_body[b, kh].cpu().numpy()
            hc.v_body[i, 0] = cache.v_body[b, kh].cpu().numpy()
            hc.k_resid[i, 0] = cache.k_resid[b, kh].view(torch_int16()).cpu().numpy().view(np.uint16)
            hc.v_resid[i, 0] = cache.v_resid[b, kh].view(torch_int16()).cpu().numpy().view(np.uint16)
            hc.seq_len[i] = int(cache.seq_len[b])
            qh[i] = q[b, kh * g:(kh + 1) * g].view(torch_int16()).cpu().numpy().view(np.uint16)
        return hc, qh

    hc, qh = sample(1)
    t0 = time.perf_counter()
    oracle.decode(hc, qh, scale)
    one = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    n = int(max(1, min(total_streams, target_s / one * threads)))
    n = max(threads, (n // threads) * threads) if n >= threads else n
    hc, qh = sample(n)
    t0 = time.perf_counter()
    oracle.decode(hc, qh, scale)
    t = time.perf_counter() - t0
    step_s = t * total_streams / n
    return {"value": round(built.spec["batch"] / step_s, 4), "unit": "tokens/s", "cores": min(threads, n),
            "kind": "oracle",
            "sample": f"{n} of {total_streams} (sequence, kv head) streams at length {int(hc.seq_len[0])}, "
                      f"decode only, {t:.1f} s wall, scaled linearly to the full step"}


def torch_int16():
    import torch
    return torch.int16


if __name__ == "__main__":
    main()
