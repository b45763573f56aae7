"""Build the synthetic workloads on the GPU through the library's own entry points.

A cache is filled the way a serving loop would fill it: the prefix that makes whole 128-token
groups is quantized with ``kvarn_quantize_block`` straight into the body (a prefill), and any
remaining tokens go through ``kvarn_append_token``.  Inputs come from ``datagen``.  Nothing
here computes any part of the quantizer or the attention.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import datagen
from . import kvarn as K


@dataclass
class Built:
    params: K.kvarn_params
    cache: K.Cache
    n_q: int
    length: int          # common length of every sequence
    dtype: torch.dtype   # K/V/q dtype
    spec: dict


def _dtype(spec) -> torch.dtype:
    return torch.float32 if spec["dtype"] == "fp32" else torch.bfloat16


def build(name: str, device="cuda", bits: int | None = None, n_sink: int = 0, context: int | None = None,
          layers: int | None = None, batch: int | None = None, extra_blocks: int = 0, seed: int | None = None,
          keep_inputs: bool = False, best_iter: bool = False, n_q: int | None = None, n_kv: int | None = None,
          aux: int = 0, rotate: int = 1, varn_iters: int | None = None):
    """Create and fill the cache of workload `name` (see datagen.WORKLOADS).

    Overrides (bits, context, layers, batch, n_sink, n_q, n_kv) make variants of the same shape;
    aux selects the tile's aux format (0 fp32, 1 compact); rotate = 0 and varn_iters select the
    ablation quantizers (no rotation, K = 0: KIVI-style RTN; no rotation, K > 0: VarN alone).
    Returns (Built, inputs) where inputs holds the K/V/best-iteration tensors if keep_inputs.
    """
    spec = dict(datagen.WORKLOADS[name])
    if bits is not None:
        spec["bits"] = bits
    if context is not None:
        spec["context"] = context
    if layers is not None:
        spec["layers"] = layers
    if batch is not None:
        spec["batch"] = batch
    if n_q is not None:
        spec["n_q"] = n_q
    if n_kv is not None:
        spec["n_kv"] = n_kv
    seed = datagen.SEEDS[name] if seed is None else seed
    dt = _dtype(spec)
    p = K.kvarn_params_init(spec["bits"])
    p.n_sink = n_sink
    p.aux_format = aux
    p.rotate = rotate
    if varn_iters is not None:
        p.varn_iters = varn_iters
    L, B, n_kv, T = spec["layers"], spec["batch"], spec["n_kv"], spec["context"]
    prefill = n_sink + ((T - n_sink) // 128) * 128 if T > n_sink else T
    tail = T - prefill
    body_blocks = max(prefill - n_sink, 0) // 128
    max_blocks = body_blocks + (tail + 127) // 128 + extra_blocks
    cache = K.Cache(p, L * B, n_kv, max(max_blocks, 1), device=device)
    inputs = {"K": [], "V": [], "best_k": [], "best_v": []}
    for layer in range(L):
        lseed = seed * 1000 + layer
        sig = datagen.channel_log_scales(lseed, n_kv, spec["dist"], device=device)
        Kx, Vx = datagen.kv_tokens(lseed, 0, B, n_kv, T, spec["dist"], dtype=dt, device=device, sigma_c=sig)
        rows = slice(layer * B, (layer + 1) * B)
        if n_sink and T > 0:
            ns = min(n_sink, T)
            cache.k_sink[rows, :, :ns] = Kx[:, :, :ns].to(torch.bfloat16)
            cache.v_sink[rows, :, :ns] = Vx[:, :, :ns].to(torch.bfloat16)
        if body_blocks:
            kb = Kx[:, :, n_sink:n_sink + body_blocks * 128].contiguous().view(B * n_kv, body_blocks * 128, 128)
            vb = Vx[:, :, n_sink:n_sink + body_blocks * 128].contiguous().view(B * n_kv, body_blocks * 128, 128)
            bik = torch.empty(B * n_kv * body_blocks, dtype=torch.int32, device=device) if best_iter else None
            biv = torch.empty(B * n_kv * body_blocks, dtype=torch.int32, device=device) if best_iter else None
            K.quantize_into_body(p, K.KVARN_KEYS, kb, cache.k_body[rows].view(B * n_kv, cache.max_blocks, -1),
                                 best_iter=bik)
            K.quantize_into_body(p, K.KVARN_VALUES, vb, cache.v_body[rows].view(B * n_kv, cache.max_blocks, -1),
                                 best_iter=biv)
            if best_iter:
                inputs["best_k"].append(bik)
                inputs["best_v"].append(biv)
        if keep_inputs:
            inputs["K"].append(Kx)
            inputs["V"].append(Vx)
        del Kx, Vx
    cache.seq_len.fill_(prefill if T > n_sink else T)
    if n_sink and T <= n_sink:
        cache.seq_len.fill_(T)
    built = Built(p, cache, spec["n_q"], T, dt, spec)
    # tail tokens through the append path (one call per token, all sequences in lock step)
    if tail:
        for t in range(prefill, T):
            kt, vt = _token(built, seed, t, inputs if keep_inputs else None)
            K.kvarn_append_token(p, cache, kt, vt, K.KVARN_BF16 if dt == torch.bfloat16 else K.KVARN_F32, t)
    built.length = T
    return built, inputs


def _token(built: Built, seed: int, t: int, inputs):
    """Token t of every (sequence, kv head), [L*B, n_kv, 128], from the kept inputs or redrawn."""
    spec = built.spec
    L, B, n_kv = spec["layers"], spec["batch"], spec["n_kv"]
    if inputs is not None and inputs["K"]:
        kt = torch.cat([k[:, :, t] for k in inputs["K"]]).contiguous()
        vt = torch.cat([v[:, :, t] for v in inputs["V"]]).contiguous()
        return kt, vt
    ks, vs = [], []
    for layer in range(L):
        lseed = seed * 1000 + layer
        sig = datagen.channel_log_scales(lseed, n_kv, spec["dist"], device=built.cache.k_body.device)
        kx, vx = datagen.kv_tokens(lseed, 1 + t, B, n_kv, 1, spec["dist"], dtype=built.dtype,
                                   device=built.cache.k_body.device, sigma_c=sig)
        ks.append(kx[:, :, 0])
        vs.append(vx[:, :, 0])
    return torch.cat(ks).contiguous(), torch.cat(vs).contiguous()


def step_tokens(built: Built, seed: int, step: int):
    """Fresh K/V tokens for decode step `step`: [L*B, n_kv, 128] each (independent draws)."""
    return _token(built, seed + 7777, 1_000_000 + step, None)


def decode_queries(built: Built, seed: int, step: int = 0) -> torch.Tensor:
    spec = built.spec
    return datagen.queries(seed, step, spec["layers"] * spec["batch"], spec["n_q"], dtype=built.dtype,
                           device=built.cache.k_body.device)
