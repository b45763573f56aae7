"""Seeded synthetic K/V/q generators for the KVarN workloads.

This module only draws random tensors; it holds none of the quantizer's or the attention's
arithmetic.  The same generators feed the GPU path and, after a copy of the exact bytes to
the host, the CPU oracle, so parity never depends on random-number portability.

Distributions (Llama-3-8B-shaped synthetic KV; no model weights or datasets are used):
  "llama":  K[t, c] = z * exp(sigma_c) * exp(tau_t),  V[t, c] = z' * exp(tau_t)
            z, z' ~ N(0, 1); sigma_c ~ N(0, 1) per (layer, kv head, channel), shared by every
            sequence and token of that layer; tau_t ~ N(0, 0.5^2) per (sequence, kv head,
            token), applied to both K and V of that token.
  "stress": K[t, c] = t3 * exp(sigma_c) with t3 ~ Student-t(3) and sigma_c ~ N(0, 1.5^2) per
            (layer, kv head, channel); V ~ N(0, 1).
  q ~ N(0, 1).
Student-t(3) is drawn exactly as z / sqrt(chi2_3 / 3) with chi2_3 a sum of three squared
standard normals.
"""
from __future__ import annotations

import torch

D = 128

# Seeds of the five workloads (the tiny case's seed is 0).
SEEDS = {"tiny": 0, "llama": 1, "throughput": 2, "streaming": 3, "stress": 4, "gqa8": 5}


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFF_FFFF_FFFF_FFFF)
    return g


def channel_log_scales(seed: int, n_kv: int, dist: str, device="cpu") -> torch.Tensor:
    """Per-(kv head, channel) log-scale sigma_c of one layer: [n_kv, 128] fp32."""
    g = _gen(seed * 7919 + 17, device)
    std = 1.5 if dist == "stress" else 1.0
    return torch.randn(n_kv, D, generator=g, device=device, dtype=torch.float32) * std


def kv_tokens(seed: int, chunk: int, batch: int, n_kv: int, n_tok: int, dist: str, dtype=torch.bfloat16,
              device="cpu", sigma_c: torch.Tensor | None = None):
    """Draw K, V for `n_tok` tokens of every (sequence, kv head): each [batch, n_kv, n_tok, 128].

    `chunk` selects an independent stream of draws (e.g. a block index or a decode step), so
    a long context can be produced piece by piece.  `sigma_c` ([n_kv, 128]) is the layer's
    channel log-scale from `channel_log_scales`.
    """
    if sigma_c is None:
        sigma_c = channel_log_scales(seed, n_kv, dist, device)
    g = _gen(seed * 1_000_003 + chunk * 7 + 1, device)
    shape = (batch, n_kv, n_tok, D)
    z = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if dist == "stress":
        chi2 = torch.zeros(shape, device=device, dtype=torch.float32)
        for _ in range(3):
            chi2 += torch.randn(shape, generator=g, device=device, dtype=torch.float32) ** 2
        K = z / torch.sqrt(chi2 / 3.0) * torch.exp(sigma_c)[None, :, None, :]
        V = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    else:
        tau = torch.randn((batch, n_kv, n_tok, 1), generator=g, device=device, dtype=torch.float32) * 0.5
        z2 = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        K = z * torch.exp(sigma_c)[None, :, None, :] * torch.exp(tau)
        V = z2 * torch.exp(tau)
    return K.to(dtype), V.to(dtype)


def queries(seed: int, step: int, batch: int, n_q: int, dtype=torch.bfloat16, device="cpu") -> torch.Tensor:
    """q ~ N(0, 1): [batch, n_q, 128]."""
    g = _gen(seed * 1_000_033 + step * 13 + 5, device)
    return torch.randn((batch, n_q, D), generator=g, device=device, dtype=torch.float32).to(dtype)


# Workload shapes (name -> dict).  `layers` independent layers are flattened into the batch
# (sequence index = layer * batch + b).
WORKLOADS = {
    "tiny": dict(layers=1, batch=1, n_q=1, n_kv=1, context=256, dtype="fp32", dist="llama", bits=2),
    "llama": dict(layers=1, batch=1, n_q=32, n_kv=8, context=8192, dtype="bf16", dist="llama", bits=2,
                  append=1),
    "throughput": dict(layers=32, batch=32, n_q=32, n_kv=8, context=32768, dtype="bf16", dist="llama", bits=2),
    "streaming": dict(layers=1, batch=64, n_q=32, n_kv=8, context=32768, dtype="bf16", dist="llama", bits=2),
    "stress": dict(layers=1, batch=128, n_q=40, n_kv=8, context=16384, dtype="bf16", dist="stress", bits=2),
    # query groups of 8 (64 q / 8 kv heads, the layout of 70B-class models), batch 128, 16k
    "gqa8": dict(layers=1, batch=128, n_q=64, n_kv=8, context=16384, dtype="bf16", dist="llama", bits=2),
}
