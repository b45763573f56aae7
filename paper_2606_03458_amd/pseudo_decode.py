"""Error accumulation of a quantized KV cache through depth and time (Sec. 3.2, Fig. 5, and
the attention-output proxy of Sec. 3.4, Fig. 6), on a random residual attention stack.

No model weights are involved.  Layer l is a pre-norm attention block with random Gaussian
projections (n_q query / n_kv key-value heads of 128):
    h = x_l / rms(x_l),  q = h W_Q,  k = (h W_K) g_t,  v = (h W_V) g_t
    x_{l+1} = x_l + attn(q, K_cache, V_cache) W_O
The columns of W_K carry log-normal scales (keys with outlier channels) and g_t is a
log-normal gain of token t (outlier tokens): the two structures Sec. 3.1 attributes the large
errors to.  The inputs x_0 share a mean vector (a common direction of the residual stream),
which gives keys per-channel offsets and the attention outputs a component that does not
average away.  The norm keeps the stack from amplifying perturbations by itself.

Tokens are processed one at a time through the library: each layer appends the token's
K/V with ``kvarn_append_token`` (a 128-token block is quantized as soon as it is complete:
the paper's block size b is the tile height) and decodes it with ``kvarn_decode_attention``.
Two settings run side by side with separate caches:
  static   every layer's K, V and q come from the full-precision activations (the
           prefill-like case of prior work: errors do not propagate);
  dynamic  each layer's quantized attention output feeds the next layer and, through the
           cache, every later token (the pseudo-decode case: errors accumulate).
The reference is exact causal attention in fp32 on K, V rounded to bf16 (the precision the
residual stores), so the error measured is that of quantization alone.  Everything here is
argument marshalling plus plain torch projections; all quantization and attention runs in
the library's kernels.
"""
from __future__ import annotations

import math

import torch

from . import kvarn as K

QUANTIZERS = {"KIVI": dict(rotate=0, varn_iters=0), "KVarN": dict(rotate=1, varn_iters=8)}


def make_stack(layers: int, batch: int, T: int, d_model: int = 1024, n_q: int = 32, n_kv: int = 8,
               seed: int = 5, device="cuda") -> dict:
    """Random projections, token gains and inputs of the stack (seeded, on `device`)."""
    D = 128
    g = torch.Generator(device=device).manual_seed(seed)
    r = lambda *s: torch.randn(s, generator=g, device=device)
    WK = r(layers, d_model, n_kv * D) / math.sqrt(d_model) * torch.exp(r(layers, 1, n_kv * D))
    return dict(WQ=r(layers, d_model, n_q * D) / math.sqrt(d_model), WK=WK,
                WV=r(layers, d_model, n_kv * D) / math.sqrt(d_model),
                WO=r(layers, n_q * D, d_model) / math.sqrt(n_q * D),
                x0=r(1, 1, d_model) + r(batch, T, d_model), gain=torch.exp(0.5 * r(batch, T, 1)),
                n_q=n_q, n_kv=n_kv, layers=layers)


def _bf(t):
    return t.to(torch.bfloat16).float()


def _qkv(st: dict, l: int, x, gain):
    """Projections of layer l for inputs x [..., d_model] with token gains [..., 1]."""
    h = x * torch.rsqrt((x * x).mean(dim=-1, keepdim=True))
    return h @ st["WQ"][l], (h @ st["WK"][l]) * gain, (h @ st["WV"][l]) * gain


def reference(st: dict):
    """Full-precision forward of the stack: per-layer inputs x_l [B, T, d] and causal attention
    outputs o_l [B, T, n_q, 128] (fp32 math, K/V rounded to bf16)."""
    x0, nq, nkv, D = st["x0"], st["n_q"], st["n_kv"], 128
    B, T, _ = x0.shape
    mask = torch.triu(torch.full((T, T), float("-inf"), device=x0.device), 1)
    xs, outs = [x0], []
    for l in range(st["layers"]):
        x = xs[-1]
        q, k, v = _qkv(st, l, x, st["gain"])
        q = q.view(B, T, nq, D).permute(0, 2, 1, 3)
        k = _bf(k).view(B, T, nkv, D).permute(0, 2, 1, 3).repeat_interleave(nq // nkv, dim=1)
        v = _bf(v).view(B, T, nkv, D).permute(0, 2, 1, 3).repeat_interleave(nq // nkv, dim=1)
        s = torch.matmul(q.contiguous(), k.transpose(-1, -2).contiguous()) / math.sqrt(D) + mask
        o = torch.matmul(torch.softmax(s, dim=-1), v.contiguous()).permute(0, 2, 1, 3)
        outs.append(o)
        xs.append(x + o.reshape(B, T, nq * D) @ st["WO"][l])
    return xs, outs


def run(st: dict, ref, quantizer: str, bits: int = 2, keep_outputs: bool = False):
    """Relative error ||o - o_ref|| / ||o_ref|| of every layer's attention output, per token,
    averaged over the batch: {"static": [layers, T], "dynamic": [layers, T]} (fp32, device).
    With keep_outputs, also returns the attention outputs themselves,
    {"static" | "dynamic": [layers, T, B, n_q, 128]} (fp32, host), and the caches
    {"static" | "dynamic": [one kvarn.Cache per layer]}."""
    xs, o_ref = ref
    x0, nq, nkv, D, layers = st["x0"], st["n_q"], st["n_kv"], 128, st["layers"]
    B, T, _ = x0.shape
    dev = x0.device
    p = K.kvarn_params_init(bits, **QUANTIZERS[quantizer])
    caches = {m: [K.Cache(p, B, nkv, T // 128 + 1, device=dev) for _ in range(layers)] for m in ("static", "dynamic")}
    err = {m: torch.zeros((layers, T), device=dev) for m in caches}
    outs = {m: torch.zeros((layers, T, B, nq, D)) for m in caches} if keep_outputs else None
    ws_bytes = K.kvarn_decode_workspace_bytes(p, caches["static"][0], nq, T)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
    out = torch.empty((B, nq, D), dtype=torch.float32, device=dev)
    scale = 1.0 / math.sqrt(D)
    for t in range(T):
        xd = x0[:, t]
        for l in range(layers):
            for m in ("static", "dynamic"):
                xin = xs[l][:, t] if m == "static" else xd
                qt, kt, vt = _qkv(st, l, xin, st["gain"][:, t])
                qt = qt.view(B, nq, D).contiguous()
                kt = kt.view(B, nkv, D).to(torch.bfloat16).contiguous()
                vt = vt.view(B, nkv, D).to(torch.bfloat16).contiguous()
                c = caches[m][l]
                K.kvarn_append_token(p, c, kt, vt, K.KVARN_BF16, t)
                K.kvarn_decode_attention(p, c, nq, qt, K.KVARN_F32, out, K.KVARN_F32, scale, T, ws, ws_bytes)
                r = o_ref[l][:, t]
                err[m][l, t] = ((out - r).norm(dim=(1, 2)) / r.norm(dim=(1, 2))).mean()
                if keep_outputs:
                    outs[m][l, t] = out.cpu()
                if m == "dynamic":
                    xd = xd + out.reshape(B, nq * D) @ st["WO"][l]
    for m in caches:
        for c in caches[m]:
            if int(c.err_word.item()) != 0:
                raise RuntimeError(f"cache error word {int(c.err_word.item())}")
    return (err, outs, caches) if keep_outputs else err
