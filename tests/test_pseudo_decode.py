"""The pseudo-decode error-accumulation harness (Sec. 3.2, Fig. 5; the proxy of Sec. 3.4, Fig. 6).

CPU: the harness's full-precision reference is pre-norm causal attention, checked against a
per-token loop on a tiny stack.  GPU: the static and dynamic settings through the library, with the
properties the construction fixes: layer 0 sees identical inputs in both settings, nothing is
quantized before the first 128-token block completes, and past layer 0 the dynamic setting's
error exceeds the static one (errors accumulate through depth)."""
import math

import pytest
import torch

from paper_2606_03458_amd import pseudo_decode as PD


def test_reference_is_causal_attention():
    st = PD.make_stack(layers=2, batch=2, T=9, d_model=64, n_q=4, n_kv=2, seed=1, device="cpu")
    xs, outs = PD.reference(st)
    bf = lambda t: t.to(torch.bfloat16).double()
    for l in range(2):
        x = xs[l].double()
        for b in range(2):
            for t in range(9):
                for h in range(4):
                    hk = h // 2
                    hx = x[b, :t + 1] / x[b, :t + 1].pow(2).mean(dim=1, keepdim=True).sqrt()
                    gn = st["gain"][b, :t + 1].double()
                    q = (hx[t] @ st["WQ"][l].double())[h * 128:(h + 1) * 128]
                    ks = bf((hx @ st["WK"][l].double()) * gn)[:, hk * 128:(hk + 1) * 128]
                    vs = bf((hx @ st["WV"][l].double()) * gn)[:, hk * 128:(hk + 1) * 128]
                    w = torch.softmax(ks @ q / math.sqrt(128), dim=0)
                    want = w @ vs
                    # bf16 rounding of K/V products computed in another order may flip a last bit
                    assert float((outs[l][b, t, h].double() - want).norm() / want.norm()) < 1e-2
        # the residual update
        o = outs[l].reshape(2, 9, -1).double()
        assert torch.allclose(xs[l + 1].double(), x + o @ st["WO"][l].double(), rtol=1e-4, atol=1e-4)


@pytest.fixture(scope="module")
def gpu_errors():
    from paper_2606_03458_amd import kvarn
    kvarn.lib()
    st = PD.make_stack(layers=3, batch=2, T=512, d_model=512, seed=3, device="cuda:0")
    ref = PD.reference(st)
    return {q: {m: e.cpu() for m, e in PD.run(st, ref, q, bits=4).items()} for q in PD.QUANTIZERS}


@pytest.mark.gpu
def test_layer0_identical_and_exact_before_first_block(gpu_errors):
    for q, e in gpu_errors.items():
        assert torch.equal(e["static"][0], e["dynamic"][0]), q
        # the first 127 tokens live in the bf16 residual (the 128th completes the block and
        # is quantized by the same append), so only rounding separates the static outputs from
        # the reference; in the dynamic setting later layers see that rounding through their
        # inputs (amplified by peaked softmax rows), still far below the quantization error
        assert float(e["static"][:, :127].max()) < 5e-3, q
        assert float(e["dynamic"][:, :127].mean()) < 0.2 * float(e["dynamic"][:, 128:].mean()), q
        assert float(e["static"][:, 128:].mean()) > 1e-2, q  # quantization shows after the first block


@pytest.mark.gpu
def test_errors_accumulate_through_depth(gpu_errors):
    """Past layer 0 the dynamic setting adds the propagated error to each layer's own."""
    for q, e in gpu_errors.items():
        for l in range(1, e["static"].shape[0]):
            assert float(e["dynamic"][l, 128:].mean()) > float(e["static"][l, 128:].mean()), (q, l)
