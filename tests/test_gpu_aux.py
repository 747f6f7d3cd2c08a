"""GPU parity of the global-level load-balancing loss against the oracle.

The loss value, the saved router probabilities, and the layer's dx and dW_r
with the loss's gradient added are compared with the fp64 oracle on the
softmax router families (top-k then renormalise, top-k softmax, logit bias),
in fp32 and bf16, with experts padded for the router-dx product (E = 8, 32)
and not (E = 128).  Large coefficients make the loss's share of dW_r and dx
large (asserted), so that the comparison sees its paths; the loss's own part
of dW_r (the difference of runs with and without it, float32) is compared
separately.
Given batch fractions replace this call's counts.  The layer backward halves
stay bitwise equal to the whole call with the loss on.  No tokens: loss 0."""
import numpy as np
import pytest

from moe_inputs import layer_inputs, variant
from tests.helpers import TOL, check_routing, dev, device_params, host, oracle_run, rel

pytestmark = pytest.mark.gpu

# Coefficients chosen so that the loss's gradient is a large share of the
# router's dx and dW_r on these inputs (near-uniform routing makes it small:
# f - sum f p nearly vanishes), so that the comparisons exercise its paths.
CASES = {
    "tiny": (variant("tiny", T=96), 100.0),
    "qwen3": (variant("qwen3", T=640), 1e5),
    "gptoss": (variant("gptoss", T=384), 1e5),
    "stress": (variant("stress", T=2048), 3e3),
}


def run(cfg, inp, coef, aux_f=None):
    import torch
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer
    shape = L.shape_from_config(dict(cfg, aux_coef=coef))
    layer = MoELayer(shape)
    p = device_params(inp, cfg)
    if aux_f is not None:
        p["aux_f"] = torch.from_numpy(aux_f.astype(np.float32)).cuda()
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    layer.forward(p, x)
    grads = layer.alloc_grads()
    dx = layer.backward(p, x, dy, grads)
    torch.cuda.synchronize()
    return layer, dx, grads


@pytest.mark.parametrize("name", list(CASES))
def test_aux_loss_parity(name):
    cfg, coef = CASES[name]
    tol = TOL[cfg["dtype"]]
    inp = layer_inputs(cfg, seed=0)
    fwd, bwd = oracle_run(cfg, inp, aux_coef=coef)
    _, bwd0 = oracle_run(cfg, inp)
    print("aux loss", name, flush=True)
    layer, dx, grads = run(cfg, inp, coef)
    _, _, grads0 = run(cfg, inp, 0.0)
    amb, _ = check_routing(cfg, fwd, host(layer.saved["topk_idx"]))
    assert not amb.any()
    aux = fwd["aux"]
    errs = {
        "loss": abs(float(host(layer.saved["aux_loss"])[0]) - aux["loss"]) / abs(aux["loss"]),
        "router_probs": rel(host(layer.saved["router_probs"]), aux["probs"]),
        "dx": rel(host(dx), bwd["dx"]),
        "dw_r": rel(host(grads["dw_r"]), bwd["dw_r"]),
        "dw_r aux part": rel(host(grads["dw_r"]) - host(grads0["dw_r"]), bwd["dw_r"] - bwd0["dw_r"]),
    }
    share = np.linalg.norm(bwd["dw_r"] - bwd0["dw_r"]) / np.linalg.norm(bwd["dw_r"])
    dx_share = np.linalg.norm(bwd["dx"] - bwd0["dx"]) / np.linalg.norm(bwd["dx"])
    print(name, "aux share of dW_r %.2f, of dx %.3f" % (share, dx_share), {k: "%.2e" % v for k, v in errs.items()})
    assert share > 0.1 and dx_share > 0.1  # the loss's gradient weighs in the comparison
    assert errs["loss"] <= 1e-5 and errs["router_probs"] <= 1e-6
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad


def test_aux_loss_given_fractions():
    cfg, coef = CASES["qwen3"]
    inp = layer_inputs(cfg, seed=0)
    f = np.random.default_rng(3).dirichlet(np.ones(cfg["E"]))
    fwd, bwd = oracle_run(cfg, inp, aux_coef=coef, aux_f=f.astype(np.float32).astype(np.float64))
    print("aux loss, given fractions", flush=True)
    layer, dx, grads = run(cfg, inp, coef, aux_f=f)
    assert abs(float(host(layer.saved["aux_loss"])[0]) - fwd["aux"]["loss"]) <= 1e-5 * abs(fwd["aux"]["loss"])
    assert rel(host(grads["dw_r"]), bwd["dw_r"]) <= TOL[cfg["dtype"]]
    assert rel(host(dx), bwd["dx"]) <= TOL[cfg["dtype"]]


def test_aux_split_equals_whole_backward():
    import torch
    cfg, coef = CASES["gptoss"]
    inp = layer_inputs(cfg, seed=0)
    print("aux loss, backward halves", flush=True)
    layer, dx1, g1 = run(cfg, inp, coef)
    dx1 = dx1.clone()
    p = device_params(inp, cfg)
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    g2 = layer.alloc_grads()
    dx2 = layer.backward_dgrad(p, x, dy).clone()
    layer.backward_wgrad(p, x, dy, g2)
    torch.cuda.synchronize()
    assert torch.equal(dx1.view(torch.int8), dx2.view(torch.int8))
    for n in g1:
        assert torch.equal(g1[n].view(torch.int8), g2[n].view(torch.int8)), n


def test_aux_loss_without_tokens_is_zero():
    cfg = variant("qwen3", T=0, d=128, f=128, E=16, k=4)
    inp = layer_inputs(cfg, seed=1)
    print("aux loss, no tokens", flush=True)
    layer, dx, grads = run(cfg, inp, 1.0)
    assert float(host(layer.saved["aux_loss"])[0]) == 0.0
    assert float(np.abs(host(grads["dw_r"])).max()) == 0.0
