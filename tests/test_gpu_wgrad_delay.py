"""GPU tests of the layer backward split into its input-gradient and
weight-gradient halves (weight-gradient delay) and of gradient accumulation.

  * moe_layer_bwd_dgrad then moe_layer_bwd_wgrad (accumulate = 0) gives the
    same bits as moe_layer_bwd, on every router family, with expert biases
    and with a shared expert;
  * accumulate = 1 adds to what the gradient buffers hold: starting from
    random values G0 the result matches G0 + the oracle's gradients (same bar
    as the other parity tests), and two accumulating calls from zero match
    twice the oracle's gradients;
  * with no tokens, accumulating leaves the buffers bit for bit unchanged."""
import numpy as np
import pytest

from moe_inputs import layer_inputs, variant
from tests.helpers import TOL, dev, device_params, host, oracle_run, rel

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": variant("tiny"),
    "qwen3": variant("qwen3", T=640),
    "gptoss": variant("gptoss", T=384),
    "dsv3": variant("dsv3", T=384, d=512, f=256, f_shared=256),
}
GRADS = ("dw_r", "dw_gate", "dw_up", "dw_down", "db_gate", "db_up", "db_down", "dws_gate", "dws_up", "dws_down")


def setup_layer(cfg, inp):
    import torch
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer
    layer = MoELayer(L.shape_from_config(cfg))
    p = device_params(inp, cfg)
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    layer.forward(p, x)
    torch.cuda.synchronize()
    return layer, p, x, dy


def oracle_grads(cfg, bwd):
    E = cfg["E"]
    g = {"dw_r": bwd["dw_r"]}
    names = ["dw_gate", "dw_up", "dw_down"] + (["db_gate", "db_up", "db_down"] if cfg["expert_bias"] else [])
    for n in names:
        g[n] = np.stack([bwd["experts"][e][n] for e in range(E)])
    if cfg["n_shared"]:
        for n, m in (("dws_gate", "dw_gate"), ("dws_up", "dw_up"), ("dws_down", "dw_down")):
            g[n] = bwd["shared"][m]
    return g


@pytest.mark.parametrize("name", list(CASES))
def test_split_equals_layer_bwd(name):
    import torch
    cfg = CASES[name]
    inp = layer_inputs(cfg, seed=0)
    print("split vs whole backward", name, flush=True)
    layer, p, x, dy = setup_layer(cfg, inp)
    g1 = layer.alloc_grads()
    dx1 = layer.backward(p, x, dy, g1).clone()
    g2 = layer.alloc_grads()
    layer.dx.zero_()
    dx2 = layer.backward_dgrad(p, x, dy).clone()
    layer.backward_wgrad(p, x, dy, g2, accumulate=False)
    torch.cuda.synchronize()
    assert torch.equal(dx1.view(torch.int8), dx2.view(torch.int8))
    for n in g1:
        assert torch.equal(g1[n].view(torch.int8), g2[n].view(torch.int8)), n


@pytest.mark.parametrize("name", ["tiny", "gptoss", "dsv3"])
def test_accumulate_adds_to_grads(name):
    import torch
    cfg = CASES[name]
    tol = TOL[cfg["dtype"]]
    inp = layer_inputs(cfg, seed=0)
    _, bwd = oracle_run(cfg, inp)
    og = oracle_grads(cfg, bwd)
    print("accumulate", name, flush=True)
    layer, p, x, dy = setup_layer(cfg, inp)
    grads = layer.alloc_grads()
    rng = np.random.default_rng(7)
    g0 = {}
    for n, t in grads.items():
        # random starting values of the gradient's own scale, in the buffer's type
        init = rng.standard_normal(t.shape) * float(np.std(og[n]) + 1e-30)
        t.copy_(torch.from_numpy(init).to(t.dtype))
        g0[n] = host(t)
    layer.backward_dgrad(p, x, dy)
    layer.backward_wgrad(p, x, dy, grads, accumulate=True)
    torch.cuda.synchronize()
    errs = {n: rel(host(grads[n]), g0[n] + og[n]) for n in grads}
    # two accumulating calls from zero: twice the gradient
    for t in grads.values():
        t.zero_()
    layer.backward_wgrad(p, x, dy, grads, accumulate=True)
    layer.backward_wgrad(p, x, dy, grads, accumulate=True)
    torch.cuda.synchronize()
    errs.update({n + " x2": rel(host(grads[n]), 2 * og[n]) for n in grads})
    print(name, {k: "%.2e" % v for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad


def test_accumulate_without_tokens_keeps_grads():
    import torch
    cfg = variant("qwen3", T=0, d=128, f=128, E=16, k=4)
    inp = layer_inputs(cfg, seed=1)
    print("accumulate, no tokens", flush=True)
    layer, p, x, dy = setup_layer(cfg, inp)
    grads = layer.alloc_grads()
    for t in grads.values():
        t.copy_(torch.randn(t.shape, device="cuda").to(t.dtype))
    before = {n: t.clone() for n, t in grads.items()}
    layer.backward_dgrad(p, x, dy)
    layer.backward_wgrad(p, x, dy, grads, accumulate=True)
    torch.cuda.synchronize()
    for n, t in grads.items():
        assert torch.equal(t.view(torch.int8), before[n].view(torch.int8)), n
