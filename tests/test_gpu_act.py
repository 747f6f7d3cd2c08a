"""GPU parity of the clamped GLU expert activation (the GPT-OSS release's
variant: gc = min(g, 7), uc = clamp(u, -7, 7), h = gc sig(1.702 gc) (uc + 1))
against the fp64 oracle.

Expert weights are scaled up (std 1.0 at d = 128, 0.2 at d = 2880, 0.27 at
d = 2048) so that about a quarter of the gate values and half of the up values
lie beyond the clamps, and both branches of every mask are exercised; one case
keeps the workload's weights (nothing clamps: the sigmoid slope alone).  The
forward's h uses the float32 g and u; the bf16 gu keeps each value on its
side of the clamp bounds, so that the backward's masks agree with the
forward's (checked: the stored values decide every mask as the oracle's fp64
values do, except within 1e-5 of a bound).  Compared: y, dx, dW_r and the
expert weight and bias gradients; the backward halves equal the whole call.

Bar: normwise relative error <= 2e-2 (bf16), <= 1e-4 (fp32)."""
import numpy as np
import pytest

from moe_inputs import layer_inputs, to_f64, variant
from tests.helpers import TOL, check_routing, dev, device_params, host, oracle_run, rel

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": variant("tiny", act="clamped_glu", w_std=1.0),
    "tiny_bias": variant("tiny", act="clamped_glu", w_std=1.0, expert_bias=True, b_std=2.0),
    "gptoss": variant("gptoss", T=256, act="clamped_glu", w_std=0.2),
    "gptoss_unclamped": variant("gptoss", T=256, act="clamped_glu"),
    "qwen3": variant("qwen3", T=640, act="clamped_glu", w_std=0.27),
}

_CACHE = {}


def case(name):
    if name not in _CACHE:
        cfg = CASES[name]
        inp = layer_inputs(cfg, seed=0)
        fwd, bwd = oracle_run(cfg, inp)
        _CACHE[name] = (cfg, inp, fwd, bwd)
    return _CACHE[name]


def run_layer(cfg, inp, split=False):
    import torch
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer
    print("layer", cfg["name"], "split" if split else "", flush=True)
    layer = MoELayer(L.shape_from_config(cfg))
    p = device_params(inp, cfg)
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    y = layer.forward(p, x)
    grads = layer.alloc_grads()
    if split:
        dx = layer.backward_dgrad(p, x, dy)
        layer.backward_wgrad(p, x, dy, grads)
    else:
        dx = layer.backward(p, x, dy, grads)
    torch.cuda.synchronize()
    return layer, y, dx, grads


@pytest.mark.parametrize("name", list(CASES))
def test_clamped_glu_parity(name):
    cfg, inp, fwd, bwd = case(name)
    tol = TOL[cfg["dtype"]]
    layer, y, dx, grads = run_layer(cfg, inp)
    amb, _ = check_routing(cfg, fwd, host(layer.saved["topk_idx"]))
    E, L = cfg["E"], cfg["act_limit"]
    g = np.concatenate([fwd["g"][e] for e in range(E) if e in fwd["g"]])
    u = np.concatenate([fwd["u"][e] for e in range(E) if e in fwd["u"]])
    frac_g, frac_u = float((g > L).mean()), float((np.abs(u) > L).mean())
    if name != "gptoss_unclamped":
        assert frac_g > 0.1 and frac_u > 0.1
    # the stored gate/up values decide every clamp mask as the fp64 values do
    # (outside 1e-5 of a bound, where float32 and fp64 may differ)
    f = cfg["f"]
    gu = host(layer.saved["gu"])
    gs, us = gu[:, :f], gu[:, f:]
    gref = np.concatenate([fwd["g"][e] for e in range(E) if e in fwd["g"]])
    uref = np.concatenate([fwd["u"][e] for e in range(E) if e in fwd["u"]])
    if np.array_equal(host(layer.saved["token_of"]), fwd["maps"]["token_of"]):
        far_g = np.abs(gref - L) > 1e-5
        far_u = np.abs(np.abs(uref) - L) > 1e-5
        assert np.array_equal((gs <= L)[far_g], (gref <= L)[far_g])
        assert np.array_equal((np.abs(us) <= L)[far_u], (np.abs(uref) <= L)[far_u])
    errs = {
        "y": rel(host(y), fwd["y"]),
        "dx": rel(host(dx), bwd["dx"]),
        "dw_r": rel(host(grads["dw_r"]), bwd["dw_r"]),
    }
    names = ("dw_gate", "dw_up", "dw_down") + (("db_gate", "db_up", "db_down") if cfg["expert_bias"] else ())
    for n in names:
        errs[n] = rel(host(grads[n]), np.stack([bwd["experts"][e][n] for e in range(E)]))
    print(name, "clamped: g %.3f, u %.3f;" % (frac_g, frac_u), "ambiguous", int(amb.sum()),
          {n: "%.2e" % v for n, v in errs.items()}, flush=True)
    bad = {n: v for n, v in errs.items() if not v <= tol}
    assert not bad, bad


def test_clamped_glu_split_equals_whole():
    import torch
    cfg, inp, fwd, bwd = case("qwen3")
    _, _, dx1, g1 = run_layer(cfg, inp)
    dx1 = dx1.clone()
    _, _, dx2, g2 = run_layer(cfg, inp, split=True)
    assert torch.equal(dx1.view(torch.int8), dx2.view(torch.int8))
    for n in g1:
        assert torch.equal(g1[n].view(torch.int8), g2[n].view(torch.int8)), n
