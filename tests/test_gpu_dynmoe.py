"""GPU parity of the threshold router (the DynMoE task of appendix B.3:
per-expert sigmoid gates, learned thresholds, a variable number of active
experts per token) against the fp64 oracle.

Cases: tiny fp32 (up to 4 of 8 experts), Qwen3 widths (128 experts, at most 8
active, about 3 on average), GPT-OSS widths with expert biases (32 experts, at
most 4), each also with the variable-k load-balancing loss (coefficients large
enough that its gradient weighs in the comparison); the full-size Qwen3-shaped
layer (T = 8192) against the whole oracle; the backward halves against the
whole call and accumulation; no tokens.  Compared: the selection (ids with
-1 in the empty slots, bit-exact outside the 1e-6 margin of the keys and of
the thresholds), the maps, weights and sigmoid scores, y, dx, dW_r, the
thresholds' straight-through gradient, the expert weight gradients.

Bar: normwise relative error <= 2e-2 (bf16), <= 1e-4 (fp32)."""
import numpy as np
import pytest

from moe_inputs import config, layer_inputs, to_f64, variant
from tests.helpers import TOL, check_maps_valid, check_routing, dev, device_params, host, oracle_run, rel

pytestmark = pytest.mark.gpu

TINY = variant("tiny", router="sigmoid_threshold", k=4, theta_mean=0.1, theta_std=0.1)
QWEN = variant("dynmoe", T=640)
GPTOSS = variant("gptoss", T=256, router="sigmoid_threshold", theta_mean=1.6, theta_std=0.1)
CASES = {
    "tiny": (TINY, 0.0),
    "tiny_aux": (TINY, 30.0),
    "qwen3": (QWEN, 0.0),
    "qwen3_aux": (QWEN, 3e4),
    "gptoss": (GPTOSS, 0.0),
}

_CACHE = {}


def case(name):
    if name not in _CACHE:
        cfg, coef = CASES[name]
        inp = layer_inputs(cfg, seed=0)
        fwd, bwd = oracle_run(cfg, inp, aux_coef=coef)
        _CACHE[name] = (cfg, coef, inp, fwd, bwd)
    return _CACHE[name]


def run_layer(cfg, inp, coef=0.0):
    import torch
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer
    print("layer", cfg["name"], "aux", coef, flush=True)
    layer = MoELayer(L.shape_from_config(dict(cfg, aux_coef=coef)))
    p = device_params(inp, cfg)
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    y = layer.forward(p, x)
    grads = layer.alloc_grads()
    dx = layer.backward(p, x, dy, grads)
    torch.cuda.synchronize()
    return layer, p, x, dy, y, dx, grads


def compare(cfg, inp, fwd, bwd, layer, y, dx, grads, coef):
    E, k = cfg["E"], cfg["k"]
    sv = {n: host(v) for n, v in layer.saved.items()
          if v is not None and n not in ("x_perm", "gu", "h", "o")}
    amb, all_equal = check_routing(cfg, fwd, sv["topk_idx"])
    n_act = (sv["topk_idx"] >= 0).sum(1)
    assert n_act.min() >= 1 and n_act.max() <= k and len(set(n_act.tolist())) >= 3
    mp = fwd["maps"]
    if all_equal:
        n = int(mp["offsets"][E])
        assert np.array_equal(sv["expert_offsets"], mp["offsets"])
        assert np.array_equal(sv["row_of"], mp["row_of"])
        assert np.array_equal(sv["token_of"][:n], mp["token_of"])
    else:
        check_maps_valid(sv["topk_idx"], sv["expert_offsets"], sv["row_of"], sv["token_of"], E)
    n = int(sv["expert_offsets"][E])
    x64 = to_f64(inp["x"], cfg["dtype"])
    assert np.array_equal(host(layer.saved["x_perm"][:n]), x64[sv["token_of"][:n] // k])
    keep = ~amb
    errs = {
        "topk_w": rel(sv["topk_w"][keep], fwd["route"]["topk_w"][keep]),
        "s_sel": rel(sv["s_sel"][keep], fwd["route"]["s_sel"][keep]),
        "y": rel(host(y), fwd["y"]),
        "dx": rel(host(dx), bwd["dx"]),
        "dw_r": rel(host(grads["dw_r"]), bwd["dw_r"]),
        "d_threshold": rel(host(grads["d_threshold"]), bwd["dtheta"]),
    }
    for nm in ("dw_gate", "dw_up", "dw_down") + (("db_gate", "db_up", "db_down") if cfg["expert_bias"] else ()):
        errs[nm] = rel(host(grads[nm]), np.stack([bwd["experts"][e][nm] for e in range(E)]))
    if coef:
        aux = fwd["aux"]
        errs["aux_loss"] = abs(float(host(layer.saved["aux_loss"])[0]) - aux["loss"]) / abs(aux["loss"])
        errs["router_probs (sigmoid)"] = rel(host(layer.saved["router_probs"]), aux["sig"])
    return amb, n_act, errs


@pytest.mark.parametrize("name", list(CASES))
def test_threshold_router_parity(name):
    cfg, coef, inp, fwd, bwd = case(name)
    tol = TOL[cfg["dtype"]]
    layer, p, x, dy, y, dx, grads = run_layer(cfg, inp, coef)
    amb, n_act, errs = compare(cfg, inp, fwd, bwd, layer, y, dx, grads, coef)
    if coef:
        _, bwd0 = oracle_run(cfg, inp)
        share = np.linalg.norm(bwd["dw_r"] - bwd0["dw_r"]) / np.linalg.norm(bwd["dw_r"])
        assert share > 0.1, share
        errs["aux share of dW_r"] = share
    print(name, "ambiguous", int(amb.sum()), "active experts per token: mean %.2f, counts %s" %
          (n_act.mean(), np.bincount(n_act).tolist()), {n_: "%.2e" % v for n_, v in errs.items()}, flush=True)
    errs.pop("aux share of dW_r", None)
    bad = {n_: v for n_, v in errs.items() if not v <= tol}
    assert not bad, bad


def test_threshold_split_and_accumulate():
    import torch
    cfg, coef, inp, fwd, bwd = case("qwen3_aux")
    layer, p, x, dy, y, dx1, g1 = run_layer(cfg, inp, coef)
    dx1 = dx1.clone()
    g2 = layer.alloc_grads()
    dx2 = layer.backward_dgrad(p, x, dy).clone()
    layer.backward_wgrad(p, x, dy, g2)
    torch.cuda.synchronize()
    assert torch.equal(dx1.view(torch.int8), dx2.view(torch.int8))
    for n in g1:
        assert torch.equal(g1[n].view(torch.int8), g2[n].view(torch.int8)), n
    layer.backward_wgrad(p, x, dy, g2, accumulate=True)
    torch.cuda.synchronize()
    for n in ("dw_r", "d_threshold", "dw_down"):
        assert rel(host(g2[n]), 2.0 * host(g1[n])) <= 1e-2, n


def test_threshold_without_tokens():
    cfg = dict(TINY, T=0)
    inp = layer_inputs(cfg, seed=1)
    layer, p, x, dy, y, dx, grads = run_layer(cfg, inp, 1.0)
    for n in ("dw_r", "d_threshold", "dw_gate"):
        assert float(np.abs(host(grads[n])).max()) == 0.0, n


def test_threshold_fullsize_whole_oracle():
    cfg = config("dynmoe")
    tol = TOL[cfg["dtype"]]
    inp = layer_inputs(cfg, seed=0)
    print("full-size dynmoe layer", flush=True)
    layer, p, x, dy, y, dx, grads = run_layer(cfg, inp)
    print("oracle, whole layer", flush=True)
    fwd, bwd = oracle_run(cfg, inp)
    amb, n_act, errs = compare(cfg, inp, fwd, bwd, layer, y, dx, grads, 0.0)
    print("dynmoe full size: ambiguous", int(amb.sum()), "mean active %.2f" % n_act.mean(),
          {n: "%.2e" % v for n, v in errs.items()}, flush=True)
    bad = {n: v for n, v in errs.items() if not v <= tol}
    assert not bad, bad


def test_threshold_route_bwd_entry_point():
    """moe_route_bwd on the oracle's omega with the threshold router's empty
    slots (id -1): dW_r and the router dx skip them."""
    import torch
    from paper_2605_31463_amd import _lib as L
    for name in ("tiny", "qwen3"):
        cfg, coef, inp, fwd, bwd = case(name)
        layer, p, x, dy, y, dx, grads = run_layer(cfg, inp)
        sv = layer.saved
        assert np.array_equal(host(sv["topk_idx"]), fwd["route"]["topk_idx"])
        assert (host(sv["topk_idx"]) < 0).any()
        omt = torch.from_numpy(bwd["omega"].astype(np.float32)).cuda()
        dwr = torch.empty(cfg["d"], cfg["E"], dtype=torch.float32, device="cuda")
        dxr = torch.empty(cfg["T"], cfg["d"], dtype=torch.float32, device="cuda")
        L.moe_route_bwd(layer.shape, x, p["w_r"], sv["topk_idx"], sv["topk_w"], sv["s_sel"], omt,
                        sv["expert_offsets"], sv["token_of"], dwr, dxr, layer.ws_bwd)
        torch.cuda.synchronize()
        tol = TOL[cfg["dtype"]]
        e1, e2 = rel(host(dwr), bwd["dw_r"]), rel(host(dxr), bwd["dx_router"])
        print(name, "route_bwd entry point: dw_r %.2e, dx_router %.2e" % (e1, e2), flush=True)
        assert e1 <= tol and e2 <= tol
