"""GPU parity of the MoE++ zero-computation experts (appendix B.3: zero, copy
and constant experts in the pool, the router widened over them, the
load-balancing loss weighting them) against the fp64 oracle.

Cases: fp32 and bf16; softmax over the top-k after a softmax over all experts
(Qwen3 widths with 8 zero, 8 copy and 16 constant experts next to the 128 FFN
experts, the pool of 160 on the MFMA router path) and softmax over the
selected logits with expert biases (GPT-OSS widths, a pool of 40 on the
general router path); a pool where most slots pick a zero-computation expert
and some FFN experts get no rows.  Compared: routing and the maps over the
whole pool (bit-exact outside the 1e-6 margin), the FFN rows of x_perm
(exact copies), y, dx, dW_r (every pool column), the expert weight
gradients, and the constant experts' dv and dW_c; with the load-balancing
loss on (zero-computation terms weighted 0.5), its value too.  The backward
halves give the bits of the whole backward, accumulation adds, and the Qwen3
-shaped workload is compared in full at T = 8192.  No tokens: zero gradients.

Bar: normwise relative error <= 2e-2 (bf16), <= 1e-4 (fp32)."""
import numpy as np
import pytest

from moe_inputs import config, layer_inputs, pool_size, to_f64, variant
from tests.helpers import TOL, check_maps_valid, check_routing, dev, device_params, host, oracle_run, rel

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": (variant("tiny", n_zero=1, n_copy=1, n_const=2, zc_aux_weight=0.5), 0.0),
    "tiny_aux": (variant("tiny", n_zero=1, n_copy=1, n_const=2, zc_aux_weight=0.5), 100.0),
    # half the pool without computation, few tokens: FFN experts without rows
    "tiny_zc_heavy": (variant("tiny", T=9, E=16, k=4, n_zero=6, n_copy=6, n_const=4), 0.0),
    "moepp": (variant("moepp", T=640), 0.0),
    "moepp_aux": (variant("moepp", T=640), 1e5),
    "gptoss": (variant("gptoss", T=256, n_zero=2, n_copy=2, n_const=4), 0.0),
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
    E, k, Ep = cfg["E"], cfg["k"], pool_size(cfg)
    sv = {n: host(v) for n, v in layer.saved.items()
          if v is not None and n not in ("x_perm", "gu", "h", "o")}
    amb, all_equal = check_routing(cfg, fwd, sv["topk_idx"])
    mp = fwd["maps"]
    if all_equal:
        for a, b in (("expert_offsets", "offsets"), ("row_of", "row_of"), ("token_of", "token_of")):
            assert np.array_equal(sv[a], mp[b]), a
    else:
        check_maps_valid(sv["topk_idx"], sv["expert_offsets"], sv["row_of"], sv["token_of"], Ep)
    n_ffn = int(sv["expert_offsets"][E])
    assert 0 < n_ffn < cfg["T"] * k                     # both kinds of slot present
    x64 = to_f64(inp["x"], cfg["dtype"])
    # (the rows after the FFN experts' hold no data)
    assert np.array_equal(host(layer.saved["x_perm"][:n_ffn]), x64[sv["token_of"][:n_ffn] // k])
    keep = ~amb
    errs = {
        "topk_w": rel(sv["topk_w"][keep], fwd["route"]["topk_w"][keep]),
        "y": rel(host(y), fwd["y"]),
        "dx": rel(host(dx), bwd["dx"]),
        "dw_r": rel(host(grads["dw_r"]), bwd["dw_r"]),
        "dw_r zc columns": rel(host(grads["dw_r"])[:, E:], bwd["dw_r"][:, E:]),
    }
    for n in ("dw_gate", "dw_up", "dw_down") + (("db_gate", "db_up", "db_down") if cfg["expert_bias"] else ()):
        errs[n] = rel(host(grads[n]), np.stack([bwd["experts"][e][n] for e in range(E)]))
    if cfg["n_const"]:
        errs["dzc_v"] = rel(host(grads["dzc_v"]), bwd["zc"]["dv"])
        errs["dzc_wc"] = rel(host(grads["dzc_wc"]), bwd["zc"]["dwc"])
    if coef:
        aux = fwd["aux"]
        errs["aux_loss"] = abs(float(host(layer.saved["aux_loss"])[0]) - aux["loss"]) / abs(aux["loss"])
        errs["router_probs"] = rel(host(layer.saved["router_probs"]), aux["probs"])
    return amb, errs


@pytest.mark.parametrize("name", list(CASES))
def test_zc_layer_parity(name):
    cfg, coef, inp, fwd, bwd = case(name)
    tol = TOL[cfg["dtype"]]
    layer, p, x, dy, y, dx, grads = run_layer(cfg, inp, coef)
    amb, errs = compare(cfg, inp, fwd, bwd, layer, y, dx, grads, coef)
    idx = fwd["route"]["topk_idx"]
    print(name, "ambiguous tokens:", int(amb.sum()), "zero-computation slots: %d of %d" %
          (int((idx >= cfg["E"]).sum()), idx.size), {n: "%.2e" % v for n, v in errs.items()}, flush=True)
    bad = {n: v for n, v in errs.items() if not v <= tol}
    assert not bad, bad
    if coef:
        assert errs["aux_loss"] <= 1e-5 and errs["router_probs"] <= 1e-6


def test_zc_split_and_accumulate():
    """dgrad then wgrad gives the whole backward's bits; a second accumulating
    wgrad doubles every gradient (within rounding)."""
    import torch
    cfg, coef, inp, fwd, bwd = case("moepp_aux")
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
    for n in ("dw_r", "dzc_v", "dzc_wc", "dw_down"):
        a, b = host(g2[n]), 2.0 * host(g1[n])
        assert rel(a, b) <= 1e-2, n


def test_zc_without_tokens():
    cfg = variant("tiny", T=0, n_zero=1, n_copy=2, n_const=2)
    inp = layer_inputs(cfg, seed=1)
    layer, p, x, dy, y, dx, grads = run_layer(cfg, inp, 1.0)
    for n in ("dw_r", "dzc_v", "dzc_wc", "dw_gate"):
        assert float(np.abs(host(grads[n])).max()) == 0.0, n
    assert float(host(layer.saved["aux_loss"])[0]) == 0.0


def test_zc_fullsize_moepp_whole_oracle():
    cfg = config("moepp")
    tol = TOL[cfg["dtype"]]
    inp = layer_inputs(cfg, seed=0)
    print("full-size moepp layer", flush=True)
    layer, p, x, dy, y, dx, grads = run_layer(cfg, inp)
    print("oracle, whole layer", flush=True)
    fwd, bwd = oracle_run(cfg, inp)
    amb, errs = compare(cfg, inp, fwd, bwd, layer, y, dx, grads, 0.0)
    print("moepp full size: ambiguous tokens", int(amb.sum()), {n: "%.2e" % v for n, v in errs.items()},
          flush=True)
    bad = {n: v for n, v in errs.items() if not v <= tol}
    assert not bad, bad
