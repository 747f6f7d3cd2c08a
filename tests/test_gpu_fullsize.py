"""GPU parity at the full sizes of the four bf16 workloads, through the fused
layer entry points in the configuration the benchmark times (MoELayer
forward then backward on one stream).

Qwen3 shape (T=8192, d=2048, E=128, k=8, f=768): the whole fp64 oracle runs
and every output is compared.

GPT-OSS (T=16384, d=2880, E=32, k=4, f=2880), DeepSeek-V3 (T=8192, d=7168,
E=256 + shared, k=8, f=2048) and the Zipf stress layer (T=32768, Qwen3
widths): the oracle routes every token, so indices, weights, counts and maps
are compared in full; its per-token evaluation (routing, combine, expert rows
and input gradient of each token, experts visited once each with all their
tokens) gives y and dx of every token, so every output tile of the forward
and data-gradient GEMMs meets the oracle, and with it the whole dW_r; the
expert weight gradients are compared
  * for every expert, with plain torch float32 products of the routed rows
    (each output tile of the weight-gradient GEMMs is covered), and
  * against the oracle, for the most- and least-loaded experts and a random
    one at sampled intermediate indices (the SwiGLU columns are independent),
    and the shared expert's at sampled indices;
and properties are checked at every row: permuted rows are exact copies of
their tokens, weights are non-negative and sum to the route scale, experts
without rows get exactly zero gradients.

Bar: as for the small shapes (routing bit-exact outside the 1e-6 margin,
normwise relative error <= 2e-2 for bf16 over each tensor, over every token
row and over every expert)."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from moe_inputs import config, layer_inputs, to_f64
from oracle import (expert_weight_grads_at, route, router_logits, sort_maps, spec_from_config,
                    token_forward_backward)
from tests.helpers import (TOL, check_maps_valid, check_routing, dev, device_params, expert_fn, group_rel,
                           host, oracle_run, rel, row_rel, shared_of)

pytestmark = pytest.mark.gpu

N_COLS = 32


def _say(*a):
    print(*a, flush=True)


def run_layer(cfg, inp):
    import torch
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer
    _say("full-size layer", cfg["name"], "T=%d d=%d E=%d k=%d f=%d" % (cfg["T"], cfg["d"], cfg["E"],
                                                                       cfg["k"], cfg["f"]))
    layer = MoELayer(L.shape_from_config(cfg))
    p = device_params(inp, cfg)
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    y = layer.forward(p, x)
    grads = layer.alloc_grads()
    dx = layer.backward(p, x, dy, grads)
    torch.cuda.synchronize()
    return layer, p, x, y, dx, grads


def check_properties(cfg, layer, x, grads, counts):
    """Checks that hold at every row, on the device."""
    import torch
    k = cfg["k"]
    sv = layer.saved
    tok = (sv["token_of"].long() // k)
    assert torch.equal(sv["x_perm"].view(torch.int16), x[tok].view(torch.int16))
    w = sv["topk_w"]
    assert bool((w >= 0).all())
    np.testing.assert_allclose(w.sum(1).cpu().numpy(), cfg["route_scale"], rtol=1e-5)
    for e in np.nonzero(counts == 0)[0]:
        for n in ("dw_gate", "dw_up", "dw_down", "db_gate", "db_up", "db_down"):
            if n in grads:
                assert torch.count_nonzero(grads[n][int(e)]).item() == 0, (e, n)
        assert torch.count_nonzero(grads["dw_r"][:, int(e)]).item() == 0


class Prefetch:
    """expert_fn that converts experts to float64 ahead of use, in the order
    they will be asked for, a bounded number at a time."""

    def __init__(self, fn, order, depth=16):
        self.fn, self.order, self.depth = fn, [int(e) for e in order], depth
        self.pool = ThreadPoolExecutor(depth)
        self.fut = {}
        self.next = 0
        self._fill()

    def _fill(self):
        while self.next < len(self.order) and len(self.fut) < self.depth:
            e = self.order[self.next]
            self.fut[e] = self.pool.submit(self.fn, e)
            self.next += 1

    def __call__(self, e):
        r = self.fut.pop(e).result()
        self._fill()
        return r

    def close(self):
        self.pool.shutdown()


def test_fullsize_qwen3_whole_oracle():
    cfg = config("qwen3")
    tol = TOL[cfg["dtype"]]
    inp = layer_inputs(cfg, seed=0)
    layer, p, x, y, dx, grads = run_layer(cfg, inp)
    _say("oracle, whole layer")
    fwd, bwd = oracle_run(cfg, inp)
    sv = {n: host(v) for n, v in layer.saved.items() if v is not None and n in
          ("topk_idx", "topk_w", "expert_offsets", "row_of", "token_of")}
    amb, all_equal = check_routing(cfg, fwd, sv["topk_idx"])
    mp = fwd["maps"]
    if all_equal:
        for a, b in (("expert_offsets", "offsets"), ("row_of", "row_of"), ("token_of", "token_of")):
            assert np.array_equal(sv[a], mp[b])
    else:
        check_maps_valid(sv["topk_idx"], sv["expert_offsets"], sv["row_of"], sv["token_of"], cfg["E"])
    check_properties(cfg, layer, x, grads, np.diff(sv["expert_offsets"]))
    E = cfg["E"]
    errs = {
        "topk_w": rel(sv["topk_w"][~amb], fwd["route"]["topk_w"][~amb]),
        "y": rel(host(y), fwd["y"]),
        "dx": rel(host(dx), bwd["dx"]),
        "dw_r": rel(host(grads["dw_r"]), bwd["dw_r"]),
    }
    for n in ("dw_gate", "dw_up", "dw_down"):
        ref = np.stack([bwd["experts"][e][n] for e in range(E)])
        errs[n] = rel(host(grads[n]), ref)
        errs[n + "[worst expert]"] = group_rel(host(grads[n]), ref)
    same = np.all(sv["topk_idx"] == fwd["route"]["topk_idx"], axis=1)
    errs["y[worst row]"] = row_rel(host(y), fwd["y"], same)
    errs["dx[worst row]"] = row_rel(host(dx), bwd["dx"], same)
    errs["dw_r[worst expert]"] = row_rel(host(grads["dw_r"]).T, bwd["dw_r"].T)
    if all_equal:
        errs["o[worst row]"] = row_rel(host(layer.saved["o"]), fwd["o"])
    _say("qwen3 full size: ambiguous tokens", int(amb.sum()), {n: "%.2e" % v for n, v in errs.items()})
    bad = {n: v for n, v in errs.items() if not v <= tol}
    assert not bad, bad


def torch_expert_weight_grads(cfg, layer, p, x, dy, grads):
    """Every expert's weight (and bias) gradients against plain torch float32
    products, so that every output tile of the weight-gradient GEMMs is checked
    at full size, whatever order the kernels deal the tiles in.  Built from the
    rows' tokens and gating weights (checked against the oracle beforehand),
    x, dy and the weights; none of the layer's saved activations is used.
    Returns, per tensor, the largest per-expert normwise error and its expert
    (one wrong 256 x 256 tile moves its expert's error well past the bar)."""
    import torch
    k, bias = cfg["k"], cfg["expert_bias"]
    sv = layer.saved
    offs = sv["expert_offsets"].long().cpu().tolist()
    slot = sv["token_of"].long()
    tok = slot // k
    wrow = sv["topk_w"].reshape(-1).float()[slot]
    names = ["dw_gate", "dw_up", "dw_down"] + (["db_gate", "db_up", "db_down"] if bias else [])
    worst = {n: (0.0, -1) for n in names}
    for e in range(cfg["E"]):
        lo, hi = offs[e], offs[e + 1]
        if hi == lo:
            continue  # exact zeros, checked by check_properties
        te = tok[lo:hi]
        xe = x[te].float()
        do = wrow[lo:hi, None] * dy[te].float()
        g = xe @ p["w_gate"][e].float()
        u = xe @ p["w_up"][e].float()
        if bias:
            g = g + p["b_gate"][e].float()
            u = u + p["b_up"][e].float()
        sg = torch.sigmoid(g)
        h = g * sg * u
        dh = do @ p["w_down"][e].float().t().contiguous()
        dg = dh * u * sg * (1.0 + g * (1.0 - sg))
        du = dh * g * sg
        xt = xe.t().contiguous()
        ref = {"dw_gate": xt @ dg, "dw_up": xt @ du, "dw_down": h.t().contiguous() @ do}
        if bias:
            ref.update(db_gate=dg.sum(0), db_up=du.sum(0), db_down=do.sum(0))
        for n, r in ref.items():
            err = (torch.linalg.vector_norm(grads[n][e].float() - r) / torch.linalg.vector_norm(r)).item()
            if not err <= worst[n][0]:
                worst[n] = (err, e)
    return worst


def _expert_rows(mp, e, k):
    toks = mp["token_of"][mp["offsets"][e]:mp["offsets"][e + 1]]
    return toks // k, toks % k


@pytest.mark.parametrize("name", ["gptoss", "dsv3", "stress"])
def test_fullsize_every_token(name):
    import torch
    cfg = config(name)
    dt = cfg["dtype"]
    tol = TOL[dt]
    T, E, k, f = cfg["T"], cfg["E"], cfg["k"], cfg["f"]
    _say("inputs", name)
    inp = layer_inputs(cfg, seed=0)
    layer, p, xd, y, dx, grads = run_layer(cfg, inp)
    _say("oracle routing of every token")
    spec = spec_from_config(cfg)
    x64 = to_f64(inp["x"], dt)
    dy64 = to_f64(inp["dy"], dt)
    w_r = inp["w_r"].astype(np.float64)
    beta = None if inp["router_bias"] is None else inp["router_bias"].astype(np.float64)
    rt = route(spec, router_logits(x64, w_r), beta)
    fwd_like = {"route": rt}
    sv = {n: host(layer.saved[n]) for n in ("topk_idx", "topk_w", "expert_offsets", "row_of", "token_of")}
    amb, all_equal = check_routing(cfg, fwd_like, sv["topk_idx"])
    errs = {"topk_w": rel(sv["topk_w"][~amb], rt["topk_w"][~amb])}
    if cfg["router"] == "sigmoid_grouped":
        errs["s_sel"] = rel(host(layer.saved["s_sel"])[~amb], rt["s_sel"][~amb])
    mp = sort_maps(rt["topk_idx"], E)
    if all_equal:
        for a, b in (("expert_offsets", "offsets"), ("row_of", "row_of"), ("token_of", "token_of")):
            assert np.array_equal(sv[a], mp[b])
    else:
        check_maps_valid(sv["topk_idx"], sv["expert_offsets"], sv["row_of"], sv["token_of"], E)
    counts = np.diff(sv["expert_offsets"])
    check_properties(cfg, layer, xd, grads, counts)
    _say("torch float32 weight gradients of every expert")
    for n, (err, e) in torch_expert_weight_grads(cfg, layer, p, xd, dev(inp["dy"], dt), grads).items():
        errs["%s[every expert, worst e=%d]" % (n, e)] = err
    # tokens routed differently from the oracle (ambiguous ones) and the experts they touch
    differ = np.nonzero(np.any(sv["topk_idx"] != rt["topk_idx"], axis=1))[0]
    touched = set(np.unique(np.concatenate([sv["topk_idx"][differ].ravel(),
                                            rt["topk_idx"][differ].ravel()])).tolist()) if differ.size else set()

    # ---- per-token results of every token: y, dx (every row), dW_r
    efn = expert_fn(inp, cfg)
    shared = shared_of(inp, cfg)
    _say("oracle per-token results of all", T, "tokens over", E, "experts")
    pf = Prefetch(efn, np.unique(rt["topk_idx"]))
    try:
        r = token_forward_backward(spec, x64, dy64, w_r, beta, pf, shared)
    finally:
        pf.close()
    keep = np.ones(T, dtype=bool)
    keep[differ] = False
    yh, dxh = host(y), host(dx)
    errs["y"] = rel(yh[keep], r["y"][keep])
    errs["dx"] = rel(dxh[keep], r["dx"][keep])
    errs["y[worst row]"] = row_rel(yh, r["y"], keep)
    errs["dx[worst row]"] = row_rel(dxh, r["dx"], keep)
    dwr_ref = x64.T @ r["dl_dense"]
    ecols = np.array([e for e in range(E) if e not in touched])  # dW_r columns of experts no flip touches
    dwr = host(grads["dw_r"])
    errs["dw_r"] = rel(dwr[:, ecols], dwr_ref[:, ecols])
    errs["dw_r[worst expert]"] = row_rel(dwr[:, ecols].T, dwr_ref[:, ecols].T)
    del r

    # ---- expert weight gradients at sampled intermediate indices
    ocounts = mp["counts"]
    usable = [e for e in range(E) if ocounts[e] > 0 and e not in touched]
    e_min = min(usable, key=lambda e: (ocounts[e], e))
    e_max = max(usable, key=lambda e: (ocounts[e], -e))
    rng = np.random.default_rng(1234)
    e_rand = int(rng.choice([e for e in usable if e not in (e_min, e_max)]))
    cols = np.unique(np.concatenate([[0, f - 1, f // 2], rng.choice(f, N_COLS, replace=False)]))
    ct = torch.from_numpy(cols).cuda()
    bias = cfg["expert_bias"]
    for tag, e in (("e_max", e_max), ("e_min", e_min), ("e_rand", e_rand)):
        tt, ss = _expert_rows(mp, e, k)
        _say("oracle weight gradients of expert", e, "rows", tt.size)
        wg, wu, wd, bg, bu, _ = efn(e)
        do = rt["topk_w"][tt, ss][:, None] * dy64[tt]
        g = expert_weight_grads_at(x64[tt], do, wg, wu, wd, bg, bu, cols=cols, with_bias=bias)
        errs["dw_gate[%s]" % tag] = rel(host(grads["dw_gate"][e][:, ct]), g["dw_gate"])
        errs["dw_up[%s]" % tag] = rel(host(grads["dw_up"][e][:, ct]), g["dw_up"])
        errs["dw_down[%s]" % tag] = rel(host(grads["dw_down"][e][ct, :]), g["dw_down"])
        if bias:
            errs["db_gate[%s]" % tag] = rel(host(grads["db_gate"][e][ct]), g["db_gate"])
            errs["db_up[%s]" % tag] = rel(host(grads["db_up"][e][ct]), g["db_up"])
            errs["db_down[%s]" % tag] = rel(host(grads["db_down"][e]), g["db_down"])
    if shared is not None:
        fs = cfg["f_shared"]
        scols = np.unique(np.concatenate([[0, fs - 1], rng.choice(fs, N_COLS, replace=False)]))
        sct = torch.from_numpy(scols).cuda()
        _say("oracle shared-expert weight gradients")
        g = expert_weight_grads_at(x64, dy64, *shared, cols=scols)
        errs["dws_gate"] = rel(host(grads["dws_gate"][:, sct]), g["dw_gate"])
        errs["dws_up"] = rel(host(grads["dws_up"][:, sct]), g["dw_up"])
        errs["dws_down"] = rel(host(grads["dws_down"][sct, :]), g["dw_down"])
    _say(name, "full size: ambiguous tokens", int(amb.sum()), "routed differently", differ.size,
         "experts e_min/e_max/e_rand", (e_min, int(ocounts[e_min])), (e_max, int(ocounts[e_max])),
         (e_rand, int(ocounts[e_rand])), {n: "%.2e" % v for n, v in errs.items()})
    bad = {n: v for n, v in errs.items() if not v <= tol}
    assert not bad, bad
