"""GPU parity of the FP8 (E4M3) forward of the routed experts against the fp64
oracle's FP8 layer.

  * the weight cache: every code bit-exact against the oracle's per-column
    quantisation, every scale equal (the row quantisers of x and h share its
    conversion and scale arithmetic);
  * the layer (moe_layer_fwd / moe_layer_bwd with shape.fp8 = 1): gu, y, dx,
    dW_r and the expert weight gradients against the oracle's FP8 layer (bar:
    2e-2 normwise), and gu farther than that from the bf16 forward (so that the
    comparison sees the quantisation), on both GEMM tile shapes (Qwen3 widths
    with 32 experts: 32 rows per expert, 128-row tiles; with 16 experts: 512
    rows, 256-row tiles), with expert biases, with the clamped GLU, and
    DeepSeek-V3 widths with the (bf16) shared expert;
  * the cache is reused across calls (two forwards, one build);
  * MoE++ (zero-computation experts in the pool) at both levels, and a
    sparse batch (16 tokens over 32 experts: most experts without rows);
  * with shape.fp8 = 2 the data-gradient GEMMs also run on E4M3 operands: the
    cache's row codes of W_down and [W_gate | W_up] bit-exact against the
    oracle's row quantisation, and the same layer cases against the oracle's
    FP8 backward, with dx farther than the bar from the backward of FP8
    forward GEMMs only."""
import numpy as np
import pytest

from moe_inputs import layer_inputs, to_f64, variant
from oracle import quantize_cols, quantize_rows
from tests.helpers import TOL, check_routing, dev, device_params, host, oracle_run, rel

pytestmark = pytest.mark.gpu

CASES = {
    "qwen3_small_tiles": variant("qwen3", T=256, E=32, k=4, fp8=True),
    # 32 slots over 32 experts: many experts without rows, one- and two-row experts
    "qwen3_sparse": variant("qwen3", T=16, E=32, k=2, fp8=True),
    "qwen3_e16": variant("qwen3", T=1024, E=16, fp8=True),
    "qwen3_e16_bias": variant("qwen3", T=1024, E=16, expert_bias=True, fp8=True),
    "qwen3_e16_clamped": variant("qwen3", T=1024, E=16, act="clamped_glu", w_std=0.27, fp8=True),
    "dsv3": variant("dsv3", T=384, d=512, f=256, f_shared=256, fp8=True),
    # zero-computation experts in the pool: d_o rows quantised by their own pass
    "moepp": variant("moepp", T=256, E=32, d=512, f=256, fp8=True),
    # the threshold router: 1 to k filled slots per token, rows quantised as usual
    "dynmoe": variant("dynmoe", T=256, E=32, d=512, f=256, fp8=True),
}


LEVELS = [(n, 1) for n in CASES] + [(n, 2) for n in CASES]


def setup(cfg, inp):
    import torch
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer
    layer = MoELayer(L.shape_from_config(cfg))
    p = device_params(inp, cfg)
    layer.build_fp8_cache(p)
    torch.cuda.synchronize()
    return layer, p


def test_weight_cache_codes_bit_exact():
    import torch
    from paper_2605_31463_amd import _lib as L
    cfg = variant("qwen3", T=64, E=3, k=2, d=256, f=128, fp8=2)
    inp = layer_inputs(cfg, seed=2)
    # add exact zeros, a zero column and wide magnitudes to the weights
    for n in ("w_gate", "w_up", "w_down"):
        w = to_f64(inp[n], "bf16")
        w[:, :, 0] = 0.0
        w[:, 3, :] *= 1e3
        inp[n] = (np.asarray(w, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    print("weight cache, E=3 d=256 f=128", flush=True)
    layer, p = setup(cfg, inp)
    E, d, f = cfg["E"], cfg["d"], cfg["f"]
    raw = layer.fp8_cache.cpu().numpy()
    off = 0

    def region(nbytes):
        nonlocal off
        r = raw[off:off + nbytes]
        off += (nbytes + 255) // 256 * 256
        return r
    qg, qu, qd = region(E * f * d), region(E * f * d), region(E * d * f)
    for n_ in (f, f, d):
        region(E * n_ * 4)                             # column maxima
    sg, su, sd = (region(E * n * 4).view(np.float32) for n in (f, f, d))
    for name, q, s, K, N in (("w_gate", qg, sg, d, f), ("w_up", qu, su, d, f), ("w_down", qd, sd, f, d)):
        for e in range(E):
            w = to_f64(inp[name][e], "bf16")
            codes, scale, _ = quantize_cols(w)               # codes [K][N]
            got = q[e * N * K:(e + 1) * N * K].reshape(N, K)  # transposed
            assert np.array_equal(got, codes.T), (name, e, int((got != codes.T).sum()))
            assert np.array_equal(s[e * N:(e + 1) * N].astype(np.float64), scale), (name, e)
    # the data-gradient GEMMs' row codes: [W_gate | W_up] [E][d][2f], W_down [E][f][d]
    qgu, qd_r = region(E * d * 2 * f), region(E * f * d)
    sgu, sd_r = region(E * d * 4).view(np.float32), region(E * f * 4).view(np.float32)
    for e in range(E):
        wgu = np.concatenate([to_f64(inp["w_gate"][e], "bf16"), to_f64(inp["w_up"][e], "bf16")], axis=1)
        codes, scale, _ = quantize_rows(wgu)
        assert np.array_equal(qgu[e * d * 2 * f:(e + 1) * d * 2 * f].reshape(d, 2 * f), codes), ("w_gu rows", e)
        assert np.array_equal(sgu[e * d:(e + 1) * d].astype(np.float64), scale), ("w_gu scales", e)
        codes, scale, _ = quantize_rows(to_f64(inp["w_down"][e], "bf16"))
        assert np.array_equal(qd_r[e * f * d:(e + 1) * f * d].reshape(f, d), codes), ("w_down rows", e)
        assert np.array_equal(sd_r[e * f:(e + 1) * f].astype(np.float64), scale), ("w_down scales", e)
    assert off == len(raw)                            # every region of the cache checked
    torch.cuda.synchronize()


@pytest.mark.parametrize("name,level", LEVELS)
def test_fp8_layer_parity(name, level):
    import torch
    cfg = dict(CASES[name], fp8=level)
    tol = TOL[cfg["dtype"]]
    inp = layer_inputs(cfg, seed=0)
    print("fp8 layer", name, "level", level, flush=True)
    layer, p = setup(cfg, inp)
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    layer.forward(p, x)
    y = layer.forward(p, x)            # the cache serves repeated calls
    grads = layer.alloc_grads()
    dx = layer.backward(p, x, dy, grads)
    torch.cuda.synchronize()
    fwd, bwd = oracle_run(cfg, inp)
    fwd0, _ = oracle_run(dict(cfg, fp8=False), inp)
    amb, all_equal = check_routing(cfg, fwd, host(layer.saved["topk_idx"]))
    assert all_equal
    E, f = cfg["E"], cfg["f"]
    n = int(host(layer.saved["expert_offsets"])[E])
    gu = host(layer.saved["gu"][:n])
    g_ref = np.concatenate([fwd["g"][e] for e in range(E) if e in fwd["g"]])
    u_ref = np.concatenate([fwd["u"][e] for e in range(E) if e in fwd["u"]])
    g_bf = np.concatenate([fwd0["g"][e] for e in range(E) if e in fwd0["g"]])
    errs = {
        "g": rel(gu[:, :f], g_ref), "u": rel(gu[:, f:], u_ref),
        "y": rel(host(y), fwd["y"]), "dx": rel(host(dx), bwd["dx"]),
        "dw_r": rel(host(grads["dw_r"]), bwd["dw_r"]),
    }
    for nm in ("dw_gate", "dw_up", "dw_down") + (("db_gate", "db_up", "db_down") if cfg["expert_bias"] else ()):
        errs[nm] = rel(host(grads[nm]), np.stack([bwd["experts"][e][nm] for e in range(E)]))
    if cfg["n_shared"]:
        errs["dws_down"] = rel(host(grads["dws_down"]), bwd["shared"]["dw_down"])
    dist_bf16 = rel(g_bf, g_ref)
    print(name, "fp8 vs bf16 forward (oracle): g %.2e, y %.2e;" % (dist_bf16, rel(fwd0["y"], fwd["y"])),
          {k: "%.2e" % v for k, v in errs.items()}, flush=True)
    assert dist_bf16 > 2 * errs["g"]          # the comparison resolves the quantisation
    if level == 2:
        # the comparison resolves the data-gradient quantisation: in dW_gate
        # (through dh) and, where the FFN experts carry dx, in dx
        _, bwd1 = oracle_run(dict(cfg, fp8=1), inp)
        dist_dx = rel(bwd1["dx"], bwd["dx"])
        dist_dwg = rel(np.stack([bwd1["experts"][e]["dw_gate"] for e in range(E)]),
                       np.stack([bwd["experts"][e]["dw_gate"] for e in range(E)]))
        print(name, "fp8 dgrad vs forward-only FP8 (oracle): dx %.2e, dw_gate %.2e" % (dist_dx, dist_dwg), flush=True)
        assert dist_dwg > 2 * errs["dw_gate"]
        if cfg["n_zero"] + cfg["n_copy"] + cfg["n_const"] == 0:
            assert dist_dx > 2 * errs["dx"]
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad


# (workload, sampled tokens, experts whose weight gradients are sampled): the
# oracle's E4M3 quantisation of one DeepSeek-V3 expert (five 7168 x 2048 weight
# quantisations) takes ~18 s on the host, so that workload samples one token
# (its 8 experts) and one expert's weight-gradient columns
FP8_FULLSIZE = {"qwen3": (6, ("e_min", "e_max", "e_rand")), "dsv3": (1, ("e_min",))}


@pytest.mark.parametrize("name", list(FP8_FULLSIZE))
def test_fp8_fullsize_sampled(name):
    """A workload at full size (the bench's launch configuration) with
    fp8 = 2: routing and maps of every token against the oracle; y and dx of
    sampled tokens (each row on its own too) against the oracle's per-token
    FP8 evaluation (with the bf16 shared expert where there is one); the
    expert weight gradients at sampled intermediate columns against its
    per-column FP8 evaluation."""
    import torch
    from moe_inputs import config
    from oracle import (expert_weight_grads_at, route, router_logits, sort_maps, spec_from_config,
                        token_forward_backward)
    from tests.helpers import check_maps_valid, expert_fn, row_rel, shared_of
    n_tok, experts = FP8_FULLSIZE[name]
    cfg = dict(config(name), fp8=2)
    T, E, k, f = cfg["T"], cfg["E"], cfg["k"], cfg["f"]
    tol = TOL[cfg["dtype"]]
    inp = layer_inputs(cfg, seed=0)
    print("full-size", name, "fp8 layer", flush=True)
    layer, p = setup(cfg, inp)
    x = dev(inp["x"], "bf16")
    dy = dev(inp["dy"], "bf16")
    y = layer.forward(p, x)
    grads = layer.alloc_grads()
    dx = layer.backward(p, x, dy, grads)
    torch.cuda.synchronize()
    print("oracle routing of every token", flush=True)
    spec = spec_from_config(cfg)
    x64, dy64 = to_f64(inp["x"], "bf16"), to_f64(inp["dy"], "bf16")
    w_r = inp["w_r"].astype(np.float64)
    beta = None if inp["router_bias"] is None else inp["router_bias"].astype(np.float64)
    rt = route(spec, router_logits(x64, w_r), beta)
    sv = {n: host(layer.saved[n]) for n in ("topk_idx", "expert_offsets", "row_of", "token_of")}
    amb, all_equal = check_routing(cfg, {"route": rt}, sv["topk_idx"])
    mp = sort_maps(rt["topk_idx"], E)
    if all_equal:
        for a, b in (("expert_offsets", "offsets"), ("row_of", "row_of"), ("token_of", "token_of")):
            assert np.array_equal(sv[a], mp[b]), a
    else:
        check_maps_valid(sv["topk_idx"], sv["expert_offsets"], sv["row_of"], sv["token_of"], E)
    differ = np.nonzero(np.any(sv["topk_idx"] != rt["topk_idx"], axis=1))[0]
    rng = np.random.default_rng(7)
    sample = np.sort(rng.choice(np.setdiff1d(np.arange(T), differ), n_tok, replace=False))
    efn = expert_fn(inp, cfg)
    print("oracle per-token FP8 results of", sample.size, "tokens", flush=True)
    r = token_forward_backward(spec, x64[sample], dy64[sample], w_r, beta, efn, shared_of(inp, cfg), fp8=2)
    st = torch.from_numpy(sample).cuda()
    errs = {"y[sample]": rel(host(y[st]), r["y"]), "dx[sample]": rel(host(dx[st]), r["dx"]),
            "y[sample, worst row]": row_rel(host(y[st]), r["y"]),
            "dx[sample, worst row]": row_rel(host(dx[st]), r["dx"])}
    touched = set(np.unique(np.concatenate([sv["topk_idx"][differ].ravel(),
                                            rt["topk_idx"][differ].ravel()])).tolist()) if differ.size else set()
    counts = mp["counts"]
    usable = [e for e in range(E) if counts[e] > 0 and e not in touched]
    e_min = min(usable, key=lambda e: (counts[e], e))
    e_max = max(usable, key=lambda e: (counts[e], -e))
    e_rand = int(rng.choice([e for e in usable if e not in (e_min, e_max)]))
    cols = np.unique(np.concatenate([[0, f - 1, f // 2], rng.choice(f, 13, replace=False)]))
    ct = torch.from_numpy(cols).cuda()
    picked = {"e_min": e_min, "e_max": e_max, "e_rand": e_rand}
    for tag, e in ((t, picked[t]) for t in experts):
        rows = mp["token_of"][mp["offsets"][e]:mp["offsets"][e + 1]]
        tt, ss = rows // k, rows % k
        print("oracle FP8 weight gradients of expert", e, "rows", tt.size, flush=True)
        wg, wu, wd, _, _, _ = efn(e)
        do = rt["topk_w"][tt, ss][:, None] * dy64[tt]
        g = expert_weight_grads_at(x64[tt], do, wg, wu, wd, cols=cols, fp8=2)
        errs["dw_gate[%s]" % tag] = rel(host(grads["dw_gate"][e][:, ct]), g["dw_gate"])
        errs["dw_up[%s]" % tag] = rel(host(grads["dw_up"][e][:, ct]), g["dw_up"])
        errs["dw_down[%s]" % tag] = rel(host(grads["dw_down"][e][ct, :]), g["dw_down"])
    print(name, "fp8 full size: ambiguous tokens", int(amb.sum()), "routed differently", differ.size,
          {n: "%.2e" % v for n, v in errs.items()}, flush=True)
    bad = {n: v for n, v in errs.items() if not v <= tol}
    assert not bad, bad



def test_fp8_zero_rows_and_zero_gradients():
    """Tokens whose x row is zero and whose dy row is zero: their rows quantise
    with scale 1 to zero codes (no division by zero), the layer stays finite
    and within the bar of the oracle at both levels."""
    import torch
    for level in (1, 2):
        cfg = variant("qwen3", T=64, E=8, k=2, d=256, f=128, fp8=level)
        inp = layer_inputs(cfg, seed=3)
        inp["x"][[0, 5, 17]] = 0
        inp["dy"][[0, 9, 33]] = 0
        print("fp8 zero rows, level", level, flush=True)
        layer, p = setup(cfg, inp)
        x = dev(inp["x"], cfg["dtype"])
        y = layer.forward(p, x)
        grads = layer.alloc_grads()
        dx = layer.backward(p, x, dev(inp["dy"], cfg["dtype"]), grads)
        torch.cuda.synchronize()
        fwd, bwd = oracle_run(cfg, inp)
        check_routing(cfg, fwd, host(layer.saved["topk_idx"]))
        hy, hdx = host(y), host(dx)
        assert np.isfinite(hy).all() and np.isfinite(hdx).all()
        for n in ("dw_gate", "dw_down"):
            assert np.isfinite(host(grads[n])).all(), n
        errs = {"y": rel(hy, fwd["y"]), "dx": rel(hdx, bwd["dx"]),
                "dw_gate": rel(host(grads["dw_gate"]), np.stack([bwd["experts"][e]["dw_gate"] for e in range(8)]))}
        print("level", level, {k: "%.2e" % v for k, v in errs.items()}, flush=True)
        assert all(v <= TOL[cfg["dtype"]] for v in errs.values()), errs
