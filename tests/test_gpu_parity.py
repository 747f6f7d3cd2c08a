"""GPU parity of every libmoe entry point against the fp64 oracle, on the five
workload shapes at sizes the oracle finishes in seconds (several tiles and
ragged expert tails), plus edge cases and run-to-run determinism.

Bar: routing indices and maps bit-exact except on tokens whose top-k margin
(oracle, fp64, selection-key space) is below 1e-6; floating-point outputs
within a normwise relative error of 2e-2 (bf16) or 1e-4 (fp32), both over the
whole tensor and for every row (token rows of y and dx, permuted rows of gu,
h, o, d_o, dgu and dx_perm; rows far below the typical norm are measured
against 5% of it) and every expert's weight gradients on their own."""
import numpy as np
import pytest

from moe_inputs import config, layer_inputs, to_f64, variant
from oracle import (combine, combine_backward, expert_backward, expert_forward, route,
                    router_backward, router_logits, sort_maps, spec_from_config, unpermute)
from tests.helpers import (TOL, check_maps_valid, check_routing, dev, device_params, group_rel, host,
                           oracle_run, rel, row_rel)

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": config("tiny"),
    "tiny_ragged": variant("tiny", T=37),
    "qwen3": variant("qwen3", T=640),
    "gptoss": variant("gptoss", T=384),
    "dsv3": variant("dsv3", T=384, d=512, f=256, f_shared=256),
    "stress": variant("stress", T=2048),
    # >= 384 rows per expert: the 256 x 256 tiles of the row-tiled GEMMs
    "qwen3_e16": variant("qwen3", T=1024, E=16),
    "gptoss_big": variant("gptoss", T=3072),
    # bf16 with E a multiple of 32: the layer's selection builds the maps
    # (block counts, last-arrival scan); T ends mid selection block and mid
    # 256-token block
    "dsv3_odd": variant("dsv3", T=1001, d=512, f=256, f_shared=256),
    # the selection builds the maps while the last arrival's pass stays within
    # 512 blocks of 256 tokens: exactly 512 here; one block more and the layer
    # falls back to the permutation's own histogram, scan and rank
    "long_maps": variant("tiny", T=131072, E=32, k=2, d=64, f=64, dtype="bf16"),
    "long": variant("tiny", T=133120, E=32, k=2, d=64, f=64, dtype="bf16"),
    # the selection's maps at the extremes of k: 16 slots per token (every
    # lane of a token's 16-lane row holds one) and a single slot
    "k16": variant("tiny", T=777, E=32, k=16, d=64, f=64, dtype="bf16"),
    "k1": variant("tiny", T=999, E=64, k=1, d=128, f=64, dtype="bf16"),
}

_CACHE = {}


def case(name):
    if name not in _CACHE:
        cfg = CASES[name]
        inp = layer_inputs(cfg, seed=0)
        fwd, bwd = oracle_run(cfg, inp)
        _CACHE[name] = (cfg, inp, fwd, bwd)
    return _CACHE[name]


def run_layer(cfg, inp):
    import torch
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer
    print("layer", cfg["name"], flush=True)
    shape = L.shape_from_config(cfg)
    layer = MoELayer(shape)
    p = device_params(inp, cfg)
    x = dev(inp["x"], cfg["dtype"])
    dy = dev(inp["dy"], cfg["dtype"])
    y = layer.forward(p, x)
    grads = layer.alloc_grads()
    dx = layer.backward(p, x, dy, grads)
    torch.cuda.synchronize()
    return layer, y, dx, grads


def per_expert(bwd, name, E):
    return np.stack([bwd["experts"][e][name] for e in range(E)])


@pytest.mark.parametrize("name", list(CASES))
def test_layer_fwd_bwd(name):
    cfg, inp, fwd, bwd = case(name)
    tol = TOL[cfg["dtype"]]
    layer, y, dx, grads = run_layer(cfg, inp)
    sv = {k: host(v) for k, v in layer.saved.items() if v is not None}
    amb, all_equal = check_routing(cfg, fwd, sv["topk_idx"])
    mp = fwd["maps"]
    if all_equal:
        assert np.array_equal(sv["expert_offsets"], mp["offsets"])
        assert np.array_equal(sv["row_of"], mp["row_of"])
        assert np.array_equal(sv["token_of"], mp["token_of"])
    else:
        check_maps_valid(sv["topk_idx"], sv["expert_offsets"], sv["row_of"], sv["token_of"], cfg["E"])
    # the permuted rows are exact copies
    x64 = to_f64(inp["x"], cfg["dtype"])
    assert np.array_equal(sv["x_perm"], x64[sv["token_of"] // cfg["k"]])
    keep = ~amb
    errs = {
        "topk_w": rel(sv["topk_w"][keep], fwd["route"]["topk_w"][keep]),
        "y": rel(host(y), fwd["y"]),
        "dx": rel(host(dx), bwd["dx"]),
        "dw_r": rel(host(grads["dw_r"]), bwd["dw_r"]),
        "dw_gate": rel(host(grads["dw_gate"]), per_expert(bwd, "dw_gate", cfg["E"])),
        "dw_up": rel(host(grads["dw_up"]), per_expert(bwd, "dw_up", cfg["E"])),
        "dw_down": rel(host(grads["dw_down"]), per_expert(bwd, "dw_down", cfg["E"])),
    }
    if cfg["expert_bias"]:
        for n in ("db_gate", "db_up", "db_down"):
            errs[n] = rel(host(grads[n]), per_expert(bwd, n, cfg["E"]))
    if cfg["n_shared"]:
        for n, m in (("dws_gate", "dw_gate"), ("dws_up", "dw_up"), ("dws_down", "dw_down")):
            errs[n] = rel(host(grads[n]), bwd["shared"][m])
    if cfg["router"] == "sigmoid_grouped":
        errs["s_sel"] = rel(sv["s_sel"][keep], fwd["route"]["s_sel"][keep])
    # every row and every expert on its own (tokens routed as the oracle routes them)
    same = np.all(sv["topk_idx"] == fwd["route"]["topk_idx"], axis=1)
    errs["y[worst row]"] = row_rel(host(y), fwd["y"], same)
    errs["dx[worst row]"] = row_rel(host(dx), bwd["dx"], same)
    if all_equal:
        errs["o[worst row]"] = row_rel(sv["o"], fwd["o"])
    for n in ("dw_gate", "dw_up", "dw_down"):
        errs[n + "[worst expert]"] = group_rel(host(grads[n]), per_expert(bwd, n, cfg["E"]))
    print(name, "ambiguous tokens:", int(amb.sum()), {k: "%.2e" % v for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad
    # routing-trace rules: ids in range, weights non-negative summing to route_scale
    assert sv["topk_idx"].min() >= 0 and sv["topk_idx"].max() < cfg["E"]
    assert np.all(sv["topk_w"] >= 0)
    np.testing.assert_allclose(sv["topk_w"].sum(1), cfg["route_scale"], rtol=1e-5)


@pytest.mark.parametrize("name", ["tiny", "qwen3", "gptoss", "dsv3"])
def test_entry_points(name):
    """Each component entry point on oracle-provided inputs vs the oracle."""
    import torch
    from paper_2605_31463_amd import _lib as L
    cfg, inp, fwd, bwd = case(name)
    print("entry points", name, flush=True)
    dt = cfg["dtype"]
    tol = TOL[dt]
    T, d, E, k, f = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["f"]
    R = T * k
    shape = L.shape_from_config(cfg)
    fws, _, bws = L.moe_workspace_size(shape)
    ws_f = torch.empty(max(fws, 1), dtype=torch.uint8, device="cuda")
    ws_b = torch.empty(max(bws, 1), dtype=torch.uint8, device="cuda")
    act = torch.bfloat16 if dt == "bf16" else torch.float32
    i32, f32 = torch.int32, torch.float32
    p = device_params(inp, cfg)
    x = dev(inp["x"], dt)

    def store(a):  # oracle float64 value -> storage dtype on the device
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).float()
        return t.to(act).cuda()

    def ex(a):  # value the device stores for an oracle float64 array
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).float().to(act)
        return host(t)

    def ok(gpu, ref, what):  # whole tensor and every row
        e, er = rel(gpu, ref), row_rel(gpu, ref)
        assert e <= tol and er <= tol, (what, e, er)

    # route
    idx = torch.empty(T, k, dtype=i32, device="cuda")
    w = torch.empty(T, k, dtype=f32, device="cuda")
    ssel = torch.empty(T, k, dtype=f32, device="cuda")
    cnt = torch.empty(E, dtype=i32, device="cuda")
    L.moe_route(shape, x, p["w_r"], p["router_bias"], idx, w, ssel, cnt, ws_f)
    torch.cuda.synchronize()
    amb, all_eq = check_routing(cfg, fwd, host(idx))
    if all_eq:
        assert np.array_equal(host(cnt), fwd["maps"]["counts"])
    assert rel(host(w)[~amb], fwd["route"]["topk_w"][~amb]) <= tol
    # permute on the oracle's selection: maps bit-exact
    mp = fwd["maps"]
    idx_o = torch.from_numpy(fwd["route"]["topk_idx"].astype(np.int32)).cuda()
    offs = torch.empty(E + 1, dtype=i32, device="cuda")
    row_of = torch.empty(T, k, dtype=i32, device="cuda")
    token_of = torch.empty(R, dtype=i32, device="cuda")
    x_perm = torch.empty(R, d, dtype=act, device="cuda")
    L.moe_permute(shape, x, idx_o, offs, row_of, token_of, x_perm, ws_f)
    torch.cuda.synchronize()
    assert np.array_equal(host(offs), mp["offsets"])
    assert np.array_equal(host(row_of), mp["row_of"])
    assert np.array_equal(host(token_of), mp["token_of"])
    assert np.array_equal(host(x_perm), fwd["x_perm"])
    # grouped gemm forward on the exact permuted rows
    gu = torch.empty(R, 2 * f, dtype=act, device="cuda")
    h = torch.empty(R, f, dtype=act, device="cuda")
    o = torch.empty(R, d, dtype=act, device="cuda")
    L.moe_grouped_gemm_fwd(shape, x_perm, offs, p["w_gate"], p["w_up"], p["w_down"], p["b_gate"],
                           p["b_up"], p["b_down"], gu, h, o)
    torch.cuda.synchronize()
    g_ref = np.zeros((R, f))
    u_ref = np.zeros((R, f))
    h_ref = np.zeros((R, f))
    for e in range(E):
        r0, r1 = mp["offsets"][e], mp["offsets"][e + 1]
        if r1 > r0:
            g_ref[r0:r1], u_ref[r0:r1], h_ref[r0:r1] = fwd["g"][e], fwd["u"][e], fwd["h"][e]
    guh = host(gu)
    ok(guh[:, :f], g_ref, "g")
    ok(guh[:, f:], u_ref, "u")
    ok(host(h), h_ref, "h")
    # the down GEMM sees the device h, so compare it with the oracle down GEMM of that h
    hd = host(h)
    o_ref = np.zeros((R, d))
    from tests.helpers import expert_fn
    efn = expert_fn(inp, cfg)
    for e in range(E):
        r0, r1 = mp["offsets"][e], mp["offsets"][e + 1]
        if r1 > r0:
            wd = efn(e)[2]
            bd = efn(e)[5]
            o_ref[r0:r1] = hd[r0:r1] @ wd + (0 if bd is None else bd)
    ok(host(o), o_ref, "o")
    # combine forward / backward on the oracle's o (rounded to storage)
    o_st = store(fwd["o"])
    o_ex = ex(fwd["o"])
    wt = torch.from_numpy(fwd["route"]["topk_w"].astype(np.float32)).cuda()
    w32 = fwd["route"]["topk_w"].astype(np.float32).astype(np.float64)
    rowt = torch.from_numpy(mp["row_of"].astype(np.int32)).cuda()
    y = torch.empty(T, d, dtype=act, device="cuda")
    sh_o = store(fwd["shared"]["o"]) if cfg["n_shared"] else None
    L.moe_combine_fwd(shape, o_st, wt, rowt, sh_o, y)
    torch.cuda.synchronize()
    y_ref = combine(o_ex, w32, mp["row_of"], None if sh_o is None else host(sh_o))
    ok(host(y), y_ref, "y")
    dy = dev(inp["dy"], dt)
    dy64 = to_f64(inp["dy"], dt)
    d_o = torch.empty(R, d, dtype=act, device="cuda")
    om = torch.empty(T, k, dtype=f32, device="cuda")
    L.moe_combine_bwd(shape, dy, o_st, wt, rowt, d_o, om)
    torch.cuda.synchronize()
    do_ref, om_ref = combine_backward(dy64, o_ex, w32, mp["row_of"])
    ok(host(d_o), do_ref, "d_o")
    ok(host(om), om_ref, "omega")
    # grouped gemm backward (both passes) on oracle-derived inputs
    gu_st = store(np.concatenate([g_ref, u_ref], axis=1))
    h_st = store(h_ref)
    do_st = store(bwd["do"])
    dgu = torch.empty(R, 2 * f, dtype=act, device="cuda")
    dxp = torch.empty(R, d, dtype=act, device="cuda")
    dwg = torch.empty(E, d, f, dtype=act, device="cuda")
    dwu = torch.empty(E, d, f, dtype=act, device="cuda")
    dwd = torch.empty(E, f, d, dtype=act, device="cuda")
    bias = cfg["expert_bias"]
    dbg = torch.empty(E, f, dtype=act, device="cuda") if bias else None
    dbu = torch.empty(E, f, dtype=act, device="cuda") if bias else None
    dbd = torch.empty(E, d, dtype=act, device="cuda") if bias else None
    L.moe_grouped_gemm_bwd(shape, L.MOE_DGRAD | L.MOE_WGRAD, x_perm, offs, gu_st, h_st, do_st,
                           p["w_gate"], p["w_up"], p["w_down"], dgu, dxp, dwg, dwu, dwd, dbg, dbu, dbd)
    torch.cuda.synchronize()
    gex, uex, hex_, doex = host(gu_st)[:, :f], host(gu_st)[:, f:], host(h_st), host(do_st)
    dg_ref = np.zeros((R, f))
    du_ref = np.zeros((R, f))
    dxp_ref = np.zeros((R, d))
    for e in range(E):
        r0, r1 = mp["offsets"][e], mp["offsets"][e + 1]
        wg, wu, wd = efn(e)[:3]
        gb = expert_backward(fwd["x_perm"][r0:r1], gex[r0:r1], uex[r0:r1], hex_[r0:r1], doex[r0:r1],
                             wg, wu, wd, with_bias=bias)
        dg_ref[r0:r1], du_ref[r0:r1], dxp_ref[r0:r1] = gb["dg"], gb["du"], gb["dx"]
        for n, t in (("dw_gate", dwg), ("dw_up", dwu), ("dw_down", dwd)):
            if r1 > r0:
                assert rel(host(t[e]), gb[n]) <= tol, (e, n)
            else:
                assert np.all(host(t[e]) == 0), (e, n)
        if bias:
            for n, t in (("db_gate", dbg), ("db_up", dbu), ("db_down", dbd)):
                assert rel(host(t[e]), gb[n]) <= tol, (e, n)
    dguh = host(dgu)
    ok(dguh[:, :f], dg_ref, "dg")
    ok(dguh[:, f:], du_ref, "du")
    # dx_perm is computed from the device dgu: compare with the oracle product of that dgu
    dxp_dev = np.zeros((R, d))
    for e in range(E):
        r0, r1 = mp["offsets"][e], mp["offsets"][e + 1]
        wg, wu = efn(e)[:2]
        dxp_dev[r0:r1] = dguh[r0:r1, :f] @ wg.T + dguh[r0:r1, f:] @ wu.T
    ok(host(dxp), dxp_dev, "dx_perm")
    ok(dxp_dev, dxp_ref, "dx_perm (oracle product of the device dgu)")
    # router backward on the oracle's omega
    spec = spec_from_config(cfg)
    omt = torch.from_numpy(bwd["omega"].astype(np.float32)).cuda()
    ss = None
    if cfg["router"] == "sigmoid_grouped":
        ss = torch.from_numpy(fwd["route"]["s_sel"].astype(np.float32)).cuda()
    dwr = torch.empty(d, E, dtype=f32, device="cuda")
    dxr = torch.empty(T, d, dtype=f32, device="cuda")
    L.moe_route_bwd(shape, x, p["w_r"], idx_o, wt, ss, omt, offs, token_of, dwr, dxr, ws_b)
    torch.cuda.synchronize()
    assert rel(host(dwr), bwd["dw_r"]) <= tol
    assert rel(host(dwr).T, bwd["dw_r"].T) <= tol and row_rel(host(dwr).T, bwd["dw_r"].T) <= tol  # every expert column
    ok(host(dxr), bwd["dx_router"], "dx_router")
    # unpermute on the oracle's dx_perm and router dx
    dxp_st = store(bwd["dx_perm"])
    dxr_t = torch.from_numpy(bwd["dx_router"].astype(np.float32)).cuda()
    dxo = torch.empty(T, d, dtype=act, device="cuda")
    L.moe_unpermute_bwd(shape, dxp_st, rowt, dxr_t, None, dxo)
    torch.cuda.synchronize()
    ref = unpermute(host(dxp_st), mp["row_of"]) + bwd["dx_router"].astype(np.float32)
    ok(host(dxo), ref, "dx (unpermute)")
    # shared expert
    if cfg["n_shared"]:
        fs = cfg["f_shared"]
        gsh = torch.empty(T, 2 * fs, dtype=act, device="cuda")
        hsh = torch.empty(T, fs, dtype=act, device="cuda")
        osh = torch.empty(T, d, dtype=act, device="cuda")
        L.moe_shared_expert_fwd(shape, x, p["ws_gate"], p["ws_up"], p["ws_down"], gsh, hsh, osh)
        torch.cuda.synchronize()
        shf = fwd["shared"]
        assert rel(host(gsh)[:, :fs], shf["g"]) <= tol
        assert rel(host(gsh)[:, fs:], shf["u"]) <= tol
        assert rel(host(hsh), shf["h"]) <= tol
        assert rel(host(osh), shf["o"]) <= tol
        dxs = torch.empty(T, d, dtype=act, device="cuda")
        dsg = torch.empty(d, fs, dtype=act, device="cuda")
        dsu = torch.empty(d, fs, dtype=act, device="cuda")
        dsd = torch.empty(fs, d, dtype=act, device="cuda")
        L.moe_shared_expert_bwd(shape, x, dy, gsh, hsh, p["ws_gate"], p["ws_up"], p["ws_down"], dxs, dsg,
                                dsu, dsd, ws_b)
        torch.cuda.synchronize()
        shared_w = tuple(to_f64(inp[n], dt) for n in ("ws_gate", "ws_up", "ws_down"))
        gb = expert_backward(to_f64(inp["x"], dt), host(gsh)[:, :fs], host(gsh)[:, fs:], host(hsh), dy64,
                             *shared_w)
        assert rel(host(dsg), gb["dw_gate"]) <= tol
        assert rel(host(dsu), gb["dw_up"]) <= tol
        assert rel(host(dsd), gb["dw_down"]) <= tol
        assert rel(host(dxs), gb["dx"]) <= tol


def test_dgrad_then_wgrad_equals_both():
    """The delayed weight-gradient pass gives the same bits as the combined call."""
    import torch
    from paper_2605_31463_amd import _lib as L
    cfg, inp, fwd, bwd = case("qwen3")
    print("dgrad/wgrad split", flush=True)
    layer, _, _, _ = run_layer(cfg, inp)
    shape = L.shape_from_config(cfg)
    p = device_params(inp, cfg)
    sv = layer.saved
    T, d, E, k, f = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["f"]
    R = T * k
    act = torch.bfloat16
    d_o = torch.randn(R, d, device="cuda").to(act)
    outs = []
    for passes in ((L.MOE_DGRAD | L.MOE_WGRAD,), (L.MOE_DGRAD, L.MOE_WGRAD)):
        dgu = torch.empty(R, 2 * f, dtype=act, device="cuda")
        dxp = torch.empty(R, d, dtype=act, device="cuda")
        dw = [torch.empty(E, d, f, dtype=act, device="cuda") for _ in range(2)] + \
             [torch.empty(E, f, d, dtype=act, device="cuda")]
        for ps in passes:
            L.moe_grouped_gemm_bwd(shape, ps, sv["x_perm"], sv["expert_offsets"], sv["gu"], sv["h"], d_o,
                                   p["w_gate"], p["w_up"], p["w_down"], dgu, dxp, dw[0], dw[1], dw[2],
                                   None, None, None)
        torch.cuda.synchronize()
        outs.append([dgu, dxp] + dw)
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("name", ["tiny", "dsv3"])
def test_determinism(name):
    import torch
    cfg, inp, _, _ = case(name)
    print("determinism", name, flush=True)
    r1 = run_layer(cfg, inp)
    a = [r1[1].clone(), r1[2].clone()] + [v.clone() for v in r1[3].values()]
    r2 = run_layer(cfg, inp)
    b = [r2[1], r2[2]] + list(r2[3].values())
    for u, v in zip(a, b):
        assert torch.equal(u, v)


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

def _run_custom(cfg, inp):
    fwd, bwd = oracle_run(cfg, inp)
    layer, y, dx, grads = run_layer(cfg, inp)
    return fwd, bwd, layer, y, dx, grads


def test_empty_tokens():
    import torch
    cfg = variant("qwen3", T=0, d=128, f=128, E=16, k=4)
    inp = layer_inputs(cfg, seed=1)
    print("empty tokens", flush=True)
    layer, y, dx, grads = run_layer(cfg, inp)
    assert host(layer.saved["expert_offsets"]).tolist() == [0] * 17
    for n in ("dw_r", "dw_gate", "dw_up", "dw_down"):
        assert torch.count_nonzero(grads[n]).item() == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_expert(dtype):
    cfg = variant("tiny", E=1, k=1, T=50, dtype=dtype)
    inp = layer_inputs(cfg, seed=2)
    print("single expert", dtype, flush=True)
    fwd, bwd, layer, y, dx, grads = _run_custom(cfg, inp)
    assert np.all(host(layer.saved["topk_idx"]) == 0)
    assert np.all(host(layer.saved["topk_w"]) == 1.0)
    assert np.all(host(grads["dw_r"]) == 0.0)
    tol = TOL[dtype]
    assert rel(host(y), fwd["y"]) <= tol
    assert rel(host(dx), bwd["dx"]) <= tol


def test_k_equals_E_full_softmax():
    cfg = variant("tiny", E=8, k=8, T=40)
    inp = layer_inputs(cfg, seed=3)
    print("k == E", flush=True)
    fwd, bwd, layer, y, dx, grads = _run_custom(cfg, inp)
    amb, _ = check_routing(cfg, fwd, host(layer.saved["topk_idx"]))
    assert rel(host(y), fwd["y"]) <= 1e-4
    assert rel(host(grads["dw_r"]), bwd["dw_r"]) <= 1e-4
    assert rel(host(dx), bwd["dx"]) <= 1e-4


def test_zero_router_ties_to_lower_index():
    cfg = variant("tiny", T=33)
    inp = layer_inputs(cfg, seed=4)
    inp["w_r"] = np.zeros_like(inp["w_r"])
    print("zero router", flush=True)
    fwd, bwd, layer, y, dx, grads = _run_custom(cfg, inp)
    assert host(layer.saved["topk_idx"]).tolist() == [[0, 1]] * 33
    assert np.all(host(layer.saved["topk_w"]) == 0.5)
    assert host(layer.saved["expert_offsets"]).tolist() == [0, 33, 66] + [66] * 6
    assert rel(host(y), fwd["y"]) <= 1e-4
    assert rel(host(dx), bwd["dx"]) <= 1e-4


def test_bad_arguments_enqueue_nothing():
    import torch
    from paper_2605_31463_amd import _lib as L
    shape = L.make_shape(T=16, d=128, E=8, k=2, f=128)
    x = torch.zeros(16, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(L.MoeError) as ei:
        L.moe_route(shape, x, None, None, None, None, None, None)
    assert ei.value.status == L.MOE_ERR_INVALID_ARG
    with pytest.raises(L.MoeError) as ei:
        L.moe_permute(shape, x, torch.zeros(16, 2, dtype=torch.int32, device="cuda"),
                      torch.zeros(9, dtype=torch.int32, device="cuda"),
                      torch.zeros(16, 2, dtype=torch.int32, device="cuda"),
                      torch.zeros(32, dtype=torch.int32, device="cuda"),
                      torch.zeros(32, 128, dtype=torch.bfloat16, device="cuda"), None)
    assert ei.value.status == L.MOE_ERR_WORKSPACE
