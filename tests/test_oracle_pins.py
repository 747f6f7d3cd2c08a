"""Pins of the fp64 oracle against facts that do not come from the oracle itself:
hand-worked examples, a dense every-expert brute force, torch autograd on an
independently written dense masked formulation, central finite differences,
closed-form special cases, brute-force enumeration of the group-limited
router, a library sort for the permutation maps, and the routing-trace
invariants (ids in range, weights non-negative and summing to one over the
top-k; appendix B.2.2, "Collect Routing Trace")."""
import itertools
import json
import os

import numpy as np
import pytest
import torch

from oracle import (RouterSpec, aux_loss, aux_loss_backward, expert_backward, expert_forward,
                    expert_weight_grads_at, layer_backward, layer_forward, route, router_logits,
                    router_probs, sort_maps, token_forward_backward)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SPECS = {
    "softmax_topk": RouterSpec("softmax_topk", E=8, k=2),
    "topk_softmax": RouterSpec("topk_softmax", E=8, k=3),
    "softmax_logit_bias": RouterSpec("softmax_topk", E=8, k=2, bias_mode="logit"),
    "sigmoid_grouped": RouterSpec("sigmoid_grouped", E=16, k=4, n_groups=4, topk_groups=2,
                                  route_scale=2.5, bias_mode="select"),
}


def make_case(spec, T=24, d=16, f=12, seed=0, expert_bias=False, shared=False, wr_std=0.3):
    rng = np.random.default_rng(seed)
    E = spec.E
    c = dict(
        x=rng.standard_normal((T, d)),
        w_r=rng.standard_normal((d, E)) * wr_std,
        beta=(rng.standard_normal(E) * 0.1 if spec.bias_mode != "none" else None),
        wg=rng.standard_normal((E, d, f)) * 0.3,
        wu=rng.standard_normal((E, d, f)) * 0.3,
        wd=rng.standard_normal((E, f, d)) * 0.3,
        bg=rng.standard_normal((E, f)) * 0.1 if expert_bias else None,
        bu=rng.standard_normal((E, f)) * 0.1 if expert_bias else None,
        bd=rng.standard_normal((E, d)) * 0.1 if expert_bias else None,
        dy=rng.standard_normal((T, d)),
        shared=((rng.standard_normal((d, f)) * 0.3, rng.standard_normal((d, f)) * 0.3,
                 rng.standard_normal((f, d)) * 0.3) if shared else None),
    )
    return c


def efn(c):
    def fn(e):
        return (c["wg"][e], c["wu"][e], c["wd"][e],
                None if c["bg"] is None else c["bg"][e],
                None if c["bu"] is None else c["bu"][e],
                None if c["bd"] is None else c["bd"][e])
    return fn


def run(spec, c):
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c), c["shared"])
    bwd = layer_backward(spec, c["x"], c["w_r"], c["beta"], efn(c), fwd, c["dy"], c["shared"],
                         with_bias=c["bg"] is not None)
    return fwd, bwd


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


# ---------------------------------------------------------------------------
# Hand-worked examples
# ---------------------------------------------------------------------------

def test_worked_example_softmax():
    g = json.load(open(os.path.join(GOLDEN, "route_worked_examples.json")))["softmax"]
    spec = RouterSpec("topk_softmax", E=g["E"], k=g["k"])
    l = np.log(np.asarray(g["logits_ln"], np.float64))
    rt = route(spec, l)
    assert rt["topk_idx"].tolist() == g["topk_idx"]
    want = np.array([[n / m for n, m in row] for row in g["topk_w_frac"]])
    np.testing.assert_allclose(rt["topk_w"], want, rtol=0, atol=1e-15)
    mp = sort_maps(rt["topk_idx"], g["E"])
    assert mp["counts"].tolist() == g["counts"]
    assert mp["offsets"].tolist() == g["offsets"]
    assert mp["row_of"].tolist() == g["row_of"]
    assert mp["token_of"].tolist() == g["token_of"]
    # the softmax-then-renormalise family is the same function
    rt2 = route(RouterSpec("softmax_topk", E=g["E"], k=g["k"]), l)
    assert rt2["topk_idx"].tolist() == g["topk_idx"]
    np.testing.assert_allclose(rt2["topk_w"], want, rtol=0, atol=1e-15)


def test_worked_example_sigmoid_grouped():
    g = json.load(open(os.path.join(GOLDEN, "route_worked_examples.json")))["sigmoid_grouped"]
    spec = RouterSpec("sigmoid_grouped", E=g["E"], k=g["k"], n_groups=g["n_groups"],
                      topk_groups=g["topk_groups"], route_scale=g["route_scale"], bias_mode="select")
    l = np.zeros((1, g["E"]))
    rt = route(spec, l, np.asarray(g["beta"]))
    assert rt["topk_idx"].tolist() == g["topk_idx"]
    want = np.array([[n / m for n, m in row] for row in g["topk_w_frac"]])
    np.testing.assert_allclose(rt["topk_w"], want, rtol=0, atol=1e-15)


# ---------------------------------------------------------------------------
# Dense every-expert brute force of the forward
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(SPECS))
def test_forward_matches_dense_bruteforce(name):
    spec = SPECS[name]
    c = make_case(spec, expert_bias=True, shared=(name == "sigmoid_grouped"))
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c), c["shared"])
    T = c["x"].shape[0]
    gate = np.zeros((T, spec.E))
    for t in range(T):
        for s in range(spec.k):
            gate[t, fwd["route"]["topk_idx"][t, s]] = fwd["route"]["topk_w"][t, s]
    y = np.zeros_like(c["x"])
    for e in range(spec.E):
        g = c["x"] @ c["wg"][e] + c["bg"][e]
        u = c["x"] @ c["wu"][e] + c["bu"][e]
        o = (g / (1 + np.exp(-g)) * u) @ c["wd"][e] + c["bd"][e]
        y += gate[:, e:e + 1] * o
    if c["shared"] is not None:
        a, b, w = c["shared"]
        g, u = c["x"] @ a, c["x"] @ b
        y += (g / (1 + np.exp(-g)) * u) @ w
    assert rel(fwd["y"], y) < 1e-12


# ---------------------------------------------------------------------------
# torch autograd on a dense masked formulation (independent of the oracle)
# ---------------------------------------------------------------------------

def torch_dense_loss(spec, c, params):
    x, w_r, wg, wu, wd = (params[n] for n in ("x", "w_r", "wg", "wu", "wd"))
    l = x @ w_r
    T, E = l.shape
    beta = None if c["beta"] is None else torch.tensor(c["beta"], dtype=torch.float64)
    if spec.router in ("softmax_topk", "topk_softmax"):
        key = l + beta if spec.bias_mode in ("logit", "select") else l
        wl = l + beta if spec.bias_mode == "logit" else l
        sel = torch.topk(key.detach(), spec.k, dim=1).indices
        mask = torch.zeros(T, E, dtype=torch.bool).scatter(1, sel, True)
        gate = spec.route_scale * torch.softmax(wl.masked_fill(~mask, float("-inf")), dim=1)
    else:
        s = torch.sigmoid(l)
        key = (s + beta).detach()
        per = E // spec.n_groups
        gs = key.view(T, spec.n_groups, per).topk(2, dim=2).values.sum(-1)
        gsel = gs.topk(spec.topk_groups, dim=1).indices
        gmask = torch.zeros(T, spec.n_groups, dtype=torch.bool).scatter(1, gsel, True)
        emask = gmask.repeat_interleave(per, dim=1)
        sel = key.masked_fill(~emask, float("-inf")).topk(spec.k, dim=1).indices
        mask = torch.zeros(T, E, dtype=torch.bool).scatter(1, sel, True)
        sm = s * mask
        gate = spec.route_scale * sm / sm.sum(1, keepdim=True)
    y = torch.zeros_like(x)
    for e in range(E):
        g = x @ wg[e]
        u = x @ wu[e]
        if "bg" in params:
            g = g + params["bg"][e]
            u = u + params["bu"][e]
        o = (torch.nn.functional.silu(g) * u) @ wd[e]
        if "bd" in params:
            o = o + params["bd"][e]
        y = y + gate[:, e:e + 1] * o
    if "sg" in params:
        g = x @ params["sg"]
        u = x @ params["su"]
        y = y + (torch.nn.functional.silu(g) * u) @ params["sd"]
    dy = torch.tensor(c["dy"], dtype=torch.float64)
    return (dy * y).sum(), sel


@pytest.mark.parametrize("name", list(SPECS))
def test_backward_matches_torch_autograd(name):
    spec = SPECS[name]
    shared = name == "sigmoid_grouped"
    c = make_case(spec, expert_bias=True, shared=shared, seed=1)
    fwd, bwd = run(spec, c)
    params = {n: torch.tensor(c[n], dtype=torch.float64, requires_grad=True)
              for n in ("x", "w_r", "wg", "wu", "wd", "bg", "bu", "bd")}
    if shared:
        for n, a in zip(("sg", "su", "sd"), c["shared"]):
            params[n] = torch.tensor(a, dtype=torch.float64, requires_grad=True)
    loss, sel = torch_dense_loss(spec, c, params)
    loss.backward()
    # same selected sets
    assert [sorted(r) for r in sel.tolist()] == [sorted(r) for r in fwd["route"]["topk_idx"].tolist()]
    assert abs(loss.item() - (c["dy"] * fwd["y"]).sum()) < 1e-10 * abs(loss.item())
    assert rel(bwd["dx"], params["x"].grad.numpy()) < 1e-11
    assert rel(bwd["dw_r"], params["w_r"].grad.numpy()) < 1e-11
    for e in range(spec.E):
        ge = bwd["experts"][e]
        for ours, theirs in (("dw_gate", "wg"), ("dw_up", "wu"), ("dw_down", "wd"),
                             ("db_gate", "bg"), ("db_up", "bu"), ("db_down", "bd")):
            want = params[theirs].grad[e].numpy()
            if np.linalg.norm(want) == 0:
                assert np.linalg.norm(ge[ours]) == 0
            else:
                assert rel(ge[ours], want) < 1e-11, (e, ours)
    if shared:
        for ours, theirs in (("dw_gate", "sg"), ("dw_up", "su"), ("dw_down", "sd")):
            assert rel(bwd["shared"][ours], params[theirs].grad.numpy()) < 1e-11


# ---------------------------------------------------------------------------
# Central finite differences along random directions
# ---------------------------------------------------------------------------

def _loss(spec, c):
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c), c["shared"])
    return float((c["dy"] * fwd["y"]).sum()), fwd["route"]["topk_idx"]


@pytest.mark.parametrize("name", list(SPECS))
def test_gradients_match_finite_differences(name):
    spec = SPECS[name]
    shared = name == "sigmoid_grouped"
    c = make_case(spec, T=12, d=8, f=6, expert_bias=True, shared=shared, seed=2)
    fwd, bwd = run(spec, c)
    rng = np.random.default_rng(5)
    grads = {"x": bwd["dx"], "w_r": bwd["dw_r"]}
    for ours, key in (("dw_gate", "wg"), ("dw_up", "wu"), ("dw_down", "wd"),
                      ("db_gate", "bg"), ("db_up", "bu"), ("db_down", "bd")):
        grads[key] = np.stack([bwd["experts"][e][ours] for e in range(spec.E)])
    h = 1e-6
    for key, gr in grads.items():
        for _ in range(3):
            v = rng.standard_normal(c[key].shape)
            v /= np.linalg.norm(v)
            cp, cm = dict(c), dict(c)
            cp[key] = c[key] + h * v
            cm[key] = c[key] - h * v
            lp, ip = _loss(spec, cp)
            lm, im = _loss(spec, cm)
            if not (np.array_equal(ip, fwd["route"]["topk_idx"])
                    and np.array_equal(im, fwd["route"]["topk_idx"])):
                continue  # the step crossed a selection boundary; draw again
            fd = (lp - lm) / (2 * h)
            an = float((gr * v).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (key, fd, an)
    if shared:
        for i, ours in enumerate(("dw_gate", "dw_up", "dw_down")):
            v = rng.standard_normal(c["shared"][i].shape)
            v /= np.linalg.norm(v)
            sp = list(c["shared"])
            sm = list(c["shared"])
            sp[i] = sp[i] + h * v
            sm[i] = sm[i] - h * v
            lp, _ = _loss(spec, dict(c, shared=tuple(sp)))
            lm, _ = _loss(spec, dict(c, shared=tuple(sm)))
            fd = (lp - lm) / (2 * h)
            an = float((bwd["shared"][ours] * v).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an))


# ---------------------------------------------------------------------------
# Closed-form special cases
# ---------------------------------------------------------------------------

def test_single_expert_is_plain_swiglu_mlp():
    spec = RouterSpec("softmax_topk", E=1, k=1)
    c = make_case(spec, seed=3)
    fwd, bwd = run(spec, c)
    x, wg, wu, wd = c["x"], c["wg"][0], c["wu"][0], c["wd"][0]
    g, u = x @ wg, x @ wu
    h = g / (1 + np.exp(-g)) * u
    assert rel(fwd["y"], h @ wd) < 1e-13
    assert np.all(fwd["route"]["topk_w"] == 1.0)
    assert np.all(bwd["dl"] == 0.0)
    assert np.all(bwd["dw_r"] == 0.0)
    # dx of a plain MLP, written with the chain rule for silu'(g) = sig(g)(1+g(1-sig(g)))
    sg = 1 / (1 + np.exp(-g))
    dh = c["dy"] @ wd.T
    dx = (dh * u * sg * (1 + g * (1 - sg))) @ wg.T + (dh * g * sg) @ wu.T
    assert rel(bwd["dx"], dx) < 1e-13


def test_k_equals_E_gives_full_softmax():
    from scipy.special import softmax
    spec = RouterSpec("softmax_topk", E=8, k=8)
    c = make_case(spec, seed=4)
    l = router_logits(c["x"], c["w_r"])
    rt = route(spec, l)
    full = softmax(l, axis=1)
    got = np.zeros_like(full)
    np.put_along_axis(got, rt["topk_idx"], rt["topk_w"], axis=1)
    assert rel(got, full) < 1e-14
    assert np.all(np.diff(np.take_along_axis(l, rt["topk_idx"], 1), axis=1) <= 0)


def test_zero_router_ties_go_to_lower_index():
    spec = RouterSpec("softmax_topk", E=8, k=3)
    c = make_case(spec, seed=5)
    c["w_r"][:] = 0.0
    fwd, bwd = run(spec, c)
    T = c["x"].shape[0]
    assert fwd["route"]["topk_idx"].tolist() == [[0, 1, 2]] * T
    assert np.all(fwd["route"]["topk_w"] == 1.0 / 3.0)
    assert fwd["maps"]["counts"].tolist() == [T, T, T, 0, 0, 0, 0, 0]
    assert fwd["maps"]["token_of"].tolist() == [t * 3 + s for s in range(3) for t in range(T)]


def test_zero_router_sigmoid_selects_by_bias_alone():
    spec = SPECS["sigmoid_grouped"]
    c = make_case(spec, seed=6)
    c["w_r"][:] = 0.0
    fwd, _ = run(spec, c)
    beta = c["beta"]
    per = spec.E // spec.n_groups
    gscore = [sum(sorted(beta[g * per:(g + 1) * per], reverse=True)[:2]) for g in range(spec.n_groups)]
    keep = sorted(range(spec.n_groups), key=lambda g: (-gscore[g], g))[:spec.topk_groups]
    cand = [e for g in keep for e in range(g * per, (g + 1) * per)]
    want = sorted(cand, key=lambda e: (-beta[e], e))[:spec.k]
    T = c["x"].shape[0]
    assert fwd["route"]["topk_idx"].tolist() == [want] * T
    np.testing.assert_allclose(fwd["route"]["topk_w"], 2.5 / spec.k, rtol=0, atol=1e-15)


# ---------------------------------------------------------------------------
# Brute-force enumeration of the group-limited router
# ---------------------------------------------------------------------------

def test_grouped_router_matches_subset_enumeration():
    spec = SPECS["sigmoid_grouped"]
    c = make_case(spec, T=40, seed=7)
    l = router_logits(c["x"], c["w_r"])
    rt = route(spec, l, c["beta"])
    per = spec.E // spec.n_groups
    for t in range(l.shape[0]):
        s = [1.0 / (1.0 + np.exp(-v)) for v in l[t]]
        key = [s[e] + c["beta"][e] for e in range(spec.E)]
        score = [sum(sorted(key[g * per:(g + 1) * per], reverse=True)[:2]) for g in range(spec.n_groups)]
        best = max(itertools.combinations(range(spec.n_groups), spec.topk_groups),
                   key=lambda sub: sum(score[g] for g in sub))
        cand = [e for g in best for e in range(g * per, (g + 1) * per)]
        want = sorted(cand, key=lambda e: (-key[e], e))[:spec.k]
        assert rt["topk_idx"][t].tolist() == want
        tot = sum(s[e] for e in want)
        np.testing.assert_allclose(rt["topk_w"][t], [2.5 * s[e] / tot for e in want], rtol=1e-14)


# ---------------------------------------------------------------------------
# Permutation maps against a library sort, and the invariants
# ---------------------------------------------------------------------------

def test_maps_match_library_stable_sort():
    rng = np.random.default_rng(8)
    T, E, k = 200, 13, 4
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    mp = sort_maps(idx, E)
    t_of = np.repeat(np.arange(T), k)
    s_of = np.tile(np.arange(k), T)
    order = np.lexsort((t_of, idx.reshape(-1)))     # by expert, then token
    assert mp["token_of"].tolist() == (t_of[order] * k + s_of[order]).tolist()
    assert mp["counts"].tolist() == np.bincount(idx.reshape(-1), minlength=E).tolist()


@pytest.mark.parametrize("name", list(SPECS))
def test_invariants(name):
    spec = SPECS[name]
    c = make_case(spec, T=64, seed=9)
    fwd, bwd = run(spec, c)
    rt, mp = fwd["route"], fwd["maps"]
    T, k, E = c["x"].shape[0], spec.k, spec.E
    idx, w = rt["topk_idx"], rt["topk_w"]
    assert idx.min() >= 0 and idx.max() < E
    assert all(len(set(r)) == k for r in idx.tolist())
    assert np.all(w >= 0)
    np.testing.assert_allclose(w.sum(1), spec.route_scale, rtol=1e-14)
    assert mp["counts"].sum() == T * k == mp["offsets"][E]
    assert np.all(np.diff(mp["offsets"]) == mp["counts"])
    assert sorted(mp["token_of"].tolist()) == list(range(T * k))
    for e in range(E):
        toks = mp["token_of"][mp["offsets"][e]:mp["offsets"][e + 1]] // k
        assert np.all(np.diff(toks) > 0)
    for t in range(T):
        for s in range(k):
            assert mp["token_of"][mp["row_of"][t, s]] == t * k + s
            assert np.array_equal(fwd["x_perm"][mp["row_of"][t, s]], c["x"][t])
    if spec.router != "sigmoid_grouped":
        # softmax routers: every row of dl sums to zero, so do the rows of dW_r
        np.testing.assert_allclose(bwd["dl"].sum(1), 0.0, atol=1e-12)
        assert np.abs(bwd["dw_r"].sum(1)).max() < 1e-11 * np.abs(bwd["dw_r"]).max()


def test_unpermute_of_permute_is_identity():
    spec = RouterSpec("softmax_topk", E=8, k=4)
    c = make_case(spec, T=50, seed=10)
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c))
    back = np.zeros_like(c["x"])
    for s in range(spec.k):
        back += 0.25 * fwd["x_perm"][fwd["maps"]["row_of"][:, s]]
    assert np.array_equal(back, c["x"])


def test_margin_flags_near_ties():
    spec = RouterSpec("softmax_topk", E=4, k=2)
    l = np.array([[0.3, 0.1, 0.1 + 5e-7, -1.0], [0.3, 0.2, 0.1, -1.0]])
    rt = route(spec, l)
    assert rt["margin"][0] < 1e-6 <= rt["margin"][1]


def test_margins_of_the_sigmoid_routers_worked_by_hand():
    """The selection margin of the grouped router (group gap at the kept /
    dropped boundary, key gaps among the k+1 best candidates of the kept
    groups) and of the threshold router (key gaps, distance of a candidate's
    key from the threshold) on hand-worked one-token cases; each case is built
    so that a margin taken at a wrong index or over the wrong set differs."""
    g = json.load(open(os.path.join(GOLDEN, "route_margins.json")))
    gg = g["sigmoid_grouped"]
    spec = RouterSpec("sigmoid_grouped", E=gg["E"], k=gg["k"], n_groups=gg["n_groups"],
                      topk_groups=gg["topk_groups"], route_scale=gg["route_scale"], bias_mode="select")
    for c in gg["cases"]:
        rt = route(spec, np.asarray([c["logits"]], np.float64), np.asarray(c["beta"], np.float64))
        assert rt["topk_idx"][0].tolist() == c["topk_idx"]
        np.testing.assert_allclose(rt["topk_w"][0], [n / m for n, m in c["topk_w_frac"]], rtol=0, atol=1e-15)
        assert rt["margin"][0] == c["margin"], (rt["margin"][0], c["margin"])
    gt = g["sigmoid_threshold"]
    spec = RouterSpec("sigmoid_threshold", E=gt["E"], k=gt["k"])
    for c in gt["cases"]:
        rt = route(spec, np.asarray([c["logits"]], np.float64), theta=np.asarray(c["theta"], np.float64))
        assert rt["topk_idx"][0].tolist() == c["topk_idx"]
        assert rt["margin"][0] == c["margin"], (rt["margin"][0], c["margin"])


def test_expert_backward_matches_finite_differences_on_its_own():
    rng = np.random.default_rng(11)
    x = rng.standard_normal((5, 4))
    wg, wu, wd = (rng.standard_normal(s) for s in ((4, 3), (4, 3), (3, 4)))
    do = rng.standard_normal((5, 4))
    g, u, h, o = expert_forward(x, wg, wu, wd)
    gr = expert_backward(x, g, u, h, do, wg, wu, wd)
    eps = 1e-6
    for name, arr in (("dw_gate", wg), ("dw_up", wu), ("dw_down", wd)):
        for idx in [(0, 0), (1, 2), (2, 1)]:
            ap = arr.copy(); ap[idx] += eps
            am = arr.copy(); am[idx] -= eps
            args_p = {"dw_gate": (ap, wu, wd), "dw_up": (wg, ap, wd), "dw_down": (wg, wu, ap)}[name]
            args_m = {"dw_gate": (am, wu, wd), "dw_up": (wg, am, wd), "dw_down": (wg, wu, am)}[name]
            fp = (do * expert_forward(x, *args_p)[3]).sum()
            fm = (do * expert_forward(x, *args_m)[3]).sum()
            assert abs((fp - fm) / (2 * eps) - gr[name][idx]) < 1e-7


# ---------------------------------------------------------------------------
# Evaluation of a layer too large to run whole: per-token results on a subset
# of the tokens, weight-gradient slices along the intermediate axis
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(SPECS))
def test_token_subset_equals_whole_layer(name):
    spec = SPECS[name]
    c = make_case(spec, T=40, expert_bias=True, shared=(name == "sigmoid_grouped"), seed=7)
    fwd, bwd = run(spec, c)
    sub = np.array([39, 3, 17, 0, 22, 5])
    r = token_forward_backward(spec, c["x"][sub], c["dy"][sub], c["w_r"], c["beta"], efn(c), c["shared"])
    assert np.array_equal(r["route"]["topk_idx"], fwd["route"]["topk_idx"][sub])
    for a, b in ((r["y"], fwd["y"][sub]), (r["dx"], bwd["dx"][sub]), (r["omega"], bwd["omega"][sub]),
                 (r["dl"], bwd["dl"][sub])):
        assert rel(a, b) < 1e-12
    # every token routed to expert e: column e of dW_r
    for e in (0, spec.E - 1, int(fwd["route"]["topk_idx"][11, 0])):
        toks = np.nonzero((fwd["route"]["topk_idx"] == e).any(axis=1))[0]
        r = token_forward_backward(spec, c["x"][toks], c["dy"][toks], c["w_r"], c["beta"], efn(c),
                                   c["shared"])
        col = c["x"][toks].T @ r["dl_dense"][:, e]
        assert rel(col, bwd["dw_r"][:, e]) < 1e-12


@pytest.mark.parametrize("bias", [False, True])
def test_weight_grad_slices_equal_full_expert_backward(bias):
    rng = np.random.default_rng(11)
    M, d, f = 29, 16, 12
    xe, do = rng.standard_normal((M, d)), rng.standard_normal((M, d))
    wg, wu = rng.standard_normal((d, f)) * 0.3, rng.standard_normal((d, f)) * 0.3
    wd = rng.standard_normal((f, d)) * 0.3
    bg = rng.standard_normal(f) * 0.1 if bias else None
    bu = rng.standard_normal(f) * 0.1 if bias else None
    g, u, h, _ = expert_forward(xe, wg, wu, wd, bg, bu)
    full = expert_backward(xe, g, u, h, do, wg, wu, wd, with_bias=bias)
    cols = np.array([11, 0, 5, 6])
    part = expert_weight_grads_at(xe, do, wg, wu, wd, bg, bu, cols=cols, with_bias=bias)
    np.testing.assert_allclose(part["dw_gate"], full["dw_gate"][:, cols], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(part["dw_up"], full["dw_up"][:, cols], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(part["dw_down"], full["dw_down"][cols, :], rtol=1e-13, atol=1e-13)
    if bias:
        np.testing.assert_allclose(part["db_gate"], full["db_gate"][cols], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(part["db_up"], full["db_up"][cols], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(part["db_down"], full["db_down"], rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# Global-level load-balancing loss
# ---------------------------------------------------------------------------

AUX_SPECS = ["softmax_topk", "topk_softmax", "softmax_logit_bias"]


def run_aux(spec, c, coef, f=None):
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c), c["shared"], aux_coef=coef, aux_f=f)
    bwd = layer_backward(spec, c["x"], c["w_r"], c["beta"], efn(c), fwd, c["dy"], c["shared"],
                         with_bias=c["bg"] is not None)
    return fwd, bwd


@pytest.mark.parametrize("name", AUX_SPECS)
def test_aux_loss_matches_torch_autograd(name):
    """Loss value and its x / W_r gradients against torch autograd of an
    independent formulation (softmax over all experts, the load fractions
    counted from torch.topk of the selection logits and held fixed)."""
    spec = SPECS[name]
    c = make_case(spec, seed=11)
    coef = 0.37
    fwd, bwd = run_aux(spec, c, coef)
    _, bwd0 = run(spec, c)
    x = torch.tensor(c["x"], dtype=torch.float64, requires_grad=True)
    w = torch.tensor(c["w_r"], dtype=torch.float64, requires_grad=True)
    v = x @ w
    if c["beta"] is not None and spec.bias_mode == "logit":
        v = v + torch.tensor(c["beta"])
    T, E, k = v.shape[0], spec.E, spec.k
    sel = torch.topk(v.detach(), k, dim=1).indices
    cnt = torch.zeros(E, dtype=torch.float64).index_add_(0, sel.reshape(-1), torch.ones(T * k, dtype=torch.float64))
    loss = coef * E * (cnt / (T * k) * torch.softmax(v, dim=1).mean(0)).sum()
    loss.backward()
    assert abs(fwd["aux"]["loss"] - loss.item()) <= 1e-13 * abs(loss.item())
    assert rel(bwd["dw_r"] - bwd0["dw_r"], w.grad.numpy()) < 1e-11
    assert rel(bwd["dx"] - bwd0["dx"], x.grad.numpy()) < 1e-11


@pytest.mark.parametrize("name", AUX_SPECS)
def test_aux_loss_gradients_match_finite_differences(name):
    """d/dx and d/dW_r of sum <dy, y> + L_aux by central differences (routing,
    and so the load fractions, unchanged by the step)."""
    spec = SPECS[name]
    c = make_case(spec, T=12, d=8, f=6, seed=12)
    coef = 0.5
    fwd, bwd = run_aux(spec, c, coef)

    def total(cc):
        fw = layer_forward(spec, cc["x"], cc["w_r"], cc["beta"], efn(cc), None, aux_coef=coef)
        return float((cc["dy"] * fw["y"]).sum()) + fw["aux"]["loss"], fw["route"]["topk_idx"]

    rng = np.random.default_rng(6)
    h = 1e-6
    for key, gr in (("x", bwd["dx"]), ("w_r", bwd["dw_r"])):
        for _ in range(3):
            v = rng.standard_normal(c[key].shape)
            v /= np.linalg.norm(v)
            lp, ip = total(dict(c, **{key: c[key] + h * v}))
            lm, im = total(dict(c, **{key: c[key] - h * v}))
            if not (np.array_equal(ip, fwd["route"]["topk_idx"]) and np.array_equal(im, fwd["route"]["topk_idx"])):
                continue
            fd = (lp - lm) / (2 * h)
            an = float((gr * v).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (key, fd, an)


def test_aux_loss_uniform_router_closed_form():
    """Equal logits: every probability is 1/E, so L = coef * sum_e f_e = coef for
    any routing, and dL/dl[t][j] = coef / T * (f_j - 1/E)."""
    spec = RouterSpec("softmax_topk", E=8, k=2)
    T = 10
    p = router_probs(spec, np.zeros((T, 8)))
    counts = np.array([7, 0, 3, 2, 4, 1, 3, 0])
    coef = 1e-3
    out = aux_loss(spec, p, counts, coef)
    assert out["loss"] == pytest.approx(coef, rel=1e-15)
    f = counts / 20.0
    dl = aux_loss_backward(p, f, coef)
    np.testing.assert_allclose(dl, np.broadcast_to(coef / T * (f - 1 / 8), (T, 8)), rtol=1e-14, atol=1e-20)


def test_aux_loss_concentrated_router_is_maximal():
    """All probability and all load on one expert: L = coef * E, its largest value."""
    spec = RouterSpec("softmax_topk", E=4, k=1)
    p = router_probs(spec, np.tile(np.array([[60.0, 0.0, 0.0, 0.0]]), (5, 1)))
    out = aux_loss(spec, p, np.array([5, 0, 0, 0]), 0.25)
    assert out["loss"] == pytest.approx(0.25 * 4, rel=1e-12)


@pytest.mark.parametrize("name", AUX_SPECS)
def test_aux_gradient_rows_sum_to_zero(name):
    """Adding a constant to a token's logits leaves its softmax unchanged, so each
    row of dL_aux/dl sums to zero."""
    spec = SPECS[name]
    c = make_case(spec, seed=13)
    fwd, _ = run_aux(spec, c, 0.8)
    dl = aux_loss_backward(fwd["aux"]["probs"], fwd["aux"]["f"], 0.8)
    assert np.abs(dl.sum(axis=1)).max() <= 1e-15 * np.abs(dl).max() * spec.E


def test_aux_loss_batch_fractions_are_used():
    """Given the batch's fractions, the loss and its gradient use them instead of
    this call's counts."""
    spec = SPECS["softmax_topk"]
    c = make_case(spec, seed=14)
    f = np.full(spec.E, 1.0 / spec.E)
    fwd, _ = run_aux(spec, c, 0.3, f=f)
    assert fwd["aux"]["loss"] == pytest.approx(0.3, rel=1e-12)  # P sums to one
    assert np.array_equal(fwd["aux"]["f"], f)


# ---------------------------------------------------------------------------
# Zero-computation experts (MoE++; appendix B.3)
# ---------------------------------------------------------------------------

from oracle import ZeroComputeSpec, zc_backward, zc_forward  # noqa: E402

ZC = ZeroComputeSpec(n_zero=2, n_copy=1, n_const=2, aux_weight=0.3)


def make_zc_case(spec, zs, T=24, d=16, f=12, seed=0, wr_std=0.3):
    """A case whose router covers the E FFN experts and zs.n more."""
    rng = np.random.default_rng(seed)
    Ep = spec.E + zs.n
    c = make_case(spec, T=T, d=d, f=f, seed=seed, wr_std=wr_std)
    c["w_r"] = rng.standard_normal((d, Ep)) * wr_std
    c["beta"] = rng.standard_normal(Ep) * 0.1 if spec.bias_mode != "none" else None
    c["v"] = rng.standard_normal((zs.n_const, d))
    c["wc"] = rng.standard_normal((zs.n_const, 2, d)) * 0.4
    return c


def run_zc(spec, zs, c, coef=0.0):
    zc = (zs, c["v"], c["wc"])
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c), c["shared"], aux_coef=coef, zc=zc)
    bwd = layer_backward(spec, c["x"], c["w_r"], c["beta"], efn(c), fwd, c["dy"], c["shared"], zc=zc)
    return fwd, bwd


def test_zc_layer_rows_cover_the_pool_with_ffn_rows_first():
    """The layer sorts every slot of the pool by (expert, token) (the library
    stable sort); the FFN slots hold the first offsets[E] rows, whose x_perm
    rows are their tokens' x, and only they reach the combine."""
    spec = RouterSpec("softmax_topk", E=6, k=3)
    c = make_zc_case(spec, ZC, T=40, seed=21, wr_std=0.6)
    fwd = layer_forward(spec, c["x"], c["w_r"], None, efn(c), zc=(ZC, c["v"], c["wc"]))
    idx, mp, k = fwd["route"]["topk_idx"], fwd["maps"], spec.k
    T, Ep = idx.shape[0], spec.E + ZC.n
    flat = idx.reshape(-1)
    t_of = np.repeat(np.arange(T), k)
    s_of = np.tile(np.arange(k), T)
    order = np.lexsort((t_of, flat))
    assert mp["token_of"].tolist() == (t_of[order] * k + s_of[order]).tolist()
    assert mp["counts"].tolist() == np.bincount(flat, minlength=Ep).tolist()
    n_ffn = int((flat < spec.E).sum())
    assert 0 < n_ffn < T * k and mp["offsets"][spec.E] == n_ffn
    assert np.array_equal(mp["row_ffn"] >= 0, idx < spec.E)
    assert np.all(mp["row_ffn"][idx < spec.E] < n_ffn)
    assert np.array_equal(fwd["x_perm"], c["x"][mp["token_of"][:n_ffn] // k])


def torch_zc_loss(spec, zs, c, params, coef):
    """Independent dense formulation: every expert of the pool evaluated for
    every token, the gate a masked softmax over the pool; returns
    sum <dy, y> + the weighted balance loss, and the selection."""
    x, w_r = params["x"], params["w_r"]
    l = x @ w_r
    T, Ep = l.shape
    E = spec.E
    key = l
    sel = torch.topk(key.detach(), spec.k, dim=1).indices
    mask = torch.zeros(T, Ep, dtype=torch.bool).scatter(1, sel, True)
    gate = torch.softmax(l.masked_fill(~mask, float("-inf")), dim=1)
    outs = []
    for e in range(E):
        g = x @ params["wg"][e]
        u = x @ params["wu"][e]
        outs.append((torch.nn.functional.silu(g) * u) @ params["wd"][e])
    outs += [torch.zeros_like(x)] * zs.n_zero + [x] * zs.n_copy
    for ci in range(zs.n_const):
        a = torch.softmax(x @ params["wc"][ci].T, dim=1)          # [T][2]
        outs.append(a[:, :1] * x + a[:, 1:] * params["v"][ci])
    y = sum(gate[:, e:e + 1] * outs[e] for e in range(Ep))
    loss = (torch.tensor(c["dy"]) * y).sum()
    if coef:
        cnt = torch.zeros(Ep, dtype=torch.float64).index_add_(
            0, sel.reshape(-1), torch.ones(T * spec.k, dtype=torch.float64))
        eta = torch.cat([torch.ones(E, dtype=torch.float64),
                         torch.full((zs.n,), zs.aux_weight, dtype=torch.float64)])
        loss = loss + coef * Ep * (eta * cnt / (T * spec.k) * torch.softmax(l, dim=1).mean(0)).sum()
    return loss, sel


@pytest.mark.parametrize("coef", [0.0, 0.4])
def test_zc_layer_matches_torch_autograd(coef):
    spec = RouterSpec("softmax_topk", E=6, k=3)
    c = make_zc_case(spec, ZC, seed=22, wr_std=0.6)
    fwd, bwd = run_zc(spec, ZC, c, coef)
    idx = fwd["route"]["topk_idx"]
    assert (idx >= spec.E).sum() >= 10 and (idx < spec.E).sum() >= 10   # both kinds exercised
    for z in range(spec.E, spec.E + ZC.n):
        assert (idx == z).any(), z
    params = {n: torch.tensor(c[n], dtype=torch.float64, requires_grad=True)
              for n in ("x", "w_r", "wg", "wu", "wd", "v", "wc")}
    loss, sel = torch_zc_loss(spec, ZC, c, params, coef)
    loss.backward()
    assert [sorted(r) for r in sel.tolist()] == [sorted(r) for r in idx.tolist()]
    ours = float((c["dy"] * fwd["y"]).sum()) + (fwd["aux"]["loss"] if coef else 0.0)
    assert abs(loss.item() - ours) <= 1e-12 * abs(loss.item())
    assert rel(bwd["dx"], params["x"].grad.numpy()) < 1e-11
    assert rel(bwd["dw_r"], params["w_r"].grad.numpy()) < 1e-11
    assert rel(bwd["zc"]["dv"], params["v"].grad.numpy()) < 1e-11
    assert rel(bwd["zc"]["dwc"], params["wc"].grad.numpy()) < 1e-11
    for e in range(spec.E):
        for o_, t_ in (("dw_gate", "wg"), ("dw_up", "wu"), ("dw_down", "wd")):
            want = params[t_].grad[e].numpy()
            if np.linalg.norm(want) == 0:
                assert np.linalg.norm(bwd["experts"][e][o_]) == 0
            else:
                assert rel(bwd["experts"][e][o_], want) < 1e-11


def test_zc_gradients_match_finite_differences():
    spec = RouterSpec("topk_softmax", E=5, k=2, bias_mode="logit")
    zs = ZeroComputeSpec(n_zero=1, n_copy=2, n_const=2, aux_weight=0.0)
    c = make_zc_case(spec, zs, T=14, d=8, f=6, seed=23, wr_std=0.7)
    coef = 0.6
    fwd, bwd = run_zc(spec, zs, c, coef)
    assert (fwd["route"]["topk_idx"] >= spec.E).sum() >= 6

    def total(cc):
        fw = layer_forward(spec, cc["x"], cc["w_r"], cc["beta"], efn(cc), None, aux_coef=coef,
                           zc=(zs, cc["v"], cc["wc"]))
        return float((cc["dy"] * fw["y"]).sum()) + fw["aux"]["loss"], fw["route"]["topk_idx"]

    rng = np.random.default_rng(7)
    h = 1e-6
    grads = {"x": bwd["dx"], "w_r": bwd["dw_r"], "v": bwd["zc"]["dv"], "wc": bwd["zc"]["dwc"],
             "wd": np.stack([bwd["experts"][e]["dw_down"] for e in range(spec.E)])}
    checked = 0
    for key, gr in grads.items():
        for _ in range(3):
            v = rng.standard_normal(c[key].shape)
            v /= np.linalg.norm(v)
            lp, ip = total(dict(c, **{key: c[key] + h * v}))
            lm, im = total(dict(c, **{key: c[key] - h * v}))
            if not (np.array_equal(ip, fwd["route"]["topk_idx"]) and np.array_equal(im, fwd["route"]["topk_idx"])):
                continue
            fd = (lp - lm) / (2 * h)
            an = float((gr * v).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (key, fd, an)
            checked += 1
    assert checked >= 12


def test_zc_omega_is_the_derivative_in_the_gate_weight():
    """y_zc is linear in each gating weight, so a unit step of w[t][s] changes
    sum <dy, y_zc> by exactly omega[t][s]."""
    rng = np.random.default_rng(24)
    T, d, E, k = 7, 10, 3, 3
    zs = ZeroComputeSpec(n_zero=1, n_copy=1, n_const=2)
    idx = np.stack([rng.permutation(E + zs.n)[:k] for _ in range(T)])
    w = rng.random((T, k))
    x, dy = rng.standard_normal((T, d)), rng.standard_normal((T, d))
    v, wc = rng.standard_normal((2, d)), rng.standard_normal((2, 2, d))
    base = float((dy * zc_forward(x, idx, w, E, zs, v, wc)["y"]).sum())
    om = zc_backward(dy, x, idx, w, E, zs, v, wc)["omega"]
    for t in range(T):
        for s in range(k):
            w2 = w.copy()
            w2[t, s] += 1.0
            step = float((dy * zc_forward(x, idx, w2, E, zs, v, wc)["y"]).sum()) - base
            assert step == pytest.approx(om[t, s], rel=1e-12, abs=1e-12)
            if idx[t, s] < E + zs.n_zero:            # FFN (handled elsewhere) or zero expert
                assert om[t, s] == 0.0


def _forced_case(kind, zs, T=9, d=12):
    """Router weights that send every token to k experts of one kind."""
    spec = RouterSpec("softmax_topk", E=4, k=2)
    c = make_zc_case(spec, zs, T=T, d=d, seed=25)
    first = {"zero": spec.E, "copy": spec.E + zs.n_zero, "const": spec.E + zs.n_zero + zs.n_copy}[kind]
    c["w_r"][:, :] = 0.0
    c["beta"] = None
    c["x"][:, 0] = np.abs(c["x"][:, 0]) + 1.0
    c["w_r"][0, first] = 40.0
    c["w_r"][0, first + 1] = 39.0
    return spec, c


def test_zc_all_copy_is_identity():
    """Both slots on copy experts: y = x (the weights sum to one), and the
    router gradient vanishes (equal omega on both slots), so dx = dy."""
    zs = ZeroComputeSpec(n_zero=1, n_copy=2, n_const=1)
    spec, c = _forced_case("copy", zs)
    fwd, bwd = run_zc(spec, zs, c)
    assert np.all(fwd["route"]["topk_idx"] >= spec.E + 1)
    np.testing.assert_allclose(fwd["y"], c["x"], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(bwd["dx"], c["dy"], rtol=1e-12, atol=1e-12)
    assert np.abs(bwd["dw_r"]).max() < 1e-12
    assert all(np.abs(g["dw_gate"]).max() == 0 for g in bwd["experts"].values())


def test_zc_all_zero_is_zero():
    zs = ZeroComputeSpec(n_zero=2, n_copy=0, n_const=1)
    spec, c = _forced_case("zero", zs)
    fwd, bwd = run_zc(spec, zs, c)
    assert np.all(fwd["y"] == 0.0)
    assert np.all(bwd["dx"] == 0.0) and np.all(bwd["dw_r"] == 0.0)
    assert np.all(bwd["zc"]["dv"] == 0.0) and np.all(bwd["zc"]["dwc"] == 0.0)


def test_zc_constant_with_zero_projection_is_the_mean():
    """W_c = 0: the two mixing weights are 1/2, so a constant expert returns
    (x + v) / 2; with both slots on constant experts y = (x + w1 v1 + w2 v2) / 2."""
    zs = ZeroComputeSpec(n_zero=0, n_copy=0, n_const=2)
    spec, c = _forced_case("const", zs)
    c["wc"][:] = 0.0
    fwd, _ = run_zc(spec, zs, c)
    w = fwd["route"]["topk_w"]
    idx = fwd["route"]["topk_idx"] - spec.E
    want = 0.5 * (c["x"] + w[:, :1] * c["v"][idx[:, 0]] + w[:, 1:] * c["v"][idx[:, 1]])
    np.testing.assert_allclose(fwd["y"], want, rtol=1e-13, atol=1e-13)


def test_zc_aux_weight_one_is_the_plain_pool_loss_and_zero_drops_the_terms():
    """aux_weight = 1: the loss over the pool of E + Z experts; aux_weight = 0:
    the same loss with every zero-computation expert's term removed (checked
    by moving all their load onto them: the loss is then 0)."""
    spec = RouterSpec("softmax_topk", E=4, k=2)
    rng = np.random.default_rng(26)
    p = router_probs(spec, rng.standard_normal((11, 7)))
    counts = np.array([3, 5, 0, 2, 4, 6, 2])
    base = aux_loss(spec, p, counts, 0.2)
    one = aux_loss(spec, p, counts, 0.2, eta=np.ones(7))
    assert one["loss"] == base["loss"]
    only_zc = np.array([0, 0, 0, 0, 7, 8, 7])
    assert aux_loss(spec, p, only_zc, 0.2, eta=[1, 1, 1, 1, 0, 0, 0])["loss"] == 0.0
    dl = aux_loss_backward(p, only_zc / 22.0, 0.2, eta=[1, 1, 1, 1, 0, 0, 0])
    assert np.all(dl == 0.0)


def test_zc_token_subset_equals_whole_layer():
    """The per-token evaluation used at full size gives the whole layer's y,
    dx, omega and dl with zero-computation experts in the pool, and the
    dW_r column of a zero-computation expert from the tokens that chose it."""
    spec = RouterSpec("softmax_topk", E=6, k=3)
    c = make_zc_case(spec, ZC, T=40, seed=27, wr_std=0.6)
    fwd, bwd = run_zc(spec, ZC, c)
    zc = (ZC, c["v"], c["wc"])
    sub = np.array([39, 3, 17, 0, 22, 5, 30])
    r = token_forward_backward(spec, c["x"][sub], c["dy"][sub], c["w_r"], c["beta"], efn(c), None, zc=zc)
    assert np.array_equal(r["route"]["topk_idx"], fwd["route"]["topk_idx"][sub])
    assert (r["route"]["topk_idx"] >= spec.E).any() and (r["route"]["topk_idx"] == spec.E).any()
    for a, b in ((r["y"], fwd["y"][sub]), (r["dx"], bwd["dx"][sub]), (r["omega"], bwd["omega"][sub]),
                 (r["dl"], bwd["dl"][sub])):
        assert rel(a, b) < 1e-12
    for e in (spec.E, spec.E + ZC.n - 1):
        toks = np.nonzero((fwd["route"]["topk_idx"] == e).any(axis=1))[0]
        r = token_forward_backward(spec, c["x"][toks], c["dy"][toks], c["w_r"], c["beta"], efn(c), None, zc=zc)
        assert rel(c["x"][toks].T @ r["dl_dense"][:, e], bwd["dw_r"][:, e]) < 1e-12


# ---------------------------------------------------------------------------
# Clamped GLU expert activation (the GPT-OSS release's variant)
# ---------------------------------------------------------------------------

from oracle import glu  # noqa: E402

CLAMPED = ("clamped_glu", 1.702, 7.0)


def _clamp_case(seed, scale=12.0, T=30):
    """Expert weights scaled so that a large share of g and u fall outside +-7."""
    spec = RouterSpec("topk_softmax", E=6, k=2)
    c = make_case(spec, T=T, d=16, f=12, seed=seed, expert_bias=True)
    for n in ("wg", "wu"):
        c[n] = c[n] * scale
    return spec, c


def test_clamped_glu_layer_matches_torch_autograd():
    spec, c = _clamp_case(31)
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c), act=CLAMPED)
    bwd = layer_backward(spec, c["x"], c["w_r"], c["beta"], efn(c), fwd, c["dy"], with_bias=True, act=CLAMPED)
    g = np.concatenate([fwd["g"][e] for e in fwd["g"]])
    u = np.concatenate([fwd["u"][e] for e in fwd["u"]])
    assert 0.15 < (g > 7.0).mean() < 0.6 and 0.15 < (np.abs(u) > 7.0).mean() < 0.8   # both clamps active
    P = {n: torch.tensor(c[n], dtype=torch.float64, requires_grad=True)
         for n in ("x", "w_r", "wg", "wu", "wd", "bg", "bu", "bd")}
    l = P["x"] @ P["w_r"]
    sel = torch.topk(l.detach(), spec.k, dim=1).indices
    mask = torch.zeros_like(l, dtype=torch.bool).scatter(1, sel, True)
    gate = torch.softmax(l.masked_fill(~mask, float("-inf")), dim=1)
    y = 0
    for e in range(spec.E):
        ge = P["x"] @ P["wg"][e] + P["bg"][e]
        ue = P["x"] @ P["wu"][e] + P["bu"][e]
        gc = torch.clamp(ge, max=7.0)
        he = gc * torch.sigmoid(1.702 * gc) * (torch.clamp(ue, -7.0, 7.0) + 1.0)
        y = y + gate[:, e:e + 1] * (he @ P["wd"][e] + P["bd"][e])
    loss = (torch.tensor(c["dy"]) * y).sum()
    loss.backward()
    assert abs(loss.item() - float((c["dy"] * fwd["y"]).sum())) <= 1e-12 * abs(loss.item())
    assert rel(bwd["dx"], P["x"].grad.numpy()) < 1e-11
    assert rel(bwd["dw_r"], P["w_r"].grad.numpy()) < 1e-11
    for ours, theirs in (("dw_gate", "wg"), ("dw_up", "wu"), ("dw_down", "wd"), ("db_gate", "bg"),
                         ("db_up", "bu"), ("db_down", "bd")):
        got = np.stack([bwd["experts"][e][ours] for e in range(spec.E)])
        assert rel(got, P[theirs].grad.numpy()) < 1e-11, ours


def test_clamped_glu_gradients_match_finite_differences():
    spec, c = _clamp_case(32, T=16)
    fwd = layer_forward(spec, c["x"], c["w_r"], c["beta"], efn(c), act=CLAMPED)
    bwd = layer_backward(spec, c["x"], c["w_r"], c["beta"], efn(c), fwd, c["dy"], with_bias=True, act=CLAMPED)

    def total(cc):
        fw = layer_forward(spec, cc["x"], cc["w_r"], cc["beta"], efn(cc), act=CLAMPED)
        return float((cc["dy"] * fw["y"]).sum()), fw["route"]["topk_idx"]

    rng = np.random.default_rng(8)
    h = 1e-7
    checked = 0
    for key, gr in (("x", bwd["dx"]), ("wg", np.stack([bwd["experts"][e]["dw_gate"] for e in range(spec.E)])),
                    ("wu", np.stack([bwd["experts"][e]["dw_up"] for e in range(spec.E)])),
                    ("bu", np.stack([bwd["experts"][e]["db_up"] for e in range(spec.E)]))):
        for _ in range(3):
            v = rng.standard_normal(c[key].shape)
            v /= np.linalg.norm(v)
            lp, ip = total(dict(c, **{key: c[key] + h * v}))
            lm, im = total(dict(c, **{key: c[key] - h * v}))
            if not (np.array_equal(ip, fwd["route"]["topk_idx"]) and np.array_equal(im, fwd["route"]["topk_idx"])):
                continue
            fd = (lp - lm) / (2 * h)
            an = float((gr * v).sum())
            assert abs(fd - an) <= 1e-5 * max(1.0, abs(an)), (key, fd, an)
            checked += 1
    assert checked >= 8


def test_clamped_glu_without_clamps_is_swiglu_of_u_plus_one():
    """alpha = 1 and no clamping: h = silu(g) (u + 1), the SwiGLU layer with b_up
    raised by one."""
    spec = RouterSpec("softmax_topk", E=5, k=2)
    c = make_case(spec, T=20, seed=33, expert_bias=True)
    fwd = layer_forward(spec, c["x"], c["w_r"], None, efn(c), act=("clamped_glu", 1.0, 1e300))
    bwd = layer_backward(spec, c["x"], c["w_r"], None, efn(c), fwd, c["dy"], with_bias=True,
                         act=("clamped_glu", 1.0, 1e300))
    c1 = dict(c, bu=c["bu"] + 1.0)
    fwd1 = layer_forward(spec, c1["x"], c1["w_r"], None, efn(c1))
    bwd1 = layer_backward(spec, c1["x"], c1["w_r"], None, efn(c1), fwd1, c1["dy"], with_bias=True)
    assert rel(fwd["y"], fwd1["y"]) < 1e-14 and rel(bwd["dx"], bwd1["dx"]) < 1e-13
    for e in range(spec.E):
        for n in ("dw_gate", "dw_up", "dw_down", "db_up"):
            assert rel(bwd["experts"][e][n], bwd1["experts"][e][n]) < 1e-13


def test_clamped_glu_saturated_gate_passes_no_gradient():
    """g above the limit everywhere: h = L sig(alpha L) (clip(u) + 1), no gradient
    reaches the gate; u beyond the limits: none reaches the up projection."""
    g = np.array([[7.5, 9.0, 100.0]])
    u = np.array([[-8.0, 0.5, 7.0]])
    h, hg, hu = glu(g, u, CLAMPED)
    L, a = 7.0, 1.702
    s = 1.0 / (1.0 + np.exp(-a * L))
    np.testing.assert_allclose(h, L * s * (np.clip(u, -L, L) + 1.0), rtol=1e-15)
    assert np.all(hg == 0.0)
    assert hu[0, 0] == 0.0 and hu[0, 1] == pytest.approx(L * s) and hu[0, 2] == pytest.approx(L * s)


# ---------------------------------------------------------------------------
# Threshold router (DynMoE-style: sigmoid gates, learned thresholds, variable k)
# ---------------------------------------------------------------------------

from oracle import threshold_backward  # noqa: E402,F401

THR = RouterSpec("sigmoid_threshold", E=8, k=4)


def _thr_case(seed, T=40, theta_mean=0.6):
    c = make_case(THR, T=T, seed=seed, wr_std=0.4, expert_bias=False)
    c["theta"] = theta_mean + 0.2 * np.random.default_rng(seed + 100).standard_normal(THR.E)
    return c


def run_thr(spec, c, coef=0.0):
    fwd = layer_forward(spec, c["x"], c["w_r"], None, efn(c), aux_coef=coef, theta=c["theta"])
    bwd = layer_backward(spec, c["x"], c["w_r"], None, efn(c), fwd, c["dy"])
    return fwd, bwd


def test_threshold_routing_invariants():
    c = _thr_case(41, T=200)
    fwd, _ = run_thr(THR, c)
    rt = fwd["route"]
    idx, w, keys = rt["topk_idx"], rt["topk_w"], rt["keys"]
    n = (idx >= 0).sum(1)
    assert n.min() >= 1 and n.max() <= THR.k and len(set(n.tolist())) >= 3   # the count varies
    for t in range(idx.shape[0]):
        act = idx[t][idx[t] >= 0]
        assert np.all(idx[t][n[t]:] == -1)                        # active slots first
        kk = keys[t, act]
        assert np.all(np.diff(kk) <= 0)                           # descending key
        above = np.nonzero(keys[t] > 0)[0]
        if len(above) == 0:
            assert len(act) == 1 and act[0] == int(np.argmax(keys[t]))   # the best one
        else:
            assert set(act.tolist()) <= set(above.tolist()) and len(act) == min(len(above), THR.k)
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=1e-14)
    assert np.all(w[idx < 0] == 0) and np.all(w[idx >= 0] > 0)


def torch_threshold_loss(spec, c, P, coef):
    """Dense formulation: every expert for every token, the active mask from
    detached keys, a straight-through indicator a = M + M (theta_d - theta) for
    the thresholds, gates a s / sum(a s); plus the variable-k balance loss with
    p = s / sum s and f the share of the filled slots."""
    x, w_r, th = P["x"], P["w_r"], P["theta"]
    l = x @ w_r
    T, E = l.shape
    s = torch.sigmoid(l)
    key = (l - th).detach()
    order = torch.argsort(-key, dim=1, stable=True)[:, :spec.k]
    M = torch.zeros(T, E, dtype=torch.bool)
    for t in range(T):
        for j, e in enumerate(order[t].tolist()):
            if j == 0 or key[t, e] > 0:
                M[t, e] = True
    Mf = M.double()
    a = Mf + Mf * (th.detach() - th)
    gate = a * s / (a * s).sum(1, keepdim=True)
    y = 0
    for e in range(E):
        he = torch.nn.functional.silu(x @ P["wg"][e]) * (x @ P["wu"][e])
        y = y + gate[:, e:e + 1] * (he @ P["wd"][e])
    loss = (torch.tensor(c["dy"]) * y).sum()
    if coef:
        cnt = Mf.sum(0)
        p = s / s.sum(1, keepdim=True)
        loss = loss + coef * E * (cnt / cnt.sum() * p.mean(0)).sum()
    return loss, M


@pytest.mark.parametrize("coef", [0.0, 0.7])
def test_threshold_router_matches_torch_autograd(coef):
    c = _thr_case(42)
    fwd = layer_forward(THR, c["x"], c["w_r"], None, efn(c), aux_coef=coef, theta=c["theta"])
    bwd = layer_backward(THR, c["x"], c["w_r"], None, efn(c), fwd, c["dy"])
    P = {n: torch.tensor(c[n], dtype=torch.float64, requires_grad=True)
         for n in ("x", "w_r", "wg", "wu", "wd", "theta")}
    loss, M = torch_threshold_loss(THR, c, P, coef)
    loss.backward()
    idx = fwd["route"]["topk_idx"]
    mine = np.zeros_like(M.numpy())
    for t in range(idx.shape[0]):
        mine[t, idx[t][idx[t] >= 0]] = True
    assert np.array_equal(mine, M.numpy())
    ours = float((c["dy"] * fwd["y"]).sum()) + (fwd["aux"]["loss"] if coef else 0.0)
    assert abs(loss.item() - ours) <= 1e-12 * abs(loss.item())
    assert rel(bwd["dx"], P["x"].grad.numpy()) < 1e-11
    assert rel(bwd["dw_r"], P["w_r"].grad.numpy()) < 1e-11
    assert rel(bwd["dtheta"], P["theta"].grad.numpy()) < 1e-11
    for e in range(THR.E):
        for o_, t_ in (("dw_gate", "wg"), ("dw_up", "wu"), ("dw_down", "wd")):
            want = P[t_].grad[e].numpy()
            if np.linalg.norm(want) == 0:
                assert np.linalg.norm(bwd["experts"][e][o_]) == 0
            else:
                assert rel(bwd["experts"][e][o_], want) < 1e-11


def test_threshold_router_gradients_match_finite_differences():
    c = _thr_case(43, T=16)
    coef = 0.5
    fwd = layer_forward(THR, c["x"], c["w_r"], None, efn(c), aux_coef=coef, theta=c["theta"])
    bwd = layer_backward(THR, c["x"], c["w_r"], None, efn(c), fwd, c["dy"])

    def total(cc):
        fw = layer_forward(THR, cc["x"], cc["w_r"], None, efn(cc), aux_coef=coef, theta=cc["theta"])
        return float((cc["dy"] * fw["y"]).sum()) + fw["aux"]["loss"], fw["route"]["topk_idx"]

    rng = np.random.default_rng(9)
    h = 1e-6
    checked = 0
    for key, gr in (("x", bwd["dx"]), ("w_r", bwd["dw_r"]),
                    ("wd", np.stack([bwd["experts"][e]["dw_down"] for e in range(THR.E)]))):
        for _ in range(3):
            v = rng.standard_normal(c[key].shape)
            v /= np.linalg.norm(v)
            lp, ip = total(dict(c, **{key: c[key] + h * v}))
            lm, im = total(dict(c, **{key: c[key] - h * v}))
            if not (np.array_equal(ip, fwd["route"]["topk_idx"]) and np.array_equal(im, fwd["route"]["topk_idx"])):
                continue
            fd = (lp - lm) / (2 * h)
            an = float((gr * v).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (key, fd, an)
            checked += 1
    assert checked >= 6


def test_threshold_router_limits_reduce_to_fixed_k_routers():
    """Thresholds far above every logit: only the best expert, weight 1 (the
    top-1 softmax router).  Far below: every expert passes and the capacity
    keeps the k largest logits, weights s / sum s (the sigmoid router without
    groups or bias).  Outputs and gradients equal those routers' bit for bit
    up to rounding."""
    c = _thr_case(44)
    for theta, ref_spec in ((1e9, RouterSpec("softmax_topk", E=8, k=1)),
                            (-1e9, RouterSpec("sigmoid_grouped", E=8, k=4))):
        c1 = dict(c, theta=np.full(THR.E, theta))
        fwd, bwd = run_thr(THR, c1)
        spec_k = ref_spec
        fr = layer_forward(spec_k, c["x"], c["w_r"], None, efn(c))
        br = layer_backward(spec_k, c["x"], c["w_r"], None, efn(c), fr, c["dy"])
        act = fwd["route"]["topk_idx"][:, :spec_k.k]
        assert np.array_equal(act, fr["route"]["topk_idx"])
        assert rel(fwd["y"], fr["y"]) < 1e-14 and rel(bwd["dx"], br["dx"]) < 1e-13
        assert rel(bwd["dw_r"], br["dw_r"]) < 1e-13 if np.linalg.norm(br["dw_r"]) else np.abs(bwd["dw_r"]).max() < 1e-15
        for e in range(THR.E):
            assert rel(bwd["experts"][e]["dw_gate"], br["experts"][e]["dw_gate"]) < 1e-13 or \
                np.linalg.norm(br["experts"][e]["dw_gate"]) == 0


# ---------------------------------------------------------------------------
# FP8 (E4M3) forward of the expert GEMMs
# ---------------------------------------------------------------------------

from oracle import e4m3_round, e4m3_values, expert_backward, fp8_expert_backward, fp8_expert_forward, quantize_rows  # noqa: E402


def test_e4m3_values_and_rounding_match_torch():
    """The format's 256 values and the round-to-nearest-even of float32 values
    against torch's float8_e4m3fn (an independent implementation)."""
    v = e4m3_values()
    t = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(np.isnan(v), np.isnan(t)) and np.array_equal(v[~np.isnan(v)], t[~np.isnan(t)])
    assert np.nanmax(v) == 448.0 and np.nanmin(np.abs(v[v != 0])) == 2.0 ** -9
    rng = np.random.default_rng(51)
    x = np.concatenate([rng.uniform(-448, 448, 100000), rng.uniform(-1, 1, 100000),
                        rng.uniform(-0.02, 0.02, 50000), [0.0, -0.0, 448.0, -448.0, 2.0 ** -10, 3 * 2.0 ** -11]])
    x = x.astype(np.float32)
    assert np.array_equal(e4m3_round(x.astype(np.float64)), torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy())


def test_row_quantisation_properties():
    """Every non-zero row reaches +-448 at its largest element; the dequantised
    values are within half an E4M3 step of the inputs; a zero row stays zero."""
    rng = np.random.default_rng(52)
    a = rng.standard_normal((40, 96)) * rng.uniform(0.01, 50, (40, 1))
    a[7] = 0.0
    a = a.astype(np.float32).astype(np.float64)
    codes, scale, vals = quantize_rows(a)
    ev = e4m3_values()
    for r in range(40):
        if r == 7:
            assert np.all(vals[r] == 0) and scale[r] == 1.0
            continue
        assert np.abs(ev[codes[r]]).max() == 448.0
        # relative step of E4M3 normals is 2^-3: rounding error <= 2^-4 relative, or
        # half the smallest subnormal step (2^-10) times the scale
        err = np.abs(vals[r] - a[r])
        assert np.all(err <= np.maximum(2.0 ** -4 * np.abs(a[r]), 2.0 ** -10 * scale[r]) * (1 + 1e-6))


def test_fp8_forward_exact_on_representable_operands():
    """Operands that are E4M3 values times a power of two, with each row's and
    column's largest magnitude at 448 times that power: quantisation is exact,
    so the first GEMM of the FP8 expert equals the plain one."""
    rng = np.random.default_rng(53)
    ev = e4m3_values()
    fin = ev[np.isfinite(ev) & (np.abs(ev) <= 448)]
    x = rng.choice(fin, (12, 16)) * 2.0 ** -6
    x[:, 0] = 448 * 2.0 ** -6
    wg = rng.choice(fin, (16, 8)) * 2.0 ** -9
    wg[0, :] = 448 * 2.0 ** -9
    wu = rng.choice(fin, (16, 8)) * 2.0 ** -8
    wu[0, :] = -448 * 2.0 ** -8
    wd = rng.standard_normal((8, 16))
    g, u, h, o = fp8_expert_forward(x, wg, wu, wd)
    assert np.array_equal(g, x @ wg) and np.array_equal(u, x @ wu)


def test_fp8_layer_close_to_bf16_layer():
    """The FP8 forward differs from the plain one by quantisation noise only
    (a few percent normwise), and the backward is the plain backward of the
    FP8 forward's activations."""
    spec = RouterSpec("softmax_topk", E=6, k=2)
    c = make_case(spec, T=48, d=64, f=48, seed=54)
    f0 = layer_forward(spec, c["x"], c["w_r"], None, efn(c))
    f1 = layer_forward(spec, c["x"], c["w_r"], None, efn(c), fp8=True)
    assert 1e-3 < rel(f1["y"], f0["y"]) < 0.1
    assert np.array_equal(f1["route"]["topk_idx"], f0["route"]["topk_idx"])


def test_round_bf16_matches_torch():
    from oracle.moe_oracle import round_bf16
    rng = np.random.default_rng(55)
    a = np.concatenate([rng.standard_normal(100000) * 10.0 ** rng.integers(-8, 8, 100000), [0.0, -0.0, 1.0]])
    want = torch.from_numpy(a).to(torch.float32).to(torch.bfloat16).double().numpy()
    assert np.array_equal(round_bf16(a), want)


# ---------------------------------------------------------------------------
# FP8 (E4M3) data-gradient products of the expert backward
# ---------------------------------------------------------------------------

def _fp8_bwd_case(seed, M=10, d=16, f=8):
    from oracle.moe_oracle import round_bf16
    rng = np.random.default_rng(seed)
    xe = rng.standard_normal((M, d))
    wg, wu = rng.standard_normal((d, f)) * 0.3, rng.standard_normal((d, f)) * 0.3
    wd = rng.standard_normal((f, d)) * 0.3
    g, u = round_bf16(xe @ wg), round_bf16(xe @ wu)     # as a bf16 layer stores them
    h = g / (1 + np.exp(-g)) * u
    do = rng.standard_normal((M, d))
    return xe, g, u, h, do, wg, wu, wd


def test_fp8_dgrad_exact_first_product_on_row_representable_operands():
    """d_o rows and W_down rows that are E4M3 values times a power of two of
    their own (rows 2^12 apart, so that no column scale could hold them), each
    row reaching 448 times its power: the row quantisation of both operands is
    exact, so dh and with it dg, du and the weight gradients equal the plain
    backward's bit for bit (the stored-bf16 rounding of d_o is exact too)."""
    xe, g, u, h, do, wg, wu, wd = _fp8_bwd_case(61)
    rng = np.random.default_rng(62)
    ev = e4m3_values()
    fin = ev[np.isfinite(ev) & (np.abs(ev) <= 448)]
    M, d = do.shape
    f = wd.shape[0]
    pw_do = 2.0 ** (12 * (np.arange(M) % 2) - 6)
    do = rng.choice(fin, (M, d)) * pw_do[:, None]
    do[:, 3] = 448 * pw_do
    pw_wd = 2.0 ** (12 * (np.arange(f) % 2) - 9)
    wd = rng.choice(fin, (f, d)) * pw_wd[:, None]
    wd[:, 5] = -448 * pw_wd
    ref = expert_backward(xe, g, u, h, do, wg, wu, wd)
    got = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd)
    for n in ("dg", "du", "dw_gate", "dw_up", "dw_down"):
        assert np.array_equal(got[n], ref[n]), n
    assert not np.array_equal(got["dx"], ref["dx"])       # dx goes through the quantised [dg | du]


def test_fp8_dgrad_row_scaling_equivariance():
    """Scaling a row of d_o by 2^p scales the same row of dx by 2^p and leaves
    every other row's bits alone (row-wise scales of d_o and of [dg | du]);
    scaling row i of both W_gate and W_up by 2^p scales column i of dx by 2^p
    and leaves the other columns alone (row-wise scales of [W_gate | W_up])."""
    xe, g, u, h, do, wg, wu, wd = _fp8_bwd_case(63)
    base = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd)["dx"]
    do2 = do.copy()
    do2[4] *= 2.0 ** 7
    got = fp8_expert_backward(xe, g, u, h, do2, wg, wu, wd)["dx"]
    assert np.array_equal(got[4], base[4] * 2.0 ** 7)
    keep = np.arange(do.shape[0]) != 4
    assert np.array_equal(got[keep], base[keep])
    wg2, wu2 = wg.copy(), wu.copy()
    wg2[6] *= 2.0 ** -5
    wu2[6] *= 2.0 ** -5
    got = fp8_expert_backward(xe, g, u, h, do, wg2, wu2, wd)["dx"]
    assert np.array_equal(got[:, 6], base[:, 6] * 2.0 ** -5)
    keep = np.arange(wg.shape[0]) != 6
    assert np.array_equal(got[:, keep], base[:, keep])
    # a W_down row scaled by 2^p: dh column scales by 2^p; dx changes (through
    # the quantised [dg | du]) but dW_down does not (unquantised operands)
    wd2 = wd.copy()
    wd2[2] *= 2.0 ** 3
    a = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd)
    b = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd2)
    assert np.array_equal(b["dg"][:, 2], a["dg"][:, 2] * 8.0)
    assert np.array_equal(np.delete(b["dg"], 2, axis=1), np.delete(a["dg"], 2, axis=1))


def test_fp8_dgrad_one_scale_over_gate_and_up_halves():
    """One scale per row over both halves: with W_up 2^-24 times W_gate (below
    the smallest E4M3 step relative to the row's largest magnitude) the up
    half quantises to zero and dx is the gate half's product alone; with
    separate scales it would not be."""
    xe, g, u, h, do, wg, wu, wd = _fp8_bwd_case(64)
    tiny = fp8_expert_backward(xe, g, u, h, do, wg, wu * 2.0 ** -24, wd)
    zero = fp8_expert_backward(xe, g, u, h, do, wg, wu * 0.0, wd)
    # the [dg | du] quantisation is the same in both calls (du does not depend on W_up)
    assert np.array_equal(tiny["dx"], zero["dx"])
    sep = fp8_expert_backward(xe, g, u, h, do, wg * 0.0, wu * 2.0 ** -24, wd)["dx"]
    assert np.abs(sep).max() > 0                              # alone, the up half is representable


def test_fp8_dgrad_error_within_e4m3_bound():
    """Against the plain backward, the FP8 products differ by quantisation
    noise of E4M3's relative step (2^-3: at most 2^-4 per element) only."""
    xe, g, u, h, do, wg, wu, wd = _fp8_bwd_case(65, M=64, d=128, f=96)
    ref = expert_backward(xe, g, u, h, do, wg, wu, wd)
    got = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd)
    for n in ("dg", "dx", "dw_gate"):
        e = rel(got[n], ref[n])
        assert 1e-3 < e < 2 * 2.0 ** -4, (n, e)
    assert np.array_equal(got["dw_down"], ref["dw_down"])    # h^T d_o: unquantised operands


def test_fp8_layer_backward_uses_fp8_dgrad():
    """layer_backward(fp8=True) differs from the plain backward of the same
    forward in dx and the expert weight gradients (through dh), by
    quantisation noise, and the router gradient is untouched."""
    spec = RouterSpec("softmax_topk", E=6, k=2)
    c = make_case(spec, T=48, d=64, f=48, seed=66)
    fwd = layer_forward(spec, c["x"], c["w_r"], None, efn(c), fp8=True)
    b0 = layer_backward(spec, c["x"], c["w_r"], None, efn(c), fwd, c["dy"])
    b1 = layer_backward(spec, c["x"], c["w_r"], None, efn(c), fwd, c["dy"], fp8=True)
    assert 1e-3 < rel(b1["dx"], b0["dx"]) < 0.1
    assert 1e-3 < rel(b1["experts"][0]["dw_gate"], b0["experts"][0]["dw_gate"]) < 0.1
    assert np.array_equal(b1["experts"][0]["dw_down"], b0["experts"][0]["dw_down"])
    assert np.array_equal(b1["dw_r"], b0["dw_r"])


def test_fp8_dgrad_second_product_reads_e4m3_rows():
    """With [W_gate | W_up] 0.875 times the identity (d = 2f: each row one
    entry 448 * 2^-9, exactly representable with scale 2^-9), dx is 0.875
    times the dequantised [dg | du]: every row of dx divided by its largest
    magnitude / 448 lands on E4M3 values."""
    f, d, M = 8, 16, 12
    xe, g, u, h, do, _, _, wd = _fp8_bwd_case(67, M=M, d=d, f=f)
    eye = np.eye(d) * 448 * 2.0 ** -9
    wg, wu = eye[:, :f], eye[:, f:]
    got = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd)
    ev = set(e4m3_values()[np.isfinite(e4m3_values())].tolist())
    for r in range(M):
        s = np.abs(got["dx"][r]).max() / 448.0
        assert s > 0 and set((got["dx"][r] / s).tolist()) <= ev, r
    ref = np.concatenate([got["dg"], got["du"]], axis=1) * 0.875
    assert not np.array_equal(got["dx"], ref)               # quantised, not the plain [dg | du]


@pytest.mark.parametrize("level", [1, 2])
def test_fp8_token_subset_and_column_slices_equal_whole_layer(level):
    """With FP8 products the per-token and per-column evaluations still give
    the whole layer's values: the row quantisation is per token, the weights'
    quantisation per column (forward) or per row (data gradients) of the whole
    weight, and the slices of the weight gradients use column-local values."""
    spec = RouterSpec("softmax_topk", E=6, k=2)
    c = make_case(spec, T=40, d=32, f=24, seed=68)
    fwd = layer_forward(spec, c["x"], c["w_r"], None, efn(c), fp8=True)
    bwd = layer_backward(spec, c["x"], c["w_r"], None, efn(c), fwd, c["dy"], fp8=(level == 2))
    sub = np.array([39, 3, 17, 0, 22, 5])
    r = token_forward_backward(spec, c["x"][sub], c["dy"][sub], c["w_r"], None, efn(c), fp8=level)
    for a, b in ((r["y"], fwd["y"][sub]), (r["dx"], bwd["dx"][sub]), (r["omega"], bwd["omega"][sub])):
        assert rel(a, b) < 1e-12
    cols = np.array([23, 0, 9, 10])
    mp = fwd["maps"]
    for e in range(spec.E):
        r0, r1 = mp["offsets"][e], mp["offsets"][e + 1]
        if r1 == r0:
            continue
        wg, wu, wd, bg, bu, _ = efn(c)(e)
        part = expert_weight_grads_at(fwd["x_perm"][r0:r1], bwd["do"][r0:r1], wg, wu, wd, cols=cols, fp8=level)
        full = bwd["experts"][e]
        assert rel(part["dw_gate"], full["dw_gate"][:, cols]) < 1e-12
        assert rel(part["dw_up"], full["dw_up"][:, cols]) < 1e-12
        assert rel(part["dw_down"], full["dw_down"][cols, :]) < 1e-12



def test_fp8_dgrad_reads_stored_activations():
    """The FP8 backward takes the activation's derivatives at g and u as a
    bf16 layer stores them: g and u off the bf16 grid give the same result as
    their rounded values, and differ from the plain backward at the unrounded
    ones."""
    from oracle.moe_oracle import round_bf16
    xe, g, u, h, do, wg, wu, wd = _fp8_bwd_case(69)
    rng = np.random.default_rng(70)
    g2 = g * (1 + rng.uniform(-2.0 ** -10, 2.0 ** -10, g.shape))   # within half a bf16 step
    u2 = u * (1 + rng.uniform(-2.0 ** -10, 2.0 ** -10, u.shape))
    assert np.array_equal(round_bf16(g2), g) and np.array_equal(round_bf16(u2), u)
    a = fp8_expert_backward(xe, g2, u2, h, do, wg, wu, wd)
    b = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd)
    for n in ("dg", "du", "dx", "dw_gate", "dw_up"):
        assert np.array_equal(a[n], b[n]), n



def _clamped_glu_torch(g, u, alpha, limit):
    """The GPT-OSS release's clamped GLU written with torch primitives (an
    independent formulation): gc = min(g, L), uc = clamp(u, -L, L),
    h = gc sigmoid(alpha gc) (uc + 1)."""
    gc = torch.clamp(g, max=limit)
    uc = torch.clamp(u, min=-limit, max=limit)
    return gc * torch.sigmoid(alpha * gc) * (uc + 1.0)


def test_fp8_dgrad_clamped_glu_masks_of_the_forward_values():
    """FP8 backward with the clamped GLU (alpha 1.702, L 7) on operands whose
    row quantisation is exact, so dh = d_o W_down^T exactly: dg and du equal dh
    times torch autograd's derivatives of the clamped GLU, the smooth factors
    taken at the stored bf16 g, u and the clamp masks at the forward's own
    g, u (torch's clamp passes the gradient inside its bounds, bounds
    included).  Planted values just past a bound (7 + 2^-8, -7 - 2^-8: nearest
    rounding puts them on the bound) pass no gradient, as the forward's clamp
    cut them; autograd at the rounded value alone would pass it."""
    from oracle.moe_oracle import round_bf16
    alpha, L = 1.702, 7.0
    act = ("clamped_glu", alpha, L)
    rng = np.random.default_rng(72)
    M, d, f = 12, 16, 8
    ev = e4m3_values()
    fin = ev[np.isfinite(ev) & (np.abs(ev) <= 448)]
    do = rng.choice(fin, (M, d)) * 2.0 ** -6
    do[:, 0] = 448 * 2.0 ** -6                               # each row's largest magnitude: exact scale
    wd = rng.choice(fin, (f, d)) * 2.0 ** -9
    wd[:, 1] = -448 * 2.0 ** -9
    xe = rng.standard_normal((M, d))
    wg, wu = rng.standard_normal((d, f)), rng.standard_normal((d, f))
    g = rng.uniform(-9, 9, (M, f))
    u = rng.uniform(-9, 9, (M, f))
    g[0, :4] = [L + 2.0 ** -8, L, L - 2.0 ** -8, L + 2.0 ** -3]
    u[1, :4] = [L + 2.0 ** -8, -L - 2.0 ** -8, L, -L]
    assert round_bf16(np.array([L + 2.0 ** -8]))[0] == L     # rounding lands on the bound
    h = _clamped_glu_torch(torch.from_numpy(g), torch.from_numpy(u), alpha, L).numpy()
    got = fp8_expert_backward(xe, g, u, h, do, wg, wu, wd, act=act)
    dh = do @ wd.T
    # smooth factors: autograd at the stored values (a value inside a bound
    # stays inside when rounded: the bounds are bf16 values)
    gs = torch.tensor(round_bf16(g), requires_grad=True)
    us = torch.tensor(round_bf16(u), requires_grad=True)
    hs = _clamped_glu_torch(gs, us, alpha, L)
    dgs, dus = torch.autograd.grad(hs, (gs, us), torch.from_numpy(dh))
    # masks: autograd of the clamps at the forward's own values
    g64 = torch.tensor(g, requires_grad=True)
    u64 = torch.tensor(u, requires_grad=True)
    mg, mu = torch.autograd.grad((torch.clamp(g64, max=L) + torch.clamp(u64, min=-L, max=L)).sum(), (g64, u64))
    want_dg = dgs.numpy() * mg.numpy()
    want_du = dus.numpy() * mu.numpy()
    np.testing.assert_allclose(got["dg"], want_dg, rtol=1e-13, atol=1e-300)
    np.testing.assert_allclose(got["du"], want_du, rtol=1e-13, atol=1e-300)
    # the planted values: the forward's clamp cut them (no gradient) ...
    assert got["dg"][0, 0] == 0.0 and got["dg"][0, 3] == 0.0
    assert got["du"][1, 0] == 0.0 and got["du"][1, 1] == 0.0
    # ... the bounds themselves pass it ...
    assert got["dg"][0, 1] != 0.0 and got["du"][1, 2] != 0.0 and got["du"][1, 3] != 0.0
    # ... and autograd at the stored (rounded) value alone would have passed it
    assert dgs.numpy()[0, 0] != 0.0 and dus.numpy()[1, 0] != 0.0
