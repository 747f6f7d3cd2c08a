"""fp64 oracle of one MoE layer: router, permutation, SwiGLU experts, combine,
and the full backward (expert dgrad/wgrad, router gradient).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP implementation; it receives the same seeded inputs, upcast
exactly to float64.

What it follows.  The paper (PithTrain, arxiv 2605.31463) trains MoE models
built from a top-k router and SwiGLU experts (section 3.2, "Other
optimizations": fused SwiGLU forward and backward, EP token scatter; appendix
B.3, DynMoE task: the framework's top-k routing kernel) and checks a routing
trace by three rules: expert ids lie in [0, num_experts), gating weights are
non-negative and sum to one over the selected top-k (appendix B.2.2, "Collect
Routing Trace").  It prints no layer equations, so this oracle writes out the
standard definitions of the three router families of the workloads it is
tested on (Qwen3-30B-A3B and GPT-OSS-20B style softmax routers, DeepSeek-V3
style group-limited sigmoid router) and of a SwiGLU expert, in float64, with
no blocking, fusion or reordering beyond plain matrix products.  Every reading
the paper leaves open is listed with the design notes (ties go to the lower
index; slots are ordered by descending key; rows within an expert by
ascending token; the DeepSeek group score is the sum of the top two keys of
the group).

Conventions.  x [T][d]; W_r [d][E_pool] (E_pool = E plus any
zero-computation experts, see the last section); expert e: W_gate, W_up [d][f],
W_down [f][d], optional biases b_gate, b_up [f], b_down [d].
Routing outputs topk_idx [T][k] (slot order = descending selection key,
ties to the lower expert), topk_w [T][k].  Maps: row r of the permuted
matrix holds (token t, slot s) with token_of[r] = t*k + s and
row_of[t][s] = r; rows are grouped by expert (ascending expert), and within
an expert ordered by ascending token.
"""
from dataclasses import dataclass

import numpy as np


@dataclass
class RouterSpec:
    """Which router family and its constants.

    router:       'softmax_topk'  softmax over all experts, keep the top k,
                                  renormalise over the k (equal, in exact
                                  arithmetic, to a softmax over the k logits)
                  'topk_softmax'  top k logits, softmax over those k
                  'sigmoid_grouped'  s = sigmoid(logit), selection key s+beta,
                                  group-limited top-k, w = scale*s/sum(s)
                  'sigmoid_threshold'  DynMoE-style gating: s = sigmoid(logit),
                                  expert e active when logit - theta_e > 0 (a
                                  learned threshold per expert), at least the
                                  best one and at most k (the slot capacity),
                                  w = scale*s/sum(s) over the active ones
    k, n_groups, topk_groups, route_scale as in the workload configs;
    bias_mode:    'none', 'select' (bias in the selection key only) or
                  'logit' (bias added to the logits, for selection and weights).
    """
    router: str
    E: int
    k: int
    n_groups: int = 1
    topk_groups: int = 1
    route_scale: float = 1.0
    bias_mode: str = "none"


def spec_from_config(cfg):
    return RouterSpec(router=cfg["router"], E=cfg["E"], k=cfg["k"],
                      n_groups=cfg["n_groups"], topk_groups=cfg["topk_groups"],
                      route_scale=cfg["route_scale"], bias_mode=cfg["bias_mode"])


def sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def silu(z):
    return z * sigmoid(z)


# ----------------------------------------------------------------------------
# Router forward
# ----------------------------------------------------------------------------

def router_logits(x, w_r):
    """l[t][e] = sum_i x[t][i] * W_r[i][e], in float64."""
    return np.asarray(x, np.float64) @ np.asarray(w_r, np.float64)


def _desc_order(keys):
    """Per row, indices sorted by descending key; equal keys keep ascending index."""
    return np.argsort(-keys, axis=-1, kind="stable")


def _adjacent_gap_min(sorted_keys, upto):
    """Smallest gap between consecutive sorted keys among the first upto+1."""
    n = min(upto + 1, sorted_keys.shape[1])
    if n < 2:
        return np.full(sorted_keys.shape[0], np.inf)
    gaps = sorted_keys[:, :n - 1] - sorted_keys[:, 1:n]
    return gaps.min(axis=1)


def route(spec, logits, beta=None, theta=None):
    """Expert selection and gating weights for every token.

    Returns a dict with
      topk_idx [T][k] int64   selected experts, slot order = descending key
      topk_w   [T][k]         gating weights
      s_sel    [T][k] or None sigmoid scores of the selected experts
                              (sigmoid_grouped router only)
      keys     [T][E]         selection keys
      margin   [T]            smallest gap between consecutive keys among the
                              top k+1 candidates (and, for the grouped router,
                              between the kept and the first dropped group
                              score; for the threshold router, between a
                              candidate's key and 0); a token is ambiguous
                              when it is < 1e-6
    The threshold router (theta [E] required) fills slots past the token's
    active experts with topk_idx = -1 and zero weight and score.
    """
    l = np.asarray(logits, np.float64)
    T, E = l.shape
    k = spec.k
    b = None if beta is None else np.asarray(beta, np.float64)
    if spec.bias_mode != "none" and b is None:
        raise ValueError("router bias required")

    if spec.router in ("softmax_topk", "topk_softmax"):
        wl = l + b if spec.bias_mode == "logit" else l          # logits seen by the weights
        keys = l + b if spec.bias_mode in ("logit", "select") else l
        order = _desc_order(keys)
        idx = order[:, :k]
        sk = np.take_along_axis(keys, order, axis=1)
        margin = _adjacent_gap_min(sk, k)
        sel = np.take_along_axis(wl, idx, axis=1)
        m = sel.max(axis=1, keepdims=True)
        p = np.exp(sel - m)
        w = spec.route_scale * p / p.sum(axis=1, keepdims=True)
        return dict(topk_idx=idx, topk_w=w, s_sel=None, keys=keys, margin=margin)

    if spec.router == "sigmoid_grouped":
        lb = l + b if spec.bias_mode == "logit" else l          # biased logits
        s = sigmoid(lb)
        keys = s + b if spec.bias_mode == "select" else s.copy()
        G = spec.n_groups
        if E % G:
            raise ValueError("E must be a multiple of n_groups")
        per = E // G
        grouped = keys.reshape(T, G, per)
        top2 = -np.sort(-grouped, axis=2)[:, :, :2]
        gscore = top2.sum(axis=2) if per >= 2 else top2[:, :, 0]
        gorder = _desc_order(gscore)
        kept = gorder[:, :spec.topk_groups]
        if spec.topk_groups < G:
            sg = np.take_along_axis(gscore, gorder, axis=1)
            gmargin = sg[:, spec.topk_groups - 1] - sg[:, spec.topk_groups]
        else:
            gmargin = np.full(T, np.inf)
        allowed = np.zeros((T, G), dtype=bool)
        np.put_along_axis(allowed, kept, True, axis=1)
        allowed_e = np.repeat(allowed, per, axis=1)
        masked = np.where(allowed_e, keys, -np.inf)
        order = _desc_order(masked)
        idx = order[:, :k]
        n_cand = spec.topk_groups * per
        sk = np.take_along_axis(masked, order, axis=1)[:, :n_cand]
        margin = np.minimum(_adjacent_gap_min(sk, k), gmargin)
        ssel = np.take_along_axis(s, idx, axis=1)
        w = spec.route_scale * ssel / ssel.sum(axis=1, keepdims=True)
        return dict(topk_idx=idx, topk_w=w, s_sel=ssel, keys=keys, margin=margin)

    if spec.router == "sigmoid_threshold":
        if theta is None:
            raise ValueError("the threshold router needs theta")
        s = sigmoid(l)
        keys = l - np.asarray(theta, np.float64)[None, :]
        order = _desc_order(keys)
        cand = order[:, :k]
        sk = np.take_along_axis(keys, cand, axis=1)
        active = sk > 0.0
        active[:, 0] = True                  # the best expert even below its threshold
        idx = np.where(active, cand, -1)
        ssel = np.where(active, np.take_along_axis(s, cand, axis=1), 0.0)
        w = spec.route_scale * ssel / ssel.sum(axis=1, keepdims=True)
        sorted_keys = np.take_along_axis(keys, order, axis=1)
        margin = np.minimum(_adjacent_gap_min(sorted_keys, k), np.abs(sk).min(axis=1))
        return dict(topk_idx=idx, topk_w=w, s_sel=ssel, keys=keys, margin=margin)

    raise ValueError("unknown router " + spec.router)


# ----------------------------------------------------------------------------
# Permutation maps (stable counting sort by expert, then token)
# ----------------------------------------------------------------------------

def sort_maps(topk_idx, E):
    """Counts, offsets and the row maps of the expert-contiguous layout.

    counts[e] = number of (t, s) with topk_idx[t][s] == e;
    offsets[e] = sum of counts of experts below e (offsets[E] = T*k when
    every selected id is below E);
    the rows of expert e are offsets[e] .. offsets[e+1]-1, filled by
    ascending token t (a token holds an expert in at most one slot).  Slots
    whose expert is not below E (zero-computation experts) get no row:
    row_of = -1.
    """
    idx = np.asarray(topk_idx)
    T, k = idx.shape
    counts = np.zeros(E, dtype=np.int64)
    for e in idx.reshape(-1):
        if 0 <= e < E:
            counts[e] += 1
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    cursor = offsets[:-1].copy()
    row_of = np.full((T, k), -1, dtype=np.int64)   # -1: a slot without a row
    token_of = np.empty(int(offsets[E]), dtype=np.int64)
    for t in range(T):                       # ascending token: stable within expert
        for s in range(k):
            e = idx[t, s]
            if not 0 <= e < E:
                continue                     # an expert outside the E with rows
            r = cursor[e]
            cursor[e] += 1
            row_of[t, s] = r
            token_of[r] = t * k + s
    return dict(counts=counts, offsets=offsets, row_of=row_of, token_of=token_of)


def permute_rows(x, token_of, k):
    """x_perm[r] = x[token_of[r] // k]."""
    return np.asarray(x)[np.asarray(token_of) // k]


# ----------------------------------------------------------------------------
# SwiGLU expert
# ----------------------------------------------------------------------------

def glu(g, u, act=None):
    """The expert's gated activation h(g, u) and its partial derivatives.

    act None: SwiGLU, h = silu(g) u.
    act ("clamped_glu", alpha, limit): the GPT-OSS release's variant (the paper
      trains GPT-OSS-20B, section 5.1, without naming it): gc = min(g, limit),
      uc = clip(u, -limit, limit), h = gc sig(alpha gc) (uc + 1).  The clamps
      pass the gradient where the value lies inside them, bounds included.
    Returns h, dh/dg, dh/du (elementwise)."""
    if act is None:
        sg = sigmoid(g)
        return g * sg * u, u * sg * (1.0 + g * (1.0 - sg)), g * sg
    kind, alpha, limit = act
    if kind != "clamped_glu":
        raise ValueError("unknown activation " + str(kind))
    gc = np.minimum(g, limit)
    uc = np.clip(u, -limit, limit)
    s = sigmoid(alpha * gc)
    h = gc * s * (uc + 1.0)
    dgc = (uc + 1.0) * s * (1.0 + alpha * gc * (1.0 - s))
    return h, np.where(g <= limit, dgc, 0.0), np.where(np.abs(u) <= limit, gc * s, 0.0)


def expert_forward(xe, wg, wu, wd, bg=None, bu=None, bd=None, act=None):
    """g = x W_gate (+b_gate), u = x W_up (+b_up), h = act(g, u) (SwiGLU:
    silu(g) * u), o = h W_down (+b_down), for the rows xe [M][d]."""
    g = xe @ wg
    u = xe @ wu
    if bg is not None:
        g = g + bg
    if bu is not None:
        u = u + bu
    h = glu(g, u, act)[0]
    o = h @ wd
    if bd is not None:
        o = o + bd
    return g, u, h, o


def expert_backward(xe, g, u, h, do, wg, wu, wd, with_bias=False, act=None):
    """Gradients of sum(<do, o>) for one expert's rows.

    dh = do W_down^T; dW_down = h^T do; db_down = sum_rows do
    dg = dh * dh/dg, du = dh * dh/du (SwiGLU: dh/dg = u sig(g) (1 + g (1 - sig(g))),
    dh/du = silu(g));
    dW_gate = x^T dg; dW_up = x^T du; db_gate, db_up = row sums
    dx = dg W_gate^T + du W_up^T
    """
    dh = do @ wd.T
    _, hg, hu = glu(g, u, act)
    dg = dh * hg
    du = dh * hu
    out = dict(
        dw_down=h.T @ do,
        dw_gate=xe.T @ dg,
        dw_up=xe.T @ du,
        dx=dg @ wg.T + du @ wu.T,
        dg=dg, du=du,
    )
    if with_bias:
        out["db_down"] = do.sum(axis=0)
        out["db_gate"] = dg.sum(axis=0)
        out["db_up"] = du.sum(axis=0)
    return out


# ----------------------------------------------------------------------------
# Router backward
# ----------------------------------------------------------------------------

def router_backward(spec, rt, omega):
    """dL/dlogit on the selected experts, dl [T][k].

    omega[t][j] = dL/dw[t][j] = <dy_t, o_j(x_t)>.
    Softmax families, w_j = c * p_j with p the softmax over the selected
    (weight) logits:  dl_j = w_j * (omega_j - sum_i w_i omega_i / c).
    Sigmoid families, w_j = c * s_j / Z, Z = sum_S s over the selected (for
    the threshold router: active) slots:
        ds_j = (c * omega_j - sum_i w_i omega_i) / Z,  dl_j = ds_j s_j (1 - s_j)
    (an empty slot, s = 0, gets 0).  The bias has no gradient.
    """
    w = rt["topk_w"]
    c = spec.route_scale
    wo = (w * omega).sum(axis=1, keepdims=True)
    if spec.router in ("softmax_topk", "topk_softmax"):
        return w * (omega - wo / c)
    s = rt["s_sel"]
    Z = s.sum(axis=1, keepdims=True)
    ds = (c * omega - wo) / Z
    return ds * s * (1.0 - s)


def threshold_backward(spec, rt, omega, E):
    """dL/dtheta [E] of the threshold router, through a straight-through
    estimator of the activation indicator a_e = [logit_e - theta_e > 0]: the
    layer's output written as sum_e a_e c s_e o_e / sum_j a_j s_j gives
    dL/da_e = s_e (c omega_e - sum_j w_j omega_j) / Z on an active expert, and
    the estimator takes da_e/dtheta_e = -1 there.  Inactive experts, whose
    outputs are never computed, contribute nothing; the logits keep their exact
    gradient (router_backward)."""
    w, ssel, idx = rt["topk_w"], rt["s_sel"], rt["topk_idx"]
    c = spec.route_scale
    Z = ssel.sum(axis=1, keepdims=True)
    wo = (w * omega).sum(axis=1, keepdims=True)
    g = -ssel * (c * omega - wo) / Z
    dtheta = np.zeros(E)
    for t in range(idx.shape[0]):
        for j in range(idx.shape[1]):
            if idx[t, j] >= 0:
                dtheta[idx[t, j]] += g[t, j]
    return dtheta


# ----------------------------------------------------------------------------
# Combine and unpermute
# ----------------------------------------------------------------------------

def combine(o, topk_w, row_of, shared_o=None):
    """y_t = sum_s w[t][s] * o[row_of[t][s]] (+ shared_o[t]); slots without a
    row (row_of = -1) contribute nothing here."""
    T, k = topk_w.shape
    y = np.zeros((T, o.shape[1]))
    for s in range(k):
        has = row_of[:, s] >= 0
        y[has] += topk_w[has, s:s + 1] * o[row_of[has, s]]
    if shared_o is not None:
        y = y + shared_o
    return y


def combine_backward(dy, o, topk_w, row_of):
    """d_o[row_of[t][s]] = w[t][s] dy_t and omega[t][s] = <dy_t, o[row_of[t][s]]>
    (omega = 0 for a slot without a row)."""
    T, k = topk_w.shape
    omega = np.zeros((T, k))
    do = np.zeros_like(o, dtype=np.float64)
    for s in range(k):
        has = row_of[:, s] >= 0
        rows = row_of[has, s]
        omega[has, s] = (dy[has] * o[rows]).sum(axis=1)
        do[rows] = topk_w[has, s:s + 1] * dy[has]
    return do, omega


def unpermute(dx_perm, row_of):
    """dx_t = sum_s dx_perm[row_of[t][s]] over the slots that have a row."""
    T, k = row_of.shape
    dx = np.zeros((T, dx_perm.shape[1]))
    for s in range(k):
        has = row_of[:, s] >= 0
        dx[has] += dx_perm[row_of[has, s]]
    return dx


# ----------------------------------------------------------------------------
# Whole layer
# ----------------------------------------------------------------------------

def layer_forward(spec, x, w_r, beta, expert_fn, shared=None, aux_coef=0.0, aux_f=None, zc=None, act=None,
                  theta=None, fp8=False):
    """Forward of one MoE layer.

    x [T][d] float64; w_r [d][E_pool]; beta [E_pool] or None;
    expert_fn(e) -> (wg, wu, wd, bg, bu, bd) float64 (biases may be None);
    shared = (wsg, wsu, wsd) or None for an always-on expert of weight 1;
    aux_coef > 0 adds the load-balancing loss (aux_f: the batch's fractions);
    zc = (ZeroComputeSpec, v, wc) appends zero-computation experts to the pool
    (E_pool = spec.E + their number), else None (E_pool = spec.E);
    act: the routed experts' activation (None: SwiGLU; see glu);
    theta [E]: the threshold router's per-expert thresholds;
    fp8: the routed experts' GEMMs on E4M3 operands (see fp8_expert_forward).
    Returns routing, maps and the per-row activations (permuted order) and y
    (and the auxiliary loss, its probabilities and fractions).
    """
    x = np.asarray(x, np.float64)
    T, d = x.shape
    E, k = spec.E, spec.k
    E_pool = E + (zc[0].n if zc is not None else 0)
    if np.asarray(w_r).shape[1] != E_pool:
        raise ValueError("w_r must have one column per expert of the pool")
    l = router_logits(x, w_r)
    rt = route(spec, l, beta, theta)
    # rows over the whole pool: the FFN experts' rows come first (lower ids),
    # a zero-computation expert's rows carry no data
    mp = sort_maps(rt["topk_idx"], E_pool)
    mp["row_ffn"] = np.where(rt["topk_idx"] < E, mp["row_of"], -1)
    R = T * k
    x_perm = permute_rows(x, mp["token_of"][:mp["offsets"][E]], k)
    fwidth = None
    o = np.zeros((R, d))
    gs, us, hs = {}, {}, {}
    for e in range(E):
        r0, r1 = mp["offsets"][e], mp["offsets"][e + 1]
        if r1 == r0:
            continue
        wg, wu, wd, bg, bu, bd = expert_fn(e)
        fwd_fn = fp8_expert_forward if fp8 else expert_forward
        g, u, h, oe = fwd_fn(x_perm[r0:r1], wg, wu, wd, bg, bu, bd, act=act)
        gs[e], us[e], hs[e] = g, u, h
        o[r0:r1] = oe
        fwidth = wg.shape[1]
    sh = None
    if shared is not None:
        g, u, h, osh = expert_forward(x, *shared)
        sh = dict(g=g, u=u, h=h, o=osh)
    y = combine(o, rt["topk_w"], mp["row_ffn"], None if sh is None else sh["o"])
    zf = None
    if zc is not None:
        zf = zc_forward(x, rt["topk_idx"], rt["topk_w"], E, *zc)
        y = y + zf["y"]
    aux = None
    if aux_coef:
        probs = router_probs(spec, l, beta)
        eta = None if zc is None else zc_aux_weights(E, zc[0])
        aux = aux_loss(spec, probs, mp["counts"], aux_coef, aux_f, eta)
        aux.update(probs=probs, coef=aux_coef, eta=eta,
                   sig=sigmoid(l) if spec.router == "sigmoid_threshold" else None)
    return dict(logits=l, route=rt, maps=mp, x_perm=x_perm, o=o, g=gs, u=us,
                h=hs, y=y, shared=sh, f=fwidth, aux=aux, zc=zf)


def layer_backward(spec, x, w_r, beta, expert_fn, fwd, dy, shared=None, with_bias=False, zc=None, act=None,
                   fp8=False):
    """Backward of L = sum_t <dy_t, y_t> (+ the auxiliary loss) through the
    whole layer.

    Returns dx [T][d], dw_r [d][E_pool], per-expert dict of dW/db,
    shared-expert grads, omega [T][k], dl [T][k], with zc the
    zero-computation experts' dict (dv, dwc), and for the threshold router
    dtheta [E].  fp8: the routed experts' data-gradient products on E4M3
    operands (fp8_expert_backward).
    """
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    T, d = x.shape
    E, k = spec.E, spec.k
    E_pool = np.asarray(w_r).shape[1]
    rt, mp = fwd["route"], fwd["maps"]
    w = rt["topk_w"]
    o = fwd["o"]
    do, omega = combine_backward(dy, o, w, mp["row_ffn"])
    zb = None
    if zc is not None:
        zb = zc_backward(dy, x, rt["topk_idx"], w, E, *zc)
        omega = omega + zb["omega"]
    # experts
    dx = np.zeros((T, d))
    dx_perm = np.zeros((T * k, d))
    grads = {}
    for e in range(E):
        r0, r1 = mp["offsets"][e], mp["offsets"][e + 1]
        wg, wu, wd, bg, bu, bd = expert_fn(e)
        if r1 == r0:
            grads[e] = dict(dw_gate=np.zeros_like(wg), dw_up=np.zeros_like(wu),
                            dw_down=np.zeros_like(wd))
            if with_bias:
                grads[e].update(db_gate=np.zeros(wg.shape[1]), db_up=np.zeros(wu.shape[1]),
                                db_down=np.zeros(wd.shape[1]))
            continue
        bwd_fn = fp8_expert_backward if fp8 else expert_backward
        ge = bwd_fn(fwd["x_perm"][r0:r1], fwd["g"][e], fwd["u"][e], fwd["h"][e],
                    do[r0:r1], wg, wu, wd, with_bias=with_bias, act=act)
        dx_perm[r0:r1] = ge.pop("dx")
        ge.pop("dg")
        ge.pop("du")
        grads[e] = ge
    dx += unpermute(dx_perm, mp["row_ffn"])
    # router
    dl = router_backward(spec, rt, omega)
    dl_dense = _scatter_slots(dl, rt["topk_idx"], E_pool)
    aux = fwd.get("aux")
    if aux is not None:
        dl_dense = dl_dense + aux_loss_backward(aux["probs"], aux["f"], aux["coef"], aux.get("eta"),
                                                aux.get("sig"))
    dw_r = x.T @ dl_dense
    dx_router = dl_dense @ np.asarray(w_r, np.float64).T
    dx += dx_router
    if zb is not None:
        dx += zb["dx"]
    sh = None
    if shared is not None:
        wsg, wsu, wsd = shared
        s_ = fwd["shared"]
        gsh = expert_backward(x, s_["g"], s_["u"], s_["h"], dy, wsg, wsu, wsd)
        dx += gsh.pop("dx")
        gsh.pop("dg")
        gsh.pop("du")
        sh = gsh
    dtheta = threshold_backward(spec, rt, omega, E) if spec.router == "sigmoid_threshold" else None
    return dict(dx=dx, dw_r=dw_r, experts=grads, shared=sh, omega=omega, dl=dl,
                dx_perm=dx_perm, do=do, dx_router=dx_router,
                zc=None if zb is None else dict(dv=zb["dv"], dwc=zb["dwc"]), dtheta=dtheta)


def _scatter_slots(v, idx, E):
    """dense [T][E] with v[t][s] at column idx[t][s] (empty slots, idx < 0, dropped)."""
    out = np.zeros((idx.shape[0], E))
    t, s = np.nonzero(idx >= 0)
    out[t, idx[t, s]] = v[t, s]
    return out


# ----------------------------------------------------------------------------
# Load-balancing auxiliary loss, global level
# ----------------------------------------------------------------------------
# The paper pretrains Qwen3-30B-A3B with a global-level load-balancing loss of
# coefficient 1e-3 (appendix A.1, training-configuration figure) and defers its
# definition to the work it cites.  Written out here as that standard loss:
# over the batch, L = coef * E * sum_e f_e P_e, with P_e the mean over tokens of
# the router's probability of expert e (softmax over all E logits) and f_e the
# fraction of the T*k routed slots that chose e; "global level" means f_e is
# taken over the whole batch, so a caller splitting a batch can pass the
# batch's f.  f is a count and carries no gradient.  Softmax routers only.

def router_probs(spec, logits, beta=None):
    """p [T][E]: softmax over all E experts of the logits (plus beta when the
    bias is added to the logits); for the threshold router the sigmoid scores
    normalised over all experts, p_e = s_e / sum_j s_j (its variable-k form:
    the gates are independent sigmoids, their shares are what balance)."""
    if spec.router == "sigmoid_grouped":
        raise ValueError("the auxiliary loss is defined for the softmax and threshold routers")
    if spec.router == "sigmoid_threshold":
        sg = sigmoid(np.asarray(logits, np.float64))
        return sg / sg.sum(axis=1, keepdims=True)
    v = np.asarray(logits, np.float64)
    if beta is not None and spec.bias_mode == "logit":
        v = v + np.asarray(beta, np.float64)[None, :]
    z = np.exp(v - v.max(axis=1, keepdims=True))
    return z / z.sum(axis=1, keepdims=True)


def aux_loss(spec, p, counts, coef, f=None, eta=None):
    """Global-level load-balancing loss.  p [T][E] from router_probs; counts
    [E] routed slots per expert; f [E] the batch's fractions if given, else
    counts / (T*k); eta [E] per-expert weights of the balance terms (None:
    all one), L = coef * E * sum_e eta_e f_e P_e.  Returns dict(loss, P, f)."""
    p = np.asarray(p, np.float64)
    T, E = p.shape
    if f is None:
        # the routed slots: T*k, or for the threshold router (a variable number
        # of experts per token) the slots actually filled
        n = float(np.sum(counts)) if spec.router == "sigmoid_threshold" else float(T * spec.k)
        f = np.asarray(counts, np.float64) / max(n, 1.0)
    f = np.asarray(f, np.float64)
    ef = f if eta is None else np.asarray(eta, np.float64) * f
    P = p.mean(axis=0)
    return dict(loss=coef * E * float(np.dot(ef, P)), P=P, f=f)


def aux_loss_backward(p, f, coef, eta=None, sig=None):
    """dL/dlogit [T][E] of aux_loss with f held fixed: through P_e = mean_t
    p[t][e] and the softmax Jacobian dp_e/dl_j = p_e (delta_ej - p_j), with
    q = eta * f (q = f without weights),
    dl[t][j] = coef * E / T * p[t][j] * (q_j - sum_e q_e p[t][e]).
    sig: the sigmoid scores of the threshold router, whose p = s / sum s has
    dp_e/dl_j = p_e (delta_ej - p_j) (1 - s_j), so the same expression carries
    the factor (1 - s_j)."""
    p = np.asarray(p, np.float64)
    T, E = p.shape
    q = np.asarray(f, np.float64)
    if eta is not None:
        q = np.asarray(eta, np.float64) * q
    F = p @ q
    dl = coef * E / T * p * (q[None, :] - F[:, None])
    return dl if sig is None else dl * (1.0 - np.asarray(sig, np.float64))


# ----------------------------------------------------------------------------
# Evaluation of a layer too large to run whole
# ----------------------------------------------------------------------------

def token_forward_backward(spec, x, dy, w_r, beta, expert_fn, shared=None, zc=None, act=None, theta=None,
                           fp8=0):
    """Every per-token result of the layer for a batch of tokens: routing, y,
    omega, dl and dx (no weight gradients).

    Routing, the combine, the expert rows and the input gradient of a token
    depend only on that token, so running the plain definitions on a subset
    of the tokens gives exactly their values in the whole layer.  Experts are
    visited in ascending order, each once, with all of the batch's tokens
    that selected it.  dl_dense [T][E] holds dl at the selected experts and
    zero elsewhere: for a batch that contains every token routed to expert e,
    column e of dW_r is x_batch^T dl_dense[:, e].  fp8: 1 the experts' forward
    products on E4M3 operands, 2 their data-gradient products too (the row
    quantisation of x, h, d_o and [dg | du] is per token, the weights'
    quantisation per column or row of the whole weight).
    """
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    T, d = x.shape
    E, k = spec.E, spec.k
    E_pool = np.asarray(w_r).shape[1]
    rt = route(spec, router_logits(x, w_r), beta, theta)
    idx, w = rt["topk_idx"], rt["topk_w"]
    y = np.zeros((T, d))
    dx = np.zeros((T, d))
    omega = np.zeros((T, k))
    if zc is not None:
        y += zc_forward(x, idx, w, E, *zc)["y"]
        zb = zc_backward(dy, x, idx, w, E, *zc)
        omega += zb["omega"]
        dx += zb["dx"]
    for e in np.unique(idx):
        if e >= E or e < 0:
            continue                         # zero-computation experts (above), empty slots
        t, s = np.nonzero(idx == e)          # a token holds e in at most one slot
        wg, wu, wd, bg, bu, bd = expert_fn(int(e))
        g, u, h, o = (fp8_expert_forward if fp8 else expert_forward)(x[t], wg, wu, wd, bg, bu, bd, act=act)
        we = w[t, s][:, None]
        y[t] += we * o
        omega[t, s] = (dy[t] * o).sum(axis=1)
        bwd_fn = fp8_expert_backward if fp8 == 2 else expert_backward
        dx[t] += bwd_fn(x[t], g, u, h, we * dy[t], wg, wu, wd, act=act)["dx"]
    dl = router_backward(spec, rt, omega)
    dl_dense = _scatter_slots(dl, idx, E_pool)
    dx += dl_dense @ np.asarray(w_r, np.float64).T
    if shared is not None:
        g, u, h, osh = expert_forward(x, *shared)
        y += osh
        dx += expert_backward(x, g, u, h, dy, *shared)["dx"]
    return dict(route=rt, y=y, dx=dx, omega=omega, dl=dl, dl_dense=dl_dense)


def expert_weight_grads_at(xe, do, wg, wu, wd, bg=None, bu=None, cols=None, with_bias=False, act=None, fp8=0):
    """Weight gradients of one expert restricted to the intermediate indices
    `cols`: dW_gate[:, cols], dW_up[:, cols], dW_down[cols, :] (and db_gate,
    db_up at cols, db_down whole).

    Along the intermediate axis the SwiGLU expert is a set of independent
    columns (g_j, u_j and h_j use only column j of W_gate and W_up, and
    dh_j only row j of W_down), so the plain expert forward and backward on
    the sliced weights give exactly those slices of the full gradients.
    xe [M][d] are the expert's rows and do [M][d] their output gradients.
    fp8 (1: forward products on E4M3 operands, 2: data-gradient products too)
    keeps this: x and d_o are quantised per row over d, W_gate and W_up per
    column, W_down per row (fp8 = 2), so g_j, u_j, h_j and dh_j still use only
    column j (the quantisation of h and [dg | du] rows spans every column, but
    feeds only o and dx, which are not returned).
    """
    cols = np.asarray(cols)
    wg_c, wu_c, wd_c = wg[:, cols], wu[:, cols], wd[cols, :]
    fwd_fn = fp8_expert_forward if fp8 else expert_forward
    bwd_fn = fp8_expert_backward if fp8 == 2 else expert_backward
    g, u, h, _ = fwd_fn(xe, wg_c, wu_c, wd_c,
                        None if bg is None else bg[cols], None if bu is None else bu[cols], act=act)
    out = bwd_fn(xe, g, u, h, do, wg_c, wu_c, wd_c, with_bias=with_bias, act=act)
    out.pop("dx")
    out.pop("dg")
    out.pop("du")
    return out


# ----------------------------------------------------------------------------
# Zero-computation experts (MoE++)
# ----------------------------------------------------------------------------
# Appendix B.3 describes the MoE++ task: the expert pool gains three kinds of
# experts that do no feed-forward work (zero, copy, constant), the router's
# output widens to cover them, and the load-balancing loss treats them
# explicitly.  The expert functions are the ones of the MoE++ work it cites,
# written out here:
#   zero      out(x) = 0
#   copy      out(x) = x
#   constant  out(x) = a0 x + a1 v,  (a0, a1) = softmax(W_c x),
#             with a trainable vector v [d] and matrix W_c [2][d] per expert.
# Pool order: the E FFN experts (ids 0 .. E-1), then n_zero zero, n_copy copy
# and n_const constant experts.  The router is the layer's softmax router
# over the whole pool; a slot that picks a zero-computation expert adds
# w * out(x_t) to y_t.  The permutation sorts every slot of the pool by
# (expert, token), so the FFN experts' rows come first; a zero-computation
# expert's rows only list its tokens (no activations are copied there).  In the balance
# loss every zero-computation expert's term carries the weight aux_weight
# (1: the plain loss over the pool, 0: excluded), FFN experts weight 1.

@dataclass
class ZeroComputeSpec:
    n_zero: int = 0
    n_copy: int = 0
    n_const: int = 0
    aux_weight: float = 1.0

    @property
    def n(self):
        return self.n_zero + self.n_copy + self.n_const


def zc_kind(e, E, zs):
    """('ffn' | 'zero' | 'copy' | 'const', index within its kind) of pool id e."""
    if e < E:
        return "ffn", e
    j = e - E
    if j < zs.n_zero:
        return "zero", j
    j -= zs.n_zero
    if j < zs.n_copy:
        return "copy", j
    j -= zs.n_copy
    if j < zs.n_const:
        return "const", j
    raise ValueError("expert id outside the pool")


def zc_aux_weights(E, zs):
    """eta [E_pool]: 1 for the FFN experts, aux_weight for the others."""
    return np.concatenate([np.ones(E), np.full(zs.n, float(zs.aux_weight))])


def zc_const_alpha(x_t, wc_c):
    """(a0, a1) = softmax(W_c x_t) for one token and one constant expert."""
    z = np.asarray(wc_c, np.float64) @ np.asarray(x_t, np.float64)
    ez = np.exp(z - z.max())
    return ez / ez.sum()


def zc_forward(x, topk_idx, topk_w, E, zs, v, wc):
    """y_zc[t] = sum over the slots s of token t whose expert is a
    zero-computation one of w[t][s] * out(x_t).  v [n_const][d],
    wc [n_const][2][d].  Returns dict(y, alpha [T][k][2], nan where the slot
    is not a constant expert)."""
    x = np.asarray(x, np.float64)
    T, d = x.shape
    k = topk_idx.shape[1]
    y = np.zeros((T, d))
    alpha = np.full((T, k, 2), np.nan)
    for t in range(T):
        for s in range(k):
            kind, c = zc_kind(int(topk_idx[t, s]), E, zs)
            wts = topk_w[t, s]
            if kind == "copy":
                y[t] += wts * x[t]
            elif kind == "const":
                a = zc_const_alpha(x[t], wc[c])
                alpha[t, s] = a
                y[t] += wts * (a[0] * x[t] + a[1] * np.asarray(v[c], np.float64))
    return dict(y=y, alpha=alpha)


def zc_backward(dy, x, topk_idx, topk_w, E, zs, v, wc):
    """Gradients of sum_t <dy_t, y_zc[t]> with the gating weights held fixed,
    and omega = dL/dw on the zero-computation slots.

    Per slot with g = w dy_t:
      copy:     omega = <dy_t, x_t>,  dx_t += g
      constant: out = a0 x + a1 v, omega = <dy_t, out>;
                da = (<g, x_t>, <g, v>), dz = a * (da - <a, da>) (softmax
                Jacobian), dx_t += a0 g + W_c^T dz, dv += a1 g, dW_c += dz x_t^T
      zero:     nothing.
    Returns dict(omega [T][k] (zero on FFN slots), dx [T][d],
    dv [n_const][d], dwc [n_const][2][d])."""
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    T, d = x.shape
    k = topk_idx.shape[1]
    omega = np.zeros((T, k))
    dx = np.zeros((T, d))
    dv = np.zeros((zs.n_const, d))
    dwc = np.zeros((zs.n_const, 2, d))
    for t in range(T):
        for s in range(k):
            kind, c = zc_kind(int(topk_idx[t, s]), E, zs)
            g = topk_w[t, s] * dy[t]
            if kind == "copy":
                omega[t, s] = float(dy[t] @ x[t])
                dx[t] += g
            elif kind == "const":
                vc = np.asarray(v[c], np.float64)
                wcc = np.asarray(wc[c], np.float64)
                a = zc_const_alpha(x[t], wcc)
                omega[t, s] = float(dy[t] @ (a[0] * x[t] + a[1] * vc))
                da = np.array([g @ x[t], g @ vc])
                dz = a * (da - a @ da)
                dx[t] += a[0] * g + wcc.T @ dz
                dv[c] += a[1] * g
                dwc[c] += np.outer(dz, x[t])
    return dict(omega=omega, dx=dx, dv=dv, dwc=dwc)


# ----------------------------------------------------------------------------
# FP8 forward of the expert GEMMs
# ----------------------------------------------------------------------------
# The paper trains with FP8 GEMMs (the Qwen3 FP8 row of its B200 results; its
# framework fuses the quantisation and caches quantised weights across
# micro-batches) without stating the scaling recipe.  Reading written out
# here: OCP FP8 E4M3 (1 sign, 4 exponent bits of bias 7, 3 mantissa bits, no
# infinities, largest finite 448); each row of an activation operand (a token
# row of x_perm, or of h) gets the scale amax_row / 448 and each output column
# of a weight matrix the scale amax_column / 448; a value v of a row with
# largest magnitude amax is stored as the E4M3 value nearest to
# min(max(v * (448 / amax), -448), 448), ties to the even mantissa, where
# 448 / amax and the product are float32 operations (the quantised codes are
# decided in float32 on both sides); an all-zero row or column gets scale 1.
# The activations are quantised from their stored bf16 values (FP8 runs bf16
# layers): x is stored bf16 already, h is rounded to float32 and then to bf16
# (nearest even) before its row is quantised.  The GEMMs multiply the
# dequantised operands (code value times scale).  With FP8 forward GEMMs only,
# the backward uses the bf16 operands and weights as if the quantisation were
# the identity (straight-through), with the activations gu and h of the FP8
# forward.  With FP8 data-gradient GEMMs as well (fp8_expert_backward), the two
# products that carry the gradient back to the input, dh = d_o W_down^T and
# dx = [dg | du] [W_gate | W_up]^T, take E4M3 operands quantised in the same
# way: the stored bf16 rows of d_o and of [dg | du] per row (one scale over a
# row's gate and up halves together), W_down per row (an output column of dh)
# and the concatenated rows of [W_gate | W_up] per row (an output column of dx,
# again one scale over both halves).  The weight-gradient products stay on the
# unquantised operands.  The smooth factors of the activation's derivative are
# evaluated at g and u as a bf16 layer stores them (rounded to nearest even), so
# that the codes of [dg | du] are decided on the values a bf16 layer holds, as
# the codes of h are; the clamped GLU's clamp masks (which values pass a
# gradient) are those of the forward's own values g and u: a clamp's derivative
# belongs to the value it clamped, not to its stored rounding.

_E4M3_MAX = 448.0


def e4m3_values():
    """The 256 E4M3 codes' values (NaN for the two NaN codes), float64."""
    out = np.empty(256)
    for code in range(256):
        s = -1.0 if code & 0x80 else 1.0
        e = (code >> 3) & 0xF
        m = code & 0x7
        if e == 0xF and m == 0x7:
            out[code] = np.nan
        elif e == 0:
            out[code] = s * m * 2.0 ** -9
        else:
            out[code] = s * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return out


_E4M3 = None


def e4m3_round(v):
    """Codes (uint8) of the E4M3 values nearest to v (|v| <= 448 assumed),
    ties to the even code (the even mantissa), the sign of v kept (a negative
    value that rounds to zero gives -0)."""
    global _E4M3
    if _E4M3 is None:
        _E4M3 = e4m3_values()
    v = np.asarray(v, np.float64)
    pos = np.arange(0, 127)                      # finite non-negative codes 0x00..0x7e
    pv = _E4M3[pos]
    a = np.abs(v).reshape(-1)
    # nearest by distance; ties to the even code
    idx = np.searchsorted(pv, a)                 # pv ascending
    lo = np.clip(idx - 1, 0, len(pv) - 1)
    hi = np.clip(idx, 0, len(pv) - 1)
    dlo = a - pv[lo]
    dhi = pv[hi] - a
    pick = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(pos[lo] % 2 == 0, lo, hi)))
    code = pos[pick].astype(np.uint8)
    neg = np.signbit(v.reshape(-1))              # the sign is kept, also on a zero result
    code = np.where(neg, code | 0x80, code).astype(np.uint8)
    return code.reshape(np.shape(v))


def quantize_rows(a):
    """Row-wise E4M3 quantisation: (codes [M][K] uint8, scale [M] float64 of the
    float32 scale amax/448, dequantised values [M][K])."""
    a32 = np.asarray(a, np.float32)
    amax = np.abs(a32).max(axis=1) if a32.shape[1] else np.zeros(a32.shape[0], np.float32)
    amax = np.where(amax > 0, amax, np.float32(_E4M3_MAX)).astype(np.float32)   # all-zero row: scale 1
    inv = (np.float32(_E4M3_MAX) / amax).astype(np.float32)
    x = (a32 * inv[:, None]).astype(np.float32)
    x = np.clip(x, np.float32(-_E4M3_MAX), np.float32(_E4M3_MAX))
    codes = e4m3_round(x.astype(np.float64))
    scale = (amax / np.float32(_E4M3_MAX)).astype(np.float32).astype(np.float64)
    vals = e4m3_values()[codes] * scale[:, None]
    return codes, scale, vals


def quantize_cols(w):
    """Column-wise quantisation of a weight [K][N] (each output column its scale):
    (codes [K][N], scale [N], dequantised [K][N])."""
    c, s, v = quantize_rows(np.asarray(w).T)
    return c.T, s, v.T


def round_bf16(a):
    """float64 values rounded to float32, then to bfloat16 (nearest, ties to
    even), returned as float64."""
    u = np.ascontiguousarray(np.asarray(a, np.float32)).view(np.uint32)
    r = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)) << np.uint32(16)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def fp8_expert_forward(xe, wg, wu, wd, bg=None, bu=None, bd=None, act=None):
    """expert_forward with both GEMMs on E4M3 operands: x rows and the stored
    (bf16) h rows quantised per row, the weights per output column."""
    _, _, xq = quantize_rows(xe)
    _, _, wgq = quantize_cols(wg)
    _, _, wuq = quantize_cols(wu)
    _, _, wdq = quantize_cols(wd)
    g = xq @ wgq
    u = xq @ wuq
    if bg is not None:
        g = g + bg
    if bu is not None:
        u = u + bu
    h = glu(g, u, act)[0]
    _, _, hq = quantize_rows(round_bf16(h))
    o = hq @ wdq
    if bd is not None:
        o = o + bd
    return g, u, h, o


def fp8_expert_backward(xe, g, u, h, do, wg, wu, wd, with_bias=False, act=None):
    """expert_backward with its two data-gradient products on E4M3 operands:
    dh from the row-quantised stored d_o and W_down, dx from the row-quantised
    stored [dg | du] and [W_gate | W_up]; the activation's smooth derivative
    factors at the stored (bf16) g and u, the clamp masks of the clamped GLU at
    the forward's g and u; the weight gradients from the unquantised d_o and
    the resulting dg, du (see the comment above e4m3_values)."""
    _, _, doq = quantize_rows(round_bf16(do))
    _, _, wdq = quantize_rows(wd)                        # [f][d]: a scale per output column j of dh
    dh = doq @ wdq.T
    gs, us = round_bf16(g), round_bf16(u)
    if act is None:
        _, hg, hu = glu(gs, us)
    else:
        # the smooth factors at the stored values (gc, uc clipped as in the
        # forward) ...
        kind, alpha, lim = act
        if kind != "clamped_glu":
            raise ValueError("unknown activation " + str(kind))
        gc = np.minimum(gs, lim)
        uc = np.clip(us, -lim, lim)
        sg = sigmoid(alpha * gc)
        # ... and the masks of the forward's own g, u (bounds included)
        hg = np.where(g <= lim, (uc + 1.0) * sg * (1.0 + alpha * gc * (1.0 - sg)), 0.0)
        hu = np.where(np.abs(u) <= lim, gc * sg, 0.0)
    dg = dh * hg
    du = dh * hu
    _, _, dguq = quantize_rows(round_bf16(np.concatenate([dg, du], axis=1)))
    _, _, wguq = quantize_rows(np.concatenate([wg, wu], axis=1))   # [d][2f]: a scale per output column of dx
    out = dict(
        dw_down=h.T @ do,
        dw_gate=xe.T @ dg,
        dw_up=xe.T @ du,
        dx=dguq @ wguq.T,
        dg=dg, du=du,
    )
    if with_bias:
        out["db_down"] = do.sum(axis=0)
        out["db_gate"] = dg.sum(axis=0)
        out["db_up"] = du.sum(axis=0)
    return out
