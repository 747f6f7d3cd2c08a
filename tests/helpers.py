"""Shared test plumbing: seeded inputs to device tensors, oracle runs, and the
parity measures (normwise relative error; routing equality outside the 1e-6
top-k margin)."""
import numpy as np

from moe_inputs import f32_from_bf16_bits, layer_inputs, to_f64
from oracle import ZeroComputeSpec, layer_backward, layer_forward, spec_from_config

MARGIN = 1e-6
TOL = {"bf16": 2e-2, "f32": 1e-4}


def dev(a, dtype):
    """Storage array (bf16 bit patterns or float32) -> torch tensor on cuda:0."""
    import torch
    if a is None:
        return None
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t):
    """torch tensor (any device) -> numpy float64 (bf16 read exactly)."""
    import torch
    if t is None:
        return None
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return f32_from_bf16_bits(t.view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    if t.dtype in (torch.int32, torch.int64):
        return t.numpy()
    return t.float().numpy().astype(np.float64)


def rel(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    nr = np.linalg.norm(ref)
    if nr == 0:
        return float(np.linalg.norm(gpu))
    return float(np.linalg.norm(gpu - ref) / nr)


ROW_FLOOR = 0.05


def row_rel(gpu, ref, rows=None):
    """Largest per-row normwise error: the maximum over rows r of
    ||gpu_r - ref_r|| / max(||ref_r||, floor), floor = ROW_FLOOR times the RMS of
    the reference's row norms (a row far below the typical size is measured
    against 5% of that size).  rows: optional mask or indices of the rows to
    compare.  One wrong row (a token of y or dx, a permuted row of o or dx_perm)
    shows here at full weight, where the whole-tensor measure would dilute it
    by the square root of the row count."""
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    g = g.reshape(g.shape[0], -1)
    r = r.reshape(r.shape[0], -1)
    if rows is not None:
        g, r = g[rows], r[rows]
    if r.shape[0] == 0:
        return 0.0
    nr = np.linalg.norm(r, axis=1)
    nd = np.linalg.norm(g - r, axis=1)
    floor = ROW_FLOOR * float(np.sqrt(np.mean(nr ** 2)))
    if floor == 0.0:
        return float(nd.max())
    return float((nd / np.maximum(nr, floor)).max())


def group_rel(gpu, ref):
    """Largest normwise error over the leading index (one expert's gradient per
    index): max_e rel(gpu[e], ref[e]); an expert whose reference is zero (no
    rows) counts the norm of the device value, which must then be 0."""
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    return max((rel(g[e], r[e]) for e in range(r.shape[0])), default=0.0)


def expert_fn(inp, cfg):
    dt = cfg["dtype"]

    def fn(e):
        b = cfg["expert_bias"]
        return (to_f64(inp["w_gate"][e], dt), to_f64(inp["w_up"][e], dt), to_f64(inp["w_down"][e], dt),
                to_f64(inp["b_gate"][e], dt) if b else None,
                to_f64(inp["b_up"][e], dt) if b else None,
                to_f64(inp["b_down"][e], dt) if b else None)
    return fn


def shared_of(inp, cfg):
    if not cfg["n_shared"]:
        return None
    dt = cfg["dtype"]
    return (to_f64(inp["ws_gate"], dt), to_f64(inp["ws_up"], dt), to_f64(inp["ws_down"], dt))


def zc_of(inp, cfg):
    """(ZeroComputeSpec, v, W_c) of a config with zero-computation experts, else None."""
    nz, ncp, nc = cfg.get("n_zero", 0), cfg.get("n_copy", 0), cfg.get("n_const", 0)
    if nz + ncp + nc == 0:
        return None
    zs = ZeroComputeSpec(n_zero=nz, n_copy=ncp, n_const=nc, aux_weight=cfg.get("zc_aux_weight", 1.0))
    d = cfg["d"]
    v = inp["zc_v"].astype(np.float64) if nc else np.zeros((0, d))
    wc = inp["zc_wc"].astype(np.float64) if nc else np.zeros((0, 2, d))
    return (zs, v, wc)


def oracle_run(cfg, inp, aux_coef=0.0, aux_f=None):
    spec = spec_from_config(cfg)
    dt = cfg["dtype"]
    x = to_f64(inp["x"], dt)
    w_r = inp["w_r"].astype(np.float64)
    beta = None if inp["router_bias"] is None else inp["router_bias"].astype(np.float64)
    efn = expert_fn(inp, cfg)
    shared = shared_of(inp, cfg)
    zc = zc_of(inp, cfg)
    act = act_of(cfg)
    theta = None if inp.get("gate_threshold") is None else inp["gate_threshold"].astype(np.float64)
    fwd = layer_forward(spec, x, w_r, beta, efn, shared, aux_coef=aux_coef, aux_f=aux_f, zc=zc, act=act,
                        theta=theta, fp8=bool(cfg.get("fp8", 0)))
    bwd = layer_backward(spec, x, w_r, beta, efn, fwd, to_f64(inp["dy"], dt), shared,
                         with_bias=cfg["expert_bias"], zc=zc, act=act, fp8=cfg.get("fp8", 0) == 2)
    return fwd, bwd


def act_of(cfg):
    """The oracle's activation argument for a config (None: SwiGLU)."""
    if cfg.get("act", "swiglu") == "swiglu":
        return None
    return (cfg["act"], float(np.float32(cfg["act_alpha"])), float(np.float32(cfg["act_limit"])))


def device_params(inp, cfg):
    import torch
    dt = cfg["dtype"]
    p = dict(
        w_r=torch.from_numpy(inp["w_r"]).cuda(),
        router_bias=None if inp["router_bias"] is None else torch.from_numpy(inp["router_bias"]).cuda(),
        w_gate=dev(inp["w_gate"], dt), w_up=dev(inp["w_up"], dt), w_down=dev(inp["w_down"], dt),
        b_gate=dev(inp.get("b_gate"), dt), b_up=dev(inp.get("b_up"), dt), b_down=dev(inp.get("b_down"), dt),
        ws_gate=dev(inp.get("ws_gate"), dt), ws_up=dev(inp.get("ws_up"), dt), ws_down=dev(inp.get("ws_down"), dt),
        zc_v=None if inp.get("zc_v") is None else torch.from_numpy(inp["zc_v"]).cuda(),
        zc_wc=None if inp.get("zc_wc") is None else torch.from_numpy(inp["zc_wc"]).cuda(),
        gate_threshold=None if inp.get("gate_threshold") is None else torch.from_numpy(inp["gate_threshold"]).cuda(),
    )
    return p


def check_routing(cfg, fwd, topk_idx_gpu):
    """Routing parity: equal outside the margin.  Returns (ambiguous mask, all_equal)."""
    ref = fwd["route"]["topk_idx"]
    amb = fwd["route"]["margin"] < MARGIN
    gpu = np.asarray(topk_idx_gpu)
    same = np.all(gpu == ref, axis=1)
    bad = np.where(~same & ~amb)[0]
    assert bad.size == 0, "topk_idx differs on %d non-ambiguous tokens, first %s: gpu %s oracle %s" % (
        bad.size, bad[:5], gpu[bad[0]], ref[bad[0]])
    return amb, bool(np.all(same))


def check_maps_valid(topk_idx, offsets, row_of, token_of, E):
    """Maps are the stable (expert, token) counting sort of the given topk_idx
    (empty slots, id -1, get no row)."""
    T, k = topk_idx.shape
    flat = topk_idx.reshape(-1)
    filled = np.nonzero(flat >= 0)[0]
    n = filled.size
    counts = np.bincount(flat[filled], minlength=E)
    assert np.array_equal(np.diff(offsets), counts)
    assert offsets[0] == 0 and offsets[E] == n
    token_of = token_of[:n]
    assert np.array_equal(np.sort(token_of), filled)
    t_of = token_of // k
    s_of = token_of % k
    assert np.array_equal(topk_idx[t_of, s_of], np.repeat(np.arange(E), counts))
    for e in range(E):
        seg = t_of[offsets[e]:offsets[e + 1]]
        assert np.all(np.diff(seg) > 0)
    assert np.array_equal(row_of[t_of, s_of], np.arange(n))
    assert np.all(row_of.reshape(-1)[flat < 0] == -1)


def small_inputs(cfg, seed=0):
    return layer_inputs(cfg, seed=seed)
