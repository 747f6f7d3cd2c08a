"""Seeded generators for the MoE layer inputs.

Recipe (one child stream per tensor slice):
  * stream = PCG64(SeedSequence([seed, cfg_id, tensor_id, slice_id])), drawn
    with standard_normal in float32 and scaled by the tensor's standard
    deviation in float32;
  * per-expert tensors (w_gate, w_up, w_down, b_*) use slice_id = expert;
  * token-major tensors (x, dy) use one slice per block of ROW_BLOCK rows;
  * bf16 tensors are rounded from that float32 value to nearest-even and kept
    as their 16-bit patterns (numpy has no bf16); fp32 tensors stay float32;
  * the router weight W_r [d][E] and any router bias are always fp32.

Distributions follow the workload statement: x ~ N(0,1), W_r ~ N(0,0.02),
expert weights and biases ~ N(0,0.02), DeepSeek-style selection bias
~ N(0,0.1), upstream gradient dy ~ N(0,1) (the second argument of N is the
standard deviation); constant zero-computation experts: v ~ N(0,1),
W_c ~ N(0,0.02), both float32; the threshold router's thresholds
~ N(theta_mean, theta_std) float32.  The stress config's logit bias is stored data (see
``stress_router_bias``).
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import TENSOR_IDS

ROW_BLOCK = 256
_HERE = os.path.dirname(os.path.abspath(__file__))
STRESS_BIAS_FILE = os.path.join(_HERE, "stress_bias_seed0.txt")


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def bf16_bits_from_f32(a):
    """Round float32 values to bfloat16 (nearest, ties to even); 16-bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def f32_from_bf16_bits(b):
    """Exact float32 values of bfloat16 bit patterns."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_f64(a, dtype):
    """Exact float64 values of a stored tensor ('bf16' bit patterns or 'f32')."""
    if a is None:
        return None
    if dtype == "bf16":
        return f32_from_bf16_bits(a).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def _stream(seed, cfg_id, tensor, slice_id):
    ss = np.random.SeedSequence([int(seed), int(cfg_id), TENSOR_IDS[tensor], int(slice_id)])
    return np.random.Generator(np.random.PCG64(ss))


def _draw(seed, cfg_id, tensor, slice_id, shape, std):
    g = _stream(seed, cfg_id, tensor, slice_id)
    z = g.standard_normal(size=shape, dtype=np.float32)
    z *= np.float32(std)
    return z


def _store(a32, dtype):
    return bf16_bits_from_f32(a32) if dtype == "bf16" else a32


def gen_tensor(seed, cfg, tensor, shape, std, dtype, slice_id=0):
    """One tensor slice in its storage format (bf16 bits or float32)."""
    return _store(_draw(seed, cfg["cfg_id"], tensor, slice_id, shape, std), dtype)


def gen_rows(seed, cfg, tensor, rows, width, std, dtype, threads=None):
    """A token-major tensor [rows][width], one child stream per ROW_BLOCK rows."""
    nblk = (rows + ROW_BLOCK - 1) // ROW_BLOCK
    out = np.empty((rows, width), dtype=np.uint16 if dtype == "bf16" else np.float32)

    def one(b):
        r0 = b * ROW_BLOCK
        r1 = min(rows, r0 + ROW_BLOCK)
        out[r0:r1] = gen_tensor(seed, cfg, tensor, (r1 - r0, width), std, dtype, slice_id=b)

    with ThreadPoolExecutor(threads or _threads()) as ex:
        list(ex.map(one, range(nblk)))
    return out


def _expert_shape(cfg, tensor):
    d, f = cfg["d"], cfg["f"]
    return {"w_gate": (d, f), "w_up": (d, f), "w_down": (f, d),
            "b_gate": (f,), "b_up": (f,), "b_down": (d,)}[tensor]


def gen_expert_tensor(seed, cfg, tensor, e):
    """Expert e's slice of w_gate / w_up / w_down / b_* in storage format."""
    std = cfg["b_std"] if tensor.startswith("b_") else cfg["w_std"]
    return gen_tensor(seed, cfg, tensor, _expert_shape(cfg, tensor), std, cfg["dtype"], slice_id=e)


def gen_expert_stack(seed, cfg, tensor, experts=None, threads=None, out=None):
    """[len(experts)][...] stack of per-expert slices, generated in parallel.

    ``out`` may be a preallocated array (for instance a pinned host buffer
    viewed through numpy) of the right shape and storage dtype.
    """
    experts = list(range(cfg["E"])) if experts is None else list(experts)
    shp = _expert_shape(cfg, tensor)
    if out is None:
        out = np.empty((len(experts),) + shp,
                       dtype=np.uint16 if cfg["dtype"] == "bf16" else np.float32)

    def one(i):
        out[i] = gen_expert_tensor(seed, cfg, tensor, experts[i])

    with ThreadPoolExecutor(threads or _threads()) as ex:
        list(ex.map(one, range(len(experts))))
    return out


def stress_router_bias(cfg):
    """The stored per-expert logit bias of the Zipf stress workload (float32 [E]).

    The values were fitted once against the seed-0 stress inputs by the
    oracle's data script and are kept as input data so that every consumer
    sees the same bias.
    """
    vals = []
    with open(STRESS_BIAS_FILE) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            vals.append(float(line))
    b = np.asarray(vals, dtype=np.float32)
    if b.shape[0] != cfg["E"]:
        raise ValueError("stored stress bias has %d entries, config wants E=%d"
                         % (b.shape[0], cfg["E"]))
    return b


def pool_size(cfg):
    """Experts the router covers: E plus any zero-computation experts."""
    return cfg["E"] + cfg.get("n_zero", 0) + cfg.get("n_copy", 0) + cfg.get("n_const", 0)


def router_bias(seed, cfg):
    if cfg["bias_mode"] == "none":
        return None
    if cfg["bias_mode"] == "select":
        return _draw(seed, cfg["cfg_id"], "router_bias", 0, (pool_size(cfg),), cfg["beta_std"])
    if cfg["bias_mode"] == "logit":
        return stress_router_bias(cfg)
    raise ValueError(cfg["bias_mode"])


def layer_inputs(cfg, seed=0, experts=True, with_dy=True, threads=None):
    """Every input of one layer forward+backward, in storage format.

    Returns a dict: x [T][d], w_r [d][E_pool] (f32), router_bias [E_pool] (f32 or None),
    w_gate/w_up [E][d][f], w_down [E][f][d], b_gate/b_up [E][f] and
    b_down [E][d] (or None), ws_gate/ws_up [d][fs], ws_down [fs][d] (or None),
    dy [T][d], and with constant experts zc_v [n_const][d], zc_wc [n_const][2][d]
    (f32).  bf16 tensors are uint16 bit patterns.  With experts=False the
    per-expert stacks are omitted (generate them with gen_expert_stack).
    """
    T, d, E, dt = cfg["T"], cfg["d"], cfg["E"], cfg["dtype"]
    out = {"cfg": cfg, "seed": seed}
    out["x"] = gen_rows(seed, cfg, "x", T, d, cfg["x_std"], dt, threads)
    out["w_r"] = _draw(seed, cfg["cfg_id"], "w_r", 0, (d, pool_size(cfg)), cfg["w_r_std"])
    out["router_bias"] = router_bias(seed, cfg)
    if experts:
        for t in ("w_gate", "w_up", "w_down"):
            out[t] = gen_expert_stack(seed, cfg, t, threads=threads)
        for t in ("b_gate", "b_up", "b_down"):
            out[t] = gen_expert_stack(seed, cfg, t, threads=threads) if cfg["expert_bias"] else None
    if cfg["n_shared"]:
        fs = cfg["f_shared"]
        out["ws_gate"] = gen_tensor(seed, cfg, "ws_gate", (d, fs), cfg["w_std"], dt)
        out["ws_up"] = gen_tensor(seed, cfg, "ws_up", (d, fs), cfg["w_std"], dt)
        out["ws_down"] = gen_tensor(seed, cfg, "ws_down", (fs, d), cfg["w_std"], dt)
    else:
        out["ws_gate"] = out["ws_up"] = out["ws_down"] = None
    out["gate_threshold"] = None
    if cfg["router"] == "sigmoid_threshold":
        th = _draw(seed, cfg["cfg_id"], "gate_threshold", 0, (E,), cfg["theta_std"])
        out["gate_threshold"] = (th + np.float32(cfg["theta_mean"])).astype(np.float32)
    nc = cfg.get("n_const", 0)
    out["zc_v"] = _draw(seed, cfg["cfg_id"], "zc_v", 0, (nc, d), cfg["zc_v_std"]) if nc else None
    out["zc_wc"] = _draw(seed, cfg["cfg_id"], "zc_wc", 0, (nc, 2, d), cfg["zc_wc_std"]) if nc else None
    if with_dy:
        out["dy"] = gen_rows(seed, cfg, "dy", T, d, cfg["dy_std"], dt, threads)
    return out
