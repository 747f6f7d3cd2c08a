"""Throughput of one MoE layer forward + backward on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload dsv3] [--no-cpu-baseline]

A step is moe_layer_fwd + moe_layer_bwd over one batch of synthetic input
already resident in HBM (routing, permutation, grouped SwiGLU expert GEMMs,
combine, expert dgrad/wgrad, router gradient, unpermute).  Prints one JSON
line: algorithmic TFLOP/s (value, forward plus backward FLOPs over the step
time), tokens/s, the dominant kernel against its roofline (average launch time
from HIP events recorded on the launch stream during the timed steps), and the
fp64 CPU oracle timed on a bounded sample of the same workload on this host.
The default workload is the DeepSeek-V3-shaped layer, the largest of the
workloads that fit one GPU.

Only one GPU: the layer's one-GPU share is the workload; --gpus above 1 is
refused.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE layer fwd+bwd TFLOP/s and tokens/s on 1 MI355X; % of MFMA/HBM roofline"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0    # MI355X dense fp8 MFMA
FP8_KERNELS = {1: ("gemm_gateup_fwd", "gemm_down_fwd"),
               2: ("gemm_gateup_fwd", "gemm_down_fwd", "gemm_down_dgrad", "gemm_gateup_dgrad")}
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
GEMM_SOURCE = os.path.join(ROOT, "paper_2605_31463_amd", "csrc", "gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def pool(cfg):
    return cfg["E"] + cfg.get("n_zero", 0) + cfg.get("n_copy", 0) + cfg.get("n_const", 0)


def layer_flops(cfg, rows=None):
    """Algorithmic FLOPs (2 per multiply-add) as (fwd, bwd):
    fwd = 2 T d E_pool + 6 R d f (+ 6 T d f_shared), bwd = 2 fwd (every product of
    the forward has a data-gradient and a weight-gradient product of the same
    size), with R = T k rows through the FFN experts (fewer when zero-computation
    experts take some slots: then the routed FFN rows of the batch).  A step
    (forward and backward) is fwd + bwd = 3 fwd."""
    T, d, k, f = cfg["T"], cfg["d"], cfg["k"], cfg["f"]
    R = T * k if rows is None else rows
    fwd = 2 * T * d * pool(cfg) + 6 * R * d * f
    if cfg["n_shared"]:
        fwd += 6 * T * d * cfg["f_shared"]
    return fwd, 2 * fwd


def kernel_work(cfg, rows=None):
    """Per-launch algorithmic work of the layer's main kernels: (bound, amount, unit).
    rows: routed FFN rows when zero-computation experts take some slots (the GEMMs
    and the row gathers touch only those; the counts below are then lower bounds
    for the gathers, which also read x or dy for such slots)."""
    T, d, E, k, f = cfg["T"], cfg["d"], pool(cfg), cfg["k"], cfg["f"]
    R = T * k if rows is None else rows
    eb = 2 if cfg["dtype"] == "bf16" else 4
    gu = 2.0 * R * d * 2 * f
    dn = 2.0 * R * f * d
    extra = {}
    if cfg["n_shared"]:
        # the shared expert's dense passes over all T tokens (kernel ids of their own)
        fs = cfg["f_shared"]
        sgu, sdn = 2.0 * T * d * 2 * fs, 2.0 * T * fs * d
        extra.update({"gemm_shared_gateup_fwd": ("mfma", sgu), "gemm_shared_down_fwd": ("mfma", sdn),
                      "gemm_shared_down_dgrad": ("mfma", sdn), "gemm_shared_gateup_dgrad": ("mfma", sgu),
                      "gemm_shared_down_wgrad": ("mfma", sdn), "gemm_shared_gateup_wgrad": ("mfma", sgu)})
    return dict(extra, **{
        "gemm_gateup_fwd": ("mfma", gu), "gemm_down_fwd": ("mfma", dn),
        "gemm_down_dgrad": ("mfma", dn), "gemm_gateup_dgrad": ("mfma", gu),
        "gemm_down_wgrad": ("mfma", dn), "gemm_gateup_wgrad": ("mfma", gu),
        # router logits: bf16 x times the three bf16 parts of W_r
        "route": ("mfma", 2.0 * T * d * E * 3),
        # bytes: reads + writes of the HBM operands, once each (FP8: the
        # permutation also writes the E4M3 rows of x_perm and their scales,
        # the combine backward at level 2 those of d_o)
        "route_select": ("hbm", T * E * 8 + T * k * 8),
        "scatter": ("hbm", T * d * eb + R * d * eb + T * k * 4 * 3 + (R * (d + 4) if cfg.get("fp8") else 0)),
        # (with a shared expert the combine also reads its output rows and the
        # unpermute its input gradient rows)
        "combine_fwd": ("hbm", R * d * eb + T * d * eb * (2 if cfg["n_shared"] else 1) + T * k * 8),
        "combine_bwd": ("hbm", T * d * eb + 2 * R * d * eb + T * k * 12
                        + (R * (d + 4) if int(cfg.get("fp8") or 0) == 2 else 0)),
        "unpermute": ("hbm", R * d * eb + T * d * eb * (2 if cfg["n_shared"] else 1) + T * k * 12),
    })


def gemm_hbm_floor(cfg, counts, rows=None):
    """Smallest HBM traffic (bytes) of each expert GEMM pass: every operand read
    once, every output written once.  The weights of an expert are read only if
    it holds rows; every expert's weight gradient is written (zero for an expert
    without rows).  counts: rows per routed expert.  FP8 passes read one-byte
    codes of the weights and of the activation operand."""
    T, d, E, k, f = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["f"]
    R = T * k if rows is None else rows
    eb = 2 if cfg["dtype"] == "bf16" else 4
    act = sum(1 for c in counts if c > 0)
    fp8 = int(cfg.get("fp8") or 0)
    q = lambda name: 1 if fp8 and name in FP8_KERNELS[fp8] else eb  # noqa: E731
    out = {
        "gemm_gateup_fwd": act * 2 * d * f * q("gemm_gateup_fwd") + R * d * q("gemm_gateup_fwd") + R * 3 * f * eb,
        "gemm_down_fwd": act * f * d * q("gemm_down_fwd") + R * f * q("gemm_down_fwd") + R * d * eb,
        "gemm_down_dgrad": act * f * d * q("gemm_down_dgrad") + R * d * q("gemm_down_dgrad") + R * 4 * f * eb,
        "gemm_gateup_dgrad": act * 2 * d * f * q("gemm_gateup_dgrad") + R * 2 * f * q("gemm_gateup_dgrad")
        + R * d * eb,
        "gemm_down_wgrad": E * f * d * eb + R * (f + d) * eb,
        "gemm_gateup_wgrad": E * 2 * d * f * eb + R * (d + 2 * f) * eb,
    }
    if cfg["n_shared"]:
        fs = cfg["f_shared"]
        out.update({
            "gemm_shared_gateup_fwd": 2 * d * fs * eb + T * (d + 3 * fs) * eb,
            "gemm_shared_down_fwd": fs * d * eb + T * (fs + d) * eb,
            "gemm_shared_down_dgrad": fs * d * eb + T * (d + 4 * fs) * eb,
            "gemm_shared_gateup_dgrad": 2 * d * fs * eb + T * (2 * fs + d) * eb,
            "gemm_shared_down_wgrad": fs * d * eb + T * (fs + d) * eb,
            "gemm_shared_gateup_wgrad": 2 * d * fs * eb + T * (d + 2 * fs) * eb,
        })
    return out


def gemm_roof(flops, floor_bytes, secs, mfma_peak_tflops, hbm_peak_gbs=PEAK_HBM_GBS):
    """Two-sided roofline of one GEMM launch of `secs` seconds: the binding side
    is the one whose peak takes longer for the launch's work (flops at the MFMA
    peak, or its smallest HBM traffic at the HBM peak).  Returns the binding
    side's achieved rate, peak and fraction, the other side's, and mfma_ceiling,
    the largest MFMA fraction the HBM floor leaves: t_mfma / max(t_mfma, t_hbm)."""
    t_c = flops / (mfma_peak_tflops * 1e12)
    t_m = floor_bytes / (hbm_peak_gbs * 1e9)
    mf = {"achieved": flops / secs / 1e12, "peak": mfma_peak_tflops, "unit": "TFLOP/s"}
    mf["frac"] = mf["achieved"] / mf["peak"]
    hb = {"achieved": floor_bytes / secs / 1e9, "peak": hbm_peak_gbs, "unit": "GB/s", "bytes": floor_bytes}
    hb["frac"] = hb["achieved"] / hb["peak"]
    r = dict(mf if t_c >= t_m else hb, bound="mfma" if t_c >= t_m else "hbm")
    r["other_side"] = dict(hb, bound="hbm") if t_c >= t_m else dict(mf, bound="mfma")
    r["mfma_ceiling"] = min(1.0, t_c / max(t_c, t_m))
    return r


def file_hash(path):
    with open(path, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


def traffic_for(kernel, workload):
    """HBM bytes per launch of a kernel on a workload from the committed
    rocprofv3 counter summary (profiles/traffic.json), if it was taken on the
    current GEMM source; else None."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256_16") != file_hash(GEMM_SOURCE):
        return None
    ent = t.get("workloads", {}).get(workload, {}).get("kernels", {}).get(kernel)
    return None if ent is None else ent.get("bytes_per_launch")


# Bounded CPU samples: the DeepSeek-V3-shaped layer whole (256 experts of
# 352 MB of float64 weights and weight gradients each) is far beyond a few
# minutes of the oracle, so its sample keeps d, f, k, the group-limited router
# (8 groups, 4 kept) and the shared expert and cuts T and E together, so that
# the experts still hold ~256 rows each on average, as at full size.
CPU_SAMPLES = {"dsv3": dict(T=1024, E=32)}


def cpu_baseline(cfg, seed, tokens=0, reps=1):
    """The fp64 oracle, as it stands, on a bounded sample of the workload: the
    first `tokens` tokens (0: the workload's sample from CPU_SAMPLES, else all of
    them), fwd+bwd repeated `reps` times on the same inputs (so that the timed
    CPU work is long enough to measure).  Its value counts the sample's own
    algorithmic FLOPs (forward + backward)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from moe_inputs import layer_inputs, variant
    from oracle import ZeroComputeSpec, layer_backward, layer_forward, spec_from_config
    from moe_inputs import to_f64

    base = cfg["name"].split("[")[0]
    over = dict(T=tokens) if tokens else dict(CPU_SAMPLES.get(base, dict(T=cfg["T"])))
    scfg = variant(base, **over)
    inp = layer_inputs(scfg, seed=seed)
    dt = scfg["dtype"]
    spec = spec_from_config(scfg)
    x = to_f64(inp["x"], dt)
    dy = to_f64(inp["dy"], dt)
    w_r = inp["w_r"].astype(np.float64)
    beta = None if inp["router_bias"] is None else inp["router_bias"].astype(np.float64)

    def efn(e):
        b = scfg["expert_bias"]
        return (to_f64(inp["w_gate"][e], dt), to_f64(inp["w_up"][e], dt), to_f64(inp["w_down"][e], dt),
                to_f64(inp["b_gate"][e], dt) if b else None, to_f64(inp["b_up"][e], dt) if b else None,
                to_f64(inp["b_down"][e], dt) if b else None)

    shared = None
    if scfg["n_shared"]:
        shared = tuple(to_f64(inp[n], dt) for n in ("ws_gate", "ws_up", "ws_down"))
    zc = None
    if pool(scfg) > scfg["E"]:
        nc = scfg["n_const"]
        zc = (ZeroComputeSpec(scfg["n_zero"], scfg["n_copy"], nc, scfg["zc_aux_weight"]),
              inp["zc_v"].astype(np.float64) if nc else np.zeros((0, scfg["d"])),
              inp["zc_wc"].astype(np.float64) if nc else np.zeros((0, 2, scfg["d"])))
    coef = cfg.get("aux_coef", 0.0)
    theta = None if inp.get("gate_threshold") is None else inp["gate_threshold"].astype(np.float64)
    t0 = time.perf_counter()
    for _ in range(reps):
        fwd = layer_forward(spec, x, w_r, beta, efn, shared, aux_coef=coef, zc=zc, theta=theta,
                            fp8=bool(cfg.get("fp8")))
        layer_backward(spec, x, w_r, beta, efn, fwd, dy, shared, with_bias=scfg["expert_bias"], zc=zc,
                       fp8=cfg.get("fp8") == 2)
    wall = time.perf_counter() - t0
    ff, fb = layer_flops(scfg, rows=int(fwd["maps"]["offsets"][scfg["E"]]))
    blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    threads = max([p.get("num_threads", 1) for p in blas] or [1])
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            cpu = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), cpu)
    except OSError:
        pass
    cut = ("%d of %d tokens" % (scfg["T"], cfg["T"]) if scfg["E"] == cfg["E"] else
           "%d of %d tokens and %d of %d routed experts (~%d rows per expert on average, as at full size)"
           % (scfg["T"], cfg["T"], scfg["E"], cfg["E"], scfg["T"] * scfg["k"] // scfg["E"]))
    return {"value": round(reps * (ff + fb) / wall / 1e12, 6), "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "cpu": cpu,
            "blas": ",".join(sorted({"%s %s" % (p.get("internal_api"), p.get("version")) for p in blas})),
            "sample": "fp64 oracle fwd+bwd of %s (otherwise the workload's shapes, seed %d), %d times, "
                      "%.1f s wall" % (cut, seed, reps, wall),
            "tokens_per_s": round(reps * scfg["T"] / wall, 1)}


def memory_kernels(cfg, L, layer, params, x, dy, reps=20, cold_reps=10, scrub_mib=1024):
    """Warm and cold times of the HBM-bound kernels, each driven through its
    C-ABI entry point on the layer's own saved buffers and timed with the
    library's events around that kernel's launch.  Warm: back-to-back calls
    (operands partly left in the 256 MB MALL by the previous call).  Cold: a
    read of a 1 GiB scrub buffer before every timed call (a read, so that no
    dirty lines drain during the timed kernel).  The unpermute entry point sums
    dx_perm rows only: the layer fuses the router's dx into the same kernel."""
    import torch
    T, d, k, E = cfg["T"], cfg["d"], cfg["k"], cfg["E"]
    R = T * k
    sv, sh = layer.saved, layer.shape
    act = layer.act
    d_o = torch.empty(R, d, dtype=act, device="cuda")
    d_w = torch.empty(T, k, dtype=torch.float32, device="cuda")
    counts = torch.empty(E, dtype=torch.int32, device="cuda")
    y = torch.empty(T, d, dtype=act, device="cuda")
    dx = torch.empty(T, d, dtype=act, device="cuda")
    scrub = torch.ones(scrub_mib << 18, dtype=torch.float32, device="cuda")
    ws = layer.ws_fwd
    calls = {
        "route_select": lambda: L.moe_route(sh, x, params["w_r"], params["router_bias"], sv["topk_idx"],
                                            sv["topk_w"], sv["s_sel"], counts, ws),
        "scatter": lambda: L.moe_permute(sh, x, sv["topk_idx"], sv["expert_offsets"], sv["row_of"],
                                         sv["token_of"], sv["x_perm"], ws),
        "combine_fwd": lambda: L.moe_combine_fwd(sh, sv["o"], sv["topk_w"], sv["row_of"], sv["o_sh"], y),
        "combine_bwd": lambda: L.moe_combine_bwd(sh, dy, sv["o"], sv["topk_w"], sv["row_of"], d_o, d_w),
        "unpermute": lambda: L.moe_unpermute_bwd(sh, sv["x_perm"], sv["row_of"], None, None, dx),
    }
    work = kernel_work(cfg)
    out = {}
    for name, call in calls.items():
        kid = L.kernel_id(name)
        res = {}
        for mode in ("warm", "cold"):
            for _ in range(2):
                call()
            torch.cuda.synchronize()
            L.moe_timing_select(kid)
            for _ in range(reps if mode == "warm" else cold_reps):
                if mode == "cold":
                    scrub.sum()
                call()
            torch.cuda.synchronize()
            ms, n = L.moe_timing_read()
            L.moe_timing_select(-1)
            us = ms / max(n, 1) * 1e3
            gbs = work[name][1] / (us / 1e6) / 1e9
            res[mode] = {"avg_us": round(us, 2), "GB/s": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)}
        out[name] = res
    del scrub
    return out


def gpu_clocks():
    """Current and available clocks from rocm-smi, as text (None when it is not there)."""
    import shutil
    import subprocess
    exe = shutil.which("rocm-smi")
    if not exe:
        return None
    try:
        r = subprocess.run([exe, "--showclocks"], capture_output=True, text=True, timeout=30)
    except (OSError, subprocess.SubprocessError):
        return None
    lines = [ln.strip() for ln in r.stdout.splitlines() if "clk" in ln.lower() and ":" in ln]
    return lines or None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dsv3")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-tokens", type=int, default=0,
                    help="tokens of the workload the CPU oracle runs (0: the workload's bounded sample)")
    ap.add_argument("--cpu-reps", type=int, default=0,
                    help="repetitions of the oracle's fwd+bwd (0: 3)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--aux-coef", type=float, default=0.0,
                    help="add the global-level load-balancing loss of this coefficient (the paper "
                         "pretrains with 1e-3); 0: without it")
    ap.add_argument("--fp8", nargs="?", const="fwd", choices=("fwd", "all"), default=None,
                    help="the routed experts' GEMMs on FP8 (E4M3) operands: the forward ones (fwd, the "
                         "default) or the forward and data-gradient ones (all); the weight cache is built "
                         "once before the steps (as once per optimizer step) and its build time reported")
    ap.add_argument("--memory-kernels", action="store_true",
                    help="instead of the step benchmark: warm and cold (after a 1 GiB read scrub) times "
                         "of the HBM-bound kernels through their entry points, and the GPU clocks")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="before the timed steps, run a plain torch copy of this many MiB three times "
                         "(a kernel of known size for scaling rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the MoE layer's one-GPU share is the workload "
              "(no collectives are built); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from moe_inputs import config, layer_inputs
    from paper_2605_31463_amd import _lib as L
    from paper_2605_31463_amd.layer import MoELayer

    cfg = config(args.workload)
    if args.aux_coef:
        cfg = dict(cfg, aux_coef=args.aux_coef)
    if args.fp8:
        cfg = dict(cfg, fp8=1 if args.fp8 == "fwd" else 2)
    dt = cfg["dtype"]
    torch.cuda.set_device(0)
    inp = layer_inputs(cfg, seed=args.seed)

    def dev(a):
        import numpy as np
        if a is None:
            return None
        if dt == "bf16" and a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    params = {n: dev(inp.get(n)) for n in ("w_r", "router_bias", "w_gate", "w_up", "w_down", "b_gate",
                                           "b_up", "b_down", "ws_gate", "ws_up", "ws_down", "zc_v", "zc_wc",
                                           "gate_threshold")}
    x = dev(inp["x"])
    dy = dev(inp["dy"])
    del inp
    layer = MoELayer(L.shape_from_config(cfg))
    grads = layer.alloc_grads()
    stream = torch.cuda.current_stream()
    cache_ms = None
    if cfg.get("fp8"):
        layer.build_fp8_cache(params)
        torch.cuda.synchronize()
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        c0.record(stream)
        layer.build_fp8_cache(params)
        c1.record(stream)
        torch.cuda.synchronize()
        cache_ms = c0.elapsed_time(c1)

    def step():
        layer.forward(params, x)
        layer.backward(params, x, dy, grads)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    zc = pool(cfg) > cfg["E"]
    variable = zc or cfg["router"] == "sigmoid_threshold"
    # routed FFN rows (every slot when every slot holds an FFN expert)
    ffn_rows = int(layer.saved["expert_offsets"][cfg["E"]].item()) if variable else cfg["T"] * cfg["k"]
    if args.memory_kernels and variable:
        print("--memory-kernels drives the component entry points, which take neither zero-computation "
              "experts nor the threshold router", file=sys.stderr)
        sys.exit(2)
    if args.memory_kernels:
        workload = "%s moe layer T=%d d=%d E=%d k=%d f=%d" % (cfg["name"], cfg["T"], cfg["d"], cfg["E"],
                                                             cfg["k"], cfg["f"])
        res = memory_kernels(cfg, L, layer, params, x, dy)
        print(json.dumps({"memory_kernels": res, "peak_GB/s": PEAK_HBM_GBS, "dtype": dt,
                          "config": {"workload": workload}, "clocks": gpu_clocks()}), flush=True)
        return
    if args.copy_calibration_mb > 0:
        n = args.copy_calibration_mb << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # per-kernel times over a few untimed steps, to pick the dominant kernel
    work = kernel_work(cfg, rows=ffn_rows)
    per_kernel = {}
    for name in work:
        L.moe_timing_select(L.kernel_id(name))
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        ms, n = L.moe_timing_read()
        if n:  # (a kernel the workload does not launch is left out)
            per_kernel[name] = ms / n
    L.moe_timing_select(-1)
    dominant = max(per_kernel, key=lambda n: per_kernel[n])

    # timed region: exactly K steps, the dominant kernel's launches timed with events
    L.moe_timing_select(L.kernel_id(dominant))
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dom_ms, dom_n = L.moe_timing_read()
    L.moe_timing_select(-1)
    ms_per_step = ev0.elapsed_time(ev1) / args.steps

    # after the timed region: forward and backward separately, per step (events
    # at the step's start, between the two calls and at its end)
    n_ph = max(10, args.steps)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_ph)]
    for e in evs:
        e[0].record(stream)
        layer.forward(params, x)
        e[1].record(stream)
        layer.backward(params, x, dy, grads)
        e[2].record(stream)
    torch.cuda.synchronize()
    f_ms = [e[0].elapsed_time(e[1]) for e in evs][-10:]
    b_ms = [e[1].elapsed_time(e[2]) for e in evs][-10:]
    s_ms = [e[0].elapsed_time(e[2]) for e in evs][-10:]
    med = lambda v: sorted(v)[len(v) // 2]  # noqa: E731

    ff, fb = layer_flops(cfg, rows=ffn_rows)
    tflops = (ff + fb) / (ms_per_step / 1e3) / 1e12
    dom_avg_s = dom_ms / max(dom_n, 1) / 1e3
    fp8 = int(cfg.get("fp8") or 0)
    mfma_peak = lambda name: PEAK_FP8_TFLOPS if fp8 and name in FP8_KERNELS[fp8] else PEAK_BF16_TFLOPS  # noqa: E731
    # expert GEMMs: two-sided roofline, the larger of the MFMA time of their
    # flops and the HBM time of their smallest traffic (the binding side is
    # the kernel's bound; the other side is reported beside it)
    counts = (layer.saved["expert_offsets"][1:cfg["E"] + 1] - layer.saved["expert_offsets"][:cfg["E"]]).tolist()
    floor_b = gemm_hbm_floor(cfg, counts, rows=ffn_rows)

    def roof(name, secs):
        b, amt = work[name]
        if b != "mfma" or name not in floor_b:
            rate = amt / secs / (1e12 if b == "mfma" else 1e9)
            peak = mfma_peak(name) if b == "mfma" else PEAK_HBM_GBS
            return {"bound": b, "achieved": rate, "peak": peak, "unit": "TFLOP/s" if b == "mfma" else "GB/s",
                    "frac": rate / peak}
        return gemm_roof(amt, floor_b[name], secs, mfma_peak(name))

    rdom = roof(dominant, dom_avg_s)
    bound, achieved, peak, unit = rdom["bound"], rdom["achieved"], rdom["peak"], rdom["unit"]
    workload = "%s moe layer T=%d d=%d E=%d k=%d f=%d" % (cfg["name"], cfg["T"], cfg["d"], cfg["E"],
                                                         cfg["k"], cfg["f"])
    kernels = {}
    for name, ms in per_kernel.items():
        r = roof(name, ms / 1e3)
        kernels[name] = {"avg_us": round(ms * 1e3, 2), "bound": r["bound"], "achieved": round(r["achieved"], 1),
                         "unit": r["unit"], "frac": round(r["frac"], 4)}
        if "other_side" in r:
            o = r["other_side"]
            kernels[name]["other_side"] = {"bound": o["bound"], "achieved": round(o["achieved"], 1),
                                           "unit": o["unit"], "frac": round(o["frac"], 4)}
            kernels[name]["mfma_ceiling"] = round(r["mfma_ceiling"], 4)
    out = {
        "metric": METRIC, "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": ("fp8 e4m3 (forward expert GEMMs) + bf16" if fp8 == 1 else
                  "fp8 e4m3 (forward and data-gradient expert GEMMs) + bf16") if fp8 else dt,
        "data": "synthetic (seeded; shapes and distributions of the workload)",
        "config": dict({"workload": workload, "T": cfg["T"], "d": cfg["d"], "E": cfg["E"], "k": cfg["k"],
                        "f": cfg["f"], "router": cfg["router"], "aux_coef": cfg.get("aux_coef", 0.0)},
                       **({"n_zero": cfg["n_zero"], "n_copy": cfg["n_copy"], "n_const": cfg["n_const"],
                           "zc_aux_weight": cfg["zc_aux_weight"]} if zc else {}),
                       **({"ffn_rows": ffn_rows} if variable else {}),
                       **({"fp8": "forward" if fp8 == 1 else "forward+dgrad"} if fp8 else {})),
        "tokens_per_s": round(cfg["T"] / (ms_per_step / 1e3), 1),
        "phases_median_of_last_10": {"fwd_ms": round(med(f_ms), 4), "bwd_ms": round(med(b_ms), 4),
                                     "step_ms": round(med(s_ms), 4),
                                     "fwd_tflops": round(ff / (med(f_ms) / 1e3) / 1e12, 2),
                                     "bwd_tflops": round(fb / (med(b_ms) / 1e3) / 1e12, 2)},
        "wall_s_timed": round(wall, 4),
        "roofline": dict({"bound": bound, "kernel": dominant, "achieved": round(achieved, 2), "peak": peak,
                          "unit": unit, "frac": round(achieved / peak, 4),
                          "avg_launch_us": round(dom_avg_s * 1e6, 2), "launches": dom_n,
                          "traffic": traffic_for(dominant, workload)},
                         **({"hbm_floor_bytes": floor_b[dominant],
                             "other_side": {k2: (round(v2, 4) if isinstance(v2, float) else v2)
                                            for k2, v2 in rdom["other_side"].items() if k2 != "bytes"},
                             "mfma_ceiling": round(rdom["mfma_ceiling"], 4)} if "other_side" in rdom else {})),
        "kernels": kernels,
    }
    if fp8:
        out["fp8_cache_build_ms"] = round(cache_ms, 4)
    if not args.no_cpu_baseline:
        reps = args.cpu_reps or 3
        out["cpu_baseline"] = cpu_baseline(cfg, args.seed, args.cpu_tokens, reps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
