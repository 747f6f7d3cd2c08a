"""Writes the stored per-expert logit bias of the Zipf load-imbalance workload.

TEST INFRASTRUCTURE (data script).  Run once:  python -m oracle.fit_stress_bias
It reads the seed-0 stress inputs from the shared generators, computes router
logits and selections with this oracle only, and writes
moe_inputs/stress_bias_seed0.txt, which every consumer then loads as input
data.

Target law.  Expert token counts follow Zipf(s=1.2) over the ranks of the 120
non-empty experts, capped at T because a token holds an expert at most once:
counts_r = min(T, a * r**-1.2) with a chosen so that the counts add up to
T*k.  Eight experts receive no token: their bias is -1e4.  Which expert gets
which rank is a seeded permutation.  The bias of the others is fitted by a
fixed number of multiplicative (log-ratio) updates on the fp64 logits.
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

from moe_inputs import config, layer_inputs, to_f64  # noqa: E402
from moe_inputs.gen import STRESS_BIAS_FILE  # noqa: E402
from oracle.moe_oracle import RouterSpec, router_logits, route  # noqa: E402

EMPTY_BIAS = -1.0e4
ITERS = 200
STEP = 0.5


def zipf_targets(T, k, n_ranked, s):
    """Capped Zipf counts over ranks 1..n_ranked adding up to T*k (water-filling)."""
    r = np.arange(1, n_ranked + 1, dtype=np.float64)
    shape = r ** -s
    lo, hi = 0.0, float(T * k) * 10
    for _ in range(200):
        a = 0.5 * (lo + hi)
        tot = np.minimum(T, a * shape).sum()
        if tot < T * k:
            lo = a
        else:
            hi = a
    return np.minimum(T, hi * shape)


def main(seed=0):
    cfg = config("stress")
    T, E, k = cfg["T"], cfg["E"], cfg["k"]
    n_empty = cfg["n_empty"]
    inp = layer_inputs(dict(cfg, bias_mode="none"), seed=seed, experts=False, with_dy=False)
    l = router_logits(to_f64(inp["x"], cfg["dtype"]), inp["w_r"].astype(np.float64))
    perm = np.random.default_rng([seed, cfg["cfg_id"], 99]).permutation(E)
    ranked, empty = perm[:E - n_empty], perm[E - n_empty:]
    targets = np.zeros(E)
    targets[ranked] = zipf_targets(T, k, E - n_empty, cfg["zipf_s"])
    beta = np.zeros(E)
    beta[empty] = EMPTY_BIAS
    spec = RouterSpec(router="softmax_topk", E=E, k=k, bias_mode="logit")
    for _ in range(ITERS):
        rt = route(spec, l, beta.astype(np.float32).astype(np.float64))
        counts = np.bincount(rt["topk_idx"].reshape(-1), minlength=E)
        beta[ranked] += STEP * np.log(targets[ranked] / (counts[ranked] + 0.5))
    b32 = beta.astype(np.float32)
    rt = route(spec, l, b32.astype(np.float64))
    counts = np.bincount(rt["topk_idx"].reshape(-1), minlength=E)
    order = np.argsort(-counts, kind="stable")
    with open(STRESS_BIAS_FILE, "w") as fh:
        fh.write("# Zipf(1.2) stress workload: per-expert router logit bias (float32), seed %d\n" % seed)
        fh.write("# written by oracle/fit_stress_bias.py; %d fitting steps of size %g\n" % (ITERS, STEP))
        fh.write("# achieved counts (descending): max %d, min nonzero %d, zero-token experts %d\n"
                 % (counts.max(), counts[counts > 0].min(), int((counts == 0).sum())))
        fh.write("# top counts: %s\n" % " ".join(str(int(c)) for c in counts[order[:12]]))
        for v in b32:
            fh.write("%.9g\n" % v)
    print("wrote", STRESS_BIAS_FILE, "max", counts.max(), "min>0", counts[counts > 0].min(),
          "zeros", int((counts == 0).sum()))


if __name__ == "__main__":
    main()
