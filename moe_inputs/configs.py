"""Workload shapes for the single-GPU MoE layer.

The paper trains Qwen3-30B-A3B and GPT-OSS-20B (section 5.1, training
throughput table) and names DeepSeek-V3 as the frontier MoE whose DualPipe
schedule it builds on (sections 1 and 3.2).  Five layer shapes stand in for
those models' MoE layers on one GPU:

  0 tiny      fp32 oracle-scale layer, softmax router with renormalised top-k
  1 qwen3     Qwen3-30B-A3B-shaped, bf16, softmax router, renormalised top-k
  2 gptoss    GPT-OSS-20B-shaped, bf16, softmax over the selected top-k
              logits, per-expert bias vectors in the experts
  3 dsv3      DeepSeek-V3-shaped, bf16, sigmoid scores with a selection-only
              bias, group-limited routing (8 groups, keep 4), weights
              renormalised and scaled by 2.5, one always-on shared expert
  4 stress    Qwen3 dims at T=32768 with a per-expert logit bias that makes the
              expert token counts follow a capped Zipf(1.2) law, 8 experts
              receive no token
  5 moepp     Qwen3 dims with MoE++ zero-computation experts added to the pool
              (appendix B.3 lists MoE++ among the new-feature tasks): 128 FFN
              experts plus 8 zero, 8 copy and 16 constant experts, one
              zero-computation expert per four FFN experts and zero : copy :
              constant = 1 : 1 : 2 as in the MoE++ work's configurations
  6 dynmoe    Qwen3 dims with DynMoE-style threshold gating (appendix B.3
              lists DynMoE among the new-feature tasks): sigmoid gates on the
              128 experts, per-expert thresholds ~ N(1.8, 0.1) on the logits,
              at most k = 8 active experts per token (on average about 3)

Fields:
  T, d, E, k, f          tokens, hidden, routed experts, top-k, expert width
  router                 'softmax_topk' | 'topk_softmax' | 'sigmoid_grouped' |
                         'sigmoid_threshold'
  n_groups, topk_groups  expert groups and groups kept (1, 1 = no group limit)
  route_scale            factor on the renormalised weights
  bias_mode              'none' | 'select' (selection key only) | 'logit'
                         (added to the logits for selection and weights)
  expert_bias            experts carry b_gate, b_up (f) and b_down (d)
  n_shared, f_shared     always-on shared expert and its width
  dtype                  'f32' or 'bf16' storage of x, weights, activations
  n_zero, n_copy, n_const  zero-computation experts after the E FFN experts
                         (the router covers E + their number)
  zc_aux_weight          their weight in the load-balancing loss
  theta_mean, theta_std  thresholds of the 'sigmoid_threshold' router
  fp8                    the routed experts' GEMMs on E4M3 operands: 0 none,
                         1 (or True) the forward ones, 2 the forward and the
                         data-gradient ones
  act, act_alpha, act_limit  routed experts' activation: 'swiglu' or
                         'clamped_glu' (the GPT-OSS release's variant; its
                         slope and clamp bound)
"""
import copy

# Tensor ids of the seeded child streams: [seed, cfg_id, tensor_id, expert_id].
TENSOR_IDS = {
    "x": 0, "w_r": 1, "w_gate": 2, "w_up": 3, "w_down": 4,
    "b_gate": 5, "b_up": 6, "b_down": 7, "router_bias": 8, "dy": 9,
    "ws_gate": 10, "ws_up": 11, "ws_down": 12, "zc_v": 13, "zc_wc": 14, "gate_threshold": 15,
}

_BASE = dict(
    n_groups=1, topk_groups=1, route_scale=1.0, bias_mode="none",
    expert_bias=False, n_shared=0, f_shared=0,
    x_std=1.0, w_r_std=0.02, w_std=0.02, b_std=0.02, beta_std=0.1, dy_std=1.0,
    n_zero=0, n_copy=0, n_const=0, zc_aux_weight=1.0, zc_v_std=1.0, zc_wc_std=0.02,
    act="swiglu", act_alpha=1.702, act_limit=7.0, theta_mean=1.8, theta_std=0.1, fp8=0,
)


def _mk(**kw):
    c = dict(_BASE)
    c.update(kw)
    return c


CONFIGS = [
    _mk(cfg_id=0, name="tiny", T=64, d=128, E=8, k=2, f=256,
        router="softmax_topk", dtype="f32"),
    _mk(cfg_id=1, name="qwen3", T=8192, d=2048, E=128, k=8, f=768,
        router="softmax_topk", dtype="bf16"),
    _mk(cfg_id=2, name="gptoss", T=16384, d=2880, E=32, k=4, f=2880,
        router="topk_softmax", expert_bias=True, dtype="bf16"),
    _mk(cfg_id=3, name="dsv3", T=8192, d=7168, E=256, k=8, f=2048,
        router="sigmoid_grouped", n_groups=8, topk_groups=4, route_scale=2.5,
        bias_mode="select", n_shared=1, f_shared=2048, dtype="bf16"),
    _mk(cfg_id=4, name="stress", T=32768, d=2048, E=128, k=8, f=768,
        router="softmax_topk", bias_mode="logit", dtype="bf16",
        zipf_s=1.2, n_empty=8),
    _mk(cfg_id=5, name="moepp", T=8192, d=2048, E=128, k=8, f=768,
        router="softmax_topk", dtype="bf16", n_zero=8, n_copy=8, n_const=16, zc_aux_weight=0.5),
    _mk(cfg_id=6, name="dynmoe", T=8192, d=2048, E=128, k=8, f=768,
        router="sigmoid_threshold", dtype="bf16"),
]


def config(name_or_id):
    """A copy of one of the workload configs, by name or id."""
    for c in CONFIGS:
        if c["name"] == name_or_id or c["cfg_id"] == name_or_id:
            return copy.deepcopy(c)
    raise KeyError(name_or_id)


def variant(name_or_id, **overrides):
    """A config with some fields replaced (smaller T, d, f, E for parity runs).

    The seeds stay those of the base config, so a variant draws its tensors
    from the same child streams with its own shapes.
    """
    c = config(name_or_id)
    c.update(overrides)
    if overrides:
        c["name"] = c["name"] + "[" + ",".join(
            "%s=%s" % kv for kv in sorted(overrides.items())) + "]"
    return c
