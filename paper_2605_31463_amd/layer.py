"""Buffers for one MoE layer and thin calls of the fused entry points.

MoELayer allocates (with torch, on the GPU) the saved tensors, the
workspaces and the gradients for a moe_shape, and calls moe_layer_fwd /
moe_layer_bwd.  Every computation happens in libmoe's kernels.
"""
import torch

from . import _lib as L


class MoELayer:
    def __init__(self, shape, device="cuda"):
        self.shape = shape
        self.device = device
        s = shape
        T, d, E, k, f = s.T, s.d, s.E, s.k, s.f
        Ep = L.pool_size(s)
        R = T * k
        self.act = torch.bfloat16 if s.dtype == L.MOE_BF16 else torch.float32
        fwd, _, bwd = L.moe_workspace_size(shape)
        self.ws_fwd = torch.empty(max(fwd, 1), dtype=torch.uint8, device=device)
        self.ws_bwd = torch.empty(max(bwd, 1), dtype=torch.uint8, device=device)
        i32, f32, a = torch.int32, torch.float32, self.act
        e = lambda *shp, dt=a: torch.empty(*shp, dtype=dt, device=device)  # noqa: E731
        self.saved = dict(
            topk_idx=e(T, k, dt=i32), topk_w=e(T, k, dt=f32),
            s_sel=e(T, k, dt=f32) if s.router in (L.MOE_ROUTER_SIGMOID_GROUPED, L.MOE_ROUTER_SIGMOID_THRESHOLD)
            else None,
            expert_offsets=e(Ep + 1, dt=i32), row_of=e(T, k, dt=i32), token_of=e(R, dt=i32),
            x_perm=e(R, d), gu=e(R, 2 * f), h=e(R, f), o=e(R, d),
            gu_sh=e(T, 2 * s.f_shared) if s.n_shared else None,
            h_sh=e(T, s.f_shared) if s.n_shared else None,
            o_sh=e(T, d) if s.n_shared else None,
            router_probs=e(T, Ep, dt=f32) if s.aux_coef > 0 else None,
            aux_loss=torch.zeros(1, dtype=f32, device=device) if s.aux_coef > 0 else None,
        )
        self.y = e(T, d)
        self.dx = e(T, d)

    def alloc_grads(self):
        s = self.shape
        a = self.act
        e = lambda *shp, dt=a: torch.empty(*shp, dtype=dt, device=self.device)  # noqa: E731
        g = dict(dw_r=e(s.d, L.pool_size(s), dt=torch.float32), dw_gate=e(s.E, s.d, s.f),
                 dw_up=e(s.E, s.d, s.f), dw_down=e(s.E, s.f, s.d))
        if s.expert_bias:
            g.update(db_gate=e(s.E, s.f), db_up=e(s.E, s.f), db_down=e(s.E, s.d))
        if s.n_shared:
            g.update(dws_gate=e(s.d, s.f_shared), dws_up=e(s.d, s.f_shared), dws_down=e(s.f_shared, s.d))
        if s.n_const:
            g.update(dzc_v=e(s.n_const, s.d, dt=torch.float32), dzc_wc=e(s.n_const, 2, s.d, dt=torch.float32))
        if s.router == L.MOE_ROUTER_SIGMOID_THRESHOLD:
            g.update(d_threshold=e(s.E, dt=torch.float32))
        return g

    def build_fp8_cache(self, params, stream=None):
        """shape.fp8: quantise the expert weights into a cache (reused by every
        forward until the weights change) and point params at it."""
        if getattr(self, "fp8_cache", None) is None:
            n = L.moe_fp8_cache_size(self.shape)
            self.fp8_cache = torch.empty(max(n, 1), dtype=torch.uint8, device=self.device)
        L.moe_fp8_cache_build(self.shape, params["w_gate"], params["w_up"], params["w_down"], self.fp8_cache, stream)
        params["fp8_cache"] = self.fp8_cache
        params["fp8_cache_bytes"] = self.fp8_cache.numel()
        return params

    def forward(self, params, x, stream=None):
        L.moe_layer_fwd(self.shape, params, x, self.saved, self.y, self.ws_fwd, stream)
        return self.y

    def backward(self, params, x, dy, grads, stream=None):
        L.moe_layer_bwd(self.shape, params, x, self.saved, dy, self.dx, grads, self.ws_bwd, stream)
        return self.dx

    def backward_dgrad(self, params, x, dy, stream=None):
        """Input gradient only; the weight gradients follow with backward_wgrad
        (the backward workspace carries what it needs in between)."""
        L.moe_layer_bwd_dgrad(self.shape, params, x, self.saved, dy, self.dx, self.ws_bwd, stream)
        return self.dx

    def backward_wgrad(self, params, x, dy, grads, accumulate=False, stream=None):
        """Weight gradients of the last backward_dgrad; accumulate adds them to grads."""
        L.moe_layer_bwd_wgrad(self.shape, params, x, self.saved, dy, grads, accumulate, self.ws_bwd, stream)
        return grads
