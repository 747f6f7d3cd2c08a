"""ctypes binding of libmoe (include/moe.h): same entry-point names, argument
marshalling only.  Tensors are torch tensors on the GPU (or None for optional
pointers); the stream is torch's current stream unless one is given.

The library is the in-tree libmoe.so built by paper_2605_31463_amd.build;
importing this module fails loudly when it is missing.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe.so")

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_UNSUPPORTED = -2
MOE_ERR_HIP = -3
MOE_ERR_WORKSPACE = -4

MOE_ROUTER_SOFTMAX_TOPK = 0
MOE_ROUTER_TOPK_SOFTMAX = 1
MOE_ROUTER_SIGMOID_GROUPED = 2
MOE_ROUTER_SIGMOID_THRESHOLD = 3
ROUTERS = {"softmax_topk": MOE_ROUTER_SOFTMAX_TOPK, "topk_softmax": MOE_ROUTER_TOPK_SOFTMAX,
           "sigmoid_grouped": MOE_ROUTER_SIGMOID_GROUPED, "sigmoid_threshold": MOE_ROUTER_SIGMOID_THRESHOLD}
MOE_BIAS_NONE = 0
MOE_BIAS_SELECT_ONLY = 1
MOE_BIAS_LOGIT = 2
BIAS_MODES = {"none": MOE_BIAS_NONE, "select": MOE_BIAS_SELECT_ONLY, "logit": MOE_BIAS_LOGIT}
MOE_F32 = 0
MOE_BF16 = 1
DTYPES = {"f32": MOE_F32, "bf16": MOE_BF16}
MOE_ACT_SWIGLU = 0
MOE_ACT_CLAMPED_GLU = 1
ACTS = {"swiglu": MOE_ACT_SWIGLU, "clamped_glu": MOE_ACT_CLAMPED_GLU}
MOE_DGRAD = 1
MOE_WGRAD = 2
MOE_ACCUMULATE = 4


class MoeError(RuntimeError):
    def __init__(self, fn, status, detail):
        super().__init__("%s failed: %s (%d): %s" % (fn, _status_string(status), status, detail))
        self.status = status


class moe_shape(ctypes.Structure):
    _fields_ = [
        ("T", ctypes.c_int64), ("d", ctypes.c_int64), ("E", ctypes.c_int64),
        ("k", ctypes.c_int64), ("f", ctypes.c_int64),
        ("n_groups", ctypes.c_int32), ("topk_groups", ctypes.c_int32),
        ("n_shared", ctypes.c_int32), ("f_shared", ctypes.c_int64),
        ("router", ctypes.c_int32), ("renorm", ctypes.c_int32),
        ("route_scale", ctypes.c_float), ("bias_mode", ctypes.c_int32),
        ("expert_bias", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("aux_coef", ctypes.c_float),
        ("n_zero", ctypes.c_int32), ("n_copy", ctypes.c_int32), ("n_const", ctypes.c_int32),
        ("zc_aux_weight", ctypes.c_float),
        ("act", ctypes.c_int32), ("act_alpha", ctypes.c_float), ("act_limit", ctypes.c_float),
        ("fp8", ctypes.c_int32),
    ]


_VP = ctypes.c_void_p


class moe_params(ctypes.Structure):
    _fields_ = [(n, _VP) for n in ("w_r", "router_bias", "w_gate", "w_up", "w_down", "b_gate",
                                   "b_up", "b_down", "ws_gate", "ws_up", "ws_down", "aux_f",
                                   "zc_v", "zc_wc", "gate_threshold", "fp8_cache")] + \
                [("fp8_cache_bytes", ctypes.c_size_t)]


class moe_saved(ctypes.Structure):
    _fields_ = [(n, _VP) for n in ("topk_idx", "topk_w", "s_sel", "expert_offsets", "row_of",
                                   "token_of", "x_perm", "gu", "h", "o", "gu_sh", "h_sh", "o_sh",
                                   "router_probs", "aux_loss")]


class moe_grads(ctypes.Structure):
    _fields_ = [(n, _VP) for n in ("dw_r", "dw_gate", "dw_up", "dw_down", "db_gate", "db_up",
                                   "db_down", "dws_gate", "dws_up", "dws_down", "dzc_v", "dzc_wc",
                                   "d_threshold")]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libmoe.so is not built (%s); run python -m paper_2605_31463_amd.build"
                          % LIB_PATH)
    # torch carries its own copy of the HIP runtime, whose file name differs
    # from the one libmoe.so asks for.  Loading torch first makes the dynamic
    # linker satisfy libmoe's libamdhip64.so.7 with torch's already-loaded copy
    # (same soname): one runtime in the process, sharing torch's streams and
    # memory.  Loaded the other way round, the process would hold two runtimes
    # and the second finds no device.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    S = ctypes.POINTER(moe_shape)
    sz = ctypes.c_size_t
    szp = ctypes.POINTER(ctypes.c_size_t)
    i32 = ctypes.c_int32
    sigs = {
        "moe_workspace_size": [S, szp, szp, szp],
        "moe_route": [S, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, sz, _VP],
        "moe_permute": [S, _VP, _VP, _VP, _VP, _VP, _VP, _VP, sz, _VP],
        "moe_permute_noalloc": [S, _VP, _VP, _VP, _VP, _VP, _VP, _VP],
        "moe_grouped_gemm_fwd": [S, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP],
        "moe_grouped_gemm_bwd": [S, i32] + [_VP] * 16 + [_VP],
        "moe_combine_fwd": [S, _VP, _VP, _VP, _VP, _VP, _VP],
        "moe_combine_bwd": [S, _VP, _VP, _VP, _VP, _VP, _VP, _VP],
        "moe_route_bwd": [S] + [_VP] * 11 + [sz, _VP],
        "moe_unpermute_bwd": [S, _VP, _VP, _VP, _VP, _VP, _VP],
        "moe_shared_expert_fwd": [S, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP],
        "moe_shared_expert_bwd": [S] + [_VP] * 12 + [sz, _VP],
        "moe_layer_fwd": [S, ctypes.POINTER(moe_params), _VP, ctypes.POINTER(moe_saved), _VP, _VP, sz, _VP],
        "moe_layer_bwd": [S, ctypes.POINTER(moe_params), _VP, ctypes.POINTER(moe_saved), _VP, _VP,
                          ctypes.POINTER(moe_grads), _VP, sz, _VP],
        "moe_layer_bwd_dgrad": [S, ctypes.POINTER(moe_params), _VP, ctypes.POINTER(moe_saved), _VP, _VP,
                                _VP, sz, _VP],
        "moe_layer_bwd_wgrad": [S, ctypes.POINTER(moe_params), _VP, ctypes.POINTER(moe_saved), _VP,
                                ctypes.POINTER(moe_grads), i32, _VP, sz, _VP],
        "moe_fp8_cache_size": [S, szp],
        "moe_fp8_cache_build": [S, _VP, _VP, _VP, _VP, sz, _VP],
        "moe_kernel_count": [],
        "moe_kernel_name": [ctypes.c_int],
        "moe_timing_select": [ctypes.c_int],
        "moe_timing_read": [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int)],
        "moe_status_string": [ctypes.c_int],
        "moe_last_error": [],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.moe_status_string.restype = ctypes.c_char_p
    lib.moe_last_error.restype = ctypes.c_char_p
    lib.moe_kernel_name.restype = ctypes.c_char_p
    return lib


LIB = _load()


def _status_string(st):
    return LIB.moe_status_string(st).decode()


def last_error():
    return LIB.moe_last_error().decode()


def _check(fn, st):
    if st != MOE_OK:
        raise MoeError(fn, st, last_error())
    return st


def P(t):
    """Device pointer of a tensor (None -> NULL)."""
    return None if t is None else t.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def make_shape(T, d, E, k, f, router="softmax_topk", n_groups=1, topk_groups=1, n_shared=0,
               f_shared=0, route_scale=1.0, bias_mode="none", expert_bias=False, dtype="bf16",
               renorm=1, aux_coef=0.0, n_zero=0, n_copy=0, n_const=0, zc_aux_weight=1.0,
               act="swiglu", act_alpha=1.702, act_limit=7.0, fp8=False):
    return moe_shape(T=T, d=d, E=E, k=k, f=f, n_groups=n_groups, topk_groups=topk_groups,
                     n_shared=n_shared, f_shared=f_shared, router=ROUTERS[router], renorm=renorm,
                     route_scale=route_scale, bias_mode=BIAS_MODES[bias_mode],
                     expert_bias=int(bool(expert_bias)), dtype=DTYPES[dtype], aux_coef=aux_coef,
                     n_zero=n_zero, n_copy=n_copy, n_const=n_const, zc_aux_weight=zc_aux_weight,
                     act=ACTS[act], act_alpha=act_alpha, act_limit=act_limit, fp8=int(fp8))


def pool_size(shape):
    """Experts the router chooses from: E plus the zero-computation experts."""
    return shape.E + shape.n_zero + shape.n_copy + shape.n_const


def shape_from_config(cfg, T=None):
    return make_shape(T=cfg["T"] if T is None else T, d=cfg["d"], E=cfg["E"], k=cfg["k"],
                      f=cfg["f"], router=cfg["router"], n_groups=cfg["n_groups"],
                      topk_groups=cfg["topk_groups"], n_shared=cfg["n_shared"],
                      f_shared=cfg["f_shared"], route_scale=cfg["route_scale"],
                      bias_mode=cfg["bias_mode"], expert_bias=cfg["expert_bias"],
                      dtype=cfg["dtype"], aux_coef=cfg.get("aux_coef", 0.0),
                      n_zero=cfg.get("n_zero", 0), n_copy=cfg.get("n_copy", 0),
                      n_const=cfg.get("n_const", 0), zc_aux_weight=cfg.get("zc_aux_weight", 1.0),
                      act=cfg.get("act", "swiglu"), act_alpha=cfg.get("act_alpha", 1.702),
                      act_limit=cfg.get("act_limit", 7.0), fp8=cfg.get("fp8", False))


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def moe_workspace_size(shape):
    a, b, c = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check("moe_workspace_size", LIB.moe_workspace_size(ctypes.byref(shape), ctypes.byref(a),
                                                         ctypes.byref(b), ctypes.byref(c)))
    return a.value, b.value, c.value


def _ws(ws):
    return (None, 0) if ws is None else (ws.data_ptr(), ws.numel() * ws.element_size())


def moe_route(shape, x, w_r, router_bias, topk_idx, topk_w, s_sel, expert_counts, ws=None, stream=None):
    wp, wb = _ws(ws)
    return _check("moe_route", LIB.moe_route(ctypes.byref(shape), P(x), P(w_r), P(router_bias),
                                             P(topk_idx), P(topk_w), P(s_sel), P(expert_counts),
                                             wp, wb, _stream(stream)))


def moe_permute(shape, x, topk_idx, expert_offsets, row_of, token_of, x_perm, ws, stream=None):
    wp, wb = _ws(ws)
    return _check("moe_permute", LIB.moe_permute(ctypes.byref(shape), P(x), P(topk_idx),
                                                 P(expert_offsets), P(row_of), P(token_of),
                                                 P(x_perm), wp, wb, _stream(stream)))


def moe_permute_noalloc(shape, x, topk_idx, expert_offsets, row_of, token_of, x_perm, stream=None):
    return _check("moe_permute_noalloc", LIB.moe_permute_noalloc(ctypes.byref(shape), P(x), P(topk_idx),
                                                                 P(expert_offsets), P(row_of), P(token_of),
                                                                 P(x_perm), _stream(stream)))


def moe_grouped_gemm_fwd(shape, x_perm, expert_offsets, w_gate, w_up, w_down, b_gate, b_up, b_down,
                         gu, h, o, stream=None):
    return _check("moe_grouped_gemm_fwd", LIB.moe_grouped_gemm_fwd(
        ctypes.byref(shape), P(x_perm), P(expert_offsets), P(w_gate), P(w_up), P(w_down),
        P(b_gate), P(b_up), P(b_down), P(gu), P(h), P(o), _stream(stream)))


def moe_grouped_gemm_bwd(shape, passes, x_perm, expert_offsets, gu, h, d_o, w_gate, w_up, w_down,
                         dgu, dx_perm, dw_gate, dw_up, dw_down, db_gate, db_up, db_down, stream=None):
    return _check("moe_grouped_gemm_bwd", LIB.moe_grouped_gemm_bwd(
        ctypes.byref(shape), passes, P(x_perm), P(expert_offsets), P(gu), P(h), P(d_o), P(w_gate),
        P(w_up), P(w_down), P(dgu), P(dx_perm), P(dw_gate), P(dw_up), P(dw_down), P(db_gate),
        P(db_up), P(db_down), _stream(stream)))


def moe_combine_fwd(shape, o, topk_w, row_of, shared_o, y, stream=None):
    return _check("moe_combine_fwd", LIB.moe_combine_fwd(ctypes.byref(shape), P(o), P(topk_w),
                                                         P(row_of), P(shared_o), P(y), _stream(stream)))


def moe_combine_bwd(shape, dy, o, topk_w, row_of, d_o, d_topk_w, stream=None):
    return _check("moe_combine_bwd", LIB.moe_combine_bwd(ctypes.byref(shape), P(dy), P(o), P(topk_w),
                                                         P(row_of), P(d_o), P(d_topk_w), _stream(stream)))


def moe_route_bwd(shape, x, w_r, topk_idx, topk_w, s_sel, d_topk_w, expert_offsets, token_of, dw_r,
                  dx_router, ws, stream=None):
    wp, wb = _ws(ws)
    return _check("moe_route_bwd", LIB.moe_route_bwd(
        ctypes.byref(shape), P(x), P(w_r), P(topk_idx), P(topk_w), P(s_sel), P(d_topk_w),
        P(expert_offsets), P(token_of), P(dw_r), P(dx_router), wp, wb, _stream(stream)))


def moe_unpermute_bwd(shape, dx_perm, row_of, dx_router, dx_shared, dx, stream=None):
    return _check("moe_unpermute_bwd", LIB.moe_unpermute_bwd(
        ctypes.byref(shape), P(dx_perm), P(row_of), P(dx_router), P(dx_shared), P(dx), _stream(stream)))


def moe_shared_expert_fwd(shape, x, ws_gate, ws_up, ws_down, gu_sh, h_sh, o_sh, stream=None):
    return _check("moe_shared_expert_fwd", LIB.moe_shared_expert_fwd(
        ctypes.byref(shape), P(x), P(ws_gate), P(ws_up), P(ws_down), P(gu_sh), P(h_sh), P(o_sh),
        _stream(stream)))


def moe_shared_expert_bwd(shape, x, dy, gu_sh, h_sh, ws_gate, ws_up, ws_down, dx_shared, dws_gate,
                          dws_up, dws_down, ws, stream=None):
    wp, wb = _ws(ws)
    return _check("moe_shared_expert_bwd", LIB.moe_shared_expert_bwd(
        ctypes.byref(shape), P(x), P(dy), P(gu_sh), P(h_sh), P(ws_gate), P(ws_up), P(ws_down),
        P(dx_shared), P(dws_gate), P(dws_up), P(dws_down), wp, wb, _stream(stream)))


def _struct(cls, tensors):
    """Pointer fields from tensors (or None); size fields from ints."""
    f = dict(cls._fields_)
    return cls(**{n: ((0 if t is None else int(t)) if f[n] is ctypes.c_size_t else P(t))
                  for n, t in tensors.items() if n in f})


def moe_layer_fwd(shape, params, x, saved, y, ws, stream=None):
    """params / saved: dicts of tensors keyed by the C struct field names."""
    wp, wb = _ws(ws)
    pr = _struct(moe_params, params)
    sv = _struct(moe_saved, saved)
    return _check("moe_layer_fwd", LIB.moe_layer_fwd(ctypes.byref(shape), ctypes.byref(pr), P(x),
                                                     ctypes.byref(sv), P(y), wp, wb, _stream(stream)))


def moe_layer_bwd(shape, params, x, saved, dy, dx, grads, ws, stream=None):
    wp, wb = _ws(ws)
    pr = _struct(moe_params, params)
    sv = _struct(moe_saved, saved)
    gr = _struct(moe_grads, grads)
    return _check("moe_layer_bwd", LIB.moe_layer_bwd(ctypes.byref(shape), ctypes.byref(pr), P(x),
                                                     ctypes.byref(sv), P(dy), P(dx), ctypes.byref(gr),
                                                     wp, wb, _stream(stream)))


def moe_layer_bwd_dgrad(shape, params, x, saved, dy, dx, ws, stream=None):
    wp, wb = _ws(ws)
    pr = _struct(moe_params, params)
    sv = _struct(moe_saved, saved)
    return _check("moe_layer_bwd_dgrad", LIB.moe_layer_bwd_dgrad(
        ctypes.byref(shape), ctypes.byref(pr), P(x), ctypes.byref(sv), P(dy), P(dx), wp, wb, _stream(stream)))


def moe_layer_bwd_wgrad(shape, params, x, saved, dy, grads, accumulate, ws, stream=None):
    wp, wb = _ws(ws)
    pr = _struct(moe_params, params)
    sv = _struct(moe_saved, saved)
    gr = _struct(moe_grads, grads)
    return _check("moe_layer_bwd_wgrad", LIB.moe_layer_bwd_wgrad(
        ctypes.byref(shape), ctypes.byref(pr), P(x), ctypes.byref(sv), P(dy), ctypes.byref(gr),
        int(accumulate), wp, wb, _stream(stream)))


def moe_kernel_count():
    return LIB.moe_kernel_count()


def moe_kernel_name(i):
    n = LIB.moe_kernel_name(i)
    return None if n is None else n.decode()


def moe_timing_select(i):
    return LIB.moe_timing_select(i)


def moe_timing_read():
    ms, n = ctypes.c_double(), ctypes.c_int()
    _check("moe_timing_read", LIB.moe_timing_read(ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def kernel_id(name):
    for i in range(moe_kernel_count()):
        if moe_kernel_name(i) == name:
            return i
    raise KeyError(name)


def moe_fp8_cache_size(shape):
    b = ctypes.c_size_t()
    _check("moe_fp8_cache_size", LIB.moe_fp8_cache_size(ctypes.byref(shape), ctypes.byref(b)))
    return b.value


def moe_fp8_cache_build(shape, w_gate, w_up, w_down, cache, stream=None):
    cp, cb = _ws(cache)
    return _check("moe_fp8_cache_build", LIB.moe_fp8_cache_build(ctypes.byref(shape), P(w_gate), P(w_up),
                                                                 P(w_down), cp, cb, _stream(stream)))
