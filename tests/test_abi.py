"""CPU checks of the C ABI: the library loads, exports every entry point that
include/moe.h declares, sizes its workspaces, and rejects bad arguments on
the host before enqueueing anything (no GPU needed: every call here fails
validation before any HIP call)."""
import ctypes
import os
import re

import pytest

from paper_2605_31463_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "moe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(moe_\w+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    for n in ("moe_route", "moe_permute", "moe_grouped_gemm_fwd", "moe_grouped_gemm_bwd",
              "moe_combine_fwd", "moe_combine_bwd", "moe_route_bwd", "moe_unpermute_bwd",
              "moe_layer_fwd", "moe_layer_bwd", "moe_workspace_size"):
        assert n in names, n
    lib = ctypes.CDLL(L.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_workspace_sizes_scale_with_shape():
    s1 = L.make_shape(T=1024, d=2048, E=128, k=8, f=768)
    s2 = L.make_shape(T=2048, d=2048, E=128, k=8, f=768)
    f1, v1, b1 = L.moe_workspace_size(s1)
    f2, v2, b2 = L.moe_workspace_size(s2)
    assert 0 < f1 <= f2 and 0 < v1 < v2 and 0 < b1 < b2
    R = 2048 * 8
    # backward keeps d_o, dgu and dx_perm (bf16)
    assert b2 >= R * (2048 + 2 * 768 + 2048) * 2


@pytest.mark.parametrize("kw,status", [
    (dict(k=9, E=8), L.MOE_ERR_INVALID_ARG),
    (dict(d=0), L.MOE_ERR_INVALID_ARG),
    (dict(T=-1), L.MOE_ERR_INVALID_ARG),
    (dict(E=12, n_groups=5, topk_groups=2, router="sigmoid_grouped"), L.MOE_ERR_INVALID_ARG),
    (dict(E=16, n_groups=4, topk_groups=5, router="sigmoid_grouped"), L.MOE_ERR_INVALID_ARG),
    (dict(E=16, k=9, n_groups=4, topk_groups=2, router="sigmoid_grouped"), L.MOE_ERR_INVALID_ARG),
    (dict(E=16, n_groups=4, topk_groups=2), L.MOE_ERR_INVALID_ARG),
    (dict(route_scale=0.0), L.MOE_ERR_INVALID_ARG),
    (dict(n_shared=1, f_shared=0), L.MOE_ERR_INVALID_ARG),
    (dict(renorm=0), L.MOE_ERR_UNSUPPORTED),
    (dict(E=512, k=8), L.MOE_ERR_UNSUPPORTED),
    (dict(k=17, E=32), L.MOE_ERR_UNSUPPORTED),
    (dict(d=100), L.MOE_ERR_UNSUPPORTED),
    (dict(f=96), L.MOE_ERR_UNSUPPORTED),
    (dict(aux_coef=-1.0), L.MOE_ERR_INVALID_ARG),
    (dict(aux_coef=float("nan")), L.MOE_ERR_INVALID_ARG),
    (dict(E=16, k=4, n_groups=4, topk_groups=2, router="sigmoid_grouped", aux_coef=1e-3), L.MOE_ERR_UNSUPPORTED),
    (dict(n_zero=-1), L.MOE_ERR_INVALID_ARG),
    (dict(n_const=2, zc_aux_weight=-0.5), L.MOE_ERR_INVALID_ARG),
    (dict(n_const=2, zc_aux_weight=float("inf")), L.MOE_ERR_INVALID_ARG),
    (dict(E=16, k=4, n_groups=4, topk_groups=2, router="sigmoid_grouped", n_copy=1), L.MOE_ERR_UNSUPPORTED),
    (dict(E=250, k=8, n_zero=4, n_copy=4), L.MOE_ERR_UNSUPPORTED),     # pool of 258
    (dict(E=2, k=5, n_zero=1, n_copy=1), L.MOE_ERR_INVALID_ARG),       # k above the pool of 4
    (dict(router="sigmoid_threshold", n_copy=1), L.MOE_ERR_UNSUPPORTED),
    (dict(router="sigmoid_threshold", bias_mode="select"), L.MOE_ERR_UNSUPPORTED),
    (dict(router="sigmoid_threshold", E=16, n_groups=4, topk_groups=2), L.MOE_ERR_INVALID_ARG),
    (dict(fp8=True, dtype="f32"), L.MOE_ERR_UNSUPPORTED),
    (dict(fp8=True, dtype="bf16", d=192), L.MOE_ERR_UNSUPPORTED),
    (dict(fp8=2, dtype="bf16", f=192), L.MOE_ERR_UNSUPPORTED),
    (dict(fp8=3, dtype="bf16"), L.MOE_ERR_INVALID_ARG),
    (dict(act="clamped_glu", act_alpha=0.0), L.MOE_ERR_INVALID_ARG),
    (dict(act="clamped_glu", act_limit=float("inf")), L.MOE_ERR_INVALID_ARG),
])
def test_bad_shapes_rejected(kw, status):
    base = dict(T=64, d=128, E=8, k=2, f=256)
    base.update(kw)
    s = L.make_shape(**base)
    with pytest.raises(L.MoeError) as ei:
        L.moe_workspace_size(s)
    assert ei.value.status == status
    assert L.last_error()


def test_null_pointers_rejected_before_launch():
    s = L.make_shape(T=64, d=128, E=8, k=2, f=256)
    st = L.LIB.moe_route(ctypes.byref(s), None, None, None, None, None, None, None, None, 0, None)
    assert st == L.MOE_ERR_INVALID_ARG
    st = L.LIB.moe_combine_fwd(ctypes.byref(s), None, None, None, None, None, None)
    assert st == L.MOE_ERR_INVALID_ARG
    st = L.LIB.moe_grouped_gemm_bwd(ctypes.byref(s), 3, *([None] * 16), None)
    assert st == L.MOE_ERR_INVALID_ARG
    st = L.LIB.moe_grouped_gemm_bwd(ctypes.byref(s), 4, *([None] * 16), None)
    assert st == L.MOE_ERR_INVALID_ARG
    st = L.LIB.moe_shared_expert_fwd(ctypes.byref(s), *([None] * 7), None)
    assert st == L.MOE_ERR_INVALID_ARG   # shape has no shared expert
    st = L.LIB.moe_layer_fwd(ctypes.byref(s), None, None, None, None, None, 0, None)
    assert st == L.MOE_ERR_INVALID_ARG
    assert "params" in L.last_error()


def test_workspace_too_small_is_reported():
    s = L.make_shape(T=64, d=128, E=8, k=2, f=256)
    fake = ctypes.c_void_p(16)   # never dereferenced: the size check fails first
    st = L.LIB.moe_permute(ctypes.byref(s), fake, fake, fake, fake, fake, fake, fake, 1, None)
    assert st == L.MOE_ERR_WORKSPACE
    assert "workspace" in L.last_error()


def test_status_strings_and_kernel_names():
    assert L.LIB.moe_status_string(0) == b"ok"
    assert L.LIB.moe_status_string(-4).startswith(b"workspace")
    names = [L.moe_kernel_name(i) for i in range(L.moe_kernel_count())]
    assert "gemm_gateup_fwd" in names and "route" in names and len(set(names)) == len(names)
    assert L.moe_kernel_name(L.moe_kernel_count()) is None


def test_shape_struct_layout_matches_header():
    # int64 x5, int32 x3 (+pad), int64, int32 x2, float, int32 x3, float, int32 x3,
    # float, int32, float x2, int32 (+pad) -> 128 bytes
    assert ctypes.sizeof(L.moe_shape) == 128
    assert L.moe_shape.f_shared.offset == 56
    assert L.moe_shape.aux_coef.offset == 88
    assert L.moe_shape.zc_aux_weight.offset == 104
    assert L.moe_shape.act_limit.offset == 116
    assert L.moe_shape.fp8.offset == 120
    # pointer structs: one pointer per field, in the header's order
    assert ctypes.sizeof(L.moe_params) == 17 * 8 and L.moe_params.fp8_cache.offset == 120
    assert L.moe_params.fp8_cache_bytes.offset == 128
    assert ctypes.sizeof(L.moe_saved) == 15 * 8 and L.moe_saved.aux_loss.offset == 112
    assert ctypes.sizeof(L.moe_grads) == 13 * 8 and L.moe_grads.d_threshold.offset == 96


def declared_arities():
    src = open(os.path.join(ROOT, "include", "moe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    out = {}
    for m in re.finditer(r"^\s*(?:const\s+)?\w+\**\s+\**(moe_\w+)\s*\(([^)]*)\)\s*;", src, flags=re.M | re.S):
        args = m.group(2).strip()
        out[m.group(1)] = 0 if args in ("", "void") else args.count(",") + 1
    return out


def test_binding_arity_matches_header():
    ar = declared_arities()
    assert len(ar) == len(declared_functions())
    for name, n in ar.items():
        fn = getattr(L.LIB, name)
        assert len(fn.argtypes) == n, (name, len(fn.argtypes), n)


def test_one_hip_runtime_in_process():
    """libmoe.so must bind to the HIP runtime torch already loaded: a second
    copy of the runtime in the process finds no device at its first launch."""
    import torch  # noqa: F401
    maps = open("/proc/self/maps").read().splitlines()
    hip = {ln.split()[-1] for ln in maps if "libamdhip64" in ln}
    assert len(hip) == 1, hip


def test_accumulate_arguments_rejected_on_the_host():
    """accumulate outside {0, 1}, and MOE_ACCUMULATE without the weight-gradient
    pass, fail validation before any HIP call."""
    s = L.make_shape(T=16, d=128, E=8, k=2, f=128)
    pr, sv, gr = L.moe_params(), L.moe_saved(), L.moe_grads()
    st = L.LIB.moe_layer_bwd_wgrad(ctypes.byref(s), ctypes.byref(pr), None, ctypes.byref(sv), None,
                                   ctypes.byref(gr), 2, None, 0, None)
    assert st == L.MOE_ERR_INVALID_ARG and "accumulate" in L.last_error()
    st = L.LIB.moe_grouped_gemm_bwd(ctypes.byref(s), L.MOE_DGRAD | L.MOE_ACCUMULATE, *([None] * 16), None)
    assert st == L.MOE_ERR_INVALID_ARG and "MOE_ACCUMULATE" in L.last_error()
    st = L.LIB.moe_grouped_gemm_bwd(ctypes.byref(s), 8, *([None] * 16), None)
    assert st == L.MOE_ERR_INVALID_ARG
    st = L.LIB.moe_layer_bwd_dgrad(ctypes.byref(s), None, None, None, None, None, None, 0, None)
    assert st == L.MOE_ERR_INVALID_ARG


def test_zero_computation_shapes_on_the_host():
    """The pool (E plus zero-computation experts) sizes the router's
    workspaces; the gather-side component entry points refuse such shapes;
    the layer entry points ask for the constant experts' parameters."""
    base = dict(T=512, d=256, E=16, k=4, f=128)
    f0, v0, b0 = L.moe_workspace_size(L.make_shape(**base))
    f1, v1, b1 = L.moe_workspace_size(L.make_shape(**base, n_zero=2, n_copy=2, n_const=4))
    assert f1 > f0 and v1 > v0 and b1 > b0
    s = L.make_shape(**base, n_copy=1)
    assert L.LIB.moe_combine_fwd(ctypes.byref(s), None, None, None, None, None, None) == L.MOE_ERR_UNSUPPORTED
    assert L.LIB.moe_combine_bwd(ctypes.byref(s), *([None] * 6), None) == L.MOE_ERR_UNSUPPORTED
    assert L.LIB.moe_unpermute_bwd(ctypes.byref(s), *([None] * 5), None) == L.MOE_ERR_UNSUPPORTED
    s = L.make_shape(**base, n_const=2)
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    pr = L.moe_params(w_r=fake, w_gate=fake, w_up=fake, w_down=fake)
    sv = L.moe_saved(**{n: fake for n, _ in L.moe_saved._fields_})
    st = L.LIB.moe_layer_fwd(ctypes.byref(s), ctypes.byref(pr), fake, ctypes.byref(sv), fake, fake, 1 << 40, None)
    assert st == L.MOE_ERR_INVALID_ARG and "zc_v" in L.last_error()
    gr = L.moe_grads(**{n: fake for n, _ in L.moe_grads._fields_ if not n.startswith("dzc")})
    st = L.LIB.moe_layer_bwd_wgrad(ctypes.byref(s), ctypes.byref(pr), fake, ctypes.byref(sv), fake,
                                   ctypes.byref(gr), 0, fake, 1 << 40, None)
    assert st == L.MOE_ERR_INVALID_ARG and "dzc_v" in L.last_error()


def test_threshold_router_on_the_host():
    """moe_route refuses the threshold router; the layer asks for the
    thresholds and their gradient buffer."""
    s = L.make_shape(T=64, d=128, E=8, k=4, f=128, router="sigmoid_threshold")
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    st = L.LIB.moe_route(ctypes.byref(s), fake, fake, None, fake, fake, fake, None, fake, 1 << 40, None)
    assert st == L.MOE_ERR_UNSUPPORTED and "threshold" in L.last_error()
    pr = L.moe_params(w_r=fake, w_gate=fake, w_up=fake, w_down=fake)
    sv = L.moe_saved(**{n: fake for n, _ in L.moe_saved._fields_})
    st = L.LIB.moe_layer_fwd(ctypes.byref(s), ctypes.byref(pr), fake, ctypes.byref(sv), fake, fake, 1 << 40, None)
    assert st == L.MOE_ERR_INVALID_ARG and "gate_threshold" in L.last_error()
    gr = L.moe_grads(**{n: fake for n, _ in L.moe_grads._fields_ if n != "d_threshold"})
    st = L.LIB.moe_layer_bwd_wgrad(ctypes.byref(s), ctypes.byref(pr), fake, ctypes.byref(sv), fake,
                                   ctypes.byref(gr), 0, fake, 1 << 40, None)
    assert st == L.MOE_ERR_INVALID_ARG and "d_threshold" in L.last_error()


def test_fp8_cache_on_the_host():
    """The cache size scales with the experts; building needs shape.fp8 and a
    large enough cache; the layer forward asks for the cache."""
    s = L.make_shape(T=64, d=256, E=4, k=2, f=128, dtype="bf16", fp8=True)
    n = L.moe_fp8_cache_size(s)
    assert n >= 3 * 4 * 256 * 128 + 4 * (2 * 4 * 128 + 4 * 256) * 2
    with pytest.raises(L.MoeError) as ei:
        L.moe_fp8_cache_size(L.make_shape(T=64, d=256, E=4, k=2, f=128, dtype="bf16"))
    assert ei.value.status == L.MOE_ERR_UNSUPPORTED
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    st = L.LIB.moe_fp8_cache_build(ctypes.byref(s), fake, fake, fake, fake, n - 1, None)
    assert st == L.MOE_ERR_WORKSPACE
    pr = L.moe_params(w_r=fake, w_gate=fake, w_up=fake, w_down=fake)
    sv = L.moe_saved(**{nm: fake for nm, _ in L.moe_saved._fields_})
    st = L.LIB.moe_layer_fwd(ctypes.byref(s), ctypes.byref(pr), fake, ctypes.byref(sv), fake, fake, 1 << 40, None)
    assert st == L.MOE_ERR_INVALID_ARG and "fp8_cache" in L.last_error()
    # a cache smaller than the shape's (say, built for another shape) is refused
    pr = L.moe_params(w_r=fake, w_gate=fake, w_up=fake, w_down=fake, fp8_cache=fake, fp8_cache_bytes=n - 1)
    st = L.LIB.moe_layer_fwd(ctypes.byref(s), ctypes.byref(pr), fake, ctypes.byref(sv), fake, fake, 1 << 40, None)
    assert st == L.MOE_ERR_WORKSPACE and "fp8_cache_bytes" in L.last_error()


def test_fp8_dgrad_on_the_host():
    """fp8 = 2 (data-gradient GEMMs too): the cache holds the row-quantised
    weights as well (twice the codes), the layer backward asks for the cache,
    and the standalone grouped backward refuses the FP8 data-gradient passes
    (their operands are the layer's)."""
    s1 = L.make_shape(T=64, d=256, E=4, k=2, f=128, dtype="bf16", fp8=1)
    s2 = L.make_shape(T=64, d=256, E=4, k=2, f=128, dtype="bf16", fp8=2)
    n1, n2 = L.moe_fp8_cache_size(s1), L.moe_fp8_cache_size(s2)
    assert n2 >= n1 + 3 * 4 * 256 * 128 + 4 * (4 * 256 + 4 * 128)
    fwd1, _, bwd1 = L.moe_workspace_size(s1)
    fwd2, _, bwd2 = L.moe_workspace_size(s2)
    R = 64 * 2
    assert fwd2 == fwd1 and bwd2 >= bwd1 + R * (256 + 2 * 128) + 2 * R * 4
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    pr = L.moe_params(w_r=fake, w_gate=fake, w_up=fake, w_down=fake)
    sv = L.moe_saved(**{nm: fake for nm, _ in L.moe_saved._fields_})
    st = L.LIB.moe_layer_bwd_dgrad(ctypes.byref(s2), ctypes.byref(pr), fake, ctypes.byref(sv), fake, fake,
                                   fake, 1 << 40, None)
    assert st == L.MOE_ERR_INVALID_ARG and "fp8_cache" in L.last_error()
    # a cache built at fp8 = 1 lacks the row codes fp8 = 2 reads: refused by size
    pr = L.moe_params(w_r=fake, w_gate=fake, w_up=fake, w_down=fake, fp8_cache=fake, fp8_cache_bytes=n1)
    st = L.LIB.moe_layer_bwd_dgrad(ctypes.byref(s2), ctypes.byref(pr), fake, ctypes.byref(sv), fake, fake,
                                   fake, 1 << 40, None)
    assert st == L.MOE_ERR_WORKSPACE and "fp8_cache_bytes" in L.last_error()
    st = L.LIB.moe_grouped_gemm_bwd(ctypes.byref(s2), L.MOE_DGRAD, fake, fake, fake, fake, fake, fake, fake, fake,
                                    fake, fake, None, None, None, None, None, None, None)
    assert st == L.MOE_ERR_UNSUPPORTED and "FP8" in L.last_error()


def test_operands_beyond_the_descriptor_reach_are_refused():
    """Operands staged through the kernels' 32-bit buffer descriptors must stay
    below 4 GiB: a shape whose routed rows times the row width reach 2^32
    bytes (one expert may hold every row), a shared expert whose dense gate/up
    rows do, or an expert weight that does, is refused before anything runs."""
    ok = L.make_shape(T=131072, d=8192, E=8, k=1, f=1024, dtype="bf16")          # R d 2 = 2 GiB
    L.moe_workspace_size(ok)
    for kw in (dict(T=262144, d=8192, E=8, k=1, f=1024),                          # R d 2 = 4 GiB
               dict(T=65536, d=4096, E=8, k=8, f=1024),                           # R d 2 = 4 GiB
               dict(T=16384, d=1024, E=8, k=8, f=8192),                           # R 2f 2 = 4 GiB
               dict(T=64, d=16384, E=2, k=1, f=65536)):                           # d 2f 2 = 4 GiB
        with pytest.raises(L.MoeError) as ei:
            L.moe_workspace_size(L.make_shape(dtype="bf16", **kw))
        assert ei.value.status == L.MOE_ERR_UNSUPPORTED and "4 GiB" in L.last_error(), kw
    with pytest.raises(L.MoeError) as ei:
        L.moe_workspace_size(L.make_shape(T=262144, d=4096, E=8, k=1, f=1024, dtype="bf16",
                                          n_shared=1, f_shared=4096))             # T 2 fs 2 = 4 GiB
    assert ei.value.status == L.MOE_ERR_UNSUPPORTED
