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
    # int64 x5, int32 x3 (+pad), int64, int32 x2, float, int32 x3, float (+pad) -> 96 bytes
    assert ctypes.sizeof(L.moe_shape) == 96
    assert L.moe_shape.f_shared.offset == 56
    assert L.moe_shape.aux_coef.offset == 88
    # pointer structs: one pointer per field, in the header's order
    assert ctypes.sizeof(L.moe_params) == 12 * 8 and L.moe_params.aux_f.offset == 88
    assert ctypes.sizeof(L.moe_saved) == 15 * 8 and L.moe_saved.aux_loss.offset == 112


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
