"""The allocation-free permutation entry point (moe_permute_noalloc, for
callers that cannot allocate device memory) against moe_permute on the same
inputs, through the C ABI: bitwise equal maps and permuted rows on two calls
in a row, the second with fewer tokens (the fixed scratch keeps the first
call's histograms, which the second must not read), and the size limit of its
fixed scratch refused on the host."""
import numpy as np
import pytest

from moe_inputs import layer_inputs, variant
from tests.helpers import dev, device_params

pytestmark = pytest.mark.gpu


def _permute_both(cfg, inp):
    import torch
    from paper_2605_31463_amd import _lib as L
    shape = L.shape_from_config(cfg)
    T, d, k = cfg["T"], cfg["d"], cfg["k"]
    Ep = L.pool_size(shape)
    R = T * k
    x = dev(inp["x"], cfg["dtype"])
    p = device_params(inp, cfg)
    fws, _, _ = L.moe_workspace_size(shape)
    ws = torch.empty(max(fws, 1), dtype=torch.uint8, device="cuda")
    idx = torch.empty(T, k, dtype=torch.int32, device="cuda")
    w = torch.empty(T, k, dtype=torch.float32, device="cuda")
    s_sel = torch.empty(T, k, dtype=torch.float32, device="cuda")
    L.moe_route(shape, x, p["w_r"], p["router_bias"], idx, w, s_sel, None, ws)
    act = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    outs = []
    for noalloc in (False, True):
        offs = torch.full((Ep + 1,), -7, dtype=torch.int32, device="cuda")
        row_of = torch.full((T, k), -7, dtype=torch.int32, device="cuda")
        token_of = torch.full((R,), -7, dtype=torch.int32, device="cuda")
        x_perm = torch.zeros(R, d, dtype=act, device="cuda")
        if noalloc:
            L.moe_permute_noalloc(shape, x, idx, offs, row_of, token_of, x_perm)
        else:
            L.moe_permute(shape, x, idx, offs, row_of, token_of, x_perm, ws)
        outs.append((offs, row_of, token_of, x_perm))
    torch.cuda.synchronize()
    return outs


def test_noalloc_permute_equals_permute_twice():
    import torch
    # Qwen3 widths, then fewer tokens and experts: the second call reads
    # histograms of its own blocks only
    for cfg in (variant("qwen3", T=4096), variant("qwen3", T=1000, E=64, k=4), variant("tiny", T=37)):
        print("noalloc permute", cfg["name"], flush=True)
        inp = layer_inputs(cfg, seed=5)
        ref, got = _permute_both(cfg, inp)
        for name, a, b in zip(("expert_offsets", "row_of", "token_of", "x_perm"), ref, got):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), (cfg["name"], name)
        offs = ref[0].cpu().numpy()
        assert offs[0] == 0 and offs[-1] == cfg["T"] * cfg["k"] and np.all(np.diff(offs) >= 0)


def test_noalloc_permute_refuses_shapes_beyond_its_scratch():
    from paper_2605_31463_amd import _lib as L
    import ctypes
    big = L.make_shape(T=(1 << 20) + 1, d=128, E=256, k=1, f=128)  # 4097 blocks x 256 x 4 B > 4 MiB
    fake = ctypes.c_void_p(16)   # never dereferenced: the size check fails first
    st = L.LIB.moe_permute_noalloc(ctypes.byref(big), fake, fake, fake, fake, fake, fake, None)
    assert st == L.MOE_ERR_UNSUPPORTED and "scratch" in L.last_error()
