"""linsimp_fwd_static (the forward for callers that cannot allocate) against
linsimp_fwd with a caller workspace, through the C ABI.  Named to be
collected last.

Two calls in a row on the same GPU share the library's static scratch; the
second is smaller than the first, so it runs over the first call's leftovers.
Both must give the bits of linsimp_fwd on a freshly allocated workspace filled
with NaN (the forward reads nothing it has not written).  Dims whose forward
workspace exceeds the static scratch are refused before any launch.
"""

import ctypes

import pytest
import torch

from paper_2608_09307_amd import linsimp as L
from paper_2608_09307_amd.workloads import Workload, make_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _reference(x, w):
    d = L.dims_of(x["q"], x["v"], x["omega"], w)
    ws = L.alloc_workspace(d, False, DEV)
    ws.view(torch.uint8).fill_(0xFF)                    # NaN bytes
    return L.fwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], w, workspace=ws)


@pytest.mark.parametrize("first,second", [
    (Workload("static_a", 4, 8, 2048, 64, 64, 64, 64, "bf16", "fwd", seed=81),      # 57 MiB of scratch
     Workload("static_b", 1, 2, 300, 128, 128, 128, 64, "bf16", "fwd", seed=82)),
    (Workload("static_c", 2, 2, 777, 128, 128, 256, 64, "bf16", "fwd", seed=83),
     Workload("static_d", 1, 1, 100, 32, 32, 32, 20, "f32", "fwd", seed=84)),
])
def test_fwd_static_equals_fwd_on_two_calls(first, second):
    for wl in (first, second):
        print(f"[fwd_static] {wl}", flush=True)
        x = make_inputs(wl, device=DEV, with_grad=False)
        need = L.workspace_size(L.dims_of(x["q"], x["v"], x["omega"], wl.w), False)
        assert need <= L.FWD_STATIC_MAX_BYTES, need
        o_s, s_s = L.fwd_static(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w)
        o_r, s_r = _reference(x, wl.w)
        torch.cuda.synchronize()
        assert torch.equal(o_s, o_r)
        assert torch.equal(s_s, s_r)
        assert bool(torch.isfinite(o_s.float()).all())


def test_fwd_static_refuses_dims_beyond_its_scratch():
    lib = L.lib()
    vp = ctypes.c_void_p
    d = L.make_dims(2, 16, 16384, 128, 128, 128, 64, L.BF16)      # 1.6 GiB of scratch
    assert L.workspace_size(d, False) > L.FWD_STATIC_MAX_BYTES
    ptrs = [vp(4096 * (i + 1)) for i in range(8)]
    rc = lib.linsimp_fwd_static(ctypes.byref(d), *ptrs, vp(0))
    assert rc == -3 and b"static scratch" in lib.linsimp_last_error()
