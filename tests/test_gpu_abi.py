"""GPU checks of the C ABI contract: error codes for invalid arguments (nothing is
enqueued), no writes on rejected calls, and the kernel-timing hooks."""
import ctypes

import pytest
import torch

from paper_2606_28560_amd import fibattn as F
from paper_2606_28560_amd import schedules

pytestmark = pytest.mark.gpu

FIB = schedules.FIB15


def _t(B=1, H=2, T=64, D=64, dtype=torch.bfloat16):
    return torch.randn(B, H, T, D, device="cuda").to(dtype)


def test_forward_rejects_bad_arguments():
    q, k, v = _t(), _t(), _t()
    o = torch.full_like(q, 7.0)
    lse = torch.full((1, 2, 64), 7.0, device="cuda")
    bad = [
        dict(W=-1), dict(W=129), dict(base=[2, 1]), dict(base=[0, 1]), dict(alpha=0.0),
        dict(alpha=float("nan")), dict(alpha=float("inf")), dict(base=list(range(1, 34))),
    ]
    for kw in bad:
        args = dict(W=8, base=FIB, alpha=1.0)
        args.update(kw)
        with pytest.raises(F.FibattnError):
            F.fibattn_forward(q, k, v, args["W"], args["base"], args["alpha"], o=o, lse=lse)
    L = F.lib()
    b = (ctypes.c_int32 * 15)(*FIB)
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    # null pointer, unsupported head size, misaligned pointer
    assert L.fibattn_forward(None, k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                             1, 2, 64, 64, 8, b, 15, ctypes.c_float(1.0), 1, s) == 1
    assert L.fibattn_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                             1, 2, 64, 48, 8, b, 15, ctypes.c_float(1.0), 1, s) == 2
    assert L.fibattn_forward(q.data_ptr() + 2, k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                             1, 2, 63, 64, 8, b, 15, ctypes.c_float(1.0), 1, s) == 1
    assert L.fibattn_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                             1, 2, 64, 64, 8, b, 15, ctypes.c_float(1.0), 7, s) == 1
    torch.cuda.synchronize()
    assert torch.all(o == 7.0) and torch.all(lse == 7.0), "a rejected call wrote its outputs"


def test_backward_rejects_small_workspace():
    q, k, v, g = _t(), _t(), _t(), _t()
    o, lse = F.fibattn_forward(q, k, v, 8, FIB, 1.0)
    need = F.fibattn_backward_workspace_bytes(1, 2, 64, 64, 8, 15)
    ws = torch.empty(need - 1, device="cuda", dtype=torch.uint8)
    with pytest.raises(F.FibattnError) as ei:
        F.fibattn_backward(q, k, v, o, lse, g, 8, FIB, 1.0, workspace=ws)
    assert ei.value.status == 3
    ws = torch.empty(need, device="cuda", dtype=torch.uint8)
    F.fibattn_backward(q, k, v, o, lse, g, 8, FIB, 1.0, workspace=ws)
    torch.cuda.synchronize()


def test_kernel_timing_hooks():
    q, k, v = _t(T=1024), _t(T=1024), _t(T=1024)
    F.fibattn_timing_begin("forward", 4)
    for _ in range(6):
        F.fibattn_forward(q, k, v, 8, FIB, 1.0)
    ms, n = F.fibattn_timing_end()
    assert n == 4 and ms > 0
