"""Python binding of libfibattn.so (argument marshalling only).

Every function has the name of the C entry point it calls (include/fibattn.h).
Tensors are torch CUDA (HIP) tensors used only as device memory; every step of the
attention runs in the library's HIP kernels, launched on torch's current stream.
There is no fallback: if the library is missing or a call fails, these functions
raise.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfibattn.so")

FIBATTN_FP32, FIBATTN_BF16 = 0, 1
MAX_RUNGS = 32
MAX_WINDOW = 128
KERNEL_IDS = {"rope": 0, "forward": 1, "bwd_dq": 2, "bwd_dkdv": 3, "dalpha_reduce": 4, "alpha": 5}
EXPORTED = ("fibattn_rung_table", "fibattn_forward", "fibattn_backward_workspace_bytes",
            "fibattn_backward", "fibattn_forward_gqa", "fibattn_backward_gqa",
            "fibattn_forward_strided", "fibattn_backward_strided",
            "fibattn_device_table_bytes", "fibattn_device_table", "fibattn_forward_dt",
            "fibattn_backward_dt", "fibattn_alpha_from_theta", "fibattn_dtheta", "fibattn_rope",
            "fibattn_rope_qk", "fibattn_status_string", "fibattn_timing_begin", "fibattn_timing_end",
            "fibattn_backward_noalloc", "fibattn_device_table_theta", "fibattn_rope_qk_table",
            "fibattn_forward_rope_q", "fibattn_forward_rope_q_dt", "fibattn_forward_rope_q_strided")
SCRATCH_BYTES = 64 << 20  # FIBATTN_SCRATCH_BYTES: the allocation-free backward's static scratch


class FibattnError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: status {status} ({status_string(status)})")


_lib = None


def lib():
    """The loaded libfibattn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(or python -m paper_2606_28560_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    ip = ctypes.POINTER(ctypes.c_int32)
    fp = ctypes.POINTER(ctypes.c_float)
    L.fibattn_rung_table.argtypes = [f, ip, i, i, ip, fp, ip, ctypes.POINTER(ctypes.c_int)]
    L.fibattn_rung_table.restype = i
    L.fibattn_forward.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, ip, i, f, i, vp]
    L.fibattn_forward.restype = i
    L.fibattn_backward_workspace_bytes.argtypes = [i, i, i, i, i, i]
    L.fibattn_backward_workspace_bytes.restype = sz
    L.fibattn_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                   i, i, i, i, i, ip, i, f, f, i, vp]
    L.fibattn_backward.restype = i
    L.fibattn_forward_gqa.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, ip, i, f, i, vp]
    L.fibattn_forward_gqa.restype = i
    L.fibattn_forward_rope_q.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, ip, i, f, f, i, vp]
    L.fibattn_forward_rope_q.restype = i
    L.fibattn_forward_rope_q_dt.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, vp, f, i, vp]
    L.fibattn_forward_rope_q_strided.argtypes = [vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, ip, i, f, f, i, vp]
    L.fibattn_forward_rope_q_strided.restype = i
    L.fibattn_forward_rope_q_dt.restype = i
    L.fibattn_backward_gqa.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                       i, i, i, i, i, i, ip, i, f, f, i, vp]
    L.fibattn_backward_gqa.restype = i
    L.fibattn_forward_strided.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, ip, i, f, i, vp]
    L.fibattn_forward_strided.restype = i
    L.fibattn_backward_strided.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp,
                                           i, i, i, i, i, i, ip, i, f, f, i, vp]
    L.fibattn_backward_strided.restype = i
    L.fibattn_device_table_bytes.argtypes = []
    L.fibattn_device_table_bytes.restype = sz
    L.fibattn_device_table.argtypes = [vp, ip, i, i, vp, vp]
    L.fibattn_device_table.restype = i
    L.fibattn_forward_dt.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, vp, i, vp]
    L.fibattn_forward_dt.restype = i
    L.fibattn_backward_dt.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                      i, i, i, i, i, i, vp, f, i, vp]
    L.fibattn_device_table_theta.argtypes = [vp, vp, ip, i, i, vp, vp]
    L.fibattn_device_table_theta.restype = i
    L.fibattn_rope_qk_table.argtypes = [vp, vp, vp, vp, i, i, i, i, i, f, vp, vp, ip, i, i, vp, i, vp]
    L.fibattn_rope_qk_table.restype = i
    L.fibattn_backward_dt.restype = i
    L.fibattn_alpha_from_theta.argtypes = [vp, vp, i, vp]
    L.fibattn_alpha_from_theta.restype = i
    L.fibattn_dtheta.argtypes = [vp, vp, vp, i, vp]
    L.fibattn_dtheta.restype = i
    L.fibattn_rope.argtypes = [vp, vp, i, i, i, i, f, i, i, vp]
    L.fibattn_rope.restype = i
    L.fibattn_rope_qk.argtypes = [vp, vp, vp, vp, i, i, i, i, f, i, vp]
    L.fibattn_rope_qk.restype = i
    L.fibattn_backward_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                           i, i, i, i, i, i, ip, i, f, f, i, vp]
    L.fibattn_backward_noalloc.restype = i
    L.fibattn_status_string.argtypes = [i]
    L.fibattn_status_string.restype = ctypes.c_char_p
    L.fibattn_timing_begin.argtypes = [i, i]
    L.fibattn_timing_begin.restype = i
    L.fibattn_timing_end.argtypes = [fp, ctypes.POINTER(ctypes.c_int)]
    L.fibattn_timing_end.restype = i
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().fibattn_status_string(int(status)).decode()


def _check(fn: str, status: int):
    if status != 0:
        raise FibattnError(fn, status)


def _base_array(base):
    b = np.ascontiguousarray(np.asarray(list(base), dtype=np.int32))
    return b, b.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.float32:
        return FIBATTN_FP32
    if t.dtype == torch.bfloat16:
        return FIBATTN_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; expected float32 or bfloat16")


def _stream(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check_tensor(name, t, shape, dtype, strided=False):
    """strided: any placement whose rows (last dimension) are contiguous."""
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if strided:
        if t.dim() != 4 or (t.shape[3] > 1 and t.stride(3) != 1):
            raise ValueError(f"{name} must have contiguous rows (last-dimension stride 1)")
    elif not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")


def fibattn_rung_table(alpha: float, base, W: int):
    """Host rung table: list of (floor(d_k), w_k, f_k) in increasing distance."""
    b, bp = _base_array(base)
    d0 = (ctypes.c_int32 * MAX_RUNGS)()
    w = (ctypes.c_float * MAX_RUNGS)()
    f = (ctypes.c_int32 * MAX_RUNGS)()
    n = ctypes.c_int(0)
    st = lib().fibattn_rung_table(ctypes.c_float(alpha), bp, b.size, int(W), d0, w, f, ctypes.byref(n))
    _check("fibattn_rung_table", st)
    return [(int(d0[a]), np.float32(w[a]), int(f[a])) for a in range(n.value)]


def _kv_heads(q, k):
    """Key/value head count: k, v are [B,H_kv,T,D] with H_kv dividing H (grouped heads)."""
    B, H, T, D = q.shape
    if k.dim() != 4 or k.shape[0] != B or tuple(k.shape[2:]) != (T, D) or k.shape[1] < 1 \
            or H % k.shape[1]:
        raise ValueError(f"k: shape {tuple(k.shape)} does not group q {tuple(q.shape)}")
    return k.shape[1]


def _layouts(*ts):
    """fibattn_layout_t array of the tensors' (batch, head, position) element strides."""
    arr = (ctypes.c_int64 * (3 * len(ts)))()
    for a, t in enumerate(ts):
        arr[3 * a], arr[3 * a + 1], arr[3 * a + 2] = t.stride(0), t.stride(1), t.stride(2)
    return arr


def fibattn_forward_rope_q(q, k, v, W: int, base, alpha: float, rope_base: float = 10000.0, *, o=None,
                           lse=None, q_out=None, keep_q=True, stream=None):
    """o, lse, q_out = forward of the UNROTATED q with keys k already rotated (fibattn_rope,
    same rope_base); the queries are rotated where the forward loads them.  q_out = R q
    (may be q itself), the rotated queries a later backward takes; keep_q=False writes no
    q_out (forward only) and returns None for it.  q [B,H,T,D]; k, v [B,H_kv,T,D] with
    H_kv dividing H; q, k, v, o, q_out may be views with contiguous rows (e.g. slices of
    a fused [B,T,3,H,D] projection output)."""
    import torch

    B, H, T, D = q.shape
    Hkv = _kv_heads(q, k)
    _check_tensor("q", q, q.shape, q.dtype, strided=True)
    for n_, t in (("k", k), ("v", v)):
        _check_tensor(n_, t, (B, Hkv, T, D), q.dtype, strided=True)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H, T), device=q.device, dtype=torch.float32) if lse is None else lse
    _check_tensor("o", o, q.shape, q.dtype, strided=True)
    _check_tensor("lse", lse, (B, H, T), torch.float32)
    if keep_q:
        q_out = torch.empty_like(q) if q_out is None else q_out
        _check_tensor("q_out", q_out, q.shape, q.dtype, strided=True)
    elif q_out is not None:
        raise ValueError("q_out given with keep_q=False")
    b, bp = _base_array(base)
    ptrs = (q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
            q_out.data_ptr() if keep_q else None)
    tail = (T, D, int(W), bp, b.size, ctypes.c_float(alpha), ctypes.c_float(rope_base), _dtype_code(q),
            _stream(stream))
    if all(t.is_contiguous() for t in (q, k, v, o) + ((q_out,) if keep_q else ())):
        st = lib().fibattn_forward_rope_q(*ptrs, B, H, Hkv, *tail)
        _check("fibattn_forward_rope_q", st)
    else:
        lay = _layouts(q, k, v, o, q_out if keep_q else q)
        st = lib().fibattn_forward_rope_q_strided(*ptrs, lay, B, H, Hkv, *tail)
        _check("fibattn_forward_rope_q_strided", st)
    return o, lse, q_out


def fibattn_forward_rope_q_dt(q, k, v, W: int, table, rope_base: float = 10000.0, *, o=None, lse=None,
                              q_out=None, keep_q=True, stream=None):
    """As fibattn_forward_rope_q, with the rung table built on the device."""
    import torch

    B, H, T, D = q.shape
    Hkv = _kv_heads(q, k)
    _check_tensor("q", q, q.shape, q.dtype)
    for n_, t in (("k", k), ("v", v)):
        _check_tensor(n_, t, (B, Hkv, T, D), q.dtype)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H, T), device=q.device, dtype=torch.float32) if lse is None else lse
    _check_tensor("o", o, q.shape, q.dtype)
    _check_tensor("lse", lse, (B, H, T), torch.float32)
    if keep_q:
        q_out = torch.empty_like(q) if q_out is None else q_out
        _check_tensor("q_out", q_out, q.shape, q.dtype)
    elif q_out is not None:
        raise ValueError("q_out given with keep_q=False")
    st = lib().fibattn_forward_rope_q_dt(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                                         q_out.data_ptr() if keep_q else None, B, H, Hkv, T, D, int(W),
                                         table.data_ptr(), ctypes.c_float(rope_base), _dtype_code(q),
                                         _stream(stream))
    _check("fibattn_forward_rope_q_dt", st)
    return o, lse, q_out


def fibattn_forward(q, k, v, W: int, base, alpha: float, *, o=None, lse=None, stream=None):
    """o, lse = forward of post-RoPE q, k and v (float32 or bfloat16).

    q: [B,H,T,D]; k, v: [B,H_kv,T,D] with H_kv dividing H (H_kv < H: grouped heads).
    q, k, v, o may be any views with contiguous rows (e.g. slices of a [B,T,3,H,D]
    projection output, transposed); lse is packed [B,H,T]."""
    import torch

    B, H, T, D = q.shape
    Hkv = _kv_heads(q, k)
    _check_tensor("q", q, q.shape, q.dtype, strided=True)
    for n_, t in (("k", k), ("v", v)):
        _check_tensor(n_, t, (B, Hkv, T, D), q.dtype, strided=True)
    if o is None:
        o = torch.empty((B, H, T, D), device=q.device, dtype=q.dtype)
    if lse is None:
        lse = torch.empty((B, H, T), device=q.device, dtype=torch.float32)
    _check_tensor("o", o, q.shape, q.dtype, strided=True)
    _check_tensor("lse", lse, (B, H, T), torch.float32)
    b, bp = _base_array(base)
    ptrs = (q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr())
    tail = (T, D, int(W), bp, b.size, ctypes.c_float(alpha), _dtype_code(q), _stream(stream))
    if not all(t.is_contiguous() for t in (q, k, v, o)):
        st = lib().fibattn_forward_strided(*ptrs, _layouts(q, k, v, o), B, H, Hkv, *tail)
        _check("fibattn_forward_strided", st)
    elif Hkv == H:
        st = lib().fibattn_forward(*ptrs, B, H, *tail)
        _check("fibattn_forward", st)
    else:
        st = lib().fibattn_forward_gqa(*ptrs, B, H, Hkv, *tail)
        _check("fibattn_forward_gqa", st)
    return o, lse


def fibattn_backward_workspace_bytes(B: int, H: int, T: int, d_head: int, W: int, K: int) -> int:
    return int(lib().fibattn_backward_workspace_bytes(B, H, T, d_head, int(W), int(K)))


def fibattn_backward(q, k, v, o, lse, dO, W: int, base, alpha: float, *, dq=None, dk=None, dv=None,
                     dalpha=None, workspace=None, rope_base: float = 0.0, stream=None):
    """dq, dk, dv, dalpha (a 1-element float32 device tensor).

    k, v (and dk, dv) may have fewer heads than q (grouped heads; dk, dv then sum over
    each group).  rope_base > 0: dq, dk are returned w.r.t. the unrotated q, k (R^T
    applied).  Every [B,*,T,D] tensor may be a view with contiguous rows; lse is packed."""
    import torch

    B, H, T, D = q.shape
    Hkv = _kv_heads(q, k)
    kvs = (B, Hkv, T, D)
    for n_, t, sh in (("q", q, q.shape), ("k", k, kvs), ("v", v, kvs), ("o", o, q.shape),
                      ("dO", dO, q.shape)):
        _check_tensor(n_, t, sh, q.dtype, strided=True)
    _check_tensor("lse", lse, (B, H, T), torch.float32)
    mk = lambda sh: torch.empty(sh, device=q.device, dtype=q.dtype)  # noqa: E731
    dq = mk(tuple(q.shape)) if dq is None else dq
    dk = mk(kvs) if dk is None else dk
    dv = mk(kvs) if dv is None else dv
    for n_, t, sh in (("dq", dq, q.shape), ("dk", dk, kvs), ("dv", dv, kvs)):
        _check_tensor(n_, t, sh, q.dtype, strided=True)
    if dalpha is None:
        dalpha = torch.empty(1, device=q.device, dtype=torch.float32)
    b, bp = _base_array(base)
    need = fibattn_backward_workspace_bytes(B, H, T, D, W, b.size)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=q.device, dtype=torch.uint8)
    ptrs = (q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), dO.data_ptr(),
            dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), dalpha.data_ptr(), workspace.data_ptr(),
            workspace.numel())
    tail = (T, D, int(W), bp, b.size, ctypes.c_float(alpha), ctypes.c_float(rope_base),
            _dtype_code(q), _stream(stream))
    if not all(t.is_contiguous() for t in (q, k, v, o, dO, dq, dk, dv)):
        st = lib().fibattn_backward_strided(*ptrs, _layouts(q, k, v, o, dO, dq, dk, dv), B, H, Hkv, *tail)
        _check("fibattn_backward_strided", st)
    elif Hkv == H:
        st = lib().fibattn_backward(*ptrs, B, H, *tail)
        _check("fibattn_backward", st)
    else:
        st = lib().fibattn_backward_gqa(*ptrs, B, H, Hkv, *tail)
        _check("fibattn_backward_gqa", st)
    return dq, dk, dv, dalpha


def fibattn_backward_noalloc(q, k, v, o, lse, dO, W: int, base, alpha: float, *, dq, dk, dv, dalpha,
                             rope_base: float = 0.0, stream=None):
    """As fibattn_backward on packed tensors, with the library's static device scratch
    instead of a workspace: neither this function nor the library allocates.  The
    caller passes every output (dq, dk, dv shaped like q, k, v; dalpha one float32)."""
    import torch

    B, H, T, D = q.shape
    Hkv = _kv_heads(q, k)
    kvs = (B, Hkv, T, D)
    for n_, t, sh in (("q", q, q.shape), ("k", k, kvs), ("v", v, kvs), ("o", o, q.shape),
                      ("dO", dO, q.shape), ("dq", dq, q.shape), ("dk", dk, kvs), ("dv", dv, kvs)):
        _check_tensor(n_, t, sh, q.dtype)
    _check_tensor("lse", lse, (B, H, T), torch.float32)
    if dalpha.dtype != torch.float32 or dalpha.numel() < 1 or not dalpha.is_cuda:
        raise ValueError("dalpha: a float32 device tensor")
    b, bp = _base_array(base)
    st = lib().fibattn_backward_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                        lse.data_ptr(), dO.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                        dv.data_ptr(), dalpha.data_ptr(), B, H, Hkv, T, D, int(W), bp,
                                        b.size, ctypes.c_float(alpha), ctypes.c_float(rope_base),
                                        _dtype_code(q), _stream(stream))
    _check("fibattn_backward_noalloc", st)
    return dq, dk, dv, dalpha


# ---- device-resident alpha ---------------------------------------------------------

def fibattn_device_table(alpha, base, W: int, *, table=None, stream=None):
    """Rung table of a device alpha (a 1-element float32 tensor, or one element of a
    per-layer array) built on the device; returns the table buffer (uint8 tensor)."""
    import torch

    if alpha.device.type != "cuda" or alpha.dtype != torch.float32 or alpha.numel() < 1:
        raise ValueError("alpha: a float32 device tensor")
    nb = int(lib().fibattn_device_table_bytes())
    if table is None:
        table = torch.empty(nb, device=alpha.device, dtype=torch.uint8)
    if table.numel() < nb or not table.is_contiguous():
        raise ValueError(f"table: {nb} contiguous bytes")
    b, bp = _base_array(base)
    st = lib().fibattn_device_table(alpha.data_ptr(), bp, b.size, int(W), table.data_ptr(), _stream(stream))
    _check("fibattn_device_table", st)
    return table


def fibattn_device_table_theta(theta, base, W: int, *, table=None, alpha=None, stream=None):
    """Rung table of alpha = 0.5 + sigmoid(theta) for a device theta (a 1-element float32
    tensor, or one element of a per-layer array), built on the device in one launch;
    writes alpha too when given.  Returns the table buffer (uint8 tensor)."""
    import torch

    if theta.device.type != "cuda" or theta.dtype != torch.float32 or theta.numel() < 1:
        raise ValueError("theta: a float32 device tensor")
    nb = int(lib().fibattn_device_table_bytes())
    if table is None:
        table = torch.empty(nb, device=theta.device, dtype=torch.uint8)
    if table.numel() < nb or not table.is_contiguous():
        raise ValueError(f"table: {nb} contiguous bytes")
    if alpha is not None and (alpha.dtype != torch.float32 or alpha.numel() < 1 or not alpha.is_cuda):
        raise ValueError("alpha: a float32 device tensor")
    b, bp = _base_array(base)
    st = lib().fibattn_device_table_theta(theta.data_ptr(), None if alpha is None else alpha.data_ptr(), bp,
                                          b.size, int(W), table.data_ptr(), _stream(stream))
    _check("fibattn_device_table_theta", st)
    return table


def fibattn_forward_dt(q, k, v, W: int, table, *, o=None, lse=None, stream=None):
    """As fibattn_forward, with the rung table built on the device."""
    import torch

    B, H, T, D = q.shape
    Hkv = _kv_heads(q, k)
    _check_tensor("q", q, q.shape, q.dtype)
    for n_, t in (("k", k), ("v", v)):
        _check_tensor(n_, t, (B, Hkv, T, D), q.dtype)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H, T), device=q.device, dtype=torch.float32) if lse is None else lse
    _check_tensor("o", o, q.shape, q.dtype)
    _check_tensor("lse", lse, (B, H, T), torch.float32)
    st = lib().fibattn_forward_dt(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                                  B, H, Hkv, T, D, int(W), table.data_ptr(), _dtype_code(q), _stream(stream))
    _check("fibattn_forward_dt", st)
    return o, lse


def fibattn_backward_dt(q, k, v, o, lse, dO, W: int, table, *, dq=None, dk=None, dv=None,
                        dalpha=None, dtheta=None, workspace=None, rope_base: float = 0.0, stream=None):
    """As fibattn_backward, with the rung table built on the device; with `dtheta` (a
    float32 device tensor) and a table built from theta, also dL/dtheta."""
    import torch

    B, H, T, D = q.shape
    Hkv = _kv_heads(q, k)
    kvs = (B, Hkv, T, D)
    for n_, t, sh in (("q", q, q.shape), ("k", k, kvs), ("v", v, kvs), ("o", o, q.shape),
                      ("dO", dO, q.shape)):
        _check_tensor(n_, t, sh, q.dtype)
    _check_tensor("lse", lse, (B, H, T), torch.float32)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    for n_, t, sh in (("dq", dq, q.shape), ("dk", dk, kvs), ("dv", dv, kvs)):
        _check_tensor(n_, t, sh, q.dtype)
    if dalpha is None:
        dalpha = torch.empty(1, device=q.device, dtype=torch.float32)
    need = fibattn_backward_workspace_bytes(B, H, T, D, W, 0)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=q.device, dtype=torch.uint8)
    st = lib().fibattn_backward_dt(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                                   dO.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                   dalpha.data_ptr(), None if dtheta is None else dtheta.data_ptr(),
                                   workspace.data_ptr(), workspace.numel(),
                                   B, H, Hkv, T, D, int(W), table.data_ptr(), ctypes.c_float(rope_base),
                                   _dtype_code(q), _stream(stream))
    _check("fibattn_backward_dt", st)
    return dq, dk, dv, dalpha


def fibattn_alpha_from_theta(theta, *, alpha=None, stream=None):
    """alpha = 0.5 + sigmoid(theta) elementwise (float32 device tensors)."""
    import torch

    if theta.device.type != "cuda" or theta.dtype != torch.float32 or not theta.is_contiguous():
        raise ValueError("theta: a contiguous float32 device tensor")
    alpha = torch.empty_like(theta) if alpha is None else alpha
    st = lib().fibattn_alpha_from_theta(theta.data_ptr(), alpha.data_ptr(), theta.numel(), _stream(stream))
    _check("fibattn_alpha_from_theta", st)
    return alpha


def fibattn_dtheta(theta, dalpha, *, dtheta=None, stream=None):
    """dtheta = dalpha * sigmoid(theta) (1 - sigmoid(theta)) elementwise."""
    import torch

    if dalpha.shape != theta.shape or dalpha.dtype != torch.float32 or dalpha.device != theta.device:
        raise ValueError("dalpha: float32, shaped like theta, same device")
    dtheta = torch.empty_like(theta) if dtheta is None else dtheta
    st = lib().fibattn_dtheta(theta.data_ptr(), dalpha.data_ptr(), dtheta.data_ptr(), theta.numel(),
                              _stream(stream))
    _check("fibattn_dtheta", st)
    return dtheta


def fibattn_rope(x, rope_base: float = 10000.0, transpose: bool = False, *, out=None, stream=None):
    """RoPE at true positions (out may be x itself); transpose applies R^T."""
    import torch

    B, H, T, D = x.shape
    _check_tensor("x", x, x.shape, x.dtype)
    out = torch.empty_like(x) if out is None else out
    _check_tensor("out", out, x.shape, x.dtype)
    st = lib().fibattn_rope(x.data_ptr(), out.data_ptr(), B, H, T, D, ctypes.c_float(rope_base),
                            int(bool(transpose)), _dtype_code(x), _stream(stream))
    _check("fibattn_rope", st)
    return out


def fibattn_rope_qk(q, k, rope_base: float = 10000.0, *, q_out=None, k_out=None, stream=None):
    """R q and R k (RoPE at true positions) in one launch."""
    import torch

    B, H, T, D = q.shape
    _check_tensor("q", q, q.shape, q.dtype)
    _check_tensor("k", k, q.shape, q.dtype)
    q_out = torch.empty_like(q) if q_out is None else q_out
    k_out = torch.empty_like(k) if k_out is None else k_out
    _check_tensor("q_out", q_out, q.shape, q.dtype)
    _check_tensor("k_out", k_out, q.shape, q.dtype)
    st = lib().fibattn_rope_qk(q.data_ptr(), k.data_ptr(), q_out.data_ptr(), k_out.data_ptr(), B, H, T,
                               D, ctypes.c_float(rope_base), _dtype_code(q), _stream(stream))
    _check("fibattn_rope_qk", st)
    return q_out, k_out


def fibattn_rope_qk_table(q, k, rope_base: float = 10000.0, *, theta=None, base=(), W: int = 0, table=None,
                          alpha=None, q_out=None, k_out=None, stream=None):
    """R q and R k in one launch (k may have fewer heads than q); with `theta` (a float32
    device tensor) the same launch builds the rung table of alpha = 0.5 + sigmoid(theta)
    for (base, W) into `table` (allocated when None) and writes alpha when given.
    q=None rotates k alone (q_out is then None).  Returns (q_out, k_out, table)."""
    import torch

    if q is None:
        if q_out is not None:
            raise ValueError("q_out given without q")
        B, Hkv, T, D = k.shape
        H = Hkv
        _check_tensor("k", k, k.shape, k.dtype)
    else:
        B, H, T, D = q.shape
        Hkv = _kv_heads(q, k)
        _check_tensor("q", q, q.shape, q.dtype)
        _check_tensor("k", k, (B, Hkv, T, D), q.dtype)
        q_out = torch.empty_like(q) if q_out is None else q_out
        _check_tensor("q_out", q_out, q.shape, q.dtype)
    k_out = torch.empty_like(k) if k_out is None else k_out
    _check_tensor("k_out", k_out, k.shape, k.dtype)
    b, bp = _base_array(base)
    if theta is not None:
        if theta.device.type != "cuda" or theta.dtype != torch.float32 or theta.numel() < 1:
            raise ValueError("theta: a float32 device tensor")
        nb = int(lib().fibattn_device_table_bytes())
        table = torch.empty(nb, device=k.device, dtype=torch.uint8) if table is None else table
        if table.numel() < nb or not table.is_contiguous():
            raise ValueError(f"table: {nb} contiguous bytes")
    st = lib().fibattn_rope_qk_table(None if q is None else q.data_ptr(), k.data_ptr(),
                                     None if q_out is None else q_out.data_ptr(), k_out.data_ptr(), B, H, Hkv,
                                     T, D, ctypes.c_float(rope_base),
                                     None if theta is None else theta.data_ptr(),
                                     None if alpha is None else alpha.data_ptr(), bp, b.size, int(W),
                                     None if table is None else table.data_ptr(), _dtype_code(k),
                                     _stream(stream))
    _check("fibattn_rope_qk_table", st)
    return q_out, k_out, table


def fibattn_timing_begin(kernel: str, capacity: int):
    _check("fibattn_timing_begin", lib().fibattn_timing_begin(KERNEL_IDS[kernel], int(capacity)))


def fibattn_timing_end():
    """(mean launch duration in ms, number of launches timed)."""
    ms = ctypes.c_float(0.0)
    n = ctypes.c_int(0)
    _check("fibattn_timing_end", lib().fibattn_timing_end(ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)
