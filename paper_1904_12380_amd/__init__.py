"""Python binding for the MI355X row-softmax C ABI (include/softmax_mi355x.h).

Argument marshalling only: every step of the softmax runs in the HIP kernels
of ``lib/libsoftmax_mi355x.so``.  torch supplies device memory and the
current stream.  There is no fallback: if the library is not built, or the
tensors are not on the GPU, these functions raise.

Functions keep the C names:

    softmax_fwd(x, out=None, stream=None) -> torch.Tensor
    softmax_fwd_ptr(x_ptr, y_ptr, rows, cols, stream_handle) -> int
    softmax_fwd_clip(x, clip_lo, out=None, stream=None) -> torch.Tensor
    softmax_fwd_clip_ptr(x_ptr, y_ptr, rows, cols, clip_lo, stream_handle) -> int
    softmax_fwd_approx(x, clip_lo=-64.0, out=None, stream=None) -> torch.Tensor
    softmax_fwd_approx_ptr(x_ptr, y_ptr, rows, cols, clip_lo, stream_handle) -> int
    softmax_log_fwd(x, clip_lo=-64.0, out=None, stream=None) -> torch.Tensor
    softmax_log_fwd_ptr(x_ptr, y_ptr, rows, cols, clip_lo, stream_handle) -> int
    softmax_attention_fwd(q, k, v, scale=None, clip_lo=-64.0, out=None, stream=None)
    softmax_attention_fwd_ptr(q_ptr, k_ptr, v_ptr, o_ptr, batch, lq, lk, d, dv,
                              scale, clip_lo, stream_handle) -> int
    softmax_plan(rows, cols, x_ptr=1 << 44, y_ptr=1 << 45) -> dict
    softmax_fwd_planned(x, plan, out=None, stream=None) -> torch.Tensor
    softmax_fwd_planned_ptr(x_ptr, y_ptr, rows, cols, plan, stream_handle) -> int
    softmax_exchange_status() -> dict
    softmax_exp_probe(x, m, out=None, stream=None, clip_lo=-64.0) -> torch.Tensor
    softmax_copy_probe(x, out=None, stream=None) -> torch.Tensor
    softmax_strerror(code) -> str
    softmax_last_hip_error() -> int
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "LIB_PATH", "HEADER_PATH", "SoftmaxError", "load_library", "softmax_fwd",
    "softmax_fwd_ptr", "softmax_fwd_clip", "softmax_fwd_clip_ptr", "softmax_plan",
    "softmax_fwd_approx", "softmax_fwd_approx_ptr", "softmax_log_fwd", "softmax_log_fwd_ptr",
    "softmax_nll_fwd", "softmax_nll_fwd_ptr",
    "softmax_attention_fwd", "softmax_attention_fwd_ptr", "ATTN_MAX_KEYS", "ATTN_MAX_DIM",
    "softmax_exp_probe", "softmax_copy_probe", "softmax_strerror", "softmax_last_hip_error",
    "softmax_fwd_planned", "softmax_fwd_planned_ptr", "softmax_exchange_status",
    "CLIP_LO", "CLIP_MAX", "KERNEL_NAMES",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libsoftmax_mi355x.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "softmax_mi355x.h")

CLIP_LO = -64.0
CLIP_MAX = -48.0
ATTN_MAX_KEYS = 64
ATTN_MAX_DIM = 65536
OK, ERR_INVALID_ARG, ERR_HIP, ERR_NOT_DEVICE = 0, 1, 2, 3
KERNEL_NAMES = {0: "none", 1: "packed", 2: "wave_row", 3: "block_row", 4: "split_row",
                5: "group_rows"}
KERNEL_IDS = {v: k for k, v in KERNEL_NAMES.items()}


class SoftmaxError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        msg = f"{what}: {softmax_strerror(code)} (code {code})"
        if code == ERR_HIP:
            msg += f", hipError_t {softmax_last_hip_error()}"
        super().__init__(msg)


class _Plan(ctypes.Structure):
    _fields_ = [
        ("kernel", ctypes.c_int32),
        ("vec_width", ctypes.c_int32),
        ("lanes_per_row", ctypes.c_int32),
        ("elems_per_lane", ctypes.c_int32),
        ("block_threads", ctypes.c_int32),
        ("launches", ctypes.c_int32),
        ("chunks_per_row", ctypes.c_int64),
        ("grid", ctypes.c_int64),
        ("workspace_bytes", ctypes.c_int64),
        ("store_delay_ns", ctypes.c_int64),
    ]


_lib = None


def load_library() -> ctypes.CDLL:
    """Load the built library (no HIP call happens at load time)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_1904_12380_amd.build` "
            "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.softmax_fwd.argtypes = [vp, vp, i64, i64, vp]
    lib.softmax_fwd.restype = ctypes.c_int
    lib.softmax_fwd_clip.argtypes = [vp, vp, i64, i64, ctypes.c_float, vp]
    lib.softmax_fwd_clip.restype = ctypes.c_int
    f32 = ctypes.c_float
    lib.softmax_attention_fwd.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i64, f32, f32, vp]
    lib.softmax_attention_fwd.restype = ctypes.c_int
    lib.softmax_strerror.argtypes = [ctypes.c_int]
    lib.softmax_strerror.restype = ctypes.c_char_p
    lib.softmax_last_hip_error.argtypes = []
    lib.softmax_last_hip_error.restype = ctypes.c_int
    lib.softmax_plan.argtypes = [vp, vp, i64, i64, ctypes.POINTER(_Plan)]
    lib.softmax_plan.restype = ctypes.c_int
    lib.softmax_exp_probe.argtypes = [vp, vp, vp, i64, ctypes.c_float, ctypes.c_int, vp]
    lib.softmax_fwd_approx.argtypes = [vp, vp, i64, i64, ctypes.c_float, vp]
    lib.softmax_fwd_approx.restype = ctypes.c_int
    lib.softmax_log_fwd.argtypes = [vp, vp, i64, i64, ctypes.c_float, vp]
    lib.softmax_log_fwd.restype = ctypes.c_int
    lib.softmax_nll_fwd.argtypes = [vp, vp, vp, i64, i64, ctypes.c_float, vp]
    lib.softmax_nll_fwd.restype = ctypes.c_int
    lib.softmax_exp_probe.restype = ctypes.c_int
    lib.softmax_copy_probe.argtypes = [vp, vp, i64, vp]
    lib.softmax_copy_probe.restype = ctypes.c_int
    lib.softmax_fwd_planned.argtypes = [vp, vp, i64, i64, ctypes.POINTER(_Plan), vp]
    lib.softmax_fwd_planned.restype = ctypes.c_int
    u64p = ctypes.POINTER(ctypes.c_uint64)
    lib.softmax_exchange_status.argtypes = [u64p, u64p, ctypes.POINTER(ctypes.c_int32)]
    lib.softmax_exchange_status.restype = ctypes.c_int
    _lib = lib
    return lib


def softmax_strerror(code: int) -> str:
    return load_library().softmax_strerror(int(code)).decode()


def softmax_last_hip_error() -> int:
    return int(load_library().softmax_last_hip_error())


def softmax_plan(rows: int, cols: int, x_ptr: int = 1 << 44,
                 y_ptr: int = 1 << 45) -> dict:
    """Host-only description of what softmax_fwd would launch.  The default
    pointers are 16-byte aligned placeholders; they are never dereferenced."""
    p = _Plan()
    rc = load_library().softmax_plan(x_ptr, y_ptr, rows, cols, ctypes.byref(p))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_plan")
    d = {name: int(getattr(p, name)) for name, _ in _Plan._fields_}
    d["kernel_name"] = KERNEL_NAMES[d["kernel"]]
    return d


def _plan_struct(plan: dict) -> _Plan:
    p = _Plan()
    for name, _ in _Plan._fields_:
        if name in plan:
            setattr(p, name, int(plan[name]))
    if "kernel_name" in plan:
        p.kernel = KERNEL_IDS[plan["kernel_name"]]
    if "store_delay_ns" not in plan:
        p.store_delay_ns = -1
    return p


def softmax_fwd_planned_ptr(x_ptr: int, y_ptr: int, rows: int, cols: int, plan: dict,
                            stream_handle: int = 0) -> int:
    """Raw C call; returns the C return code.  ``plan`` holds kernel (or
    kernel_name), vec_width and, for split rows, block_threads and
    elems_per_lane; store_delay_ns defaults to -1 (the library's schedule)."""
    p = _plan_struct(plan)
    return int(load_library().softmax_fwd_planned(x_ptr, y_ptr, rows, cols, ctypes.byref(p),
                                                  stream_handle))


def softmax_exchange_status() -> dict:
    """Give-up counters and held row entries of the split-row exchange on
    the current device (synchronous)."""
    f, w = ctypes.c_uint64(), ctypes.c_uint64()
    busy = ctypes.c_int32()
    rc = load_library().softmax_exchange_status(ctypes.byref(f), ctypes.byref(w),
                                                ctypes.byref(busy))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_exchange_status")
    return {"join_give_ups": int(f.value), "wait_give_ups": int(w.value),
            "entries_in_use": int(busy.value)}


def softmax_fwd_ptr(x_ptr: int, y_ptr: int, rows: int, cols: int,
                    stream_handle: int = 0) -> int:
    """Raw C call; returns the C return code."""
    return int(load_library().softmax_fwd(x_ptr, y_ptr, rows, cols, stream_handle))


def _torch():
    import torch
    return torch


def _stream_handle(stream) -> int:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _check_f32_cuda(t, name: str):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (no CPU path exists)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major, leading dim = cols)")


def softmax_fwd_clip_ptr(x_ptr: int, y_ptr: int, rows: int, cols: int, clip_lo: float,
                         stream_handle: int = 0) -> int:
    """Raw C call; returns the C return code."""
    return int(load_library().softmax_fwd_clip(x_ptr, y_ptr, rows, cols, float(clip_lo),
                                               stream_handle))


def _out_for(x, out):
    torch = _torch()
    _check_f32_cuda(x, "x")
    if x.dim() != 2:
        raise ValueError("x must be 2-D [rows, cols]")
    if out is None:
        return torch.empty_like(x)
    _check_f32_cuda(out, "out")
    if out.shape != x.shape or out.device != x.device:
        raise ValueError("out must match x in shape and device")
    return out


def softmax_fwd(x, out=None, stream=None):
    """Row-wise clipped softmax (bound -64) of a 2-D float32 GPU tensor
    [rows, cols].

    ``out`` may be ``x`` itself (in place).  Runs on ``stream`` (default: the
    current torch stream) and returns without synchronising."""
    torch = _torch()
    out = _out_for(x, out)
    rows, cols = x.shape
    with torch.cuda.device(x.device):
        rc = softmax_fwd_ptr(x.data_ptr(), out.data_ptr(), rows, cols,
                             _stream_handle(stream))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_fwd")
    return out


def softmax_fwd_planned(x, plan: dict, out=None, stream=None):
    """softmax_fwd with a caller-chosen kernel (see softmax_fwd_planned_ptr)."""
    torch = _torch()
    out = _out_for(x, out)
    rows, cols = x.shape
    with torch.cuda.device(x.device):
        rc = softmax_fwd_planned_ptr(x.data_ptr(), out.data_ptr(), rows, cols, plan,
                                     _stream_handle(stream))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_fwd_planned")
    return out


def softmax_fwd_clip(x, clip_lo: float, out=None, stream=None):
    """softmax_fwd with the clip bound as an argument: any value <= CLIP_MAX,
    or -inf for no clip."""
    torch = _torch()
    out = _out_for(x, out)
    rows, cols = x.shape
    with torch.cuda.device(x.device):
        rc = softmax_fwd_clip_ptr(x.data_ptr(), out.data_ptr(), rows, cols, clip_lo,
                                  _stream_handle(stream))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_fwd_clip")
    return out


def softmax_fwd_approx_ptr(x_ptr: int, y_ptr: int, rows: int, cols: int, clip_lo: float,
                           stream_handle: int = 0) -> int:
    """Raw C call; returns the C return code."""
    return int(load_library().softmax_fwd_approx(x_ptr, y_ptr, rows, cols, float(clip_lo),
                                                 stream_handle))


def softmax_fwd_approx(x, clip_lo: float = CLIP_LO, out=None, stream=None):
    """softmax_fwd_clip with the fast fp32 exponential (looser, stated
    bound: 2e-6 + 1.5e-7 |x - max| relative)."""
    torch = _torch()
    out = _out_for(x, out)
    rows, cols = x.shape
    with torch.cuda.device(x.device):
        rc = softmax_fwd_approx_ptr(x.data_ptr(), out.data_ptr(), rows, cols, clip_lo,
                                    _stream_handle(stream))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_fwd_approx")
    return out


def softmax_log_fwd_ptr(x_ptr: int, y_ptr: int, rows: int, cols: int, clip_lo: float,
                        stream_handle: int = 0) -> int:
    """Raw C call; returns the C return code."""
    return int(load_library().softmax_log_fwd(x_ptr, y_ptr, rows, cols, float(clip_lo),
                                              stream_handle))


def softmax_log_fwd(x, clip_lo: float = CLIP_LO, out=None, stream=None):
    """Row-wise log of the clipped softmax, y = max(x - M, clip_lo) - ln S."""
    torch = _torch()
    out = _out_for(x, out)
    rows, cols = x.shape
    with torch.cuda.device(x.device):
        rc = softmax_log_fwd_ptr(x.data_ptr(), out.data_ptr(), rows, cols, clip_lo,
                                 _stream_handle(stream))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_log_fwd")
    return out


def softmax_nll_fwd_ptr(x_ptr: int, labels_ptr: int, loss_ptr: int, rows: int, cols: int,
                        clip_lo: float, stream_handle: int = 0) -> int:
    """Raw C call; returns the C return code."""
    return int(load_library().softmax_nll_fwd(x_ptr, labels_ptr, loss_ptr, rows, cols,
                                              float(clip_lo), stream_handle))


def softmax_nll_fwd(x, labels, clip_lo: float = CLIP_LO, out=None, stream=None):
    """Per-row negative log-likelihood of ``labels`` (int64 GPU tensor
    [rows]) under the clipped softmax of ``x`` [rows, cols]:
    loss = ln S - max(x[label] - M, clip_lo).  Returns float32 [rows]; a
    label outside [0, cols) gives NaN."""
    torch = _torch()
    _check_f32_cuda(x, "x")
    if x.dim() != 2:
        raise ValueError("x must be 2-D [rows, cols]")
    rows, cols = x.shape
    if not isinstance(labels, torch.Tensor) or labels.dtype != torch.int64:
        raise TypeError("labels must be an int64 torch.Tensor")
    if labels.shape != (rows,) or labels.device != x.device or not labels.is_contiguous():
        raise ValueError("labels must be contiguous [rows] on x's device")
    if out is None:
        out = torch.empty(rows, dtype=torch.float32, device=x.device)
    _check_f32_cuda(out, "out")
    if out.shape != (rows,) or out.device != x.device:
        raise ValueError("out must be [rows] on x's device")
    with torch.cuda.device(x.device):
        rc = softmax_nll_fwd_ptr(x.data_ptr(), labels.data_ptr(), out.data_ptr(), rows, cols,
                                 clip_lo, _stream_handle(stream))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_nll_fwd")
    return out


def softmax_attention_fwd_ptr(q_ptr: int, k_ptr: int, v_ptr: int, o_ptr: int, batch: int,
                              lq: int, lk: int, d: int, dv: int, scale: float,
                              clip_lo: float = CLIP_LO, stream_handle: int = 0) -> int:
    """Raw C call; returns the C return code."""
    return int(load_library().softmax_attention_fwd(
        q_ptr, k_ptr, v_ptr, o_ptr, batch, lq, lk, d, dv, float(scale), float(clip_lo),
        stream_handle))


def softmax_attention_fwd(q, k, v, scale=None, clip_lo: float = CLIP_LO, out=None,
                          stream=None):
    """O = softmax_clip(scale * Q K^T) V per batch element, on the matrix
    cores, for float32 GPU tensors q [B, lq, d], k [B, lk, d], v [B, lk, dv].
    ``scale`` defaults to 1/sqrt(d) rounded to float32."""
    torch = _torch()
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        _check_f32_cuda(t, name)
        if t.dim() != 3:
            raise ValueError(f"{name} must be 3-D [batch, len, dim]")
    b, lq, d = q.shape
    if k.shape[0] != b or k.shape[2] != d or v.shape[:2] != k.shape[:2]:
        raise ValueError("q, k, v shapes do not match")
    lk, dv = k.shape[1], v.shape[2]
    if scale is None:
        scale = float(torch.tensor(1.0 / max(d, 1) ** 0.5, dtype=torch.float32))
    if out is None:
        out = torch.empty((b, lq, dv), dtype=torch.float32, device=q.device)
    else:
        _check_f32_cuda(out, "out")
        if tuple(out.shape) != (b, lq, dv):
            raise ValueError("out must be [batch, lq, dv]")
    with torch.cuda.device(q.device):
        rc = softmax_attention_fwd_ptr(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                       b, lq, lk, d, dv, scale, clip_lo, _stream_handle(stream))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_attention_fwd")
    return out


def softmax_exp_probe(x, m, out=None, stream=None, clip_lo: float = CLIP_LO,
                      approx=False):
    """e = exp(max(x - m, clip_lo)) elementwise through the kernels' exp
    routine (the fast approximation of softmax_fwd_approx if ``approx`` is
    true or 1); ``approx=2`` gives e = 2^x from the bare v_exp_f32
    instruction (``m`` may then be None)."""
    torch = _torch()
    _check_f32_cuda(x, "x")
    if m is None:
        if int(approx) != 2:
            raise ValueError("m is needed unless approx == 2")
    else:
        _check_f32_cuda(m, "m")
        if m.shape != x.shape:
            raise ValueError("m must match x")
    if out is None:
        out = torch.empty_like(x)
    _check_f32_cuda(out, "out")
    with torch.cuda.device(x.device):
        rc = int(load_library().softmax_exp_probe(
            x.data_ptr(), None if m is None else m.data_ptr(), out.data_ptr(), x.numel(),
            float(clip_lo), int(approx), _stream_handle(stream)))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_exp_probe")
    return out


def softmax_copy_probe(x, out=None, stream=None):
    """out = x through the library's 128-bit copy kernel (bandwidth ceiling)."""
    torch = _torch()
    _check_f32_cuda(x, "x")
    if out is None:
        out = torch.empty_like(x)
    _check_f32_cuda(out, "out")
    if out.numel() != x.numel():
        raise ValueError("out must have as many elements as x")
    with torch.cuda.device(x.device):
        rc = int(load_library().softmax_copy_probe(
            x.data_ptr(), out.data_ptr(), x.numel(), _stream_handle(stream)))
    if rc != OK:
        raise SoftmaxError(rc, "softmax_copy_probe")
    return out
