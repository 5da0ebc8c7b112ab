"""Thin Python binding of the C ABI in include/mg3m.h (libmg3m.so).

Functions carry the C names and only marshal arguments: every step of the
convolution runs in the library's HIP kernels.  Device buffers are torch
tensors (or raw device addresses as ints); torch provides device memory and
the current stream, nothing else.  There is no fallback: if libmg3m.so is
missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmg3m.so")

HWCN = 0
NCHW = 1
LAYOUTS = {"HWCN": HWCN, "NCHW": NCHW}

STATUS = {
    0: "MG3M_OK", 1: "MG3M_ERR_NULL", 2: "MG3M_ERR_SHAPE", 3: "MG3M_ERR_LAYOUT",
    4: "MG3M_ERR_TOO_LARGE", 5: "MG3M_ERR_ALIAS", 6: "MG3M_ERR_WORKSPACE", 7: "MG3M_ERR_PLAN",
    8: "MG3M_ERR_HIP", 9: "MG3M_ERR_ALIGN", 10: "MG3M_ERR_ARG",
}


class Mg3mError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"{STATUS.get(status, status)}: {detail}")


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("mt", ctypes.c_int), ("nt", ctypes.c_int), ("kt", ctypes.c_int),
        ("waves_m", ctypes.c_int), ("waves_n", ctypes.c_int),
        ("split", ctypes.c_int), ("k_tiles", ctypes.c_int), ("k_tiles_per_wg", ctypes.c_int),
        ("dp_tiles", ctypes.c_int), ("tail_tiles", ctypes.c_int), ("tail_wgs", ctypes.c_int),
        ("tiles_m", ctypes.c_int), ("tiles_n", ctypes.c_int),
        ("grid", ctypes.c_longlong), ("Mg", ctypes.c_longlong), ("Ng", ctypes.c_longlong),
        ("Kg", ctypes.c_longlong), ("workspace_bytes", ctypes.c_size_t), ("lds_bytes", ctypes.c_int),
        ("pad_efficiency", ctypes.c_double), ("est_us", ctypes.c_double),
        ("layout", ctypes.c_int), ("a_mode", ctypes.c_int), ("b_mode", ctypes.c_int),
        ("e_mode", ctypes.c_int),
        ("persistent", ctypes.c_int), ("via_hwcn", ctypes.c_int),
    ]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class Layer(ctypes.Structure):
    """mg3m_layer: one layer of a network for the executor."""
    _fields_ = [
        ("op", ctypes.c_int), ("input", ctypes.c_int), ("add", ctypes.c_int), ("relu", ctypes.c_int),
        ("K", ctypes.c_int), ("R", ctypes.c_int), ("S", ctypes.c_int),
        ("stride", ctypes.c_int), ("pad", ctypes.c_int), ("w", ctypes.c_void_p),
    ]


OP_CONV, OP_MAXPOOL = 0, 1

_lib = None


def load_library(path: str = LIB_PATH):
    """Load libmg3m.so (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2307_04941_amd.build`")
    # torch ships its own HIP and HSA runtimes under the same sonames as
    # ROCm's.  Loaded first, they satisfy the library's dependencies and one
    # runtime serves the process; loaded after the library, they come in as
    # second copies, and whichever runtime initialises the device second finds
    # none (hipErrorNoDevice at the first launch).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    i, p, sz, cp = ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_char_p
    shape = [i] * 10                     # N, C, H, W, K, R, S, stride, pad, layout
    shape_hw = [i] * 12                  # N, C, H, W, K, R, S, sh, sw, ph, pw, layout
    lib.conv2d_out_dims.argtypes = [i] * 6 + [ctypes.POINTER(i)] * 2
    lib.conv2d_out_dims_hw.argtypes = [i] * 8 + [ctypes.POINTER(i)] * 2
    lib.conv2d_fwd_f32_hw.argtypes = [p, p, p] + shape_hw + [p, sz, cp, p]
    lib.conv2d_fwd_f32_hw_workspace_bytes.argtypes = shape_hw + [cp, ctypes.POINTER(sz)]
    lib.conv2d_fwd_f32_acc64.argtypes = [p, p, p] + shape_hw + [cp, p]
    lib.conv2d_fwd_f32_fused.argtypes = [p, p, p, p, i] + shape_hw + [p, sz, cp, p]
    lib.maxpool2d_f32.argtypes = [p, p] + [i] * 11 + [p]
    lib.maxpool2d_out_dims.argtypes = [i] * 8 + [ctypes.POINTER(i)] * 2
    lib.mg3m_net_create.argtypes = [ctypes.POINTER(Layer), i, i, i, i, i, i, i, ctypes.POINTER(p)]
    lib.mg3m_net_activation.argtypes = [p, i, ctypes.POINTER(i), ctypes.POINTER(i), ctypes.POINTER(i),
                                        ctypes.POINTER(p)]
    lib.mg3m_net_memory.argtypes = [p, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    lib.mg3m_net_forward.argtypes = [p, p, p, p]
    lib.mg3m_net_forward_graph.argtypes = [p, p, p, p]
    lib.mg3m_net_destroy.argtypes = [p]
    lib.conv2d_fwd_f32_acc64_plan_string.argtypes = shape_hw + [cp, ctypes.c_char_p, sz]
    lib.conv2d_fwd_f32.argtypes = [p, p, p] + shape + [p]
    lib.conv2d_fwd_f32_noalloc.argtypes = [p, p, p] + shape + [p]
    lib.mg3m_launch_empty.argtypes = [p]
    lib.mg3m_probe_mfma_f32.argtypes = [p, i, i, p, ctypes.POINTER(ctypes.c_double)]
    lib.mg3m_probe_copy.argtypes = [p, p, sz, p]
    lib.mg3m_probe_fill.argtypes = [p, sz, p]
    lib.mg3m_timing_event_create.argtypes = [ctypes.POINTER(p)]
    lib.mg3m_timing_event_record.argtypes = [p, p]
    lib.mg3m_timing_event_elapsed_ms.argtypes = [p, p, ctypes.POINTER(ctypes.c_float)]
    lib.mg3m_timing_event_destroy.argtypes = [p]
    lib.conv2d_fwd_f32_ex.argtypes = [p, p, p] + shape + [p, sz, cp, p]
    lib.conv2d_fwd_f32_workspace_bytes.argtypes = shape + [cp, ctypes.POINTER(sz)]
    lib.conv2d_fwd_f32_plan_string.argtypes = shape + [cp, ctypes.c_char_p, sz]
    lib.conv2d_fwd_f32_plan_info.argtypes = shape + [cp, ctypes.POINTER(PlanInfo)]
    lib.mg3m_padding_overhead.argtypes = [i] * 5 + [ctypes.POINTER(ctypes.c_double)] * 2
    lib.mg3m_time_next_kernel.argtypes = [p, p]
    lib.mg3m_status_string.argtypes = [i]
    lib.mg3m_status_string.restype = ctypes.c_char_p
    lib.mg3m_last_error.argtypes = []
    lib.mg3m_last_error.restype = ctypes.c_char_p
    lib.mg3m_trim_workspace_pool.argtypes = []
    for name in ("conv2d_out_dims", "conv2d_out_dims_hw", "conv2d_fwd_f32_hw",
                 "conv2d_fwd_f32_hw_workspace_bytes", "conv2d_fwd_f32_acc64",
                 "conv2d_fwd_f32_acc64_plan_string", "conv2d_fwd_f32_fused", "maxpool2d_f32",
                 "maxpool2d_out_dims", "mg3m_net_create", "mg3m_net_activation", "mg3m_net_memory",
                 "mg3m_net_forward", "mg3m_net_forward_graph", "mg3m_net_destroy",
                 "conv2d_fwd_f32", "conv2d_fwd_f32_ex",
                 "conv2d_fwd_f32_workspace_bytes", "conv2d_fwd_f32_plan_string",
                 "conv2d_fwd_f32_plan_info", "mg3m_padding_overhead", "mg3m_time_next_kernel"):
        getattr(lib, name).restype = i
    _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        raise Mg3mError(rc, mg3m_last_error())


def _layout(layout) -> int:
    return LAYOUTS[layout] if isinstance(layout, str) else int(layout)


def _ptr(t) -> Optional[int]:
    """Device address of a tensor (must be fp32, contiguous, on a GPU) or an int."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor or an int device address")
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if t.dtype != torch.float32:
        raise TypeError("tensor must be float32")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _enc(plan):
    return plan.encode() if isinstance(plan, str) else plan


# ------------------------------------------------------------ C-named calls
def mg3m_status_string(status: int) -> str:
    return load_library().mg3m_status_string(status).decode()


def mg3m_last_error() -> str:
    return load_library().mg3m_last_error().decode()


def conv2d_out_dims(H, W, R, S, stride, pad):
    ho, wo = ctypes.c_int(), ctypes.c_int()
    _check(load_library().conv2d_out_dims(H, W, R, S, stride, pad, ctypes.byref(ho), ctypes.byref(wo)))
    return ho.value, wo.value


def conv2d_out_dims_hw(H, W, R, S, stride_h, stride_w, pad_h, pad_w):
    ho, wo = ctypes.c_int(), ctypes.c_int()
    _check(load_library().conv2d_out_dims_hw(H, W, R, S, stride_h, stride_w, pad_h, pad_w,
                                             ctypes.byref(ho), ctypes.byref(wo)))
    return ho.value, wo.value


def conv2d_fwd_f32_hw(x, w, y, N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout,
                      workspace=None, workspace_bytes=0, plan=None, stream=None):
    _check(load_library().conv2d_fwd_f32_hw(_ptr(x), _ptr(w), _ptr(y), N, C, H, W, K, R, S,
                                            stride_h, stride_w, pad_h, pad_w, _layout(layout),
                                            _ptr(workspace), workspace_bytes, _enc(plan),
                                            _stream(stream)))


def conv2d_fwd_f32_hw_workspace_bytes(N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w,
                                      layout, plan=None) -> int:
    b = ctypes.c_size_t()
    _check(load_library().conv2d_fwd_f32_hw_workspace_bytes(
        N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, _layout(layout), _enc(plan),
        ctypes.byref(b)))
    return b.value


def conv2d_fwd_f32_acc64(x, w, y, N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout,
                         plan=None, stream=None):
    _check(load_library().conv2d_fwd_f32_acc64(_ptr(x), _ptr(w), _ptr(y), N, C, H, W, K, R, S,
                                               stride_h, stride_w, pad_h, pad_w, _layout(layout),
                                               _enc(plan), _stream(stream)))


def conv2d_fwd_f32_acc64_plan_string(N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout,
                                     plan=None) -> str:
    buf = ctypes.create_string_buffer(1024)
    _check(load_library().conv2d_fwd_f32_acc64_plan_string(
        N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, _layout(layout), _enc(plan), buf,
        len(buf)))
    return buf.value.decode()


def conv2d_fwd_f32_fused(x, w, y, add, relu, N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w,
                         layout, workspace=None, workspace_bytes=0, plan=None, stream=None):
    _check(load_library().conv2d_fwd_f32_fused(
        _ptr(x), _ptr(w), _ptr(y), _ptr(add), int(relu), N, C, H, W, K, R, S, stride_h, stride_w,
        pad_h, pad_w, _layout(layout), _ptr(workspace), workspace_bytes, _enc(plan), _stream(stream)))


def maxpool2d_out_dims(H, W, R, S, stride_h, stride_w, pad_h, pad_w):
    ho, wo = ctypes.c_int(), ctypes.c_int()
    _check(load_library().maxpool2d_out_dims(H, W, R, S, stride_h, stride_w, pad_h, pad_w,
                                             ctypes.byref(ho), ctypes.byref(wo)))
    return ho.value, wo.value


def maxpool2d_f32(x, y, N, C, H, W, R, S, stride_h, stride_w, pad_h, pad_w, layout, stream=None):
    _check(load_library().maxpool2d_f32(_ptr(x), _ptr(y), N, C, H, W, R, S, stride_h, stride_w,
                                        pad_h, pad_w, _layout(layout), _stream(stream)))


def maxpool2d(x, R, S=None, stride=None, pad=0, layout="HWCN", out=None, stream=None):
    """Max pooling of a torch tensor on the GPU (allocates y unless `out`)."""
    import torch
    S = R if S is None else S
    sh, sw = _pair(R if stride is None else stride)
    ph, pw = _pair(pad)
    if _layout(layout) == HWCN:
        H, W, C, N = x.shape
    else:
        N, C, H, W = x.shape
    Ho, Wo = maxpool2d_out_dims(H, W, R, S, sh, sw, ph, pw)
    shape = (Ho, Wo, C, N) if _layout(layout) == HWCN else (N, C, Ho, Wo)
    y = out if out is not None else torch.empty(shape, dtype=torch.float32, device=x.device)
    maxpool2d_f32(x, y, N, C, H, W, R, S, sh, sw, ph, pw, layout, stream)
    return y


class Net:
    """A chain of layers run by the native executor (mg3m_net_*).

    layers: list of dicts with keys op ("conv" or "maxpool"), input (activation
    id, default: the previous layer's output), and for "conv": K, R, S, stride,
    pad, relu, add (activation id or -1) and w (a device filter tensor in the
    network's layout, kept referenced here); for "maxpool": R, S, stride, pad.
    input_shape: (N, C, H, W).  keep_all: keep every activation (inspection)."""

    def __init__(self, layers, input_shape, layout="HWCN", keep_all=False):
        lib = load_library()
        self._filters = []
        arr = (Layer * len(layers))()
        for i, d in enumerate(layers):
            conv = d["op"] == "conv"
            w = d.get("w") if conv else None
            if conv:
                self._filters.append(w)
            arr[i] = Layer(OP_CONV if conv else OP_MAXPOOL, int(d.get("input", i)), int(d.get("add", -1)),
                           int(d.get("relu", 0)), int(d.get("K", 0)), int(d["R"]), int(d.get("S", d["R"])),
                           int(d.get("stride", 1)), int(d.get("pad", 0)), _ptr(w) if w is not None else None)
        self.n_layers = len(layers)
        self.layout = layout
        self.input_shape = tuple(input_shape)
        self._h = ctypes.c_void_p()
        N, C, H, W = input_shape
        _check(lib.mg3m_net_create(arr, len(layers), N, C, H, W, _layout(layout), int(keep_all),
                                   ctypes.byref(self._h)))

    def dims(self, i):
        """(C, H, W) of activation i (0 = input, n_layers = output)."""
        c, h, w = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        _check(load_library().mg3m_net_activation(self._h, i, ctypes.byref(c), ctypes.byref(h),
                                                  ctypes.byref(w), None))
        return c.value, h.value, w.value

    def shape(self, i):
        c, h, w = self.dims(i)
        n = self.input_shape[0]
        return (h, w, c, n) if _layout(self.layout) == HWCN else (n, c, h, w)

    def activation(self, i):
        """A torch view of stored activation i (1 .. n_layers-1), valid after a
        forward pass (every one of them only with keep_all).  Stored
        activations are HWCN, shape (H, W, C, N), in every network: an NCHW
        network runs its layers in HWCN and changes layout only for x and y."""
        import torch
        c, h, w, p = ctypes.c_int(), ctypes.c_int(), ctypes.c_int(), ctypes.c_void_p()
        _check(load_library().mg3m_net_activation(self._h, i, ctypes.byref(c), ctypes.byref(h),
                                                  ctypes.byref(w), ctypes.byref(p)))
        if not p.value:
            raise ValueError("activation 0 and the last one are the caller's tensors")
        n = self.input_shape[0] * c.value * h.value * w.value
        return _device_view(p.value, n, torch).view(h.value, w.value, c.value, self.input_shape[0])

    def memory(self):
        a, b = ctypes.c_size_t(), ctypes.c_size_t()
        _check(load_library().mg3m_net_memory(self._h, ctypes.byref(a), ctypes.byref(b)))
        return a.value, b.value

    def forward(self, x, out=None, graph=False, stream=None):
        import torch
        y = out if out is not None else torch.empty(self.shape(self.n_layers), dtype=torch.float32,
                                                     device=x.device)
        fn = load_library().mg3m_net_forward_graph if graph else load_library().mg3m_net_forward
        _check(fn(self._h, _ptr(x), _ptr(y), _stream(stream)))
        return y

    def close(self):
        if self._h:
            load_library().mg3m_net_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _device_view(addr, n, torch):
    """A float32 torch tensor over n floats of device memory at addr (no copy,
    not owned)."""
    class _Holder:
        __cuda_array_interface__ = {"shape": (n,), "typestr": "<f4", "data": (addr, False), "version": 2}
    return torch.as_tensor(_Holder(), device="cuda")


def conv2d_fwd_f32(x, w, y, N, C, H, W, K, R, S, stride, pad, layout, stream=None):
    _check(load_library().conv2d_fwd_f32(_ptr(x), _ptr(w), _ptr(y), N, C, H, W, K, R, S,
                                         stride, pad, _layout(layout), _stream(stream)))


def conv2d_fwd_f32_noalloc(x, w, y, N, C, H, W, K, R, S, stride, pad, layout, stream=None):
    _check(load_library().conv2d_fwd_f32_noalloc(_ptr(x), _ptr(w), _ptr(y), N, C, H, W, K, R, S,
                                                 stride, pad, _layout(layout), _stream(stream)))


def mg3m_launch_empty(stream=None):
    _check(load_library().mg3m_launch_empty(_stream(stream)))


def mg3m_probe_mfma_f32(sink, blocks, iters, stream=None) -> float:
    """Launch the fp32-MFMA-only probe; returns the flops it performs."""
    fl = ctypes.c_double()
    _check(load_library().mg3m_probe_mfma_f32(_ptr(sink), blocks, iters, _stream(stream), ctypes.byref(fl)))
    return fl.value


def mg3m_probe_copy(src, dst, nbytes, stream=None):
    _check(load_library().mg3m_probe_copy(_ptr(src), _ptr(dst), nbytes, _stream(stream)))


def mg3m_probe_fill(dst, nbytes, stream=None):
    _check(load_library().mg3m_probe_fill(_ptr(dst), nbytes, _stream(stream)))


def conv2d_fwd_f32_ex(x, w, y, N, C, H, W, K, R, S, stride, pad, layout,
                      workspace=None, workspace_bytes=0, plan=None, stream=None):
    _check(load_library().conv2d_fwd_f32_ex(_ptr(x), _ptr(w), _ptr(y), N, C, H, W, K, R, S,
                                            stride, pad, _layout(layout), _ptr(workspace),
                                            workspace_bytes, _enc(plan), _stream(stream)))


def conv2d_fwd_f32_workspace_bytes(N, C, H, W, K, R, S, stride, pad, layout, plan=None) -> int:
    b = ctypes.c_size_t()
    _check(load_library().conv2d_fwd_f32_workspace_bytes(N, C, H, W, K, R, S, stride, pad,
                                                         _layout(layout), _enc(plan), ctypes.byref(b)))
    return b.value


def conv2d_fwd_f32_plan_string(N, C, H, W, K, R, S, stride, pad, layout, plan=None) -> str:
    buf = ctypes.create_string_buffer(1024)
    _check(load_library().conv2d_fwd_f32_plan_string(N, C, H, W, K, R, S, stride, pad,
                                                     _layout(layout), _enc(plan), buf, len(buf)))
    return buf.value.decode()


def conv2d_fwd_f32_plan_info(N, C, H, W, K, R, S, stride, pad, layout, plan=None) -> dict:
    info = PlanInfo()
    _check(load_library().conv2d_fwd_f32_plan_info(N, C, H, W, K, R, S, stride, pad,
                                                   _layout(layout), _enc(plan), ctypes.byref(info)))
    return info.as_dict()


def mg3m_time_next_kernel(start, stop):
    """start/stop: TimingEvent objects, torch.cuda.Event objects (already
    recorded once, so that they exist), raw hipEvent_t handles as ints, or
    None, None."""
    def h(e):
        if e is None or isinstance(e, int):
            return e
        if isinstance(e, TimingEvent):
            return e.handle
        return e.cuda_event
    _check(load_library().mg3m_time_next_kernel(h(start), h(stop)))


class TimingEvent:
    """A HIP timing event without the system-scope fence of a default event
    (mg3m_timing_event_*): it records a timestamp on a stream and nothing
    else, so timing a sequence of kernels does not flush the caches between
    them."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check(load_library().mg3m_timing_event_create(ctypes.byref(h)))
        self.handle = h.value

    def record(self, stream=None):
        _check(load_library().mg3m_timing_event_record(self.handle, _stream(stream)))

    def elapsed_ms(self, stop: "TimingEvent") -> float:
        """Milliseconds from this event to stop; both recorded and completed."""
        ms = ctypes.c_float()
        _check(load_library().mg3m_timing_event_elapsed_ms(self.handle, stop.handle, ctypes.byref(ms)))
        return ms.value

    def close(self):
        if self.handle is not None and _lib is not None:
            _lib.mg3m_timing_event_destroy(self.handle)
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def mg3m_padding_overhead(M, N, C, mt, nt):
    f, d = ctypes.c_double(), ctypes.c_double()
    _check(load_library().mg3m_padding_overhead(M, N, C, mt, nt, ctypes.byref(f), ctypes.byref(d)))
    return f.value, d.value


def mg3m_trim_workspace_pool():
    _check(load_library().mg3m_trim_workspace_pool())


# ------------------------------------------------------- tensor convenience
def dims_of(x, w, layout):
    """(N, C, H, W, K, R, S) from tensor shapes in `layout`."""
    lay = _layout(layout)
    if lay == HWCN:
        H, W, C, N = x.shape
        R, S, C2, K = w.shape
    else:
        N, C, H, W = x.shape
        K, C2, R, S = w.shape
    if C != C2:
        raise ValueError("input and filter channel counts differ")
    return N, C, H, W, K, R, S


def _pair(v):
    if isinstance(v, (tuple, list)):
        return int(v[0]), int(v[1])
    return int(v), int(v)


def conv2d_fwd(x, w, stride=1, pad=0, layout="HWCN", plan: Optional[str] = None,
               out=None, workspace=None, stream=None, acc64: bool = False):
    """y = conv(x, w) for torch tensors on the GPU; allocates y unless `out`
    is given.  stride and pad: an int, or (vertical, horizontal).  With
    `plan`, `workspace` or unequal per-axis values the _ex / _hw entry
    points are used (workspace allocated here when needed).  acc64=True
    uses conv2d_fwd_f32_acc64 (fp64 accumulation, no workspace)."""
    import torch
    N, C, H, W, K, R, S = dims_of(x, w, layout)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv2d_out_dims_hw(H, W, R, S, sh, sw, ph, pw)
    shape = (Ho, Wo, K, N) if _layout(layout) == HWCN else (N, K, Ho, Wo)
    y = out if out is not None else torch.empty(shape, dtype=torch.float32, device=x.device)
    if tuple(y.shape) != shape:
        raise ValueError(f"out has shape {tuple(y.shape)}, expected {shape}")
    if acc64:
        if workspace is not None:
            raise ValueError("the fp64-accumulating path takes no workspace")
        conv2d_fwd_f32_acc64(x, w, y, N, C, H, W, K, R, S, sh, sw, ph, pw, layout, plan, stream)
        return y
    square = sh == sw and ph == pw
    if square and plan is None and workspace is None:
        conv2d_fwd_f32(x, w, y, N, C, H, W, K, R, S, sh, ph, layout, stream)
        return y
    wsb = conv2d_fwd_f32_hw_workspace_bytes(N, C, H, W, K, R, S, sh, sw, ph, pw, layout, plan)
    if workspace is None and wsb > 0:
        workspace = torch.empty((wsb + 3) // 4, dtype=torch.float32, device=x.device)
    wsz = workspace.numel() * 4 if workspace is not None else 0
    if square:
        conv2d_fwd_f32_ex(x, w, y, N, C, H, W, K, R, S, sh, ph, layout, workspace, wsz, plan, stream)
    else:
        conv2d_fwd_f32_hw(x, w, y, N, C, H, W, K, R, S, sh, sw, ph, pw, layout, workspace, wsz,
                          plan, stream)
    return y
