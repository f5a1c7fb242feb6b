"""RubiConv on MI355X: boundary-respecting causal long convolution over packed sequences.

A thin ctypes binding of ``librubiconv.so`` (C ABI in ``include/rubiconv.h``).  It
only marshals arguments: every step of the convolution runs in the library's HIP
kernels.  PyTorch supplies device memory and the stream; it is imported before the
library is loaded so that both share one HIP runtime.

    plan = Plan(cu_seqlens, N=x.shape[1], D=x.shape[2], L=filters.shape[1],
                x_dtype=x.dtype, y_dtype=torch.bfloat16)
    spec = filter_spectrum(plan, filters)          # filters: cuda float32 [D, L]
    y = packed_conv(plan, x, spec)                 # x: cuda [B, N, D]

The library must be built first (``python -m paper_2605_08451_amd.build``); if it
is missing, loading fails loudly -- there is no fallback implementation.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional

import numpy as np
import torch

__all__ = ["Plan", "RubiconvError", "filter_spectrum", "packed_conv", "packed_conv_noalloc",
           "packed_conv_dx",
           "packed_conv_dk", "conv", "CTPlan", "ct_filter_spectrum", "ct_packed_conv",
           "library_path", "load_library", "EXPORTED_SYMBOLS"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "librubiconv.so")
_LIB = None

F32, BF16 = 0, 1
_STATUS = {0: "ok", 1: "invalid argument", 2: "invalid cu_seqlens", 3: "unsupported configuration",
           4: "allocation failed", 5: "HIP error or no device"}

#: Every function ``include/rubiconv.h`` and ``include/rubiconv_ct.h`` declare.
EXPORTED_SYMBOLS = ("rubiconv_plan", "rubiconv_plan_destroy", "rubiconv_spectrum_bytes",
                    "rubiconv_workspace_bytes", "rubiconv_filter_spectrum", "rubiconv_packed_conv",
                    "rubiconv_packed_conv_dx", "rubiconv_dk_workspace_bytes", "rubiconv_packed_conv_dk",
                    "rubiconv_packed_conv_backward", "rubiconv_packed_conv_noalloc",
                    "rubiconv_plan_info", "rubiconv_plan_doc_table", "rubiconv_profile_start",
                    "rubiconv_profile_read", "rubiconv_status_string",
                    "rubiconv_ct_plan", "rubiconv_ct_plan_destroy", "rubiconv_ct_spectrum_bytes",
                    "rubiconv_ct_workspace_bytes", "rubiconv_ct_filter_spectrum",
                    "rubiconv_ct_packed_conv", "rubiconv_ct_plan_doc_table")


class RubiconvError(RuntimeError):
    def __init__(self, what: str, status: int):
        super().__init__(f"{what}: {_STATUS.get(status, status)} (status {status})")
        self.status = status


class _PlanInfo(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("N", ctypes.c_int), ("D", ctypes.c_int), ("L", ctypes.c_int),
                ("n1", ctypes.c_int), ("n_docs", ctypes.c_int), ("n_classes", ctypes.c_int),
                ("n_pair_blocks", ctypes.c_int), ("grid_points", ctypes.c_int64),
                ("class_points", ctypes.c_int64), ("tokens", ctypes.c_int64),
                ("direct_max", ctypes.c_int), ("n_direct", ctypes.c_int)]


class _KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int),
                ("total_ms", ctypes.c_double)]


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load the in-tree ``librubiconv.so`` (raises if it has not been built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                           "`python -m paper_2605_08451_amd.build` (no fallback exists)")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32p, c_int, sz = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.c_int, ctypes.c_size_t
    lib.rubiconv_plan.argtypes = [ctypes.POINTER(vp), c_int, c_int, c_int, c_int, c_int, i32p,
                                  c_int, c_int, c_int, vp]
    lib.rubiconv_plan.restype = c_int
    lib.rubiconv_plan_destroy.argtypes = [vp]
    lib.rubiconv_plan_destroy.restype = None
    lib.rubiconv_spectrum_bytes.argtypes = [vp]
    lib.rubiconv_spectrum_bytes.restype = sz
    lib.rubiconv_workspace_bytes.argtypes = [vp]
    lib.rubiconv_workspace_bytes.restype = sz
    lib.rubiconv_filter_spectrum.argtypes = [vp, vp, vp, vp, vp]
    lib.rubiconv_filter_spectrum.restype = c_int
    lib.rubiconv_packed_conv.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.rubiconv_packed_conv.restype = c_int
    lib.rubiconv_packed_conv_noalloc.argtypes = [vp, vp, vp, vp, vp]
    lib.rubiconv_packed_conv_noalloc.restype = c_int
    lib.rubiconv_packed_conv_dx.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.rubiconv_packed_conv_dx.restype = c_int
    lib.rubiconv_dk_workspace_bytes.argtypes = [vp]
    lib.rubiconv_dk_workspace_bytes.restype = sz
    lib.rubiconv_packed_conv_dk.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.rubiconv_packed_conv_dk.restype = c_int
    lib.rubiconv_packed_conv_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
    lib.rubiconv_packed_conv_backward.restype = c_int
    lib.rubiconv_plan_info.argtypes = [vp, ctypes.POINTER(_PlanInfo)]
    lib.rubiconv_plan_info.restype = c_int
    lib.rubiconv_plan_doc_table.argtypes = [vp, i32p, c_int, ctypes.POINTER(c_int)]
    lib.rubiconv_plan_doc_table.restype = c_int
    lib.rubiconv_profile_start.argtypes = [vp, c_int]
    lib.rubiconv_profile_start.restype = c_int
    lib.rubiconv_profile_read.argtypes = [vp, ctypes.POINTER(_KernelTime), c_int,
                                          ctypes.POINTER(c_int)]
    lib.rubiconv_profile_read.restype = c_int
    lib.rubiconv_status_string.argtypes = [c_int]
    lib.rubiconv_status_string.restype = ctypes.c_char_p
    lib.rubiconv_ct_plan.argtypes = [ctypes.POINTER(vp), c_int, c_int, c_int, c_int, c_int, i32p,
                                     c_int, c_int]
    lib.rubiconv_ct_plan.restype = c_int
    lib.rubiconv_ct_plan_destroy.argtypes = [vp]
    lib.rubiconv_ct_plan_destroy.restype = None
    lib.rubiconv_ct_spectrum_bytes.argtypes = [vp]
    lib.rubiconv_ct_spectrum_bytes.restype = sz
    lib.rubiconv_ct_workspace_bytes.argtypes = [vp]
    lib.rubiconv_ct_workspace_bytes.restype = sz
    lib.rubiconv_ct_filter_spectrum.argtypes = [vp, vp, vp, vp, vp]
    lib.rubiconv_ct_filter_spectrum.restype = c_int
    lib.rubiconv_ct_packed_conv.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.rubiconv_ct_packed_conv.restype = c_int
    lib.rubiconv_ct_plan_doc_table.argtypes = [vp, i32p, c_int, ctypes.POINTER(c_int)]
    lib.rubiconv_ct_plan_doc_table.restype = c_int
    _LIB = lib
    return lib


def _dtype_code(dt) -> int:
    if dt in (torch.float32, "f32", "float32", F32):
        return F32
    if dt in (torch.bfloat16, "bf16", "bfloat16", BF16):
        return BF16
    raise ValueError(f"unsupported dtype {dt!r} (float32 or bfloat16)")


def _torch_dtype(code: int):
    return torch.float32 if code == F32 else torch.bfloat16


def _check(status: int, what: str):
    if status != 0:
        raise RubiconvError(what, status)


def _on_stream(stream):
    """Context in which buffers the binding allocates for a call belong to the call's
    stream: the caching allocator then reuses them only after that stream's work."""
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def _stream_handle(device, stream) -> int:
    s = torch.cuda.current_stream(device) if stream is None else stream
    return s.cuda_stream


def _cu_array(cu_seqlens) -> np.ndarray:
    if isinstance(cu_seqlens, torch.Tensor):
        cu_seqlens = cu_seqlens.detach().cpu().numpy()
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    if cu.ndim == 1:
        cu = cu[None]
    if cu.ndim != 2 or cu.shape[1] < 2:
        raise ValueError("cu_seqlens must be [B, max_docs + 1]")
    return cu


class Plan:
    """Document table, size classes and twiddles for one batch of boundaries
    (Algorithm 1's data processing; shared by every layer that sees this batch)."""

    def __init__(self, cu_seqlens, N: int, D: int, L: int, x_dtype=torch.bfloat16,
                 y_dtype=None, n1: int = 0, stream=None):
        lib = load_library()
        cu = _cu_array(cu_seqlens)
        self.B, self.max_docs = int(cu.shape[0]), int(cu.shape[1] - 1)
        self.N, self.D, self.L = int(N), int(D), int(L)
        self.x_dtype = _dtype_code(x_dtype)
        self.y_dtype = self.x_dtype if y_dtype is None else _dtype_code(y_dtype)
        self._h = ctypes.c_void_p()
        self._lib = lib
        # the device tables are uploaded on `stream` (the current stream by default);
        # without a visible GPU the plan is host-only and no stream is touched
        sh = None
        if torch.cuda.is_available():
            sh = (torch.cuda.current_stream() if stream is None else stream).cuda_stream
        _check(lib.rubiconv_plan(ctypes.byref(self._h), self.B, self.N, self.D, self.L,
                                 self.max_docs, cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                 self.x_dtype, self.y_dtype, int(n1), sh), "rubiconv_plan")
        self.cu_seqlens = cu.copy()

    @property
    def handle(self):
        if not self._h:
            raise RuntimeError("plan already destroyed")
        return self._h

    @property
    def spectrum_bytes(self) -> int:
        return int(self._lib.rubiconv_spectrum_bytes(self.handle))

    @property
    def workspace_bytes(self) -> int:
        return int(self._lib.rubiconv_workspace_bytes(self.handle))

    def info(self) -> dict:
        inf = _PlanInfo()
        _check(self._lib.rubiconv_plan_info(self.handle, ctypes.byref(inf)), "rubiconv_plan_info")
        return {name: getattr(inf, name) for name, _ in _PlanInfo._fields_}

    def doc_table(self) -> np.ndarray:
        """int32 [n_docs, 6]: row, index in row, start, length, m_i, P_i (m_i = P_i = 0 for a
        document the direct path computes)."""
        n = ctypes.c_int(0)
        _check(self._lib.rubiconv_plan_doc_table(self.handle, None, 0, ctypes.byref(n)),
               "rubiconv_plan_doc_table")
        out = np.zeros((max(n.value, 1), 6), dtype=np.int32)
        _check(self._lib.rubiconv_plan_doc_table(
            self.handle, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n.value,
            ctypes.byref(n)), "rubiconv_plan_doc_table")
        return out[:n.value].copy()

    def profile_start(self, max_calls: int):
        """Time every kernel of the next ``max_calls`` library calls with HIP events."""
        _check(self._lib.rubiconv_profile_start(self.handle, int(max_calls)),
               "rubiconv_profile_start")

    def profile_read(self) -> dict:
        """{kernel name: (launches, total milliseconds)} of the profiled calls (waits)."""
        n = ctypes.c_int(0)
        _check(self._lib.rubiconv_profile_read(self.handle, None, 0, ctypes.byref(n)),
               "rubiconv_profile_read")
        cap = max(n.value, 1)
        out = (_KernelTime * cap)()
        _check(self._lib.rubiconv_profile_read(self.handle, out, cap, ctypes.byref(n)),
               "rubiconv_profile_read")
        return {out[i].name.decode(): (out[i].launches, out[i].total_ms)
                for i in range(min(n.value, cap))}

    def new_spectrum(self, device) -> torch.Tensor:
        return torch.empty(self.spectrum_bytes, dtype=torch.uint8, device=device)

    def new_workspace(self, device) -> torch.Tensor:
        return torch.empty(self.workspace_bytes, dtype=torch.uint8, device=device)

    @property
    def dk_workspace_bytes(self) -> int:
        return int(self._lib.rubiconv_dk_workspace_bytes(self.handle))

    def new_dk_workspace(self, device) -> torch.Tensor:
        return torch.empty(self.dk_workspace_bytes, dtype=torch.uint8, device=device)

    def close(self):
        if self._h:
            self._lib.rubiconv_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _cuda_contig(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def filter_spectrum(plan: Plan, filters: torch.Tensor, spectrum: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Spectra of ``filters`` (cuda float32 [D, L]) for every size class of ``plan``."""
    _cuda_contig(filters, "filters")
    if filters.dtype != torch.float32 or tuple(filters.shape) != (plan.D, plan.L):
        raise ValueError(f"filters must be float32 [{plan.D}, {plan.L}]")
    dev = filters.device
    with _on_stream(stream):
        if spectrum is None:
            spectrum = plan.new_spectrum(dev)
        if workspace is None:
            workspace = plan.new_workspace(dev)
    if spectrum.numel() * spectrum.element_size() < plan.spectrum_bytes:
        raise ValueError("spectrum buffer too small")
    if workspace.numel() * workspace.element_size() < plan.workspace_bytes:
        raise ValueError("workspace buffer too small")
    with torch.cuda.device(dev):
        _check(plan._lib.rubiconv_filter_spectrum(plan.handle, filters.data_ptr(),
                                                  spectrum.data_ptr(), workspace.data_ptr(),
                                                  _stream_handle(dev, stream)),
               "rubiconv_filter_spectrum")
    return spectrum


def packed_conv(plan: Plan, x: torch.Tensor, spectrum: torch.Tensor,
                y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """y[b, t, d] = sum over the lags inside t's document of k[d, tau] x[b, t - tau, d]."""
    _cuda_contig(x, "x")
    if tuple(x.shape) != (plan.B, plan.N, plan.D) or x.dtype != _torch_dtype(plan.x_dtype):
        raise ValueError(f"x must be {_torch_dtype(plan.x_dtype)} [{plan.B}, {plan.N}, {plan.D}]")
    dev = x.device
    with _on_stream(stream):
        if y is None:
            y = torch.empty((plan.B, plan.N, plan.D), dtype=_torch_dtype(plan.y_dtype), device=dev)
        if workspace is None:
            workspace = plan.new_workspace(dev)
    _cuda_contig(y, "y")
    if tuple(y.shape) != (plan.B, plan.N, plan.D) or y.dtype != _torch_dtype(plan.y_dtype):
        raise ValueError("y has the wrong shape or dtype")
    if workspace.numel() * workspace.element_size() < plan.workspace_bytes:
        raise ValueError("workspace buffer too small")
    if spectrum.numel() * spectrum.element_size() < plan.spectrum_bytes:
        raise ValueError("spectrum buffer too small")
    with torch.cuda.device(dev):
        _check(plan._lib.rubiconv_packed_conv(plan.handle, x.data_ptr(), spectrum.data_ptr(),
                                              y.data_ptr(), workspace.data_ptr(),
                                              _stream_handle(dev, stream)),
               "rubiconv_packed_conv")
    return y


#: Bytes of the library's per-device scratch array (RUBICONV_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 320 << 20


def packed_conv_noalloc(plan: Plan, x: torch.Tensor, spectrum: torch.Tensor, y: torch.Tensor,
                        stream=None) -> torch.Tensor:
    """packed_conv without a workspace: the library's per-device scratch array serves as
    one (rubiconv_packed_conv_noalloc).  y must be given; nothing is allocated."""
    _check_btd(x, plan, plan.x_dtype, "x")
    _check_btd(y, plan, plan.y_dtype, "y")
    if spectrum.numel() * spectrum.element_size() < plan.spectrum_bytes:
        raise ValueError("spectrum buffer too small")
    with torch.cuda.device(x.device):
        _check(plan._lib.rubiconv_packed_conv_noalloc(plan.handle, x.data_ptr(), spectrum.data_ptr(),
                                                      y.data_ptr(), _stream_handle(x.device, stream)),
               "rubiconv_packed_conv_noalloc")
    return y


def _check_btd(t: torch.Tensor, plan: "Plan", code: int, name: str):
    _cuda_contig(t, name)
    if tuple(t.shape) != (plan.B, plan.N, plan.D) or t.dtype != _torch_dtype(code):
        raise ValueError(f"{name} must be {_torch_dtype(code)} [{plan.B}, {plan.N}, {plan.D}]")


def packed_conv_dx(plan: Plan, dy: torch.Tensor, spectrum: torch.Tensor,
                   dx: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                   stream=None) -> torch.Tensor:
    """dx[b, s, d] = sum over the lags that stay in s's document of k[d, tau] dy[b, s + tau, d]
    (dy has the plan's y dtype, dx its x dtype)."""
    _check_btd(dy, plan, plan.y_dtype, "dy")
    dev = dy.device
    with _on_stream(stream):
        if dx is None:
            dx = torch.empty((plan.B, plan.N, plan.D), dtype=_torch_dtype(plan.x_dtype), device=dev)
        if workspace is None:
            workspace = plan.new_workspace(dev)
    _check_btd(dx, plan, plan.x_dtype, "dx")
    if workspace.numel() * workspace.element_size() < plan.workspace_bytes:
        raise ValueError("workspace buffer too small")
    if spectrum.numel() * spectrum.element_size() < plan.spectrum_bytes:
        raise ValueError("spectrum buffer too small")
    with torch.cuda.device(dev):
        _check(plan._lib.rubiconv_packed_conv_dx(plan.handle, dy.data_ptr(), spectrum.data_ptr(),
                                                 dx.data_ptr(), workspace.data_ptr(),
                                                 _stream_handle(dev, stream)),
               "rubiconv_packed_conv_dx")
    return dx


def packed_conv_dk(plan: Plan, x: torch.Tensor, dy: torch.Tensor,
                   dk: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                   stream=None) -> torch.Tensor:
    """dk[d, tau] = sum over every document of dy[b, t, d] x[b, t - tau, d], float32 [D, L]."""
    _check_btd(x, plan, plan.x_dtype, "x")
    _check_btd(dy, plan, plan.y_dtype, "dy")
    dev = x.device
    with _on_stream(stream):
        if dk is None:
            dk = torch.empty((plan.D, plan.L), dtype=torch.float32, device=dev)
        if workspace is None:
            workspace = plan.new_dk_workspace(dev)
    _cuda_contig(dk, "dk")
    if tuple(dk.shape) != (plan.D, plan.L) or dk.dtype != torch.float32:
        raise ValueError(f"dk must be float32 [{plan.D}, {plan.L}]")
    if workspace.numel() * workspace.element_size() < plan.dk_workspace_bytes:
        raise ValueError("workspace buffer too small")
    with torch.cuda.device(dev):
        _check(plan._lib.rubiconv_packed_conv_dk(plan.handle, x.data_ptr(), dy.data_ptr(),
                                                 dk.data_ptr(), workspace.data_ptr(),
                                                 _stream_handle(dev, stream)),
               "rubiconv_packed_conv_dk")
    return dk


def packed_conv_backward(plan: Plan, x: torch.Tensor, dy: torch.Tensor, spectrum: torch.Tensor,
                         dx: Optional[torch.Tensor] = None, dk: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None, stream=None):
    """(dx, dk) of one backward pass in one call (``rubiconv_packed_conv_backward``): the
    results of :func:`packed_conv_dx` and :func:`packed_conv_dk`, dy's column pass shared."""
    _check_btd(x, plan, plan.x_dtype, "x")
    _check_btd(dy, plan, plan.y_dtype, "dy")
    dev = x.device
    with _on_stream(stream):
        if dx is None:
            dx = torch.empty((plan.B, plan.N, plan.D), dtype=_torch_dtype(plan.x_dtype), device=dev)
        if dk is None:
            dk = torch.empty((plan.D, plan.L), dtype=torch.float32, device=dev)
        if workspace is None:
            workspace = plan.new_dk_workspace(dev)
    _check_btd(dx, plan, plan.x_dtype, "dx")
    _cuda_contig(dk, "dk")
    if tuple(dk.shape) != (plan.D, plan.L) or dk.dtype != torch.float32:
        raise ValueError(f"dk must be float32 [{plan.D}, {plan.L}]")
    if workspace.numel() * workspace.element_size() < plan.dk_workspace_bytes:
        raise ValueError("workspace buffer too small")
    if spectrum.numel() * spectrum.element_size() < plan.spectrum_bytes:
        raise ValueError("spectrum buffer too small")
    with torch.cuda.device(dev):
        _check(plan._lib.rubiconv_packed_conv_backward(plan.handle, x.data_ptr(), dy.data_ptr(),
                                                       spectrum.data_ptr(), dx.data_ptr(), dk.data_ptr(),
                                                       workspace.data_ptr(), _stream_handle(dev, stream)),
               "rubiconv_packed_conv_backward")
    return dx, dk


def conv(x: torch.Tensor, filters: torch.Tensor, cu_seqlens, y_dtype=None, n1: int = 0):
    """One-shot convenience: plan, filter spectrum and convolution (allocates)."""
    plan = Plan(cu_seqlens, N=x.shape[1], D=x.shape[2], L=filters.shape[1], x_dtype=x.dtype,
                y_dtype=y_dtype, n1=n1)
    ws = plan.new_workspace(x.device)
    spec = filter_spectrum(plan, filters, workspace=ws)
    y = packed_conv(plan, x, spec, workspace=ws)
    torch.cuda.current_stream(x.device).synchronize()
    plan.close()
    return y


# ----------------------------------------------------------------- masked Cooley-Tukey
class CTPlan:
    """Plan of the masked Cooley-Tukey variant (Algorithm 2, ``include/rubiconv_ct.h``):
    power-of-two document sizes and the packed layout its masked stages run on."""

    def __init__(self, cu_seqlens, N: int, D: int, L: int, x_dtype=torch.bfloat16, y_dtype=None):
        lib = load_library()
        cu = _cu_array(cu_seqlens)
        self.B, self.max_docs = int(cu.shape[0]), int(cu.shape[1] - 1)
        self.N, self.D, self.L = int(N), int(D), int(L)
        self.x_dtype = _dtype_code(x_dtype)
        self.y_dtype = self.x_dtype if y_dtype is None else _dtype_code(y_dtype)
        self._h = ctypes.c_void_p()
        self._lib = lib
        _check(lib.rubiconv_ct_plan(ctypes.byref(self._h), self.B, self.N, self.D, self.L,
                                    self.max_docs, cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                    self.x_dtype, self.y_dtype), "rubiconv_ct_plan")
        self.cu_seqlens = cu.copy()

    @property
    def handle(self):
        if not self._h:
            raise RuntimeError("plan already destroyed")
        return self._h

    @property
    def spectrum_bytes(self) -> int:
        return int(self._lib.rubiconv_ct_spectrum_bytes(self.handle))

    @property
    def workspace_bytes(self) -> int:
        return int(self._lib.rubiconv_ct_workspace_bytes(self.handle))

    def doc_table(self) -> np.ndarray:
        """int32 [n_docs, 6]: row, index in row, start, length, P_i, offset in the packed array."""
        n = ctypes.c_int(0)
        _check(self._lib.rubiconv_ct_plan_doc_table(self.handle, None, 0, ctypes.byref(n)),
               "rubiconv_ct_plan_doc_table")
        out = np.zeros((max(n.value, 1), 6), dtype=np.int32)
        _check(self._lib.rubiconv_ct_plan_doc_table(
            self.handle, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n.value,
            ctypes.byref(n)), "rubiconv_ct_plan_doc_table")
        return out[:n.value].copy()

    def new_spectrum(self, device) -> torch.Tensor:
        return torch.empty(self.spectrum_bytes, dtype=torch.uint8, device=device)

    def new_workspace(self, device) -> torch.Tensor:
        return torch.empty(self.workspace_bytes, dtype=torch.uint8, device=device)

    def close(self):
        if self._h:
            self._lib.rubiconv_ct_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ct_filter_spectrum(plan: CTPlan, filters: torch.Tensor, spectrum: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Spectra of ``filters`` (cuda float32 [D, L]) for every power-of-two size of ``plan``."""
    _cuda_contig(filters, "filters")
    if filters.dtype != torch.float32 or tuple(filters.shape) != (plan.D, plan.L):
        raise ValueError(f"filters must be float32 [{plan.D}, {plan.L}]")
    dev = filters.device
    with _on_stream(stream):
        if spectrum is None:
            spectrum = plan.new_spectrum(dev)
        if workspace is None:
            workspace = plan.new_workspace(dev)
    if spectrum.numel() * spectrum.element_size() < plan.spectrum_bytes:
        raise ValueError("spectrum buffer too small")
    if workspace.numel() * workspace.element_size() < plan.workspace_bytes:
        raise ValueError("workspace buffer too small")
    with torch.cuda.device(dev):
        _check(plan._lib.rubiconv_ct_filter_spectrum(plan.handle, filters.data_ptr(),
                                                     spectrum.data_ptr(), workspace.data_ptr(),
                                                     _stream_handle(dev, stream)),
               "rubiconv_ct_filter_spectrum")
    return spectrum


def ct_packed_conv(plan: CTPlan, x: torch.Tensor, spectrum: torch.Tensor,
                   y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                   stream=None) -> torch.Tensor:
    """The packed causal convolution through the masked Cooley-Tukey transform."""
    _check_btd(x, plan, plan.x_dtype, "x")
    dev = x.device
    with _on_stream(stream):
        if y is None:
            y = torch.empty((plan.B, plan.N, plan.D), dtype=_torch_dtype(plan.y_dtype), device=dev)
        if workspace is None:
            workspace = plan.new_workspace(dev)
    _check_btd(y, plan, plan.y_dtype, "y")
    if workspace.numel() * workspace.element_size() < plan.workspace_bytes:
        raise ValueError("workspace buffer too small")
    if spectrum.numel() * spectrum.element_size() < plan.spectrum_bytes:
        raise ValueError("spectrum buffer too small")
    with torch.cuda.device(dev):
        _check(plan._lib.rubiconv_ct_packed_conv(plan.handle, x.data_ptr(), spectrum.data_ptr(),
                                                 y.data_ptr(), workspace.data_ptr(),
                                                 _stream_handle(dev, stream)),
               "rubiconv_ct_packed_conv")
    return y
