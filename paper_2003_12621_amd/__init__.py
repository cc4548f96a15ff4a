"""Python binding of libfftsplit: split-FFT 2-D convolution on MI355X (gfx950).

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI declared in include/fftsplit.h.  PyTorch supplies
device memory (``torch.empty(..., device='cuda')``) and the stream
(``torch.cuda.current_stream()``).  If the built library is missing the
import of the native entry points fails loudly; there is no fallback.

    import paper_2003_12621_amd as fs
    plan = fs.Plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28)
    wspec = plan.transform_weights(w)          # once per layer
    y = plan.conv2d(x, wspec)                  # the hot path
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfftsplit.so")

SUCCESS = 0
ERROR_INVALID_VALUE = 1
ERROR_NOT_SUPPORTED = 2
ERROR_INSUFFICIENT_WORKSPACE = 3
ERROR_DEVICE = 4
ERROR_ARCH = 5

# patch and output spectra are stored in blocks of this many channels
CHANNEL_BLOCK = 16

OVERLAP_SAVE = 0
OVERLAP_ADD = 1
BIAS = 2
RELU = 4
MAXPOOL = 8

# FFTSPLIT_NOALLOC_MAX_WORKSPACE of fftsplit.h: bytes of the static scratch
# behind fftsplit_conv2d_noalloc
NOALLOC_MAX_WORKSPACE = 256 << 20


class Problem(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int), ("cin", ctypes.c_int), ("h", ctypes.c_int), ("w", ctypes.c_int),
                ("cout", ctypes.c_int), ("k", ctypes.c_int), ("tile", ctypes.c_int), ("stride", ctypes.c_int),
                ("pad", ctypes.c_int), ("flags", ctypes.c_uint)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("tile", ctypes.c_int), ("nfft", ctypes.c_int), ("tiles_h", ctypes.c_int),
                ("tiles_w", ctypes.c_int), ("tiles", ctypes.c_int), ("tiles_padded", ctypes.c_int),
                ("bins", ctypes.c_int), ("cout_padded", ctypes.c_int), ("flags", ctypes.c_uint),
                ("wspec_bytes", ctypes.c_size_t), ("workspace_bytes", ctypes.c_size_t),
                ("xspec_offset", ctypes.c_size_t), ("xspec_bytes", ctypes.c_size_t),
                ("yspec_offset", ctypes.c_size_t), ("yspec_bytes", ctypes.c_size_t),
                ("aux_offset", ctypes.c_size_t), ("aux_bytes", ctypes.c_size_t),
                ("contract_tile_m", ctypes.c_int), ("contract_tile_n", ctypes.c_int),
                ("contract_stage_k", ctypes.c_int), ("contract_real_products", ctypes.c_int),
                ("spec_group", ctypes.c_int), ("fused_channel_sum", ctypes.c_int),
                ("direct_wspec_bytes", ctypes.c_size_t), ("contract_prefetch", ctypes.c_int),
                ("model_contract_flops", ctypes.c_double), ("model_transform_bytes", ctypes.c_double),
                ("model_seconds", ctypes.c_double),
                ("forward_band", ctypes.c_int), ("forward_sweep", ctypes.c_int), ("inverse_band", ctypes.c_int),
                ("forward_stream", ctypes.c_int)]


class FftsplitError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({detail})")


_lib = None

# Every function the header declares, with its ctypes signature.
_SIGNATURES = {
    "fftsplit_plan": (ctypes.c_int, [ctypes.POINTER(Problem), ctypes.c_int, ctypes.POINTER(ctypes.c_void_p)]),
    "fftsplit_plan_for_arch": (ctypes.c_int, [ctypes.POINTER(Problem), ctypes.c_char_p,
                                              ctypes.POINTER(ctypes.c_void_p)]),
    "fftsplit_plan_info": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(PlanInfo)]),
    "fftsplit_plan_destroy": (None, [ctypes.c_void_p]),
    "fftsplit_transform_weights": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_void_p]),
    "fftsplit_conv2d": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "fftsplit_conv2d_noalloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_void_p]),
    "fftsplit_forward": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                        ctypes.c_void_p]),
    "fftsplit_contract": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                         ctypes.c_void_p]),
    "fftsplit_inverse": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_size_t, ctypes.c_void_p]),
    "fftsplit_maxpool2x2": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                           ctypes.c_int, ctypes.c_int, ctypes.c_void_p]),
    "fftsplit_direct_transform_weights": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                         ctypes.c_void_p]),
    "fftsplit_direct_conv2d": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p, ctypes.c_void_p]),
    "fftsplit_set_timing_events": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p]),
    "fftsplit_probe_matrix": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "fftsplit_probe_stream": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_size_t,
                                             ctypes.c_void_p]),
    "fftsplit_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "fftsplit_last_error": (ctypes.c_char_p, []),
}


def lib():
    """Load libfftsplit.so (built in-tree by ``paper_2003_12621_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2003_12621_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def status_string(status: int) -> str:
    return lib().fftsplit_status_string(status).decode()


def last_error() -> str:
    return lib().fftsplit_last_error().decode()


def _check(status: int, where: str):
    if status != SUCCESS:
        raise FftsplitError(status, where, last_error())


def _torch():
    import torch
    return torch


def _stream_handle(device) -> ctypes.c_void_p:
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dev_tensor(t, name: str, dtype=None, numel: Optional[int] = None):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) torch tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    return ctypes.c_void_p(t.data_ptr())


def problem(n, cin, h, w, cout, k, tile=0, mode="os", bias=False, relu=False, stride=1, pad=None,
            pool=False) -> Problem:
    flags = ((OVERLAP_ADD if mode == "oaa" else OVERLAP_SAVE) | (BIAS if bias else 0) | (RELU if relu else 0)
             | (MAXPOOL if pool else 0))
    if mode not in ("os", "oaa"):
        raise ValueError("mode must be 'os' or 'oaa'")
    return Problem(n, cin, h, w, cout, k, tile, stride, k // 2 if pad is None else pad, flags)


def _prod(shape):
    p = 1
    for v in shape:
        p *= v
    return p


class Plan:
    """A validated layer plan (host-side).  See fftsplit.h for every field."""

    def __init__(self, n, cin, h, w, cout, k, tile=0, mode="os", bias=False, relu=False, device=None,
                 arch: Optional[str] = None, stride=1, pad=None, pool=False):
        """pool=True appends the 2x2 stride-2 max-pool (FFTSPLIT_MAXPOOL):
        outputs are [n, cout, h // 2, w // 2]."""
        self.prob = problem(n, cin, h, w, cout, k, tile, mode, bias, relu, stride, pad, pool)
        handle = ctypes.c_void_p()
        if arch is not None:
            _check(lib().fftsplit_plan_for_arch(ctypes.byref(self.prob), arch.encode(), ctypes.byref(handle)),
                   "fftsplit_plan_for_arch")
            self.device = None
        else:
            torch = _torch()
            dev = torch.device("cuda", torch.cuda.current_device() if device is None else int(device))
            _check(lib().fftsplit_plan(ctypes.byref(self.prob), dev.index, ctypes.byref(handle)), "fftsplit_plan")
            self.device = dev
        self._h = handle
        info = PlanInfo()
        _check(lib().fftsplit_plan_info(self._h, ctypes.byref(info)), "fftsplit_plan_info")
        self.info = info
        self.n, self.cin, self.h, self.w, self.cout, self.k = n, cin, h, w, cout, k
        self.mode, self.has_bias, self.relu, self.pool = mode, bias, relu, pool

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.fftsplit_plan_destroy(h)
            self._h = None

    # -- shapes ---------------------------------------------------------
    @property
    def tile(self) -> int:
        return self.info.tile

    @property
    def nfft(self) -> int:
        return self.info.nfft

    def new_workspace(self):
        torch = _torch()
        return torch.empty(self.info.workspace_bytes, dtype=torch.uint8, device=self.device)

    @property
    def out_shape(self):
        if self.pool:
            return (self.n, self.cout, self.h // 2, self.w // 2)
        return (self.n, self.cout, self.h, self.w)

    def new_output(self):
        torch = _torch()
        return torch.empty(self.out_shape, dtype=torch.float32, device=self.device)

    # -- entry points ---------------------------------------------------
    def transform_weights(self, w, out=None):
        """Filter spectra (complex64 stored as float32 pairs), once per layer."""
        torch = _torch()
        wp = _dev_tensor(w, "w", torch.float32, self.cout * self.cin * self.k * self.k)
        if out is None:
            out = torch.empty(self.info.wspec_bytes // 4, dtype=torch.float32, device=self.device)
        if out.numel() * out.element_size() < self.info.wspec_bytes:
            raise ValueError("wspec buffer too small")
        _check(lib().fftsplit_transform_weights(self._h, wp, _dev_tensor(out, "wspec"), _stream_handle(self.device)),
               "fftsplit_transform_weights")
        return out

    def _wspec(self, wspec):
        # the C ABI takes no filter-spectra size: a buffer of another plan
        # (another layer) would be read past its end on the device
        p = _dev_tensor(wspec, "wspec")
        if wspec.numel() * wspec.element_size() < self.info.wspec_bytes:
            raise ValueError(f"wspec has {wspec.numel() * wspec.element_size()} bytes, the plan needs "
                             f"{self.info.wspec_bytes}")
        return p

    def conv2d(self, x, wspec, bias=None, out=None, workspace=None):
        torch = _torch()
        xp = _dev_tensor(x, "x", torch.float32, self.n * self.cin * self.h * self.w)
        out = self.new_output() if out is None else out
        yp = _dev_tensor(out, "y", torch.float32, _prod(self.out_shape))
        ws = self.new_workspace() if workspace is None else workspace
        bp = None if bias is None else _dev_tensor(bias, "bias", torch.float32, self.cout)
        _check(lib().fftsplit_conv2d(self._h, xp, self._wspec(wspec), bp, yp, _dev_tensor(ws, "workspace"),
                                     ws.numel() * ws.element_size(), _stream_handle(self.device)),
               "fftsplit_conv2d")
        return out

    def conv2d_noalloc(self, x, wspec, bias=None, out=None):
        """conv2d with the library's static device scratch as the workspace
        (fftsplit_conv2d_noalloc): the library allocates nothing.  Needs
        info.workspace_bytes <= NOALLOC_MAX_WORKSPACE; calls overlapping on
        one device race on the shared scratch."""
        torch = _torch()
        xp = _dev_tensor(x, "x", torch.float32, self.n * self.cin * self.h * self.w)
        if out is None:
            raise ValueError("conv2d_noalloc needs a caller-allocated output (out=)")
        yp = _dev_tensor(out, "y", torch.float32, _prod(self.out_shape))
        bp = None if bias is None else _dev_tensor(bias, "bias", torch.float32, self.cout)
        _check(lib().fftsplit_conv2d_noalloc(self._h, xp, self._wspec(wspec), bp, yp, _stream_handle(self.device)),
               "fftsplit_conv2d_noalloc")
        return out

    def forward(self, x, workspace):
        torch = _torch()
        xp = _dev_tensor(x, "x", torch.float32, self.n * self.cin * self.h * self.w)
        _check(lib().fftsplit_forward(self._h, xp, _dev_tensor(workspace, "workspace"),
                                      workspace.numel() * workspace.element_size(), _stream_handle(self.device)),
               "fftsplit_forward")

    def contract(self, wspec, workspace):
        _check(lib().fftsplit_contract(self._h, self._wspec(wspec), _dev_tensor(workspace, "workspace"),
                                       workspace.numel() * workspace.element_size(), _stream_handle(self.device)),
               "fftsplit_contract")

    def inverse(self, workspace, bias=None, out=None):
        torch = _torch()
        out = self.new_output() if out is None else out
        yp = _dev_tensor(out, "y", torch.float32, _prod(self.out_shape))
        bp = None if bias is None else _dev_tensor(bias, "bias", torch.float32, self.cout)
        _check(lib().fftsplit_inverse(self._h, bp, yp, _dev_tensor(workspace, "workspace"),
                                      workspace.numel() * workspace.element_size(), _stream_handle(self.device)),
               "fftsplit_inverse")
        return out

    # -- the spatial (direct) convolution of the same layer --------------
    def direct_transform_weights(self, w, out=None):
        """Filters rearranged for fftsplit_direct_conv2d, once per layer."""
        torch = _torch()
        wp = _dev_tensor(w, "w", torch.float32, self.cout * self.cin * self.k * self.k)
        if out is None:
            out = torch.empty(self.info.direct_wspec_bytes // 4, dtype=torch.float32, device=self.device)
        if out.numel() * out.element_size() < self.info.direct_wspec_bytes:
            raise ValueError("direct weight buffer too small")
        _check(lib().fftsplit_direct_transform_weights(self._h, wp, _dev_tensor(out, "wd"),
                                                       _stream_handle(self.device)),
               "fftsplit_direct_transform_weights")
        return out

    def direct_conv2d(self, x, wd, bias=None, out=None):
        torch = _torch()
        xp = _dev_tensor(x, "x", torch.float32, self.n * self.cin * self.h * self.w)
        out = self.new_output() if out is None else out
        yp = _dev_tensor(out, "y", torch.float32, self.n * self.cout * self.h * self.w)
        bp = None if bias is None else _dev_tensor(bias, "bias", torch.float32, self.cout)
        if wd.numel() * wd.element_size() < self.info.direct_wspec_bytes:
            raise ValueError("direct weight buffer too small for this plan")
        _check(lib().fftsplit_direct_conv2d(self._h, xp, _dev_tensor(wd, "wd"), bp, yp,
                                            _stream_handle(self.device)), "fftsplit_direct_conv2d")
        return out

    # -- measurement hook ---------------------------------------------------
    def probe_matrix(self, sink=None):
        """Enqueue the matrix-core probe of this plan's contraction launch
        (fftsplit_probe_matrix): same grid and occupancy, the same fp32
        matrix operations per wave, no memory traffic.  `sink`: a CUDA
        float32 tensor of at least one element (allocated if None)."""
        torch = _torch()
        if sink is None:
            sink = torch.zeros(1, dtype=torch.float32, device=self.device)
        if sink.numel() < 1:
            raise ValueError("sink needs one element")
        _check(lib().fftsplit_probe_matrix(self._h, _dev_tensor(sink, "sink", torch.float32),
                                           _stream_handle(self.device)), "fftsplit_probe_matrix")
        return sink

    # -- views of the workspace (complex64), for stage-level tests -------
    def _unblock(self, raw, channels):
        # channel-blocked [c/16][bins][c%16][tiles_padded] -> [bins][c][tiles_padded] (a copy)
        i = self.info
        blocks = -(-channels // CHANNEL_BLOCK)
        v = raw.view(_torch().complex64).view(blocks, i.bins, CHANNEL_BLOCK, i.tiles_padded)
        return v.permute(1, 0, 2, 3).reshape(i.bins, blocks * CHANNEL_BLOCK, i.tiles_padded)[:, :channels]

    def xspec_view(self, workspace):
        """Patch spectra as [bins][cin][tiles_padded] (complex64, a copy)."""
        i = self.info
        return self._unblock(workspace[i.xspec_offset:i.xspec_offset + i.xspec_bytes], self.cin)

    def yspec_view(self, workspace):
        """Output spectra as [bins][cout_padded][tiles_padded] (complex64, a copy)."""
        i = self.info
        g = i.spec_group
        raw = workspace[i.yspec_offset:i.yspec_offset + i.yspec_bytes]
        v = raw.view(_torch().complex64).view(i.cout_padded, i.tiles_padded // g, i.bins, g)
        return v.permute(2, 0, 1, 3).reshape(i.bins, i.cout_padded, i.tiles_padded)

    def wspec_view(self, wspec):
        i = self.info
        return wspec.view(_torch().complex64)[: i.bins * self.cin * i.cout_padded].view(i.bins, self.cin,
                                                                                         i.cout_padded)


def set_timing_events(start=None, stop=None):
    """Time this thread's following fftsplit calls with two torch.cuda.Event
    objects (enable_timing=True), recorded by the kernels' own dispatch
    timestamps; set_timing_events() turns it off.  Each event must already
    exist on the device (record it once beforehand)."""
    def handle(ev):
        if ev is None:
            return None
        h = ev.cuda_event
        if not h:
            raise ValueError("event has no device handle yet; record it once first")
        return ctypes.c_void_p(h)
    _check(lib().fftsplit_set_timing_events(handle(start), handle(stop)), "fftsplit_set_timing_events")


def probe_stream(src, dst, read_bytes, write_bytes):
    """Enqueue the streaming probe (fftsplit_probe_stream): load
    `read_bytes` of src and store `write_bytes` to dst (CUDA tensors, on
    the current stream of their device)."""
    for t, nb, name in ((src, read_bytes, "src"), (dst, write_bytes, "dst")):
        if nb > t.numel() * t.element_size():
            raise ValueError(f"{name} holds fewer than {nb} bytes")
    _check(lib().fftsplit_probe_stream(_dev_tensor(src, "src"), _dev_tensor(dst, "dst"), int(read_bytes),
                                       int(write_bytes), _stream_handle(dst.device)), "fftsplit_probe_stream")


def maxpool2x2(x, out=None):
    """2x2 stride-2 max-pool (floor) on an NCHW float32 CUDA tensor."""
    torch = _torch()
    n, c, h, w = x.shape
    out = torch.empty((n, c, h // 2, w // 2), dtype=torch.float32, device=x.device) if out is None else out
    xp = _dev_tensor(x, "x", torch.float32)
    yp = _dev_tensor(out, "y", torch.float32, n * c * (h // 2) * (w // 2))
    _check(lib().fftsplit_maxpool2x2(xp, yp, n, c, h, w, _stream_handle(x.device)), "fftsplit_maxpool2x2")
    return out


def bin_coords(L: int):
    """Stored bins of an L x L real transform, in the library's order
    (fftsplit.h): a list of L*L/2 entries.  Entry f is (k1, k2) for a complex
    bin; the last two entries are pairs ((k1, k2) of the real part,
    (k1, k2) of the imaginary part) for the slots holding two real bins.
    Odd L (the OaAConv configuration): (L*L+1)/2 complex bins, none packed."""
    h2 = L // 2
    if L % 2:
        return [(k1, k2) for k2 in range(1, h2 + 1) for k1 in range(L)] + [(k1, 0) for k1 in range(h2 + 1)]
    coords = []
    for k2 in range(1, h2):
        for k1 in range(L):
            coords.append((k1, k2))
    for k1 in range(1, h2):
        coords.append((k1, 0))
    for k1 in range(1, h2):
        coords.append((k1, h2))
    coords.append(((0, 0), (h2, 0)))
    coords.append(((0, h2), (h2, h2)))
    return coords
