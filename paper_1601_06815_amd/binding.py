"""ctypes binding of liboaa.so (include/oaa.h). Argument marshalling only.

Functions carry the C names and take plain integers for device pointers and
streams. ``Plan`` wraps them for torch tensors: torch supplies device memory
(the workspace is a uint8 tensor) and the current stream; every step of every
pass runs in the library's HIP kernels. There is no fallback: if the library
is missing, ``load()`` raises.
"""

import ctypes
import os

from .build import LIB_PATH

OAA_OK = 0
STATUS = {0: "OAA_OK", 1: "OAA_ERR_INVALID_ARG", 2: "OAA_ERR_UNSUPPORTED",
          3: "OAA_ERR_NO_WORKSPACE", 4: "OAA_ERR_NO_CACHE", 5: "OAA_ERR_HIP"}
REGION_W_SPECTRUM, REGION_X_SPECTRUM, REGION_G_SPECTRUM, REGION_PRODUCT = 0, 1, 2, 3
CONTRACTION_AUTO, CONTRACTION_VALU, CONTRACTION_MFMA, CONTRACTION_NARROW, CONTRACTION_FUSED = 0, 1, 2, 3, 4
METHOD_OVERLAP_ADD, METHOD_OVERLAP_SAVE = 0, 1
STAGES = ["w_spectrum", "x_spectrum", "g_spectrum", "fwd_product", "fwd_inverse",
          "bwd_data_product", "bwd_data_inverse", "bwd_filter_product", "bwd_filter_inverse"]

# every symbol include/oaa.h declares, with its ctypes signature
_c_int, _c_size, _vp = ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p


class Geometry(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int) for k in ("B", "C", "K", "N", "n", "M", "T", "P", "L", "F", "split", "b",
                                            "method", "fused")]


SIGNATURES = {
    "oaa_plan_create": (_c_int, [ctypes.POINTER(_vp), _c_int, _c_int, _c_int, _c_int, _c_int]),
    "oaa_plan_create_tiled": (_c_int, [ctypes.POINTER(_vp), _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int]),
    "oaa_plan_create_method": (_c_int, [ctypes.POINTER(_vp), _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                        _c_int]),
    "oaa_plan_destroy": (_c_int, [_vp]),
    "oaa_plan_geometry": (_c_int, [_vp, ctypes.POINTER(Geometry)]),
    "oaa_plan_workspace_bytes": (_c_size, [_vp]),
    "oaa_plan_region": (_c_int, [_vp, _c_int, ctypes.POINTER(_c_size), ctypes.POINTER(_c_size)]),
    "oaa_plan_bind_workspace": (_c_int, [_vp, _vp, _c_size]),
    "oaa_plan_set_contraction": (_c_int, [_vp, _c_int]),
    "oaa_plan_set_timing": (_c_int, [_vp, _c_int]),
    "oaa_plan_stage_times": (_c_int, [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_c_int), _c_int]),
    "oaa_conv_forward": (_c_int, [_vp, _vp, _vp, _vp, _vp]),
    "oaa_conv_backward_data": (_c_int, [_vp, _vp, _vp, _vp, _vp]),
    "oaa_conv_backward_filter": (_c_int, [_vp, _vp, _vp, _vp, _vp]),
    "oaa_conv_forward_noalloc": (_c_int, [_vp, _vp, _vp, _vp, _vp]),
    "oaa_plan_chain_scratch_bytes": (_c_size, [_vp, _c_int]),
    "oaa_plan_set_kernel_chain": (_c_int, [_vp, _vp, _c_int, _c_int, _vp, _c_int, _vp, _c_size, _vp]),
    "oaa_status_string": (ctypes.c_char_p, [_c_int]),
    "oaa_last_error_detail": (ctypes.c_char_p, []),
}

_LIB = None


def load(path=None):
    """Load liboaa.so (once) and declare its signatures."""
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run paper_1601_06815_amd.build.build() "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path == LIB_PATH:
        _LIB = lib
    return lib


def use_library(path):
    """Load liboaa.so from `path` and make it the library every later call
    uses (for comparing builds; the default is the in-tree build)."""
    global _LIB
    _LIB = None
    lib = load(path)
    _LIB = lib
    return lib


class OaaError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


def _check(st):
    if st != OAA_OK:
        lib = load()
        raise OaaError(st, lib.oaa_last_error_detail().decode())
    return st


# ---- C names, integer pointers ------------------------------------------------

def oaa_plan_create(B, C, K, N, n):
    h = _vp()
    _check(load().oaa_plan_create(ctypes.byref(h), B, C, K, N, n))
    return h.value


def oaa_plan_create_tiled(B, C, K, N, n, L, b):
    h = _vp()
    _check(load().oaa_plan_create_tiled(ctypes.byref(h), B, C, K, N, n, L, b))
    return h.value


def oaa_plan_create_method(B, C, K, N, n, L, b, method):
    h = _vp()
    _check(load().oaa_plan_create_method(ctypes.byref(h), B, C, K, N, n, L, b, method))
    return h.value


def oaa_plan_destroy(plan):
    return _check(load().oaa_plan_destroy(plan))


def oaa_plan_geometry(plan):
    g = Geometry()
    _check(load().oaa_plan_geometry(plan, ctypes.byref(g)))
    return {k: getattr(g, k) for k, _ in Geometry._fields_}


def oaa_plan_workspace_bytes(plan):
    return load().oaa_plan_workspace_bytes(plan)


def oaa_plan_region(plan, region):
    off, size = _c_size(), _c_size()
    _check(load().oaa_plan_region(plan, region, ctypes.byref(off), ctypes.byref(size)))
    return off.value, size.value


def oaa_plan_bind_workspace(plan, dev_ptr, nbytes):
    return _check(load().oaa_plan_bind_workspace(plan, dev_ptr, nbytes))


def oaa_plan_set_contraction(plan, which):
    return _check(load().oaa_plan_set_contraction(plan, which))


def oaa_plan_set_timing(plan, enable):
    return _check(load().oaa_plan_set_timing(plan, 1 if enable else 0))


def oaa_plan_stage_times(plan):
    """{stage name: (total ms, launches)} since the last call; waits for the GPU."""
    n = len(STAGES)
    ms = (ctypes.c_double * n)()
    cnt = (_c_int * n)()
    _check(load().oaa_plan_stage_times(plan, ms, cnt, n))
    return {name: (ms[i], cnt[i]) for i, name in enumerate(STAGES)}


def oaa_conv_forward(plan, x, w, y, stream):
    return _check(load().oaa_conv_forward(plan, x, w, y, stream))


def oaa_conv_backward_data(plan, g, w, dx, stream):
    return _check(load().oaa_conv_backward_data(plan, g, w, dx, stream))


def oaa_conv_backward_filter(plan, x, g, dw, stream):
    return _check(load().oaa_conv_backward_filter(plan, x, g, dw, stream))


def oaa_conv_forward_noalloc(plan, x, w, y, stream):
    return _check(load().oaa_conv_forward_noalloc(plan, x, w, y, stream))


def oaa_plan_chain_scratch_bytes(plan, J):
    return load().oaa_plan_chain_scratch_bytes(plan, J)


def oaa_plan_set_kernel_chain(plan, w1, J, n1, w2, n2, scratch, scratch_bytes, stream):
    return _check(load().oaa_plan_set_kernel_chain(plan, w1, J, n1, w2, n2, scratch, scratch_bytes, stream))


def oaa_status_string(status):
    return load().oaa_status_string(status).decode()


def oaa_last_error_detail():
    return load().oaa_last_error_detail().decode()


# ---- torch convenience wrapper ----------------------------------------------

class Plan:
    """One layer x[B,C,N,N] (*) w[K,C,n,n]; owns a plan handle and a device
    workspace tensor. Calls enqueue on torch's current stream of the tensors'
    device and return without synchronising. The workspace is marked as used
    by every stream a call runs on, so that torch does not hand its memory
    out again before that work is done once the plan is released.
    ``generation`` counts the passes that replaced cached spectra (forward,
    backward_data, backward_filter)."""

    def __init__(self, B, C, K, N, n, device="cuda", contraction=CONTRACTION_AUTO, tiling="paper",
                 method=METHOD_OVERLAP_ADD):
        """tiling: "paper" (blocks of n, oaa_plan_create), "auto" (the
        library's choice) or an (L, b) pair (oaa_plan_create_tiled).
        method=METHOD_OVERLAP_SAVE: the output-tiled passes
        (oaa_plan_create_method); tiling "auto"/"paper" or (L, b) with b 0 or
        L - n + 1."""
        import torch
        if method != METHOD_OVERLAP_ADD:
            L, b = (0, 0) if tiling in ("paper", "auto") else tiling
            self.handle = oaa_plan_create_method(B, C, K, N, n, L, b, method)
        elif tiling == "paper":
            self.handle = oaa_plan_create(B, C, K, N, n)
        elif tiling == "auto":
            self.handle = oaa_plan_create_tiled(B, C, K, N, n, 0, 0)
        else:
            L, b = tiling
            self.handle = oaa_plan_create_tiled(B, C, K, N, n, L, b)
        self.geometry = oaa_plan_geometry(self.handle)
        self.device = torch.device(device)
        self.generation = 0
        nbytes = oaa_plan_workspace_bytes(self.handle)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        self._streams = {torch.cuda.current_stream(self.device).cuda_stream}
        oaa_plan_bind_workspace(self.handle, self.workspace.data_ptr(), self.workspace.numel())
        if contraction != CONTRACTION_AUTO:
            oaa_plan_set_contraction(self.handle, contraction)
            self.geometry = oaa_plan_geometry(self.handle)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                oaa_plan_destroy(h)
            except Exception:
                pass
            self.handle = None

    @property
    def output_side(self):
        return self.geometry["M"]

    @property
    def caches_grad_spectra(self):
        """Whether backward_filter may take gr=None after backward_data (the
        fused few-channel passes keep no gradient spectra)."""
        return not self.geometry["fused"]

    def _ptr(self, t, shape, name):
        import torch
        if t is None:
            return None
        if t.dtype != torch.float32 or not t.is_contiguous() or t.device != self.device:
            raise ValueError(f"{name} must be a contiguous float32 tensor on {self.device}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
        return t.data_ptr()

    def _stream(self):
        import torch
        s = torch.cuda.current_stream(self.device)
        if s.cuda_stream not in self._streams:
            self.workspace.record_stream(s)
            self._streams.add(s.cuda_stream)
        return s.cuda_stream

    def _empty(self, shape):
        import torch
        return torch.empty(shape, dtype=torch.float32, device=self.device)

    def forward(self, x, w, y=None):
        g = self.geometry
        B, C, K, N, n, M = g["B"], g["C"], g["K"], g["N"], g["n"], g["M"]
        y = self._empty((B, K, M, M)) if y is None else y
        oaa_conv_forward(self.handle, self._ptr(x, (B, C, N, N), "x"), self._ptr(w, (K, C, n, n), "w"),
                         self._ptr(y, (B, K, M, M), "y"), self._stream())
        self.generation += 1
        return y

    def forward_noalloc(self, x, w, y):
        """oaa_conv_forward_noalloc into the caller's y: the library's static
        scratch instead of this plan's workspace, no allocation."""
        g = self.geometry
        B, C, K, N, n, M = g["B"], g["C"], g["K"], g["N"], g["n"], g["M"]
        oaa_conv_forward_noalloc(self.handle, self._ptr(x, (B, C, N, N), "x"), self._ptr(w, (K, C, n, n), "w"),
                                 self._ptr(y, (B, K, M, M), "y"), self._stream())
        return y

    def backward_data(self, gr, w, dx=None):
        g = self.geometry
        B, C, K, N, n, M = g["B"], g["C"], g["K"], g["N"], g["n"], g["M"]
        dx = self._empty((B, C, N, N)) if dx is None else dx
        oaa_conv_backward_data(self.handle, self._ptr(gr, (B, K, M, M), "g"), self._ptr(w, (K, C, n, n), "w"),
                               self._ptr(dx, (B, C, N, N), "dx"), self._stream())
        self.generation += 1
        return dx

    def backward_filter(self, x, gr, dw=None):
        g = self.geometry
        B, C, K, N, n, M = g["B"], g["C"], g["K"], g["N"], g["n"], g["M"]
        dw = self._empty((K, C, n, n)) if dw is None else dw
        oaa_conv_backward_filter(self.handle, self._ptr(x, (B, C, N, N), "x"), self._ptr(gr, (B, K, M, M), "g"),
                                 self._ptr(dw, (K, C, n, n), "dw"), self._stream())
        self.generation += 1
        return dw

    def set_kernel_chain(self, w1, w2):
        """oaa_plan_set_kernel_chain: the plan's kernel spectra become those
        of two stacked layers, w1[J,C,n1,n1] then w2[K,J,n2,n2] with
        n1 + n2 - 1 = n; forward(x, None) then computes both layers."""
        import torch
        g = self.geometry
        J, n1, n2 = w1.shape[0], w1.shape[-1], w2.shape[-1]
        p1 = self._ptr(w1, (J, g["C"], n1, n1), "w1")
        p2 = self._ptr(w2, (g["K"], J, n2, n2), "w2")
        nbytes = oaa_plan_chain_scratch_bytes(self.handle, J)
        scratch = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        stream = self._stream()
        # scratch is allocated on, and used on, the current stream: torch
        # reuses its memory only for work ordered after these kernels
        oaa_plan_set_kernel_chain(self.handle, p1, J, n1, p2, n2, scratch.data_ptr(), scratch.numel(), stream)
        self.generation += 1

    def set_timing(self, enable):
        oaa_plan_set_timing(self.handle, enable)

    def stage_times(self):
        return oaa_plan_stage_times(self.handle)

    def region(self, which):
        """A view of one workspace region as complex64 (for stage checks)."""
        import torch
        off, size = oaa_plan_region(self.handle, which)
        return self.workspace[off:off + size].view(torch.complex64)
