"""ctypes binding of ``libconvcrf.so`` (C ABI in ``include/convcrf.h``).

Argument marshalling only: every step of mean-field inference runs in the
library's HIP kernels.  torch provides device memory and the stream; tensors
must be contiguous float32 on the context's GPU.  There is no fallback: if
the library is missing or cannot be loaded, every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libconvcrf.so")

# status codes (convcrf_status)
OK = 0
E_INVALID_ARG = -1
E_UNSUPPORTED = -2
E_NO_DEVICE = -3
E_HIP = -4
E_OOM = -5

VARIANT_FUSED = 0
VARIANT_MATERIALISED = 1
VARIANT_RESIDENT = 2

KERNEL_NAMES = ("fused_first", "fused_iter", "fused_resident", "sync_reset", "softmax", "build_kernel",
                "materialised_iter", "blur_pool", "blur_message", "blur_update",
                "bwd_point", "bwd_message", "bwd_reduce", "feature_iter", "bwd_blur_transpose",
                "blur_iteration")

EXPORTED = ("convcrf_default_params", "convcrf_validate", "convcrf_init", "convcrf_destroy",
            "convcrf_meanfield", "convcrf_meanfield_backward", "convcrf_profile_enable",
            "convcrf_profile_read", "convcrf_last_error", "convcrf_status_string",
            "convcrf_strerror", "convcrf_synchronize", "convcrf_meanfield_noalloc")

# order of grad_kernel in convcrf_meanfield_backward
KERNEL_PARAM_NAMES = ("w_app", "theta_alpha", "theta_beta", "w_smooth", "theta_gamma")


class ConvCRFError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class CParams(ctypes.Structure):
    _fields_ = [
        ("filter_size", ctypes.c_int32),
        ("blur", ctypes.c_int32),
        ("include_center", ctypes.c_int32),
        ("variant", ctypes.c_int32),
        ("w_app", ctypes.c_float),
        ("theta_alpha", ctypes.c_float),
        ("theta_beta", ctypes.c_float),
        ("w_smooth", ctypes.c_float),
        ("theta_gamma", ctypes.c_float),
        ("compat", ctypes.POINTER(ctypes.c_float)),
        ("features", ctypes.c_void_p),
        ("feature_dim", ctypes.c_int32),
    ]


@dataclass
class Params:
    """Mirror of ``convcrf_params``; ``compat`` is a C x C host sequence or
    None for Potts; ``features`` a contiguous float32 GPU tensor
    [B, D, H, W] of learnable smoothness features, or None."""
    filter_size: int = 7
    blur: int = 1
    include_center: bool = False
    variant: int = VARIANT_FUSED
    w_app: float = 10.0
    theta_alpha: float = 80.0
    theta_beta: float = 13.0
    w_smooth: float = 3.0
    theta_gamma: float = 3.0
    compat: object = None
    features: object = None
    _keep: list = field(default_factory=list, repr=False, compare=False)

    def c(self, shape=None, device=None) -> CParams:
        """The C struct.  With ``shape`` = (B, C, H, W) of the unary (and its
        ``device``), ``compat`` must be C x C and ``features`` a float32
        tensor [B, D, H, W] on that device: the library reads C*C floats from
        the compatibility pointer and B*D*H*W from the features pointer
        without being able to check either."""
        p = CParams(int(self.filter_size), int(self.blur), int(self.include_center),
                    int(self.variant), float(self.w_app), float(self.theta_alpha),
                    float(self.theta_beta), float(self.w_smooth), float(self.theta_gamma), None,
                    None, 0)
        if self.features is not None:
            import torch
            f = self.features
            if (not isinstance(f, torch.Tensor) or f.dtype != torch.float32 or not f.is_cuda
                    or not f.is_contiguous() or f.dim() != 4):
                raise ConvCRFError(E_INVALID_ARG, "features must be a contiguous 4-D float32 GPU tensor")
            if shape is not None:
                B, _, H, W = shape
                if f.shape[0] != B or f.shape[2] != H or f.shape[3] != W:
                    raise ConvCRFError(E_INVALID_ARG, f"features must be [B, D, H, W] = "
                                       f"[{B}, D, {H}, {W}], got {list(f.shape)}")
            if device is not None and f.device != device:
                raise ConvCRFError(E_INVALID_ARG, f"features are on {f.device}, the unary on {device}")
            p.features = f.data_ptr()
            p.feature_dim = int(f.shape[1])
        if self.compat is not None:
            import numpy as np
            mu = np.asarray(self.compat)
            if mu.dtype.kind not in "fiu":
                raise ConvCRFError(E_INVALID_ARG, "compat must be a real C x C array")
            mu = np.ascontiguousarray(mu, dtype=np.float32)
            if shape is not None and mu.shape != (shape[1], shape[1]):
                raise ConvCRFError(E_INVALID_ARG, f"compat must be C x C = {shape[1]} x {shape[1]}, "
                                   f"got shape {mu.shape}")
            if mu.ndim != 2 or mu.shape[0] != mu.shape[1]:
                raise ConvCRFError(E_INVALID_ARG, f"compat must be a square matrix, got shape {mu.shape}")
            self._keep[:] = [mu]
            p.compat = mu.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
        return p


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libconvcrf.so (once) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    # torch first: the library then binds the HIP runtime torch has loaded,
    # rather than a second copy that would not see torch's devices
    import torch  # noqa: F401
    if not os.path.exists(path):
        raise ConvCRFError(E_NO_DEVICE, f"{path} is not built; run "
                           "`python -m paper_1805_04777_amd.build`")
    lib = ctypes.CDLL(path)
    st = ctypes.c_int
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    lib.convcrf_default_params.restype = st
    lib.convcrf_default_params.argtypes = [P(CParams)]
    lib.convcrf_validate.restype = st
    lib.convcrf_validate.argtypes = [ctypes.c_int] * 4 + [P(CParams), ctypes.c_int]
    lib.convcrf_init.restype = st
    lib.convcrf_init.argtypes = [P(vp), ctypes.c_int]
    lib.convcrf_destroy.restype = None
    lib.convcrf_destroy.argtypes = [vp]
    lib.convcrf_meanfield.restype = st
    lib.convcrf_meanfield.argtypes = [vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int, P(CParams), ctypes.c_int, vp, vp]
    lib.convcrf_meanfield_noalloc.restype = st
    lib.convcrf_meanfield_noalloc.argtypes = lib.convcrf_meanfield.argtypes
    lib.convcrf_meanfield_backward.restype = st
    lib.convcrf_meanfield_backward.argtypes = [vp, vp, vp, ctypes.c_int, ctypes.c_int,
                                               ctypes.c_int, ctypes.c_int, P(CParams),
                                               ctypes.c_int, vp, vp, vp, vp, vp, vp]
    lib.convcrf_profile_enable.restype = st
    lib.convcrf_profile_enable.argtypes = [vp, ctypes.c_int]
    lib.convcrf_profile_read.restype = st
    lib.convcrf_profile_read.argtypes = [vp, ctypes.c_char_p, P(ctypes.c_double),
                                         P(ctypes.c_int64)]
    lib.convcrf_last_error.restype = ctypes.c_char_p
    lib.convcrf_last_error.argtypes = [vp]
    lib.convcrf_status_string.restype = ctypes.c_char_p
    lib.convcrf_status_string.argtypes = [ctypes.c_int]
    lib.convcrf_strerror.restype = ctypes.c_char_p
    lib.convcrf_strerror.argtypes = [vp, ctypes.c_int]
    lib.convcrf_synchronize.restype = st
    lib.convcrf_synchronize.argtypes = [vp, vp]
    _lib = lib
    return lib


def _check(status: int, ctx=None):
    if status != OK:
        lib = load_library()
        raise ConvCRFError(status, lib.convcrf_strerror(ctx, status).decode())


def default_params() -> Params:
    c = CParams()
    _check(load_library().convcrf_default_params(ctypes.byref(c)))
    return Params(c.filter_size, c.blur, bool(c.include_center), c.variant, c.w_app,
                  c.theta_alpha, c.theta_beta, c.w_smooth, c.theta_gamma, None)


def validate(B: int, C: int, H: int, W: int, params: Params, iters: int) -> int:
    """Status that meanfield would return for these sizes (no device needed)."""
    try:
        cp = params.c((B, C, H, W))
    except ConvCRFError as e:
        return e.status
    return int(load_library().convcrf_validate(B, C, H, W, ctypes.byref(cp), iters))


class ConvCRF:
    """A library context bound to one GPU."""

    def __init__(self, device: int = 0):
        lib = load_library()
        h = ctypes.c_void_p()
        _check(lib.convcrf_init(ctypes.byref(h), int(device)))
        self._lib = lib
        self._h = h
        self.device = int(device)

    def close(self):
        if getattr(self, "_h", None):
            self._lib.convcrf_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def meanfield(self, unary, image, params: Params, iters: int, out=None, stream=None,
                  noalloc: bool = False):
        """Q after ``iters`` mean-field rounds; unary [B,C,H,W], image
        [B,3,H,W], both contiguous float32 CUDA tensors.  Enqueued on
        ``stream`` (default: torch's current stream); returns ``out``.
        ``noalloc`` calls convcrf_meanfield_noalloc (workspace in the
        library's per-device scratch array; pass ``out`` to allocate
        nothing on the torch side either)."""
        import torch
        for name, t in (("unary", unary), ("image", image)):
            if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
                raise ConvCRFError(E_INVALID_ARG, f"{name} must be a contiguous 4-D float32 GPU tensor")
        B, C, H, W = unary.shape
        if tuple(image.shape) != (B, 3, H, W):
            raise ConvCRFError(E_INVALID_ARG, "image must be [B,3,H,W] matching unary")
        if out is None:
            out = torch.empty_like(unary)
        elif (out.dtype != torch.float32 or not out.is_contiguous()
              or tuple(out.shape) != tuple(unary.shape) or out.device != unary.device):
            raise ConvCRFError(E_INVALID_ARG, "out must match unary")
        if stream is None:
            stream = torch.cuda.current_stream(unary.device)
        sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        cp = params.c((B, C, H, W), unary.device)
        fn = self._lib.convcrf_meanfield_noalloc if noalloc else self._lib.convcrf_meanfield
        _check(fn(self._h, unary.data_ptr(), image.data_ptr(), B, C, H, W, ctypes.byref(cp),
                  int(iters), out.data_ptr(), sp), self._h)
        return out

    def meanfield_backward(self, unary, image, params: Params, iters: int, grad_q,
                           grad_compat: bool = False, grad_kernel: bool = False,
                           out=None, stream=None):
        """Derivative of a loss through ``meanfield``: returns
        (dL/dU [B,C,H,W], dL/dmu [C,C] or None, dL/d(Eq. 4 parameters) [5]
        or None) as float32 tensors on the unary's device, and with
        ``params.features`` a fourth value, dL/dfeatures; ``grad_q`` is
        dL/dQ.  Enqueued on ``stream`` (default: torch's current stream)."""
        import torch
        for name, t in (("unary", unary), ("image", image), ("grad_q", grad_q)):
            if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
                raise ConvCRFError(E_INVALID_ARG, f"{name} must be a contiguous 4-D float32 GPU tensor")
        B, C, H, W = unary.shape
        if tuple(image.shape) != (B, 3, H, W) or tuple(grad_q.shape) != (B, C, H, W):
            raise ConvCRFError(E_INVALID_ARG, "image must be [B,3,H,W] and grad_q [B,C,H,W]")
        if out is None:
            out = torch.empty_like(unary)
        elif (out.dtype != torch.float32 or not out.is_contiguous()
              or tuple(out.shape) != tuple(unary.shape) or out.device != unary.device):
            raise ConvCRFError(E_INVALID_ARG, "out must match unary")
        gmu = torch.empty((C, C), dtype=torch.float32, device=unary.device) if grad_compat else None
        gk = torch.empty(5, dtype=torch.float32, device=unary.device) if grad_kernel else None
        gf = None if params.features is None else torch.empty_like(params.features)
        if stream is None:
            stream = torch.cuda.current_stream(unary.device)
        sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        cp = params.c((B, C, H, W), unary.device)
        _check(self._lib.convcrf_meanfield_backward(
            self._h, unary.data_ptr(), image.data_ptr(), B, C, H, W, ctypes.byref(cp),
            int(iters), grad_q.data_ptr(), out.data_ptr(),
            gmu.data_ptr() if gmu is not None else None,
            gk.data_ptr() if gk is not None else None,
            gf.data_ptr() if gf is not None else None, sp), self._h)
        return (out, gmu, gk) if gf is None else (out, gmu, gk, gf)

    def last_error(self) -> str:
        """The library's last message for this context."""
        return self._lib.convcrf_last_error(self._h).decode()

    def synchronize(self, stream=None):
        """Wait for ``stream`` (default: torch's current stream on this
        context's device) and raise if a resident call's bounded neighbour
        wait gave up since the last check (its output is then invalid)."""
        import torch
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        sp = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        _check(self._lib.convcrf_synchronize(self._h, sp), self._h)

    def profile_enable(self, on: bool = True):
        _check(self._lib.convcrf_profile_enable(self._h, int(bool(on))), self._h)

    def profile_read(self, name: str):
        """(total milliseconds, launches) of kernel `name` since enabling."""
        ms = ctypes.c_double()
        n = ctypes.c_int64()
        _check(self._lib.convcrf_profile_read(self._h, name.encode(), ctypes.byref(ms),
                                              ctypes.byref(n)), self._h)
        return ms.value, n.value
