"""Double-precision CPU oracle for ConvCRF mean-field inference.

TEST INFRASTRUCTURE ONLY.  This package is the independent checker the HIP
library is compared against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it; the product package
never does, and the two share no code.

Contents
--------
- ``oracle.c`` (built to ``liboracle.so`` with gcc -O2 -fopenmp, no fast-math):
  the windowed mean-field of Alg. 1 with the Eq. 4 kernel and the Eq. 6
  message, plus the pooled ("blur", Sec. 4.2) variant, and the reverse-mode
  derivative of the unpooled mean-field (the loss gradient with respect to
  the unaries, the compatibility and the five Eq. 4 parameters, obtained by
  undoing each step of Alg. 1).  Wrapped here.
- ``bruteforce.py``: two slower, differently-structured forms used to pin
  ``oracle.c`` (dense all-pairs FullCRF mean-field, and mean-field derived by
  enumerating the Gibbs energy of Eq. 1-3).

Every array is float64, C-contiguous, layout [B][C][H][W] for class planes and
[B][3][H][W] for RGB on its 0..255 scale.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

__all__ = [
    "OracleParams", "build", "meanfield", "message", "update", "softmax",
    "avgpool", "upsample", "kernel", "num_threads", "meanfield_backward", "PARAM_NAMES",
]

# order of the Eq. 4 parameters in meanfield_backward's dparams
PARAM_NAMES = ("w_app", "theta_alpha", "theta_beta", "w_smooth", "theta_gamma")


def build(force: bool = False) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` (gcc, -O2, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _CParams(ctypes.Structure):
    _fields_ = [
        ("filter_size", ctypes.c_int),
        ("blur", ctypes.c_int),
        ("include_center", ctypes.c_int),
        ("reserved", ctypes.c_int),
        ("w_app", ctypes.c_double),
        ("theta_alpha", ctypes.c_double),
        ("theta_beta", ctypes.c_double),
        ("w_smooth", ctypes.c_double),
        ("theta_gamma", ctypes.c_double),
    ]


@dataclass
class OracleParams:
    """Eq. 4 parameters, window side k (Sec. 4), blur factor s (Sec. 4.2)."""
    filter_size: int = 7
    blur: int = 1
    include_center: bool = False
    w_app: float = 10.0
    theta_alpha: float = 80.0
    theta_beta: float = 13.0
    w_smooth: float = 3.0
    theta_gamma: float = 3.0

    def c(self) -> _CParams:
        return _CParams(int(self.filter_size), int(self.blur), int(bool(self.include_center)), 0,
                        float(self.w_app), float(self.theta_alpha), float(self.theta_beta),
                        float(self.w_smooth), float(self.theta_gamma))


_lib = None
_dp = ctypes.POINTER(ctypes.c_double)


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        lib.oracle_meanfield.restype = ctypes.c_int
        lib.oracle_meanfield.argtypes = [_dp, _dp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_int, ctypes.POINTER(_CParams), _dp,
                                         ctypes.c_int, _dp]
        lib.oracle_message.restype = None
        lib.oracle_message.argtypes = [_dp, _dp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.POINTER(_CParams), ctypes.c_double, _dp]
        lib.oracle_update.restype = None
        lib.oracle_update.argtypes = [_dp, _dp, _dp, ctypes.c_int, ctypes.c_long, _dp]
        lib.oracle_softmax.restype = None
        lib.oracle_softmax.argtypes = [_dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _dp]
        lib.oracle_avgpool.restype = None
        lib.oracle_avgpool.argtypes = [_dp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, _dp]
        lib.oracle_upsample.restype = None
        lib.oracle_upsample.argtypes = [_dp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, _dp]
        lib.oracle_kernel.restype = ctypes.c_double
        lib.oracle_kernel.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.POINTER(_CParams)]
        lib.oracle_meanfield_f.restype = ctypes.c_int
        lib.oracle_meanfield_f.argtypes = [_dp, _dp, _dp, ctypes.c_int, ctypes.c_int,
                                           ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           ctypes.POINTER(_CParams), _dp, ctypes.c_int, _dp]
        lib.oracle_meanfield_backward_f.restype = ctypes.c_int
        lib.oracle_meanfield_backward_f.argtypes = [_dp, _dp, _dp, ctypes.c_int, ctypes.c_int,
                                                    ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                    ctypes.POINTER(_CParams), _dp,
                                                    ctypes.c_int, _dp, _dp, _dp, _dp, _dp]
        lib.oracle_meanfield_backward.restype = ctypes.c_int
        lib.oracle_meanfield_backward.argtypes = [_dp, _dp, ctypes.c_int, ctypes.c_int,
                                                  ctypes.c_int, ctypes.c_int,
                                                  ctypes.POINTER(_CParams), _dp, ctypes.c_int,
                                                  _dp, _dp, _dp, _dp]
        lib.oracle_num_threads.restype = ctypes.c_int
        lib.oracle_num_threads.argtypes = []
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_dp)


def num_threads() -> int:
    """OpenMP threads the oracle will use (OMP_NUM_THREADS, else all cores)."""
    return int(_load().oracle_num_threads())


def kernel(pos_d2: float, col_d2: float, params: OracleParams) -> float:
    """Eq. 4 merged kernel for squared position / colour distances."""
    return float(_load().oracle_kernel(pos_d2, col_d2, ctypes.byref(params.c())))


def _features(F, B, H, W):
    if F is None:
        return None, 0
    F = _f64(F)
    if F.ndim != 4 or F.shape[0] != B or F.shape[2:] != (H, W) or F.shape[1] < 1:
        raise ValueError("expected features [B,d,H,W]")
    return F, F.shape[1]


def meanfield(U, I, params: OracleParams, iters: int, compat=None, features=None) -> np.ndarray:
    """Alg. 1: ``iters`` mean-field rounds from softmax(U).  U [B,C,H,W],
    I [B,3,H,W]; compat = row-major C x C mu[l][l'] or None for Potts;
    features = learnable smoothness features [B,d,H,W] (the "+T" variant of
    Sec. 4.2) or None for the positions."""
    U = _f64(U)
    I = _f64(I)
    if U.ndim != 4 or I.ndim != 4 or I.shape[1] != 3 or I.shape[0] != U.shape[0] \
            or I.shape[2:] != U.shape[2:]:
        raise ValueError("expected U [B,C,H,W] and I [B,3,H,W]")
    B, C, H, W = U.shape
    F, d = _features(features, B, H, W)
    mu = None if compat is None else _f64(compat).reshape(C, C)
    Q = np.empty_like(U)
    rc = _load().oracle_meanfield_f(_ptr(U), _ptr(I), None if F is None else _ptr(F), d,
                                    B, C, H, W, ctypes.byref(params.c()),
                                    None if mu is None else _ptr(mu), int(iters), _ptr(Q))
    if rc != 0:
        raise ValueError("oracle_meanfield rejected its arguments")
    return Q


def meanfield_backward(U, I, params: OracleParams, iters: int, G, compat=None,
                       features=None):
    """Reverse-mode derivative of ``meanfield`` for a loss whose
    derivative with respect to the returned Q is G [B,C,H,W].  Returns
    (dU [B,C,H,W], dmu [C,C], dparams [5] in PARAM_NAMES order); dmu is the
    derivative with respect to the compatibility at ``compat`` (Potts when
    None), dparams with respect to the Eq. 4 parameters; both are summed over
    the batch.  With ``features`` [B,d,H,W] a fourth value, dL/dfeatures of
    the same shape, is returned."""
    U = _f64(U)
    I = _f64(I)
    G = _f64(G)
    if U.ndim != 4 or G.shape != U.shape or I.shape != (U.shape[0], 3) + U.shape[2:]:
        raise ValueError("expected U, G [B,C,H,W] and I [B,3,H,W]")
    B, C, H, W = U.shape
    F, d = _features(features, B, H, W)
    mu = None if compat is None else _f64(compat).reshape(C, C)
    dU = np.empty_like(U)
    dmu = np.empty((C, C))
    dp = np.empty(5)
    dF = None if F is None else np.empty_like(F)
    rc = _load().oracle_meanfield_backward_f(_ptr(U), _ptr(I),
                                             None if F is None else _ptr(F), d, B, C, H, W,
                                             ctypes.byref(params.c()),
                                             None if mu is None else _ptr(mu), int(iters),
                                             _ptr(G), _ptr(dU), _ptr(dmu), _ptr(dp),
                                             None if dF is None else _ptr(dF))
    if rc != 0:
        raise ValueError("oracle_meanfield_backward rejected its arguments")
    return (dU, dmu, dp) if F is None else (dU, dmu, dp, dF)


def message(Q, I, params: OracleParams, pos_scale: float = 1.0) -> np.ndarray:
    """Eq. 6 message for one image: Q [C,H,W], I [3,H,W] -> M [C,H,W]."""
    Q = _f64(Q)
    I = _f64(I)
    C, H, W = Q.shape
    M = np.empty_like(Q)
    _load().oracle_message(_ptr(Q), _ptr(I), C, H, W, ctypes.byref(params.c()),
                           float(pos_scale), _ptr(M))
    return M


def update(U, M, compat=None) -> np.ndarray:
    """Alg. 1 compatibility + unary + softmax: U, M [C,H,W] -> Q [C,H,W]."""
    U = _f64(U)
    M = _f64(M)
    C = U.shape[0]
    mu = None if compat is None else _f64(compat).reshape(C, C)
    Q = np.empty_like(U)
    _load().oracle_update(_ptr(U), _ptr(M), None if mu is None else _ptr(mu), C,
                          int(U.size // C), _ptr(Q))
    return Q


def softmax(U) -> np.ndarray:
    """Alg. 1 initialisation: softmax over classes of U [C,H,W]."""
    U = _f64(U)
    C, H, W = U.shape
    Q = np.empty_like(U)
    _load().oracle_softmax(_ptr(U), C, H, W, _ptr(Q))
    return Q


def avgpool(X, s: int) -> np.ndarray:
    """s x s average pooling of X [n,H,W]."""
    X = _f64(X)
    n, H, W = X.shape
    Y = np.empty((n, H // s, W // s))
    _load().oracle_avgpool(_ptr(X), n, H, W, int(s), _ptr(Y))
    return Y


def upsample(X, s: int) -> np.ndarray:
    """Bilinear x s upsampling (half-pixel centres, edge clamp) of X [n,h,w]."""
    X = _f64(X)
    n, h, w = X.shape
    Y = np.empty((n, h * s, w * s))
    _load().oracle_upsample(_ptr(X), n, h, w, int(s), _ptr(Y))
    return Y
