"""Single-precision replica of the windowed mean-field, for conditioning
and storage-precision studies.  TEST CODE ONLY.

It evaluates the same update as the double oracle (Alg. 1 with the Eq. 4
kernel, the centre tap excluded, out-of-image neighbours contributing
nothing, Potts compatibility folded as softmax(U + M), which differs from
U - (sum M - M) by a per-pixel shift only), but every array operation runs
in float32, in a chosen order of the window taps.  Two replicas that differ
only in the order of the taps round differently; pixels where they leave the
double result by a wide margin are the ones whose value single precision
cannot fix, whatever the implementation.

`store` optionally rounds the stored tensors (the unary once, Q after each
round) through a narrower format, to measure what storing them in it would
cost.  Nothing here is shared with the HIP library.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned
    as float32."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    r = ((b + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def _softmax(Z: np.ndarray) -> np.ndarray:
    m = Z.max(axis=1, keepdims=True)
    e = np.exp(Z - m, dtype=np.float32)
    return (e / e.sum(axis=1, keepdims=True, dtype=np.float32)).astype(np.float32)


def taps(k: int, reverse: bool = False):
    r = (k - 1) // 2
    t = [(dy, dx) for dy in range(-r, r + 1) for dx in range(-r, r + 1) if (dy, dx) != (0, 0)]
    return t[::-1] if reverse else t


def meanfield_f32(U, I, k: int, w_app: float, theta_alpha: float, theta_beta: float,
                  w_smooth: float, theta_gamma: float, T: int, reverse: bool = False,
                  store=None) -> np.ndarray:
    """Q after T rounds, [B, C, H, W] float32; U [B, C, H, W] logits, I
    [B, 3, H, W] RGB on 0..255."""
    f = np.float32
    U = np.ascontiguousarray(U, dtype=f)
    I = np.ascontiguousarray(I, dtype=f)
    if store is not None:
        U = store(U)
    B, C, H, W = U.shape
    r = (k - 1) // 2
    # zero-padded copies so that a neighbour outside the image reads 0 and
    # carries weight 0 (the mask)
    Ip = np.zeros((B, 3, H + 2 * r, W + 2 * r), f)
    Ip[:, :, r:r + H, r:r + W] = I
    mask = np.zeros((H + 2 * r, W + 2 * r), f)
    mask[r:r + H, r:r + W] = 1
    inv_a = f(1.0 / (2.0 * theta_alpha * theta_alpha))
    inv_b = f(1.0 / (2.0 * theta_beta * theta_beta))
    inv_g = f(1.0 / (2.0 * theta_gamma * theta_gamma))
    weights = []
    for dy, dx in taps(k, reverse):
        sl = (slice(None), slice(None), slice(r + dy, r + dy + H), slice(r + dx, r + dx + W))
        d = I - Ip[sl]
        col2 = (d * d).sum(axis=1, dtype=f)
        n = f(dy * dy + dx * dx)
        w = (f(w_app) * np.exp(-n * inv_a - col2 * inv_b, dtype=f)
             + f(w_smooth) * np.exp(-n * inv_g, dtype=f)).astype(f)
        weights.append((dy, dx, w * mask[r + dy:r + dy + H, r + dx:r + dx + W]))
    Q = _softmax(U)
    for _ in range(T):
        if store is not None:
            Q = store(Q)
        Qp = np.zeros((B, C, H + 2 * r, W + 2 * r), f)
        Qp[:, :, r:r + H, r:r + W] = Q
        M = np.zeros_like(U)
        for dy, dx, w in weights:
            M += w[:, None] * Qp[:, :, r + dy:r + dy + H, r + dx:r + dx + W]
        Q = _softmax(U + M)
    return Q
