"""Slow, differently-structured forms of mean-field inference used to pin
``oracle.c``.  TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Two forms, both float64 numpy, for tiny images only:

``dense_meanfield``
    The fully-connected CRF message of Sec. 3 written as one N x N kernel
    matrix over all pixel pairs (Eq. 4), with the ConvCRF locality assumption
    of Sec. 4 applied as a 0/1 mask on that matrix (pairs farther apart than
    the window are conditionally independent, so their potential is zero).
    With the mask off it is FullCRF mean-field computed exactly, which is what
    the paper says ConvCRF message passing reproduces when the window covers
    the image (Sec. 4.1, Sec. 5.1).

``energy_meanfield``
    Mean-field derived from the Gibbs distribution itself (Eq. 1-3) instead of
    from Alg. 1: each pixel's new marginal is proportional to
    exp(-E_{x_-i ~ Q}[E(x_i = l, x_-i)]), the expectation being an explicit sum
    over every labelling of the other pixels weighted by its probability under
    the current (factorised) Q.  The pairwise sum runs over unordered pairs
    i < j, which is the convention under which Alg. 1 (no factor 2) is the
    exact coordinate update; updates are applied to all pixels at once, as in
    Alg. 1.  Cost is C^(N-1) per pixel, so N <= ~8.
"""
from __future__ import annotations

import itertools
import math

import numpy as np


def _pixels(H: int, W: int):
    ys, xs = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64),
                         indexing="ij")
    return ys.ravel(), xs.ravel()


def pair_kernel_matrix(I, w_app, theta_alpha, theta_beta, w_smooth, theta_gamma,
                       filter_size=None):
    """N x N matrix of Eq. 4 over all pixel pairs of I [3,H,W], zero diagonal
    (the energy sums over i != j, Eq. 2).  If ``filter_size`` is given, pairs
    outside the (k x k) window are zeroed (Sec. 4 conditional independence)."""
    I = np.asarray(I, dtype=np.float64)
    _, H, W = I.shape
    ys, xs = _pixels(H, W)
    pos = (ys[:, None] - ys[None, :]) ** 2 + (xs[:, None] - xs[None, :]) ** 2
    f = I.reshape(3, -1)
    col = sum((f[ch][:, None] - f[ch][None, :]) ** 2 for ch in range(3))
    K = (w_app * np.exp(-pos / (2 * theta_alpha ** 2) - col / (2 * theta_beta ** 2))
         + w_smooth * np.exp(-pos / (2 * theta_gamma ** 2)))
    np.fill_diagonal(K, 0.0)
    if filter_size is not None:
        r = (filter_size - 1) // 2
        cheb = np.maximum(np.abs(ys[:, None] - ys[None, :]), np.abs(xs[:, None] - xs[None, :]))
        K = np.where(cheb <= r, K, 0.0)
    return K


def _softmax_cols(Z):
    Z = Z - Z.max(axis=0, keepdims=True)
    E = np.exp(Z)
    return E / E.sum(axis=0, keepdims=True)


def dense_meanfield(U, I, iters, w_app, theta_alpha, theta_beta, w_smooth, theta_gamma,
                    filter_size=None, compat=None):
    """Mean-field for one image U [C,H,W], I [3,H,W] with the all-pairs kernel
    matrix; returns Q [C,H,W]."""
    U = np.asarray(U, dtype=np.float64)
    C, H, W = U.shape
    K = pair_kernel_matrix(I, w_app, theta_alpha, theta_beta, w_smooth, theta_gamma,
                           filter_size)
    mu = (1.0 - np.eye(C)) if compat is None else np.asarray(compat, dtype=np.float64)
    u = U.reshape(C, -1)
    Q = _softmax_cols(u)
    for _ in range(iters):
        M = Q @ K.T                      # M[l, i] = sum_j K[i, j] Q[l, j]
        Q = _softmax_cols(u - mu @ M)
    return Q.reshape(C, H, W)


def energy_meanfield(U, I, iters, w_app, theta_alpha, theta_beta, w_smooth, theta_gamma,
                     filter_size=None, compat=None):
    """Mean-field from the Gibbs energy by enumeration (tiny images only).

    E(x) = sum_i psi_u(x_i) + sum_{i<j} mu(x_i, x_j) k(f_i, f_j), psi_u = -U.
    ``compat`` must be symmetric for this energy to be well defined with one
    term per unordered pair."""
    U = np.asarray(U, dtype=np.float64)
    C, H, W = U.shape
    N = H * W
    if N > 9:
        raise ValueError("enumeration is only for N <= 9 pixels")
    Kmat = pair_kernel_matrix(I, w_app, theta_alpha, theta_beta, w_smooth, theta_gamma,
                              filter_size)
    mu = (1.0 - np.eye(C)) if compat is None else np.asarray(compat, dtype=np.float64)
    if not np.allclose(mu, mu.T):
        raise ValueError("energy form needs a symmetric compatibility")
    psi = -U.reshape(C, N)

    def energy(x):
        e = sum(psi[x[i], i] for i in range(N))
        for i in range(N):
            for j in range(i + 1, N):
                e += mu[x[i], x[j]] * Kmat[i, j]
        return e

    # Q0: the Gibbs marginals with the pairwise term dropped, i.e. softmax(-psi).
    Q = np.zeros((C, N))
    for i in range(N):
        z = [-psi[l, i] for l in range(C)]
        m = max(z)
        e = [math.exp(v - m) for v in z]
        Q[:, i] = [v / sum(e) for v in e]

    for _ in range(iters):
        Qn = np.zeros_like(Q)
        for i in range(N):
            others = [j for j in range(N) if j != i]
            expect = np.zeros(C)
            for labels in itertools.product(range(C), repeat=N - 1):
                prob = 1.0
                for j, lj in zip(others, labels):
                    prob *= Q[lj, j]
                x = [0] * N
                for j, lj in zip(others, labels):
                    x[j] = lj
                for l in range(C):
                    x[i] = l
                    expect[l] += prob * energy(x)
            z = -expect
            z -= z.max()
            e = np.exp(z)
            Qn[:, i] = e / e.sum()
        Q = Qn
    return Q.reshape(C, H, W)
