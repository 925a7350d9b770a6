"""Pins of the oracle's reverse-mode derivative of the mean-field (Alg. 1
unrolled over T rounds; Eq. 4 kernel, Eq. 6 message).

The derivative is checked against central finite differences of the forward
oracle, which is itself pinned by the tests in test_oracle.py: the loss is
L = sum(G * Q^T) for a seeded G, and every unary, every compatibility entry
and every Eq. 4 parameter is perturbed in turn.  A dropped term, a wrong sign,
a transposed compatibility or a wrong kernel derivative changes the result by
far more than the finite-difference error (about 1e-9 relative here).
"""
import numpy as np
import pytest

import oracle as orc


def _problem(seed, B, C, H, W, gen_mu=True):
    rng = np.random.default_rng(seed)
    U = rng.normal(0.0, 1.5, (B, C, H, W))
    # a few colour levels, so that colour differences take both small and
    # large values inside every window
    I = rng.integers(0, 4, (B, 3, H, W)) * 40.0 + rng.normal(0.0, 6.0, (B, 3, H, W))
    G = rng.normal(0.0, 1.0, (B, C, H, W))
    mu = rng.normal(0.3, 0.5, (C, C)) if gen_mu else None
    return U, I, G, mu


def _loss(U, I, params, T, G, mu):
    return float(np.sum(G * orc.meanfield(U, I, params, T, compat=mu)))


def _fd(f, x, h):
    return (f(x + h) - f(x - h)) / (2.0 * h)


CASES = [
    # (seed, B, C, H, W, k, T, include_center, general mu)
    (1, 1, 3, 4, 5, 3, 2, False, True),
    (2, 2, 2, 5, 4, 5, 3, False, False),
    (3, 1, 4, 3, 6, 3, 1, True, True),
    (4, 1, 3, 5, 5, 7, 2, True, False),
    (5, 1, 2, 2, 3, 3, 0, False, True),
]


@pytest.mark.parametrize("seed,B,C,H,W,k,T,center,gen_mu", CASES)
def test_unary_gradient_matches_finite_differences(seed, B, C, H, W, k, T, center, gen_mu):
    U, I, G, mu = _problem(seed, B, C, H, W, gen_mu)
    params = orc.OracleParams(filter_size=k, include_center=center, w_app=4.0,
                              theta_alpha=3.0, theta_beta=30.0, w_smooth=1.5,
                              theta_gamma=1.2)
    dU, _, _ = orc.meanfield_backward(U, I, params, T, G, compat=mu)
    h = 1e-5
    fd = np.empty_like(U)
    for idx in np.ndindex(U.shape):
        def f(v):
            Up = U.copy()
            Up[idx] = v
            return _loss(Up, I, params, T, G, mu)
        fd[idx] = _fd(f, U[idx], h)
    scale = np.max(np.abs(fd))
    assert scale > 1e-3
    np.testing.assert_allclose(dU, fd, rtol=0, atol=1e-7 * max(1.0, scale))


@pytest.mark.parametrize("seed,B,C,H,W,k,T,center,gen_mu", CASES)
def test_compat_gradient_matches_finite_differences(seed, B, C, H, W, k, T, center, gen_mu):
    U, I, G, mu = _problem(seed, B, C, H, W, gen_mu)
    params = orc.OracleParams(filter_size=k, include_center=center, w_app=4.0,
                              theta_alpha=3.0, theta_beta=30.0, w_smooth=1.5,
                              theta_gamma=1.2)
    _, dmu, _ = orc.meanfield_backward(U, I, params, T, G, compat=mu)
    # Potts (compat None) is mu = 1 - identity: perturb that matrix
    base = mu if mu is not None else 1.0 - np.eye(C)
    h = 1e-6
    fd = np.empty((C, C))
    for a in range(C):
        for b in range(C):
            def f(v):
                m = base.copy()
                m[a, b] = v
                return _loss(U, I, params, T, G, m)
            fd[a, b] = _fd(f, base[a, b], h)
    if T == 0:
        assert np.all(dmu == 0.0)
    else:
        assert np.max(np.abs(fd)) > 1e-3
    np.testing.assert_allclose(dmu, fd, rtol=0, atol=1e-7 * max(1.0, np.max(np.abs(fd))))


@pytest.mark.parametrize("seed,B,C,H,W,k,T,center,gen_mu", CASES)
def test_kernel_parameter_gradient_matches_finite_differences(seed, B, C, H, W, k, T, center,
                                                              gen_mu):
    U, I, G, mu = _problem(seed, B, C, H, W, gen_mu)
    vals = dict(w_app=4.0, theta_alpha=3.0, theta_beta=30.0, w_smooth=1.5, theta_gamma=1.2)
    params = orc.OracleParams(filter_size=k, include_center=center, **vals)
    _, _, dp = orc.meanfield_backward(U, I, params, T, G, compat=mu)
    fd = np.empty(5)
    for j, name in enumerate(orc.PARAM_NAMES):
        h = 1e-6 * vals[name]
        def f(v):
            kw = dict(vals)
            kw[name] = v
            return _loss(U, I, orc.OracleParams(filter_size=k, include_center=center, **kw), T,
                         G, mu)
        fd[j] = _fd(f, vals[name], h)
    if T == 0:
        assert np.all(dp == 0.0)
    else:
        assert np.min(np.abs(fd)) > 1e-6   # every parameter matters in these cases
    np.testing.assert_allclose(dp, fd, rtol=2e-6, atol=1e-9)


def test_batch_items_are_independent():
    """dU of a batch equals the per-image derivatives stacked; dmu and the
    parameter derivative add up over the batch."""
    U, I, G, mu = _problem(11, 3, 3, 5, 6, True)
    params = orc.OracleParams(filter_size=3, w_app=4.0, theta_alpha=3.0, theta_beta=30.0,
                              w_smooth=1.5, theta_gamma=1.2)
    dU, dmu, dp = orc.meanfield_backward(U, I, params, 2, G, compat=mu)
    parts = [orc.meanfield_backward(U[b:b + 1], I[b:b + 1], params, 2, G[b:b + 1], compat=mu)
             for b in range(3)]
    np.testing.assert_array_equal(dU, np.concatenate([p[0] for p in parts]))
    np.testing.assert_allclose(dmu, sum(p[1] for p in parts), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(dp, sum(p[2] for p in parts), rtol=1e-13, atol=1e-15)


def test_gradient_of_zero_pairwise_weights_is_softmax_adjoint():
    """With both kernel weights zero the messages vanish and Q^T = softmax(U):
    dU is the softmax adjoint of G in closed form, whatever T."""
    U, I, G, mu = _problem(12, 1, 4, 4, 4, True)
    params = orc.OracleParams(filter_size=3, w_app=0.0, w_smooth=0.0)
    dU, _, _ = orc.meanfield_backward(U, I, params, 3, G, compat=mu)
    Q = np.exp(U - U.max(axis=1, keepdims=True))
    Q /= Q.sum(axis=1, keepdims=True)
    want = Q * (G - np.sum(Q * G, axis=1, keepdims=True))
    np.testing.assert_allclose(dU, want, rtol=1e-12, atol=1e-14)


BLUR_CASES = [
    # (seed, B, C, H, W, k, T, s, include_center, general mu)
    (13, 1, 3, 6, 8, 3, 2, 2, False, True),
    (14, 2, 2, 8, 8, 3, 1, 4, True, False),
    (15, 1, 3, 6, 9, 5, 2, 3, False, False),
    (16, 1, 2, 16, 16, 3, 2, 8, False, True),   # s = 8: a 2 x 2 pooled grid
]


@pytest.mark.parametrize("seed,B,C,H,W,k,T,s,center,gen_mu", BLUR_CASES)
def test_blur_gradient_matches_finite_differences(seed, B, C, H, W, k, T, s, center, gen_mu):
    """The pooled message (Sec. 4.2 blur): every unary, every compatibility
    entry and every Eq. 4 parameter against central finite differences."""
    U, I, G, mu = _problem(seed, B, C, H, W, gen_mu)
    # with s = 8 the pooled cells lie 8 pixels apart: a smoothness width on
    # that scale, so that its derivative stands above the differences' noise
    vals = dict(w_app=4.0, theta_alpha=3.0, theta_beta=30.0, w_smooth=1.5,
                theta_gamma=1.2 if s < 8 else 9.0)
    params = orc.OracleParams(filter_size=k, blur=s, include_center=center, **vals)
    dU, dmu, dp = orc.meanfield_backward(U, I, params, T, G, compat=mu)
    fd = np.empty_like(U)
    for idx in np.ndindex(U.shape):
        def f(v):
            Up = U.copy()
            Up[idx] = v
            return _loss(Up, I, params, T, G, mu)
        fd[idx] = _fd(f, U[idx], 1e-5)
    np.testing.assert_allclose(dU, fd, rtol=0, atol=1e-7 * max(1.0, np.abs(fd).max()))
    base = mu if mu is not None else 1.0 - np.eye(C)
    fdm = np.empty((C, C))
    for a in range(C):
        for b in range(C):
            def g(v):
                m = base.copy()
                m[a, b] = v
                return _loss(U, I, params, T, G, m)
            fdm[a, b] = _fd(g, base[a, b], 1e-6)
    assert np.abs(fdm).max() > 1e-4
    np.testing.assert_allclose(dmu, fdm, rtol=0, atol=1e-7 * max(1.0, np.abs(fdm).max()))
    for j, name in enumerate(orc.PARAM_NAMES):
        h = 1e-6 * vals[name]
        def q(v):
            return _loss(U, I, orc.OracleParams(filter_size=k, blur=s, include_center=center,
                                                **dict(vals, **{name: v})), T, G, mu)
        fdp = _fd(q, vals[name], h)
        assert abs(fdp - dp[j]) <= 2e-6 * abs(fdp) + 1e-9, (name, fdp, dp[j])


def test_blur_of_one_is_the_unpooled_derivative():
    U, I, G, mu = _problem(16, 1, 3, 6, 6, True)
    a = orc.meanfield_backward(U, I, orc.OracleParams(filter_size=3), 2, G, compat=mu)
    b = orc.meanfield_backward(U, I, orc.OracleParams(filter_size=3, blur=1), 2, G, compat=mu)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
