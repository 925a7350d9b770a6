"""Pins of the oracle's learnable smoothness features (the "+T" variant of
Sec. 4.2: the inputs of the smoothness Gaussian of Eq. 4 are replaced by a
learnable per-pixel map, initialised to the positions).

Forward: features equal to the pixel positions reproduce the pinned forward
(Eq. 4 as written); constant features make the smoothness Gaussian 1 inside
every window, which a very wide theta_gamma reproduces; scaling the features
and theta_gamma together changes nothing.  Derivative: central finite
differences of the forward for every feature entry and, with features
present, for the unaries, the compatibility and the Eq. 4 parameters.

With blur (Sec. 4.2) the features are pooled to the s x s cells like the
colours: position features then reproduce the pooled kernel, constant ones a
flat smoothness term, only cell means matter, and the derivative (finite
differences again) is the same for every pixel of a cell.
"""
import numpy as np
import pytest

import oracle as orc

VALS = dict(w_app=4.0, theta_alpha=3.0, theta_beta=30.0, w_smooth=1.5, theta_gamma=1.2)


def _problem(seed, B, C, H, W, d=2):
    rng = np.random.default_rng(seed)
    U = rng.normal(0.0, 1.5, (B, C, H, W))
    I = rng.integers(0, 4, (B, 3, H, W)) * 40.0 + rng.normal(0.0, 6.0, (B, 3, H, W))
    G = rng.normal(0.0, 1.0, (B, C, H, W))
    yy, xx = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64),
                         indexing="ij")
    pos = np.stack([yy, xx] + [np.zeros((H, W))] * (d - 2))[None].repeat(B, axis=0)
    F = pos + rng.normal(0.0, 0.4, pos.shape)
    return U, I, G, F, pos


def positions(B, H, W):
    yy, xx = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64),
                         indexing="ij")
    return np.stack([yy, xx])[None].repeat(B, axis=0)


@pytest.mark.parametrize("k,center", [(3, False), (5, True), (7, False)])
def test_position_features_reproduce_eq4(k, center):
    U, I, _, _, pos = _problem(1, 2, 4, 9, 11)
    p = orc.OracleParams(filter_size=k, include_center=center, **VALS)
    np.testing.assert_allclose(orc.meanfield(U, I, p, 3, features=pos), orc.meanfield(U, I, p, 3),
                               rtol=0, atol=1e-13)


def test_constant_features_make_the_smoothness_term_flat():
    U, I, _, _, pos = _problem(2, 1, 3, 8, 9)
    F = np.full_like(pos, 5.0)
    p = orc.OracleParams(filter_size=5, **VALS)
    wide = orc.OracleParams(filter_size=5, **dict(VALS, theta_gamma=1e9))
    np.testing.assert_allclose(orc.meanfield(U, I, p, 2, features=F), orc.meanfield(U, I, wide, 2),
                               rtol=0, atol=1e-12)


def test_feature_scale_pairs_with_theta_gamma():
    U, I, _, F, _ = _problem(3, 1, 3, 7, 8)
    p = orc.OracleParams(filter_size=5, **VALS)
    p3 = orc.OracleParams(filter_size=5, **dict(VALS, theta_gamma=3 * VALS["theta_gamma"]))
    np.testing.assert_allclose(orc.meanfield(U, I, p3, 2, features=3 * F),
                               orc.meanfield(U, I, p, 2, features=F), rtol=0, atol=1e-13)


def _loss(U, I, p, T, G, mu, F):
    return float(np.sum(G * orc.meanfield(U, I, p, T, compat=mu, features=F)))


CASES = [(4, 1, 3, 5, 6, 3, 2, False, True, 2), (5, 2, 2, 4, 5, 5, 2, True, False, 2),
         (6, 1, 3, 6, 5, 3, 1, False, False, 3), (7, 1, 2, 4, 4, 7, 3, True, True, 1)]


@pytest.mark.parametrize("seed,B,C,H,W,k,T,center,gen_mu,d", CASES)
def test_feature_gradient_matches_finite_differences(seed, B, C, H, W, k, T, center, gen_mu, d):
    U, I, G, F, _ = _problem(seed, B, C, H, W, d=max(d, 2))
    F = np.ascontiguousarray(F[:, :d])
    mu = np.random.default_rng(seed).normal(0.3, 0.5, (C, C)) if gen_mu else None
    p = orc.OracleParams(filter_size=k, include_center=center, **VALS)
    dU, dmu, dp, dF = orc.meanfield_backward(U, I, p, T, G, compat=mu, features=F)
    h = 1e-6
    fd = np.empty_like(F)
    for idx in np.ndindex(F.shape):
        def f(v):
            Fp = F.copy()
            Fp[idx] = v
            return _loss(U, I, p, T, G, mu, Fp)
        fd[idx] = (f(F[idx] + h) - f(F[idx] - h)) / (2 * h)
    assert np.abs(fd).max() > 1e-4
    np.testing.assert_allclose(dF, fd, rtol=0, atol=1e-7 * max(1.0, np.abs(fd).max()))
    # the other derivatives with features present
    fdU = np.empty_like(U)
    for idx in list(np.ndindex(U.shape))[::3]:
        def g(v):
            Up = U.copy()
            Up[idx] = v
            return _loss(Up, I, p, T, G, mu, F)
        fdU[idx] = (g(U[idx] + 1e-5) - g(U[idx] - 1e-5)) / 2e-5
        assert abs(fdU[idx] - dU[idx]) <= 1e-7 * max(1.0, np.abs(dU).max())
    for j, name in enumerate(orc.PARAM_NAMES):
        hh = 1e-6 * VALS[name]
        def q(v):
            return _loss(U, I, orc.OracleParams(filter_size=k, include_center=center,
                                                **dict(VALS, **{name: v})), T, G, mu, F)
        fdp = (q(VALS[name] + hh) - q(VALS[name] - hh)) / (2 * hh)
        assert abs(fdp - dp[j]) <= 2e-6 * abs(fdp) + 1e-9, (name, fdp, dp[j])


def test_position_features_give_the_same_other_derivatives():
    U, I, G, _, pos = _problem(8, 1, 3, 6, 7)
    mu = np.random.default_rng(8).normal(0.3, 0.5, (3, 3))
    p = orc.OracleParams(filter_size=5, **VALS)
    a = orc.meanfield_backward(U, I, p, 2, G, compat=mu)
    b = orc.meanfield_backward(U, I, p, 2, G, compat=mu, features=pos)
    for x, y in zip(a, b[:3]):
        np.testing.assert_allclose(x, y, rtol=1e-11, atol=1e-12)


# ---- blur together with learnable features: the features are pooled to the
# s x s cells like the colours, and the smoothness Gaussian takes the pooled
# features' distance between cells.

def _blur_problem(seed, B, C, H, W, d=2):
    U, I, G, F, pos = _problem(seed, B, C, H, W, d=max(d, 2))
    return U, I, G, np.ascontiguousarray(F[:, :d]), pos


@pytest.mark.parametrize("s,k,center", [(2, 3, False), (2, 5, True), (4, 3, False)])
def test_blur_position_features_reproduce_the_pooled_kernel(s, k, center):
    # block means of the pixel coordinates are the cell centres, whose
    # differences are s times the grid offsets: the pooled Eq. 4
    U, I, _, _, pos = _blur_problem(11, 2, 3, 4 * s, 3 * s)
    p = orc.OracleParams(filter_size=k, blur=s, include_center=center, **VALS)
    np.testing.assert_allclose(orc.meanfield(U, I, p, 3, features=pos), orc.meanfield(U, I, p, 3),
                               rtol=0, atol=1e-13)


def test_blur_constant_features_make_the_smoothness_term_flat():
    U, I, _, _, pos = _blur_problem(12, 1, 3, 8, 12)
    p = orc.OracleParams(filter_size=5, blur=2, **VALS)
    wide = orc.OracleParams(filter_size=5, blur=2, **dict(VALS, theta_gamma=1e9))
    np.testing.assert_allclose(orc.meanfield(U, I, p, 2, features=np.full_like(pos, -3.0)),
                               orc.meanfield(U, I, wide, 2), rtol=0, atol=1e-12)


def test_blur_features_see_only_cell_means():
    # moving feature mass inside a cell leaves the pooled features, and so Q,
    # unchanged
    U, I, _, F, _ = _blur_problem(13, 1, 3, 8, 8)
    p = orc.OracleParams(filter_size=3, blur=2, **VALS)
    F2 = F.copy()
    F2[:, :, 0::2, 0::2] += 0.7
    F2[:, :, 1::2, 1::2] -= 0.7
    np.testing.assert_allclose(orc.meanfield(U, I, p, 2, features=F2),
                               orc.meanfield(U, I, p, 2, features=F), rtol=0, atol=1e-13)
    F3 = F.copy()
    F3[:, :, 0, 0] += 0.7                 # one cell's mean moves: Q moves
    assert np.abs(orc.meanfield(U, I, p, 2, features=F3) -
                  orc.meanfield(U, I, p, 2, features=F)).max() > 1e-6


BLUR_CASES = [(21, 1, 3, 6, 8, 2, 3, 2, False, False, 2), (22, 2, 2, 8, 8, 4, 3, 2, True, True, 1),
              (23, 1, 2, 6, 4, 2, 5, 1, False, True, 3),
              (24, 1, 2, 16, 16, 8, 3, 2, False, True, 2)]   # s = 8: a 2 x 2 pooled grid


@pytest.mark.parametrize("seed,B,C,H,W,s,k,T,center,gen_mu,d", BLUR_CASES)
def test_blur_feature_gradient_matches_finite_differences(seed, B, C, H, W, s, k, T, center,
                                                          gen_mu, d):
    U, I, G, F, _ = _blur_problem(seed, B, C, H, W, d)
    mu = np.random.default_rng(seed).normal(0.3, 0.5, (C, C)) if gen_mu else None
    # the features are positions plus noise: with s = 8 the pooled features of
    # neighbouring cells lie 8 apart, so a smoothness width on that scale
    vals = dict(VALS, theta_gamma=9.0) if s == 8 else VALS
    p = orc.OracleParams(filter_size=k, blur=s, include_center=center, **vals)
    dU, dmu, dp, dF = orc.meanfield_backward(U, I, p, T, G, compat=mu, features=F)
    h = 1e-6
    fd = np.empty_like(F)
    for idx in np.ndindex(F.shape):
        def f(v):
            Fp = F.copy()
            Fp[idx] = v
            return _loss(U, I, p, T, G, mu, Fp)
        fd[idx] = (f(F[idx] + h) - f(F[idx] - h)) / (2 * h)
    assert np.abs(fd).max() > 1e-4
    np.testing.assert_allclose(dF, fd, rtol=0, atol=1e-7 * max(1.0, np.abs(fd).max()))
    # every pixel of a cell gets the same derivative (the pooling's transpose)
    for b in range(B):
        for c in range(d):
            cells = dF[b, c].reshape(H // s, s, W // s, s)
            assert np.ptp(cells, axis=(1, 3)).max() <= 1e-15 * max(1.0, np.abs(dF).max())
    for idx in list(np.ndindex(U.shape))[::5]:
        def g(v):
            Up = U.copy()
            Up[idx] = v
            return _loss(Up, I, p, T, G, mu, F)
        fdu = (g(U[idx] + 1e-5) - g(U[idx] - 1e-5)) / 2e-5
        assert abs(fdu - dU[idx]) <= 1e-7 * max(1.0, np.abs(dU).max())
    for j, name in enumerate(orc.PARAM_NAMES):
        hh = 1e-6 * vals[name]
        def q(v):
            return _loss(U, I, orc.OracleParams(filter_size=k, blur=s, include_center=center,
                                                **dict(vals, **{name: v})), T, G, mu, F)
        fdp = (q(vals[name] + hh) - q(vals[name] - hh)) / (2 * hh)
        assert abs(fdp - dp[j]) <= 2e-6 * abs(fdp) + 1e-9, (name, fdp, dp[j])


def test_blur_position_features_give_the_same_other_derivatives():
    U, I, G, _, pos = _blur_problem(24, 1, 3, 8, 6)
    mu = np.random.default_rng(24).normal(0.3, 0.5, (3, 3))
    p = orc.OracleParams(filter_size=3, blur=2, **VALS)
    a = orc.meanfield_backward(U, I, p, 2, G, compat=mu)
    b = orc.meanfield_backward(U, I, p, 2, G, compat=mu, features=pos)
    for x, y in zip(a, b[:3]):
        np.testing.assert_allclose(x, y, rtol=1e-11, atol=1e-12)
