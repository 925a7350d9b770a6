"""Locality of the mean-field iteration, checked on the oracle (CPU).

After T iterations with window radius r, a pixel's Q depends only on the
inputs within T*r pixels (Alg. 1 applied T times to the k x k window of
Sec. 4).  The GPU parity tests rely on this to compare the largest workloads
on crops: the oracle run on a crop padded by T*r gives exactly the
full-image values inside it.
"""
import numpy as np

from oracle import OracleParams


def run(oracle_mod, U, I, T):
    p = OracleParams(filter_size=5, w_app=0.9, theta_alpha=6.0, theta_beta=30.0, w_smooth=0.5,
                     theta_gamma=3.0)
    return oracle_mod.meanfield(U, I, p, T)


def test_crop_padded_by_t_times_r_is_exact(oracle_mod):
    rng = np.random.default_rng(3)
    U = rng.normal(0.0, 2.0, size=(1, 4, 40, 44))
    I = rng.integers(0, 256, size=(1, 3, 40, 44)).astype(np.float64)
    T, m = 3, 3 * 2
    full = run(oracle_mod, U, I, T)
    y0, x0, s = 15, 17, 8
    Qo = run(oracle_mod, U[:, :, y0 - m:y0 + s + m, x0 - m:x0 + s + m],
             I[:, :, y0 - m:y0 + s + m, x0 - m:x0 + s + m], T)
    np.testing.assert_array_equal(Qo[:, :, m:m + s, m:m + s], full[:, :, y0:y0 + s, x0:x0 + s])
    # one pixel less of margin is not enough
    Qs = run(oracle_mod, U[:, :, y0 - m + 1:y0 + s + m, x0 - m:x0 + s + m],
             I[:, :, y0 - m + 1:y0 + s + m, x0 - m:x0 + s + m], T)
    assert np.abs(Qs[:, :, m - 1:m - 1 + s, m:m + s] - full[:, :, y0:y0 + s, x0:x0 + s]).max() > 0


def test_crop_at_image_corner_is_exact(oracle_mod):
    # where the crop is clipped by the image border no margin is needed
    rng = np.random.default_rng(4)
    U = rng.normal(0.0, 2.0, size=(1, 3, 30, 30))
    I = rng.integers(0, 256, size=(1, 3, 30, 30)).astype(np.float64)
    T, m, s = 4, 8, 6
    full = run(oracle_mod, U, I, T)
    Qo = run(oracle_mod, U[:, :, :s + m, :s + m], I[:, :, :s + m, :s + m], T)
    np.testing.assert_array_equal(Qo[:, :, :s, :s], full[:, :, :s, :s])
