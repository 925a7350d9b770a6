"""Single-precision conditioning of the i.i.d. 1 x 21 x 512 x 512 case.

On i.i.d. inputs (N(0, 2) logits for every class and pixel, uniform integer
colours), k = 7, T = 5 and the default Eq. 4 parameters, a few pixels cannot
be computed to 1e-4 in float32 by any implementation: they sit on decision
boundaries where the message (up to ~90 in a logit) carries float32 rounding
of ~5e-6, and five synchronous rounds amplify it.  The workload-shaped
scenes do not have such pixels (see the full-workload tests).

The evidence comes from the single-precision replica in fp32_replica.py (test
code, no GPU): two replicas that differ only in the order of the window taps
each leave the double oracle by more than 1e-4 at a few pixels (a different
few for each order).  Call S the pixels where either replica lands more than
2e-5 from the double result: single precision does not fix their value to
that accuracy.  S is 0.2% of the image.

The GPU test then applies the 1e-4 bar to every pixel outside S, bounds
the size of S and the GPU's worst error inside it, and keeps the argmax bar
(>= 99.99% of pixels) over the whole image.  (Measured on MI355X: 5.4e-5
outside S, 1.5e-4 inside, 4 pixels above 1e-4.)
"""

import numpy as np
import pytest

from fp32_replica import meanfield_f32

K, T = 7, 5
PAR = dict(w_app=10.0, theta_alpha=80.0, theta_beta=13.0, w_smooth=3.0, theta_gamma=3.0)
TOL = 1e-4
SENSITIVE = 2e-5      # a float32 replica lands farther from the double result


def iid_case():
    rng = np.random.default_rng(0)
    U = rng.normal(0.0, 2.0, (1, 21, 512, 512)).astype(np.float32)
    I = rng.integers(0, 256, (1, 3, 512, 512)).astype(np.float32)
    return U, I


@pytest.fixture(scope="module")
def analysis(oracle_mod):
    U, I = iid_case()
    Qo = oracle_mod.meanfield(U, I, oracle_mod.OracleParams(filter_size=K, **PAR), T)
    Qf = meanfield_f32(U, I, K, T=T, **PAR)
    Qr = meanfield_f32(U, I, K, T=T, reverse=True, **PAR)
    split = np.maximum(np.abs(Qf - Qo), np.abs(Qr - Qo)).max(axis=1)[0] > SENSITIVE
    return U, I, Qo, Qf, Qr, split


@pytest.mark.slow
def test_float32_alone_leaves_the_bar_on_iid_inputs(analysis):
    _, _, Qo, Qf, Qr, split = analysis
    ef = np.abs(Qf - Qo).max(axis=1)[0]
    er = np.abs(Qr - Qo).max(axis=1)[0]
    # single precision, whatever the order of the taps, misses 1e-4 somewhere
    assert max(ef.max(), er.max()) > TOL
    assert min(ef.max(), er.max()) > TOL / 2
    # at different pixels for the two orders: rounding, not a formula
    assert not np.any((ef > TOL) & (er > TOL))
    # the sensitive set is a small part of the image
    frac = split.mean()
    assert 5e-4 <= frac <= 4e-3, frac
    # the argmax bar still holds for both
    assert (Qf.argmax(1) == Qo.argmax(1)).mean() >= 0.9999
    assert (Qr.argmax(1) == Qo.argmax(1)).mean() >= 0.9999


@pytest.mark.gpu
def test_gpu_meets_the_bar_where_float32_can(analysis):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_1805_04777_amd import convcrf as cc
    U, I, Qo, Qf, Qr, split = analysis
    with cc.ConvCRF(0) as crf:
        p = cc.Params(filter_size=K, **PAR)
        Q = crf.meanfield(torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda(), p, T)
        crf.synchronize()
        Qg = Q.cpu().numpy().astype(np.float64)
    err = np.abs(Qg - Qo).max(axis=1)[0]
    assert err[~split].max() <= TOL, f"outside the sensitive set: {err[~split].max():.3e}"
    assert split.mean() <= 4e-3
    inside = err[split].max()
    assert inside <= 5e-4, f"inside the sensitive set: {inside:.3e}"
    assert (Qg.argmax(1) == Qo.argmax(1)).mean() >= 0.9999
    assert np.abs(Qg.sum(1) - 1.0).max() <= 1e-5
    print(f"i.i.d. 512^2: outside the sensitive set max |dQ| {err[~split].max():.3e}, "
          f"inside {inside:.3e} over {int(split.sum())} pixels, {int((err > TOL).sum())} above 1e-4")
