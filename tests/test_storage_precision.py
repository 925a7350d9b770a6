"""Storing Q and U in bfloat16 between rounds fails the 1e-4 bar.

The candidate was to keep fp32 arithmetic but store the unary once and Q
after every round in bfloat16, halving the bytes of every per-iteration
launch on the batched (8 x 21 x 512^2) and street (1 x 19 x 1024 x 2048)
workloads.  The paper says nothing about storage precision; the bar is the
benchmark's: every probability within 1e-4 of the double oracle, argmax on
>= 99.99% of pixels.

The single-precision replica in fp32_replica.py (test code) evaluates the
same update on batch item 0 of the batched workload (full 512 x 512) and on
a 256 x 512 window of the street frame (the oracle and the replica run on it
padded by T r = 15 pixels; after T rounds only inputs within T r pixels
matter, so the window's values are the full frame's).  In float32 it stays
within 1.1e-6 of the oracle; with bfloat16 storage it leaves 1e-4 (by 2x to
5x, at a few pixels), so the storage format is not used.
"""

import numpy as np
import pytest

from fp32_replica import meanfield_f32, round_bf16
from paper_1805_04777_amd import synth

TOL = 1e-4


def test_bf16_rounding_matches_torch():
    import torch
    x = np.concatenate([np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -3.14159, 1e-20, 65504.0,
                                  2 ** -130], np.float32),
                        np.random.default_rng(3).normal(0, 100, 1000).astype(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(round_bf16(x), ref)
    assert round_bf16(np.float32([1 + 2 ** -8]))[0] == 1.0             # tie to even
    assert round_bf16(np.float32([1 + 3 * 2 ** -8]))[0] == 1 + 2 ** -6


def cases():
    b = synth.WORKLOADS["batched"]
    U, I, _ = synth.make_inputs(b.with_(B=1))
    yield "batched item 0", b, U, I, (slice(None),) * 4
    s = synth.WORKLOADS["street"]
    U, I, _ = synth.make_inputs(s)
    m = s.iters * (s.filter_size - 1) // 2
    y0, x0 = 384, 768
    win = (slice(None), slice(None), slice(y0 - m, y0 + 256 + m), slice(x0 - m, x0 + 512 + m))
    yield "street window", s, U[win].copy(), I[win].copy(), (slice(None), slice(None),
                                                            slice(m, -m), slice(m, -m))


@pytest.mark.slow
def test_bf16_storage_misses_the_bar_where_fp32_meets_it(oracle_mod):
    worst = {}
    for name, wl, U, I, inner in cases():
        par = dict(w_app=wl.w_app, theta_alpha=wl.theta_alpha, theta_beta=wl.theta_beta,
                   w_smooth=wl.w_smooth, theta_gamma=wl.theta_gamma)
        Qo = oracle_mod.meanfield(U, I, oracle_mod.OracleParams(filter_size=wl.filter_size, **par),
                                  wl.iters)[inner]
        Q32 = meanfield_f32(U, I, wl.filter_size, T=wl.iters, **par)[inner]
        Q16 = meanfield_f32(U, I, wl.filter_size, T=wl.iters, store=round_bf16, **par)[inner]
        e32 = np.abs(Q32 - Qo).max()
        e16 = np.abs(Q16 - Qo).max()
        assert e32 <= TOL / 10, (name, e32)
        assert (Q32.argmax(1) == Qo.argmax(1)).mean() >= 0.9999
        assert e16 > 1.5 * TOL, (name, e16)
        worst[name] = (e32, e16)
    print({k: (f"{a:.2e}", f"{b:.2e}") for k, (a, b) in worst.items()})
