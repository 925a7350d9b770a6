"""GPU parity of the reverse mode (convcrf_meanfield_backward) against the
oracle's derivative, which finite differences of the forward oracle pin
(test_oracle_backward.py).

Bar: the forward bar is 1e-4 absolute on probabilities, whose scale is 1.
Gradients have no natural unit, so the same bar is taken relative to the
tensor's own scale: max |GPU - oracle| <= 1e-4 * max |oracle| for dL/dU and
dL/dmu.  Each Eq. 4 parameter derivative is one sum over every pixel pair,
compared with |GPU - oracle| <= 1e-3 * |oracle| on cases where none of them
cancels to near zero (each case asserts that), and exactly where it is zero
by construction (k = 1: no offsets, so the three scale derivatives vanish).

The reverse mode can be no more accurate than the float32 forward it
differentiates: the logits Z = U - mu M are rounded at the scale of the
message M, so with large messages (k = 15 and the default weights: |M| up to
about 170) the forward's own relative error in Q reaches about 2e-4 and the
derivative inherits it.  The main cases keep |M| below about 100; the
large-window case checks that the backward adds no error beyond the
forward's.
"""
import dataclasses

import numpy as np
import pytest

from oracle import OracleParams
from paper_1805_04777_amd import synth

pytestmark = pytest.mark.gpu

TOL_REL = 1e-4
TOL_PARAM = 1e-3


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch


@pytest.fixture(scope="module")
def crf(torch_cuda):
    from paper_1805_04777_amd import convcrf as cc
    ctx = cc.ConvCRF(0)
    yield ctx
    ctx.close()


def make_case(seed, B, C, H, W, levels=4):
    """Unaries, a piecewise-constant noisy image (so that colour distances in
    a window take small and large values), and dL/dQ."""
    rng = np.random.default_rng(seed)
    U = rng.normal(0.0, 1.5, (B, C, H, W)).astype(np.float32)
    blocks = rng.integers(0, levels, (B, 3, (H + 7) // 8, (W + 7) // 8)) * (200.0 / levels)
    I = np.repeat(np.repeat(blocks, 8, axis=2), 8, axis=3)[:, :, :H, :W]
    I = np.clip(np.rint(I + rng.normal(0.0, 8.0, I.shape)), 0, 255).astype(np.float32)
    G = rng.normal(0.0, 1.0, (B, C, H, W)).astype(np.float32)
    return U, I, G


def run_gpu(torch, crf, U, I, G, p, T, want=True):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    dU, dmu, dk = crf.meanfield_backward(t(U), t(I), p, T, t(G), grad_compat=want,
                                         grad_kernel=want)
    torch.cuda.synchronize()
    f = lambda x: None if x is None else x.cpu().numpy().astype(np.float64)
    return f(dU), f(dmu), f(dk)


def run_oracle(oracle_mod, U, I, G, p, T):
    op = OracleParams(filter_size=p.filter_size, include_center=bool(p.include_center),
                      w_app=p.w_app, theta_alpha=p.theta_alpha, theta_beta=p.theta_beta,
                      w_smooth=p.w_smooth, theta_gamma=p.theta_gamma)
    return oracle_mod.meanfield_backward(U, I, op, T, G, compat=p.compat)


def check(got, ref, what, T):
    dU, dmu, dk = got
    rU, rmu, rk = ref
    assert np.all(np.isfinite(dU)) and np.all(np.isfinite(dmu)) and np.all(np.isfinite(dk))
    eU = np.abs(dU - rU).max() / max(np.abs(rU).max(), 1e-30)
    assert eU <= TOL_REL, f"{what}: dU rel err {eU:.3e}"
    if T == 0:
        assert np.all(dmu == 0) and np.all(dk == 0), what
        return eU, 0.0, 0.0
    emu = np.abs(dmu - rmu).max() / max(np.abs(rmu).max(), 1e-30)
    assert emu <= TOL_REL, f"{what}: dmu rel err {emu:.3e}"
    zero = rk == 0.0
    assert np.all(dk[zero] == 0.0), f"{what}: structural zeros {dk[zero]}"
    nz = ~zero
    assert np.all(np.abs(rk[nz]) > 1e-6 * np.abs(rk).max()), f"{what}: a parameter derivative cancels"
    ek = np.abs(dk[nz] - rk[nz]) / np.abs(rk[nz])
    assert np.all(ek <= TOL_PARAM), f"{what}: kernel-parameter rel err {ek}"
    print(f"{what}: rel err dU {eU:.2e} dmu {emu:.2e} dk {ek.max():.2e}", flush=True)
    return eU, emu, ek.max()


def params(k, center=False, compat=None, **kw):
    from paper_1805_04777_amd import convcrf as cc
    base = dict(filter_size=k, include_center=center, w_app=10.0, theta_alpha=80.0,
                theta_beta=13.0, w_smooth=3.0, theta_gamma=3.0, compat=compat)
    base.update(kw)
    return cc.Params(**base)


CASES = [
    # (seed, B, C, H, W, k, T, include_center, general compat)
    (1, 1, 3, 20, 37, 3, 2, False, False),
    (2, 2, 5, 33, 40, 5, 3, True, True),
    (3, 1, 21, 40, 70, 7, 2, False, False),     # fused forward on iter_kernel
    (4, 1, 21, 48, 64, 7, 3, False, True),      # streamed forward, general compat
    (5, 1, 19, 24, 36, 9, 1, False, True),
    (6, 1, 4, 17, 23, 15, 2, True, False),     # weights 2 and 1 (|M| < 40)
    (7, 1, 2, 5, 6, 1, 3, True, True),          # k = 1: the centre tap only
    (8, 2, 21, 16, 24, 11, 2, False, False),
    (9, 1, 24, 19, 29, 13, 1, False, True),
    (10, 1, 6, 9, 11, 5, 0, False, True),       # T = 0: the softmax adjoint only
]


@pytest.mark.parametrize("seed,B,C,H,W,k,T,center,gen_mu", CASES)
def test_backward_matches_oracle(torch_cuda, crf, oracle_mod, seed, B, C, H, W, k, T, center,
                                 gen_mu):
    U, I, G = make_case(seed, B, C, H, W)
    mu = None
    if gen_mu:
        mu = np.random.default_rng(seed + 100).normal(0.3, 0.5, (C, C)).astype(np.float32)
    p = params(k, center, mu, **({"w_app": 2.0, "w_smooth": 1.0} if k == 15 else {}))
    print(f"case seed={seed} B={B} C={C} {H}x{W} k={k} T={T}", flush=True)
    got = run_gpu(torch_cuda, crf, U, I, G, p, T)
    ref = run_oracle(oracle_mod, U, I, G, p, T)
    check(got, ref, f"seed {seed}", T)


def test_pascal_backward_full(torch_cuda, crf, oracle_mod):
    """The headline workload, 1 x 21 x 512 x 512, k = 7, T = 5, in full."""
    wl = synth.WORKLOADS["pascal"]
    U, I, _ = synth.make_inputs(wl)
    G = np.random.default_rng(77).normal(0.0, 1.0, U.shape).astype(np.float32)
    p = params(wl.filter_size, w_app=wl.w_app, theta_alpha=wl.theta_alpha,
               theta_beta=wl.theta_beta, w_smooth=wl.w_smooth, theta_gamma=wl.theta_gamma)
    print("case pascal 1x21x512x512 k=7 T=5", flush=True)
    got = run_gpu(torch_cuda, crf, U, I, G, p, wl.iters)
    ref = run_oracle(oracle_mod, U, I, G, p, wl.iters)
    check(got, ref, "pascal", wl.iters)


def test_large_window_adds_no_error_beyond_the_forward(torch_cuda, crf, oracle_mod):
    """k = 15 with the default weights: the derivative's relative error stays
    within twice the forward's own relative error of Q (on Q > 1e-3) on the
    same inputs, and within 1e-3."""
    U, I, G = make_case(6, 1, 4, 17, 23)
    p = params(15, center=True)
    op = OracleParams(filter_size=15, include_center=True)
    Qo = oracle_mod.meanfield(U, I, op, 2)
    Qg = crf.meanfield(torch_cuda.from_numpy(U).cuda(), torch_cuda.from_numpy(I).cuda(), p,
                       2).cpu().numpy()
    fwd = (np.abs(Qg - Qo) / Qo)[Qo > 1e-3].max()
    got = run_gpu(torch_cuda, crf, U, I, G, p, 2)
    ref = run_oracle(oracle_mod, U, I, G, p, 2)
    for g, r in zip(got[:2], ref[:2]):
        e = np.abs(g - r).max() / np.abs(r).max()
        print(f"k=15: forward rel err {fwd:.2e}, backward rel err {e:.2e}", flush=True)
        assert e <= min(1e-3, max(TOL_REL, 2.0 * fwd))


BLUR_CASES = [
    # (seed, B, C, H, W, k, T, s, general compat)
    (31, 1, 3, 16, 24, 3, 2, 2, True),
    (32, 2, 21, 32, 48, 5, 2, 4, False),
    (33, 1, 19, 40, 64, 7, 3, 8, True),
    (34, 1, 5, 24, 36, 11, 1, 4, False),
    # 4 x 4 with a general compatibility: the fused recompute with mu, the
    # -dL/dZ plane and its upsampling transpose, a 9 x 11-cell grid
    (35, 1, 8, 36, 44, 7, 2, 4, True),
]


@pytest.mark.parametrize("seed,B,C,H,W,k,T,s,gen_mu", BLUR_CASES)
def test_blur_backward_matches_oracle(torch_cuda, crf, oracle_mod, seed, B, C, H, W, k, T, s,
                                      gen_mu):
    """The pooled message (Sec. 4.2 blur): the transposes of the upsampling
    and the pooling around the pooled adjoint message."""
    U, I, G = make_case(seed, B, C, H, W)
    mu = None
    if gen_mu:
        mu = np.random.default_rng(seed + 100).normal(0.3, 0.5, (C, C)).astype(np.float32)
    p = params(k, False, mu, blur=s)
    print(f"case blur seed={seed} B={B} C={C} {H}x{W} k={k} T={T} s={s}", flush=True)
    got = run_gpu(torch_cuda, crf, U, I, G, p, T)
    op = OracleParams(filter_size=k, blur=s, w_app=p.w_app, theta_alpha=p.theta_alpha,
                      theta_beta=p.theta_beta, w_smooth=p.w_smooth, theta_gamma=p.theta_gamma)
    ref = oracle_mod.meanfield_backward(U, I, op, T, G, compat=mu)
    check(got, ref, f"blur seed {seed}", T)


def test_blur_workload_backward_full(torch_cuda, crf, oracle_mod):
    """The blur workload, 1 x 21 x 512 x 512, k = 11 on the 4 x 4 pooled
    grid, T = 5, in full."""
    wl = synth.WORKLOADS["blur"]
    U, I, _ = synth.make_inputs(wl)
    G = np.random.default_rng(78).normal(0.0, 1.0, U.shape).astype(np.float32)
    p = params(wl.filter_size, blur=wl.blur, w_app=wl.w_app, theta_alpha=wl.theta_alpha,
               theta_beta=wl.theta_beta, w_smooth=wl.w_smooth, theta_gamma=wl.theta_gamma)
    print("case blur 1x21x512x512 k=11 s=4 T=5", flush=True)
    got = run_gpu(torch_cuda, crf, U, I, G, p, wl.iters)
    op = OracleParams(filter_size=wl.filter_size, blur=wl.blur, w_app=wl.w_app,
                      theta_alpha=wl.theta_alpha, theta_beta=wl.theta_beta,
                      w_smooth=wl.w_smooth, theta_gamma=wl.theta_gamma)
    ref = oracle_mod.meanfield_backward(U, I, op, wl.iters, G)
    check(got, ref, "blur workload", wl.iters)


def test_street_backward_full(torch_cuda, crf, oracle_mod):
    """The street workload, 1 x 19 x 1024 x 2048, k = 7, T = 5, in full
    (19 classes: class groups of 7, 7 and 5)."""
    wl = synth.WORKLOADS["street"]
    U, I, _ = synth.make_inputs(wl)
    G = np.random.default_rng(79).normal(0.0, 1.0, U.shape).astype(np.float32)
    p = params(wl.filter_size, w_app=wl.w_app, theta_alpha=wl.theta_alpha,
               theta_beta=wl.theta_beta, w_smooth=wl.w_smooth, theta_gamma=wl.theta_gamma)
    print("case street 1x19x1024x2048 k=7 T=5", flush=True)
    got = run_gpu(torch_cuda, crf, U, I, G, p, wl.iters)
    ref = run_oracle(oracle_mod, U, I, G, p, wl.iters)
    check(got, ref, "street", wl.iters)


def test_outputs_are_independent_of_what_is_requested(torch_cuda, crf):
    U, I, G = make_case(21, 1, 21, 48, 64)
    p = params(7)
    a = run_gpu(torch_cuda, crf, U, I, G, p, 3, want=True)
    b = run_gpu(torch_cuda, crf, U, I, G, p, 3, want=False)
    c = run_gpu(torch_cuda, crf, U, I, G, p, 3, want=True)
    np.testing.assert_array_equal(a[0], b[0])
    for x, y in zip(a, c):          # deterministic: same bits on a second call
        np.testing.assert_array_equal(x, y)


def test_empty_batch_gives_zero_sums(torch_cuda, crf):
    torch = torch_cuda
    p = params(5)
    z = torch.zeros((0, 4, 8, 8), device="cuda")
    dU, dmu, dk = crf.meanfield_backward(z, torch.zeros((0, 3, 8, 8), device="cuda"), p, 2, z,
                                         grad_compat=True, grad_kernel=True)
    torch.cuda.synchronize()
    assert dU.shape == (0, 4, 8, 8)
    assert torch.all(dmu == 0) and torch.all(dk == 0)


def test_backward_errors(torch_cuda, crf):
    from paper_1805_04777_amd import convcrf as cc
    torch = torch_cuda
    U, I, G = make_case(22, 1, 4, 16, 16)
    t = lambda a: torch.from_numpy(a).cuda()
    with pytest.raises(cc.ConvCRFError) as e:
        crf.meanfield_backward(t(U), t(I), params(5, blur=3), 2, t(G))   # s not 1, 2, 4, 8
    assert e.value.status == cc.E_INVALID_ARG
    Ut, Gt = t(U), t(G)
    with pytest.raises(cc.ConvCRFError) as e:
        crf.meanfield_backward(Ut, t(I), params(5), 2, Gt, out=Gt)   # overlaps grad_q
    assert e.value.status == cc.E_INVALID_ARG
    with pytest.raises(cc.ConvCRFError) as e:
        crf.meanfield_backward(Ut, t(I), params(4), 2, Gt)            # even window
    assert e.value.status == cc.E_INVALID_ARG


@pytest.mark.parametrize("blur,k,C,T", [(1, 7, 21, 3), (4, 5, 21, 2), (1, 5, 2, 2)])
def test_potts_compat_derivative_matches_the_explicit_matrix(torch_cuda, crf, oracle_mod,
                                                             blur, k, C, T):
    """With Potts compatibility (no matrix given, C > 1) the compatibility
    derivative takes -dL/dZ from dL/dM; with the same matrix 1 - I given
    explicitly it reads the stored -dL/dZ.  Both meet the bar against the
    oracle and agree with each other.  C = 2 is the smallest case of the
    derivation (sum dM = -sum dZ).  Weights 3 and 1 keep |M| small: with a
    matrix given, the forward forms U - mu M, which rounds at the scale of M
    (the Potts form softmax(U + M) does not cancel)."""
    U, I, G = make_case(41 + blur + C, 1, C, 32, 48)
    potts = (1.0 - np.eye(C)).astype(np.float32)
    w = dict(w_app=3.0, w_smooth=1.0)
    a = run_gpu(torch_cuda, crf, U, I, G, params(k, False, None, blur=blur, **w), T)
    b = run_gpu(torch_cuda, crf, U, I, G, params(k, False, potts, blur=blur, **w), T)
    op = OracleParams(filter_size=k, blur=blur, **w)
    ref = oracle_mod.meanfield_backward(U, I, op, T, G, compat=None)
    check(a, ref, f"Potts, blur {blur}", T)
    check(b, ref, f"explicit 1 - I, blur {blur}", T)
    for x, y, name in zip(a, b, ("dU", "dmu", "dk")):
        e = np.abs(x - y).max() / max(np.abs(y).max(), 1e-30)
        assert e <= TOL_REL, f"{name}: Potts and explicit 1 - I differ by {e:.2e}"
