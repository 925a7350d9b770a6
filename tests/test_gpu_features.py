"""GPU parity of the learnable smoothness features (the "+T" variant of
Sec. 4.2) against the oracle, forward and derivative.

Forward bar: the inference bar (1e-4 absolute per probability, argmax
agreement >= 99.99%, rows summing to 1 within 1e-5).  Derivative bar: the
reverse-mode bar (1e-4 of each tensor's largest magnitude; 1e-3 relative
per kernel parameter), with dL/dF held to the same 1e-4 of its largest
magnitude.
"""
import numpy as np
import pytest

from oracle import OracleParams

pytestmark = pytest.mark.gpu


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


def make_case(seed, B, C, H, W, D):
    rng = np.random.default_rng(seed)
    U = rng.normal(0.0, 1.5, (B, C, H, W)).astype(np.float32)
    blocks = rng.integers(0, 4, (B, 3, (H + 7) // 8, (W + 7) // 8)) * 50.0
    I = np.repeat(np.repeat(blocks, 8, axis=2), 8, axis=3)[:, :, :H, :W]
    I = np.clip(np.rint(I + rng.normal(0.0, 8.0, I.shape)), 0, 255).astype(np.float32)
    yy, xx = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64),
                         indexing="ij")
    base = [yy, xx, np.zeros((H, W)), np.zeros((H, W))][:D]
    F = (np.stack(base)[None].repeat(B, axis=0) + rng.normal(0.0, 0.5, (B, D, H, W)))
    G = rng.normal(0.0, 1.0, (B, C, H, W)).astype(np.float32)
    return U, I, F.astype(np.float32), G


def params(torch, k, F, center=False, compat=None, **kw):
    from paper_1805_04777_amd import convcrf as cc
    base = dict(filter_size=k, include_center=center, w_app=10.0, theta_alpha=80.0,
                theta_beta=13.0, w_smooth=3.0, theta_gamma=3.0, compat=compat,
                features=None if F is None else torch.from_numpy(F).cuda())
    base.update(kw)
    return cc.Params(**base)


def oparams(p):
    return OracleParams(filter_size=p.filter_size, blur=p.blur, include_center=bool(p.include_center),
                        w_app=p.w_app, theta_alpha=p.theta_alpha, theta_beta=p.theta_beta,
                        w_smooth=p.w_smooth, theta_gamma=p.theta_gamma)


CASES = [
    # (seed, B, C, H, W, k, T, D, include_center, general compat)
    (1, 1, 3, 20, 37, 3, 2, 2, False, False),
    (2, 2, 5, 33, 40, 5, 3, 2, True, True),
    (3, 1, 21, 40, 64, 7, 2, 2, False, False),
    (4, 1, 19, 24, 36, 9, 2, 3, False, True),
    (5, 1, 4, 17, 23, 13, 1, 1, True, False),
    (6, 1, 24, 16, 24, 7, 1, 4, False, False),
    # the ring kernel's feature mode (C = 19 or 21, W a multiple of 4,
    # k = 3..7): every feature count, ragged rows and columns, B = 2
    (11, 2, 19, 21, 68, 5, 3, 1, True, True),
    (12, 1, 19, 30, 44, 3, 2, 3, False, False),
    (13, 1, 21, 19, 36, 7, 3, 4, True, False),
    (14, 1, 19, 13, 72, 7, 2, 2, True, True),
]

# blur together with the features (Sec. 4.2): the features pooled to the cells
# like the colours, the pooled message taking their distance.  Weights 4 and
# 1.5 and a compatibility of 0.3 N(0.3, 0.5): with the default 10 and 3 and a
# compatibility of N(0.3, 0.5), the pooled messages drive Q to one-hot and
# every derivative below 1e-10, where a relative comparison measures nothing
# (the oracle's dL/dU of each case is checked to exceed 1e-2, its dL/dF
# 1e-4).  Blur 8: theta_gamma 12, as the pooled features of neighbouring cells
# lie 8 apart.
BLUR_W = dict(w_app=4.0, w_smooth=1.5)
BLUR_MU_SCALE = 0.3
BLUR_CASES = [
    # (seed, B, C, H, W, k, T, D, include_center, general compat, blur, theta_gamma)
    (31, 1, 21, 64, 96, 11, 3, 2, False, False, 4, 3.0),
    (32, 2, 5, 32, 48, 5, 2, 1, True, True, 2, 3.0),
    (33, 1, 19, 64, 64, 7, 2, 3, False, False, 8, 12.0),
    (34, 1, 3, 40, 24, 3, 3, 4, True, False, 4, 3.0),
]


# forward only: the fused 4 x 4 round with features on a ragged grid (Hp = 9,
# Wp = 13, so the word-by-word staging), 13 classes (the general class width),
# two window rows per wavefront (k = 9 with features) and a general compatibility
BLUR_FWD_EXTRA = [(36, 2, 13, 36, 52, 9, 2, 3, False, True, 4, 5.0),
                  # one wavefront per window row with features: 19 classes at
                  # k = 9 with four feature planes (the most registers), a
                  # general compatibility, a 10 x 12-cell grid; 6 classes (the
                  # eight-class width) at k = 11 with one plane, B = 2 and the centre
                  (37, 1, 19, 40, 48, 9, 2, 4, False, True, 4, 3.0),
                  (38, 2, 6, 32, 44, 11, 3, 1, True, False, 4, 3.0)]


@pytest.mark.parametrize("seed,B,C,H,W,k,T,D,center,gen_mu,s,tg", BLUR_CASES + BLUR_FWD_EXTRA)
def test_forward_with_features_and_blur(torch_cuda, crf, oracle_mod, seed, B, C, H, W, k, T, D,
                                        center, gen_mu, s, tg):
    torch = torch_cuda
    U, I, F, _ = make_case(seed, B, C, H, W, D)
    mu = (BLUR_MU_SCALE * np.random.default_rng(seed + 100).normal(0.3, 0.5, (C, C))).astype(
        np.float32) if gen_mu else None
    p = params(torch, k, F, center, mu, blur=s, theta_gamma=tg, **BLUR_W)
    Q = crf.meanfield(torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda(), p, T)
    torch.cuda.synchronize()
    Qg = Q.cpu().numpy().astype(np.float64)
    Qo = oracle_mod.meanfield(U, I, oparams(p), T, compat=mu, features=F)
    err = np.abs(Qg - Qo).max()
    print(f"case {seed} (blur {s}): forward max|dQ| {err:.2e}", flush=True)
    assert err <= 1e-4
    assert (Qg.argmax(1) == Qo.argmax(1)).mean() >= 0.9999
    assert np.abs(Qg.sum(1) - 1.0).max() <= 1e-5


@pytest.mark.parametrize("seed,B,C,H,W,k,T,D,center,gen_mu,s,tg", BLUR_CASES)
def test_backward_with_features_and_blur(torch_cuda, crf, oracle_mod, seed, B, C, H, W, k, T, D,
                                         center, gen_mu, s, tg):
    torch = torch_cuda
    U, I, F, G = make_case(seed, B, C, H, W, D)
    mu = (BLUR_MU_SCALE * np.random.default_rng(seed + 100).normal(0.3, 0.5, (C, C))).astype(
        np.float32) if gen_mu else None
    p = params(torch, k, F, center, mu, blur=s, theta_gamma=tg, **BLUR_W)
    t = lambda x: torch.from_numpy(x).cuda()
    dU, dmu, dk, dF = crf.meanfield_backward(t(U), t(I), p, T, t(G), grad_compat=True,
                                             grad_kernel=True)
    torch.cuda.synchronize()
    got = [x.cpu().numpy().astype(np.float64) for x in (dU, dmu, dk, dF)]
    ref = oracle_mod.meanfield_backward(U, I, oparams(p), T, G, compat=mu, features=F)
    assert np.abs(ref[0]).max() > 1e-2 and np.abs(ref[3]).max() > 1e-4   # not saturated
    errs = []
    for g, r, name in zip((got[0], got[1], got[3]), (ref[0], ref[1], ref[3]), ("dU", "dmu", "dF")):
        e = np.abs(g - r).max() / np.abs(r).max()
        errs.append(e)
        assert e <= 1e-4, f"{name}: rel err {e:.2e}"
    ek = np.abs(got[2] - ref[2]) / np.abs(ref[2])
    assert np.all(ek <= 1e-3), ek
    # every pixel of a cell carries the same derivative
    cells = got[3].reshape(B, D, H // s, s, W // s, s)
    assert np.ptp(cells, axis=(3, 5)).max() <= 1e-6 * np.abs(got[3]).max()
    print(f"case {seed} (blur {s}): backward rel err dU {errs[0]:.1e} dmu {errs[1]:.1e} "
          f"dF {errs[2]:.1e} dk {ek.max():.1e}", flush=True)


def test_position_features_with_blur_match_the_blur_path(torch_cuda, crf, oracle_mod):
    """Position features pool to the cell centres: with blur 4 the feature
    path (three kernels per round) and the fused blur launch meet the bar
    against the oracle of the pooled Eq. 4, and each other."""
    torch = torch_cuda
    U, I, _, _ = make_case(35, 1, 21, 64, 64, 2)
    yy, xx = np.meshgrid(np.arange(64, dtype=np.float32), np.arange(64, dtype=np.float32),
                         indexing="ij")
    pos = np.stack([yy, xx])[None].copy()
    Ut, It = torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda()
    a = crf.meanfield(Ut, It, params(torch, 7, pos, blur=4), 3).cpu().numpy().astype(np.float64)
    b = crf.meanfield(Ut, It, params(torch, 7, None, blur=4), 3).cpu().numpy().astype(np.float64)
    o = oracle_mod.meanfield(U, I, OracleParams(filter_size=7, blur=4), 3)
    assert np.abs(a - o).max() <= 1e-4 and np.abs(b - o).max() <= 1e-4
    assert np.abs(a - b).max() <= 1e-4


@pytest.mark.parametrize("seed,B,C,H,W,k,T,D,center,gen_mu", CASES)
def test_forward_with_features(torch_cuda, crf, oracle_mod, seed, B, C, H, W, k, T, D, center,
                               gen_mu):
    torch = torch_cuda
    U, I, F, _ = make_case(seed, B, C, H, W, D)
    mu = np.random.default_rng(seed + 100).normal(0.3, 0.5, (C, C)).astype(np.float32) \
        if gen_mu else None
    p = params(torch, k, F, center, mu)
    Q = crf.meanfield(torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda(), p, T)
    torch.cuda.synchronize()
    Qg = Q.cpu().numpy().astype(np.float64)
    Qo = oracle_mod.meanfield(U, I, oparams(p), T, compat=mu, features=F)
    err = np.abs(Qg - Qo).max()
    print(f"case {seed}: forward max|dQ| {err:.2e}", flush=True)
    assert err <= 1e-4
    assert (Qg.argmax(1) == Qo.argmax(1)).mean() >= 0.9999
    assert np.abs(Qg.sum(1) - 1.0).max() <= 1e-5


def test_position_features_match_the_fused_path(torch_cuda, crf, oracle_mod):
    """Features equal to the pixel positions reproduce Eq. 4: the feature
    kernel and the fused kernel both meet the inference bar against the
    oracle of Eq. 4, and each other."""
    torch = torch_cuda
    U, I, _, _ = make_case(7, 1, 21, 48, 64, 2)
    yy, xx = np.meshgrid(np.arange(48, dtype=np.float32), np.arange(64, dtype=np.float32),
                         indexing="ij")
    pos = np.stack([yy, xx])[None].copy()
    Ut, It = torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda()
    a = crf.meanfield(Ut, It, params(torch, 7, pos), 2).cpu().numpy().astype(np.float64)
    b = crf.meanfield(Ut, It, params(torch, 7, None), 2).cpu().numpy().astype(np.float64)
    o = oracle_mod.meanfield(U, I, OracleParams(filter_size=7), 2)
    assert np.abs(a - o).max() <= 1e-4 and np.abs(b - o).max() <= 1e-4
    assert np.abs(a - b).max() <= 1e-4


@pytest.mark.parametrize("seed,B,C,H,W,k,T,D,center,gen_mu", CASES)
def test_backward_with_features(torch_cuda, crf, oracle_mod, seed, B, C, H, W, k, T, D, center,
                                gen_mu):
    torch = torch_cuda
    U, I, F, G = make_case(seed, B, C, H, W, D)
    mu = np.random.default_rng(seed + 100).normal(0.3, 0.5, (C, C)).astype(np.float32) \
        if gen_mu else None
    p = params(torch, k, F, center, mu)
    t = lambda x: torch.from_numpy(x).cuda()
    dU, dmu, dk, dF = crf.meanfield_backward(t(U), t(I), p, T, t(G), grad_compat=True,
                                             grad_kernel=True)
    torch.cuda.synchronize()
    got = [x.cpu().numpy().astype(np.float64) for x in (dU, dmu, dk, dF)]
    ref = oracle_mod.meanfield_backward(U, I, oparams(p), T, G, compat=mu, features=F)
    errs = []
    for g, r, name in zip((got[0], got[1], got[3]), (ref[0], ref[1], ref[3]), ("dU", "dmu", "dF")):
        e = np.abs(g - r).max() / np.abs(r).max()
        errs.append(e)
        assert e <= 1e-4, f"{name}: rel err {e:.2e}"
    ek = np.abs(got[2] - ref[2]) / np.abs(ref[2])
    assert np.all(ek <= 1e-3), ek
    print(f"case {seed}: backward rel err dU {errs[0]:.1e} dmu {errs[1]:.1e} dF {errs[2]:.1e} "
          f"dk {ek.max():.1e}", flush=True)


def test_zero_iterations_give_zero_feature_derivative(torch_cuda, crf):
    torch = torch_cuda
    U, I, F, G = make_case(8, 1, 4, 12, 16, 2)
    p = params(torch, 5, F)
    t = lambda x: torch.from_numpy(x).cuda()
    out = crf.meanfield_backward(t(U), t(I), p, 0, t(G))
    torch.cuda.synchronize()
    assert torch.all(out[3] == 0)


def test_feature_errors(torch_cuda, crf):
    from paper_1805_04777_amd import convcrf as cc
    torch = torch_cuda
    U, I, F, _ = make_case(9, 1, 4, 16, 16, 2)
    Ut, It = torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda()
    F5 = np.zeros((1, 5, 16, 16), np.float32)
    with pytest.raises(cc.ConvCRFError) as e:
        crf.meanfield(Ut, It, params(torch, 5, F5), 2)
    assert e.value.status == cc.E_INVALID_ARG


def test_unaligned_output_takes_the_scalar_staging(torch_cuda, crf):
    """An output 4 bytes off a 16-byte boundary stages Q by scalars; the
    arithmetic is the same, so the result is identical to the vector path
    (20 classes: the ring kernel does not take these shapes)."""
    torch = torch_cuda
    U, I, F, _ = make_case(10, 1, 20, 32, 48, 2)
    Ut, It = torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda()
    p = params(torch, 7, F)
    a = crf.meanfield(Ut, It, p, 3)
    buf = torch.empty(U.size + 1, device="cuda")
    out = buf[1:].view(U.shape)
    assert out.data_ptr() % 16 != 0
    b = crf.meanfield(Ut, It, p, 3, out=out)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_ring_and_feature_kernel_agree(torch_cuda, crf, oracle_mod):
    """21 classes: an aligned output runs the ring kernel's feature mode, an
    output 4 bytes off an 8-byte boundary the feature kernel; both meet the
    inference bar against the oracle and each other (their rounding differs,
    so they are not bitwise equal)."""
    torch = torch_cuda
    U, I, F, _ = make_case(15, 1, 21, 40, 56, 3)
    Ut, It = torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda()
    p = params(torch, 7, F, True)
    a = crf.meanfield(Ut, It, p, 3)
    buf = torch.empty(U.size + 1, device="cuda")
    out = buf[1:].view(U.shape)
    assert out.data_ptr() % 8 != 0
    b = crf.meanfield(Ut, It, p, 3, out=out)
    torch.cuda.synchronize()
    a, b = (x.cpu().numpy().astype(np.float64) for x in (a, b))
    o = oracle_mod.meanfield(U, I, oparams(p), 3, features=F)
    ea, eb, eab = np.abs(a - o).max(), np.abs(b - o).max(), np.abs(a - b).max()
    print(f"ring {ea:.2e}, feature kernel {eb:.2e}, between {eab:.2e}", flush=True)
    assert ea <= 1e-4 and eb <= 1e-4 and eab <= 1e-4
    assert eab > 0      # two different kernels: not the same path twice


def bench_features(wl):
    """The feature planes `bench.py --features` times: the pixel coordinates
    (row, column) plus N(0, 0.5), seed 78."""
    yy, xx = np.meshgrid(np.arange(wl.H, dtype=np.float32), np.arange(wl.W, dtype=np.float32),
                         indexing="ij")
    return (np.stack([yy, xx])[None].repeat(wl.B, axis=0) + np.random.default_rng(78).normal(
        0.0, 0.5, (wl.B, 2, wl.H, wl.W))).astype(np.float32)


def workload_params(torch, wl, F):
    return params(torch, wl.filter_size, F, blur=wl.blur, w_app=wl.w_app,
                  theta_alpha=wl.theta_alpha, theta_beta=wl.theta_beta, w_smooth=wl.w_smooth,
                  theta_gamma=wl.theta_gamma)


@pytest.mark.parametrize("name", ["pascal", "blur"])
def test_feature_workload_full(torch_cuda, crf, oracle_mod, name):
    """The workloads `bench.py --features` times, every pixel and class:
    1 x 21 x 512 x 512 with two feature planes, k = 7 (the ring kernel's
    feature mode) or k = 11 on the 4 x 4 pooled grid (the fused round's)."""
    from paper_1805_04777_amd import synth
    torch = torch_cuda
    wl = synth.WORKLOADS[name]
    U, I, _ = synth.make_inputs(wl)
    F = bench_features(wl)
    p = workload_params(torch, wl, F)
    print(f"case {name} with features, full", flush=True)
    Q = crf.meanfield(torch.from_numpy(U).cuda(), torch.from_numpy(I).cuda(), p, wl.iters)
    torch.cuda.synchronize()
    Qg = Q.cpu().numpy().astype(np.float64)
    Qo = oracle_mod.meanfield(U, I, oparams(p), wl.iters, features=F)
    err = np.abs(Qg - Qo).max()
    agree = (Qg.argmax(1) == Qo.argmax(1)).mean()
    print(f"{name} with features: max|dQ| {err:.2e}, argmax agreement {agree:.6f}", flush=True)
    assert err <= 1e-4
    assert agree >= 0.9999
    assert np.abs(Qg.sum(1) - 1.0).max() <= 1e-5


@pytest.mark.parametrize("name", ["pascal", "blur"])
def test_feature_workload_backward_full(torch_cuda, crf, oracle_mod, name):
    """The derivative `bench.py --backward --features` times (1 x 21 x 512 x
    512, T = 5, two feature planes; k = 7, or k = 11 on the 4 x 4 pooled
    grid), in full."""
    from paper_1805_04777_amd import synth
    torch = torch_cuda
    wl = synth.WORKLOADS[name]
    U, I, _ = synth.make_inputs(wl)
    F = bench_features(wl)
    G = np.random.default_rng(77).normal(0.0, 1.0, U.shape).astype(np.float32)
    p = workload_params(torch, wl, F)
    print(f"case {name} with features, derivative, full", flush=True)
    t = lambda x: torch.from_numpy(x).cuda()
    dU, dmu, dk, dF = crf.meanfield_backward(t(U), t(I), p, wl.iters, t(G), grad_compat=True,
                                             grad_kernel=True)
    torch.cuda.synchronize()
    got = [x.cpu().numpy().astype(np.float64) for x in (dU, dmu, dk, dF)]
    ref = oracle_mod.meanfield_backward(U, I, oparams(p), wl.iters, G, features=F)
    for g, r, nm in zip((got[0], got[1], got[3]), (ref[0], ref[1], ref[3]), ("dU", "dmu", "dF")):
        e = np.abs(g - r).max() / np.abs(r).max()
        print(f"{name} with features: {nm} rel err {e:.2e}", flush=True)
        assert e <= 1e-4, f"{nm}: rel err {e:.2e}"
    # the five parameter derivatives as one vector, held to its own scale as
    # the tensors above are (1e-4 of its largest entry), and each entry to
    # 1e-3 relative where its sum does not cancel (at least 1e-2 of the
    # largest): with these features the theta_gamma sum over every pixel pair
    # cancels to about 1.6e-3 of the scale (0.77 against 4.9 without them)
    ek = np.abs(got[2] - ref[2]) / np.abs(ref[2])
    scale = np.abs(ref[2]).max()
    for j in range(5):
        print(f"{name} with features: parameter {j}: gpu {got[2][j]:.9e} oracle {ref[2][j]:.9e} "
              f"rel err {ek[j]:.2e}", flush=True)
    assert np.abs(got[2] - ref[2]).max() <= 1e-4 * scale
    big = np.abs(ref[2]) >= 1e-2 * scale
    assert big.sum() >= 3 and np.all(ek[big] <= 1e-3), ek
