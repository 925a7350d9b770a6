"""convcrf_meanfield_noalloc: the allocation-free variant of convcrf_meanfield.

It runs the same kernels with its workspace in the library's per-device
scratch array, so its output must equal convcrf_meanfield's bit for bit.
The calls come in a row on one context, each smaller than the one before
(the scratch array keeps the previous call's contents), and the smaller
ones are also held to the oracle's 1e-4 bar.  A request beyond the scratch
size is refused with nothing enqueued.
"""

import numpy as np
import pytest

from paper_1805_04777_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch


def _params(wl=None, **kw):
    from paper_1805_04777_amd import convcrf as cc
    base = {}
    if wl is not None:
        base = dict(filter_size=wl.filter_size, blur=wl.blur, w_app=wl.w_app,
                    theta_alpha=wl.theta_alpha, theta_beta=wl.theta_beta,
                    w_smooth=wl.w_smooth, theta_gamma=wl.theta_gamma)
    base.update(kw)
    return cc.Params(**base)


def _cases():
    # largest first: the pascal workload (22 MB of ping-pong), then smaller
    # inputs that reuse the front of the scratch array
    pascal = synth.WORKLOADS["pascal"]
    U, I, _ = synth.make_inputs(pascal)
    yield "pascal 1x21x512x512 k=7 T=5", U, I, _params(pascal), pascal.iters
    rng = np.random.default_rng(11)
    U = rng.normal(0, 2, (2, 21, 96, 160)).astype(np.float32)
    I = rng.integers(0, 256, (2, 3, 96, 160)).astype(np.float32)
    yield ("2x21x96x160 k=5 general mu T=3", U, I,
           _params(filter_size=5, compat=synth.random_compat(21, seed=5), w_app=2.0, w_smooth=0.7), 3)
    U = rng.normal(0, 2, (1, 19, 64, 96)).astype(np.float32)
    I = rng.integers(0, 256, (1, 3, 64, 96)).astype(np.float32)
    yield "1x19x64x96 k=11 blur 4 T=3", U, I, _params(filter_size=11, blur=4), 3
    U = rng.normal(0, 2, (1, 5, 33, 47)).astype(np.float32)
    I = rng.integers(0, 256, (1, 3, 33, 47)).astype(np.float32)
    yield "1x5x33x47 k=7 T=4", U, I, _params(filter_size=7), 4


def test_noalloc_matches_meanfield_on_calls_in_a_row(torch_cuda, oracle_mod):
    from oracle import OracleParams
    from paper_1805_04777_amd import convcrf as cc
    torch = torch_cuda
    with cc.ConvCRF(0) as ref, cc.ConvCRF(0) as na:
        for i, (name, U, I, p, T) in enumerate(_cases()):
            Ut = torch.from_numpy(U).cuda()
            It = torch.from_numpy(I).cuda()
            q_ref = ref.meanfield(Ut, It, p, T)
            q_na = torch.full_like(Ut, -1.0)
            torch.cuda.synchronize()
            free0 = torch.cuda.mem_get_info()[0]
            na.meanfield(Ut, It, p, T, out=q_na, noalloc=True)
            na.synchronize()
            free1 = torch.cuda.mem_get_info()[0]
            assert free1 == free0, f"{name}: device memory changed by {free0 - free1} bytes"
            a = q_ref.cpu().numpy()
            b = q_na.cpu().numpy()
            assert np.array_equal(a, b), f"{name}: max diff {np.abs(a - b).max():.3e}"
            if i > 0:   # the smaller calls are cheap for the oracle: hold them to its bar
                Qo = oracle_mod.meanfield(U, I, OracleParams(
                    filter_size=p.filter_size, blur=p.blur, w_app=p.w_app,
                    theta_alpha=p.theta_alpha, theta_beta=p.theta_beta, w_smooth=p.w_smooth,
                    theta_gamma=p.theta_gamma), T, compat=p.compat)
                assert np.abs(b - Qo).max() <= 1e-4, name
                assert (b.argmax(1) == Qo.argmax(1)).mean() >= 0.9999, name
            print(f"noalloc {name}: identical to convcrf_meanfield", flush=True)


def test_noalloc_refuses_what_does_not_fit(torch_cuda):
    from paper_1805_04777_amd import convcrf as cc
    torch = torch_cuda
    with cc.ConvCRF(0) as na:
        # 8 x 21 x 512 x 512 needs 176 MB of ping-pong: beyond the scratch array
        U = torch.zeros(8, 21, 512, 512, device="cuda")
        I = torch.zeros(8, 3, 512, 512, device="cuda")
        out = torch.full_like(U, 7.0)
        with pytest.raises(cc.ConvCRFError) as e:
            na.meanfield(U, I, _params(), 5, out=out, noalloc=True)
        assert e.value.status == cc.E_UNSUPPORTED and "scratch" in str(e.value)
        # the materialised variant needs its kernel matrix allocated
        with pytest.raises(cc.ConvCRFError) as e:
            na.meanfield(U[:1], I[:1], _params(variant=cc.VARIANT_MATERIALISED), 5, out=out[:1],
                         noalloc=True)
        assert e.value.status == cc.E_UNSUPPORTED
        na.synchronize()
        assert bool((out == 7.0).all())
