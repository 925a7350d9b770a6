"""The C ABI of libconvcrf, checked without a GPU.

The library must load, export every function that include/convcrf.h declares,
and reject invalid arguments with the documented status before touching the
device (convcrf_validate needs no context and makes no HIP call).
"""
import ctypes
import os
import re

import numpy as np

import pytest

from paper_1805_04777_amd import convcrf as cc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "convcrf.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(convcrf_[a-z_]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(cc.LIB_PATH):
        from paper_1805_04777_amd import build
        build.build()
    return cc.load_library()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("convcrf_init", "convcrf_meanfield", "convcrf_destroy", "convcrf_validate",
              "convcrf_last_error"):
        assert n in names
    assert set(names) == set(cc.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_layout_matches_header(lib):
    # 4 int32 + 5 float (+ 4 padding) + pointer + pointer + int32 (+ 4 padding)
    assert ctypes.sizeof(cc.CParams) == 4 * 4 + 5 * 4 + 4 + 8 + 8 + 4 + 4
    assert cc.CParams.compat.offset == 40
    assert cc.CParams.features.offset == 48
    assert cc.CParams.feature_dim.offset == 56


def test_default_params(lib):
    p = cc.default_params()
    assert (p.filter_size, p.blur, p.include_center, p.variant) == (7, 1, False, cc.VARIANT_FUSED)
    assert (p.w_app, p.theta_alpha, p.theta_beta, p.w_smooth, p.theta_gamma) == (10, 80, 13, 3, 3)
    assert p.compat is None and p.features is None


def test_status_strings(lib):
    for code, name in [(cc.OK, "CONVCRF_OK"), (cc.E_INVALID_ARG, "CONVCRF_E_INVALID_ARG"),
                       (cc.E_UNSUPPORTED, "CONVCRF_E_UNSUPPORTED"),
                       (cc.E_NO_DEVICE, "CONVCRF_E_NO_DEVICE"), (cc.E_HIP, "CONVCRF_E_HIP"),
                       (cc.E_OOM, "CONVCRF_E_OOM")]:
        assert lib.convcrf_status_string(code).decode() == name


def P(**kw):
    return cc.Params(**kw)


@pytest.mark.parametrize("args,status", [
    ((1, 21, 64, 64, P(), 5), cc.OK),
    ((8, 19, 1024, 2048, P(), 5), cc.OK),
    ((1, 21, 512, 512, P(filter_size=11, blur=4), 5), cc.OK),
    ((0, 21, 64, 64, P(), 5), cc.OK),                      # empty batch
    ((1, 21, 0, 64, P(), 5), cc.OK),                       # empty image
    ((1, 21, 64, 64, P(), 0), cc.OK),
    ((1, 1, 3, 3, P(filter_size=1), 2), cc.OK),
    ((1, 24, 8, 8, P(filter_size=15), 1), cc.OK),
    ((-1, 21, 64, 64, P(), 5), cc.E_INVALID_ARG),
    ((1, 0, 64, 64, P(), 5), cc.E_INVALID_ARG),
    ((1, 21, -4, 64, P(), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(), -1), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(filter_size=6), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(filter_size=0), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(filter_size=17), 5), cc.E_UNSUPPORTED),
    ((1, 25, 64, 64, P(), 5), cc.E_UNSUPPORTED),
    ((1, 21, 64, 64, P(include_center=2), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(variant=7), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(theta_alpha=0.0), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(theta_beta=-1.0), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(theta_gamma=float("inf")), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(w_smooth=float("nan")), 5), cc.E_INVALID_ARG),
    ((1, 21, 64, 64, P(w_app=-1.0), 5), cc.E_UNSUPPORTED),
    ((1, 21, 64, 64, P(blur=3), 5), cc.E_INVALID_ARG),
    ((1, 21, 66, 64, P(blur=4), 5), cc.E_UNSUPPORTED),     # H not a multiple of s
    ((1, 21, 2 * 65536, 8, P(blur=2), 5), cc.E_UNSUPPORTED),  # pooled rows beyond the grid
    ((65536, 21, 8, 8, P(blur=2), 5), cc.E_UNSUPPORTED),      # batch beyond the grid
    ((1, 21, 2 * 65535, 8, P(blur=2), 5), cc.OK),
    ((1, 21, 64, 64, P(blur=2, variant=cc.VARIANT_MATERIALISED), 5), cc.E_UNSUPPORTED),
    ((1, 21, 64, 64, P(blur=2, variant=cc.VARIANT_RESIDENT), 5), cc.OK),
    ((1, 21, 64, 64, P(variant=cc.VARIANT_RESIDENT), 5), cc.OK),
])
def test_validation(lib, args, status):
    B, C, H, W, p, T = args
    assert cc.validate(B, C, H, W, p, T) == status


def test_validation_null_params(lib):
    assert lib.convcrf_validate(1, 21, 8, 8, None, 1) == cc.E_INVALID_ARG
    assert "params" in lib.convcrf_last_error(None).decode()


def test_null_context_is_rejected(lib):
    p = P().c()
    st = lib.convcrf_meanfield(None, 1, 2, 1, 21, 8, 8, ctypes.byref(p), 1, 3, None)
    assert st == cc.E_INVALID_ARG
    assert lib.convcrf_profile_enable(None, 1) == cc.E_INVALID_ARG
    lib.convcrf_destroy(None)  # no-op


def test_init_rejects_null_out(lib):
    assert lib.convcrf_init(None, 0) == cc.E_INVALID_ARG


def test_init_without_a_gpu_reports_no_device(lib):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    h = ctypes.c_void_p(1234)
    assert lib.convcrf_init(ctypes.byref(h), 0) == cc.E_NO_DEVICE
    assert h.value is None


def test_strerror_names_the_status_and_the_message(lib):
    assert lib.convcrf_strerror(None, cc.OK).decode() == "CONVCRF_OK"
    assert lib.convcrf_validate(1, 21, 8, 8, None, 1) == cc.E_INVALID_ARG
    text = lib.convcrf_strerror(None, cc.E_INVALID_ARG).decode()
    assert text.startswith("CONVCRF_E_INVALID_ARG: ") and "params" in text


def test_synchronize_rejects_a_null_context(lib):
    assert lib.convcrf_synchronize(None, None) == cc.E_INVALID_ARG


def test_negative_smoothness_weight_is_accepted(lib):
    # Eq. 4 fixes no sign for the weights; only w_app is folded into log2
    assert cc.validate(1, 21, 64, 64, P(w_smooth=-2.0), 5) == cc.OK
    assert cc.validate(1, 21, 64, 64, P(w_app=-2.0), 5) == cc.E_UNSUPPORTED


@pytest.mark.parametrize("compat", [
    np.zeros((3, 3), np.float32),        # the wrong class count
    np.zeros(21 * 21, np.float32),       # flat, not C x C
    np.zeros((21, 20), np.float32),
    [["a"] * 21] * 21,                   # not numbers
])
def test_compat_must_be_c_by_c(lib, compat):
    assert cc.validate(1, 21, 8, 8, P(compat=compat), 1) == cc.E_INVALID_ARG
    with pytest.raises(cc.ConvCRFError) as e:
        P(compat=compat).c((1, 21, 8, 8))
    assert e.value.status == cc.E_INVALID_ARG


def test_compat_of_the_right_shape_is_passed_through(lib):
    mu = np.arange(21 * 21, dtype=np.float64).reshape(21, 21)
    p = P(compat=mu)
    c = p.c((1, 21, 8, 8))
    got = np.ctypeslib.as_array(c.compat, shape=(21 * 21,))
    assert np.array_equal(got, mu.ravel().astype(np.float32))
    assert cc.validate(1, 21, 8, 8, p, 1) == cc.OK


class _FakeFeatures:
    """Stands in for a CUDA tensor on a CPU-only host (the binding reads only
    these attributes before handing the pointer to the library)."""

    def __init__(self, shape, dtype=None, device="cuda:0"):
        import torch
        self.shape = tuple(shape)
        self.dtype = torch.float32 if dtype is None else dtype
        self.device = torch.device(device)
        self.is_cuda = True

    def is_contiguous(self):
        return True

    def dim(self):
        return len(self.shape)

    def data_ptr(self):
        return 4096


@pytest.mark.parametrize("shape,dtype,why", [
    ((1, 2, 8, 8), "int32", "dtype"),
    ((2, 2, 8, 8), None, "batch"),
    ((1, 2, 8, 9), None, "width"),
    ((1, 2, 7, 8), None, "height"),
    ((1, 2, 8), None, "rank"),
])
def test_features_must_match_the_unary(lib, monkeypatch, shape, dtype, why):
    import torch
    monkeypatch.setattr(torch, "Tensor", _FakeFeatures)
    f = _FakeFeatures(shape, getattr(torch, dtype) if dtype else None)
    with pytest.raises(cc.ConvCRFError) as e:
        P(features=f).c((1, 21, 8, 8), torch.device("cuda:0"))
    assert e.value.status == cc.E_INVALID_ARG, why


def test_features_must_be_on_the_unary_device(lib, monkeypatch):
    import torch
    monkeypatch.setattr(torch, "Tensor", _FakeFeatures)
    f = _FakeFeatures((1, 2, 8, 8), device="cuda:1")
    with pytest.raises(cc.ConvCRFError):
        P(features=f).c((1, 21, 8, 8), torch.device("cuda:0"))
    c = P(features=_FakeFeatures((1, 2, 8, 8))).c((1, 21, 8, 8), torch.device("cuda:0"))
    assert c.feature_dim == 2 and c.features == 4096
