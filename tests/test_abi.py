"""C-ABI contract checks that need no GPU.

* the library loads and exports every function include/specdiff.h declares;
* the binding declares a signature for each of them;
* invalid arguments return SD_EINVAL with a message, before any HIP call;
* the host schedule table equals the oracle's VP schedule.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_13426_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names += re.findall(r"\b(sd_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2606_13426_amd import build
        build.build()
    return _lib.load()


def test_exports_every_declared_symbol(lib):
    declared = _declared_functions()
    assert len(declared) >= 15
    for name in declared:
        assert hasattr(lib, name), name
    bound = {n for n, _, _ in _lib.SIGNATURES}
    assert set(declared) == bound


def test_abi_version(lib):
    assert _lib.sd_abi_version() == 4


def _expect_einval(status, needle):
    assert status == _lib.SD_EINVAL
    assert needle in _lib.last_error()


def test_invalid_arguments_rejected_without_gpu(lib):
    null = None
    s0 = _lib.sd_stride(0, 0)
    bad = _lib.schedule(10, churn=0.0)
    h = ctypes.c_void_p()
    mu = np.zeros((2, 3), np.float32)
    var = np.ones(2, np.float32)
    lw = np.zeros(2, np.float32)
    st = lib.sd_target_create(ctypes.byref(bad), 3, 2, mu.ctypes.data_as(ctypes.c_void_p),
                              var.ctypes.data_as(ctypes.c_void_p), lw.ctypes.data_as(ctypes.c_void_p), 0,
                              ctypes.byref(h))
    _expect_einval(st, "schedule")
    good = _lib.schedule(10)
    st = lib.sd_target_create(ctypes.byref(good), 0, 2, mu.ctypes.data_as(ctypes.c_void_p),
                              var.ctypes.data_as(ctypes.c_void_p), lw.ctypes.data_as(ctypes.c_void_p), 0,
                              ctypes.byref(h))
    _expect_einval(st, "d = 0")
    vneg = np.array([1.0, -1.0], np.float32)
    st = lib.sd_target_create(ctypes.byref(good), 3, 2, mu.ctypes.data_as(ctypes.c_void_p),
                              vneg.ctypes.data_as(ctypes.c_void_p), lw.ctypes.data_as(ctypes.c_void_p), 0,
                              ctypes.byref(h))
    _expect_einval(st, "var[1]")
    st = lib.sd_verify_block(4, 65, 8, 0, null, s0, null, s0, null, s0, null, null, null, 0, 0,
                             null, null, null, null, null, null, null)
    _expect_einval(st, "K = 65")
    st = lib.sd_verify_block(4, 8, 8, 0, null, s0, null, s0, null, s0, null, null, null, 0, 0,
                             null, null, null, null, null, null, null)
    _expect_einval(st, "NULL")
    st = lib.sd_draft_block(ctypes.byref(bad), 4, 8, 8, null, null, null, null, 0, null, s0, null, s0, null)
    _expect_einval(st, "schedule")
    st = lib.sd_sample_residual(0, 8, 8, null, s0, null, s0, null, s0, null, null, null, null, null,
                                null, null, 0, null, null)
    _expect_einval(st, "B >= 1")
    st = lib.sd_run_sampler(null, 4, 8, 0, 0, 0, null, null, 0, null, null, 0, null)
    _expect_einval(st, "target is NULL")
    for omega in (0.0, -1.0, float("inf"), float("nan"), 1e-200, 1e200):
        st = lib.sd_verify_block_tempered(4, 8, 8, 0, omega, null, s0, null, s0, null, s0, null, null,
                                          null, 0, 0, null, null, null, null, null, null, null)
        _expect_einval(st, "omega")
    st = lib.sd_sample_residual_reflection(4, 0, 8, null, s0, null, s0, null, s0, null, null, null, null,
                                           null, 0, null, null)
    _expect_einval(st, "K = 0")
    st = lib.sd_run_sampler_ex(null, 4, 8, None, 0, null, null, 0, null, null, 0, null)
    _expect_einval(st, "options are NULL")
    opts = _lib.sd_sampler_options(_lib.SD_BLOCK, 0, _lib.SD_RESIDUAL_REFLECTION, _lib.SD_DRAFTER_FREE, 1.0)
    st = lib.sd_run_sampler_ex(null, 4, 8, ctypes.byref(opts), 0, null, null, 0, null, null, 0, null)
    _expect_einval(st, "reflection residual needs sample")
    opts = _lib.sd_sampler_options(_lib.SD_TOKEN, 0, _lib.SD_RESIDUAL_REFLECTION, 7, 1.0)
    st = lib.sd_run_sampler_ex(null, 4, 8, ctypes.byref(opts), 0, null, null, 0, null, null, 0, null)
    _expect_einval(st, "unknown drafter")
    opts = _lib.sd_sampler_options(_lib.SD_TOKEN, 0, 0, _lib.SD_DRAFTER_FROZEN, 0.0)
    st = lib.sd_run_sampler_ex(null, 4, 8, ctypes.byref(opts), 0, null, null, 0, null, null, 0, null)
    _expect_einval(st, "omega")
    opts = _lib.sd_sampler_options(_lib.SD_TOKEN, 0, _lib.SD_RESIDUAL_REFLECTION, _lib.SD_DRAFTER_FROZEN, 2.0)
    st = lib.sd_run_sampler_ex(null, 4, 8, ctypes.byref(opts), 0, null, null, 0, null, null, 0, null)
    _expect_einval(st, "target is NULL")
    opts = _lib.sd_sampler_options(_lib.SD_BLOCK, 0, 0, 0, 1.0, -1, -1)
    st = lib.sd_run_sampler_ex(null, 4, 8, ctypes.byref(opts), 0, null, null, 0, null, null, 0, null)
    _expect_einval(st, "start_round must be >= 0")
    view = _lib.sd_sampler_view()
    st = lib.sd_sampler_state(null, 4, 8, null, 0, 0, ctypes.byref(view))
    _expect_einval(st, "NULL")
    st = lib.sd_run_plain_em(null, 4, 0, null, null, 0, null)
    _expect_einval(st, "target is NULL")
    assert lib.sd_plain_em_workspace(null, 4) == 0
    st = lib.sd_init_chains(0, 3, 0, null, null)
    _expect_einval(st, "B >= 1")
    assert lib.sd_sampler_workspace(null, 4, 8) == 0
    assert lib.sd_target_mean_workspace(null, 4) == 0


def test_profile_controls_without_gpu(lib):
    # the profiling switches are host state: no HIP call, no device needed
    _expect_einval(lib.sd_profile_every(0), "n < 1")
    _expect_einval(lib.sd_profile_seen(None, None), "NULL")
    assert lib.sd_profile_every(4) == _lib.SD_OK
    assert lib.sd_profile_enable(1) == _lib.SD_OK
    assert _lib.sd_profile_seen("gmm_mean_lr") == 0
    assert lib.sd_profile_enable(0) == _lib.SD_OK
    assert lib.sd_profile_every(1) == _lib.SD_OK


def test_strides_validated(lib):
    good = _lib.schedule(10)
    p = ctypes.c_void_p(256)  # never dereferenced: validation fails first
    st = lib.sd_draft_block(ctypes.byref(good), 2, 4, 16, p, p, p, p, 0, p, _lib.sd_stride(16 * 4, 16), p,
                            _lib.sd_stride(64, 16), None)
    _expect_einval(st, "x stride")


def test_schedule_table_matches_oracle(lib):
    from oracle.schedule import Schedule
    for N, eps in ((100, 1.0), (1000, 0.25)):
        tab = _lib.sd_schedule_table(_lib.schedule(N, churn=eps))
        sch = Schedule(N, churn=eps)
        n = np.arange(N + 1)
        np.testing.assert_allclose(tab[0], sch.signal(n), rtol=1e-14)
        np.testing.assert_allclose(tab[1], sch.sigma(n), rtol=1e-14)
        np.testing.assert_allclose(tab[2], sch.c1(n), rtol=1e-15)
        np.testing.assert_allclose(tab[3], sch.c2(n), rtol=1e-14)
