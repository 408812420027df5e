"""C-ABI checks that need no GPU: the library loads, exports every entry point the
header declares, and the host-side validation / workspace sizing behaves."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2212_11142_amd import gp
from workloads import Param, make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "baco_gp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gp_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    return gp.load()


def test_header_symbols_exported(lib):
    names = header_functions()
    assert len(names) >= 15
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(gp.exported_names()) == names


def test_version(lib):
    assert lib.gp_version() == 100


def space_of(name):
    return gp.Space(make_workload(name, 64).space)


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_workspace_sizes(lib, name):
    sp = space_of(name)
    a = lib.gp_fit_workspace_bytes(sp.ref(), 512, 0)
    b = lib.gp_fit_workspace_bytes(sp.ref(), 512, 1)
    assert 0 < a < b
    assert a % 256 == 0 and b % 256 == 0
    assert lib.gp_fit_workspace_bytes(sp.ref(), 0, 0) == 0
    assert lib.gp_fit_workspace_bytes(sp.ref(), 4097, 0) == 0
    assert lib.gp_debug_workspace_bytes(sp.ref(), None, 1000) > 0
    # fused fit and scoring: the fit's workspace (rounded to 256) and the scoring buffers
    f = lib.gp_fit_score_workspace_bytes(sp.ref(), 512, 1, 1 << 20)
    assert f > b + (1 << 20) * 2 * 512 * 2
    assert f > lib.gp_fit_score_workspace_bytes(sp.ref(), 512, 0, 1 << 20)
    assert lib.gp_fit_score_workspace_bytes(sp.ref(), 512, 1, 0) > b
    assert lib.gp_fit_score_workspace_bytes(sp.ref(), 512, 1, -1) == 0
    assert lib.gp_fit_score_workspace_bytes(sp.ref(), 0, 1, 10) == 0


def test_fused_workspace_bound_any_lengthscales(lib):
    """gp_fit_score_workspace_bytes takes no lengthscales, so its scoring region must hold
    the candidate codes for any of them. Categorical one-hot fields share a 32-bit code
    word only when their weights (1 / 2l^2) are equal: two 8-level categoricals fit one
    word, two 20-level ones never do. With per-parameter lengthscales (C5 draws them
    log-uniformly) the 8-level pair takes two words, so the bound must grow per candidate
    row exactly as for the 20-level pair. (A bound computed with shared words ran the
    full-size C5 fused step 4 MiB past the end of its workspace.)"""
    def per_rows(levels, rows=1 << 16, M0=1 << 20):
        sp = gp.Space([Param("a", "cat", levels=levels), Param("b", "cat", levels=levels),
                       Param("x", "real")])
        f = lambda M: lib.gp_fit_score_workspace_bytes(sp.ref(), 64, 0, M)
        return f(M0 + rows) - f(M0)
    assert per_rows(8) == per_rows(20) > 0
    c5 = space_of("C5")
    grew = (lib.gp_fit_score_workspace_bytes(c5.ref(), 2048, 0, (1 << 20) + (1 << 16)) -
            lib.gp_fit_score_workspace_bytes(c5.ref(), 2048, 0, 1 << 20))
    # C5: 8 numeric words, 2 categorical words, 2 Hamming words, 2 Spearman words
    assert grew >= (1 << 16) * 4 * 14


@pytest.mark.parametrize("name,n", [("C3", 256), ("C4", 512), ("C5", 2048)])
def test_workspace_refine_block_buffers(lib, name, n):
    """The fp64 recomputation's block path (more than 4096 flagged candidates) needs
    [ceil(n/256)][rows] partial norms and [rows] means in fp64; the scoring buffers carry
    them once the candidate rows (M rounded up to 128) exceed 4096, and grow with the rows
    from there."""
    sp = space_of(name)
    f = lambda M: lib.gp_fit_score_workspace_bytes(sp.ref(), n, 1, M)
    step = f(4096) - f(3968)  # one row tile of the other per-row buffers
    tiles = (n + 255) // 256
    cross = f(4224) - f(4096)
    assert abs(cross - step - (tiles + 1) * 4224 * 8) <= 64 * 256, (cross, step)
    above = f(4352) - f(4224)
    assert abs(above - step - (tiles + 1) * 128 * 8) <= 64 * 256, (above, step)


@pytest.mark.parametrize("name", ["C1", "C4", "C5"])
def test_hyper_workspace_sizes(lib, name):
    sp = space_of(name)
    n = 512
    a = lib.gp_hyper_workspace_bytes(sp.ref(), n, 8, 0)
    b = lib.gp_hyper_workspace_bytes(sp.ref(), n, 64, 0)
    c = lib.gp_hyper_workspace_bytes(sp.ref(), n, 1000, 0)       # batches of 64
    f = lib.gp_hyper_workspace_bytes(sp.ref(), n, 1000, 16)      # + samples and L-BFGS state
    assert 0 < a < b == c < f
    ld = 512
    assert b >= 3 * 64 * ld * ld * 8 + len(sp.params) * n * n * 8
    for bad in [(0, 8, 0), (4097, 8, 0), (n, 0, 0), (n, 8, 9), (n, 100, 65), (n, 8, -1)]:
        assert lib.gp_hyper_workspace_bytes(sp.ref(), *bad) == 0, bad


def test_invalid_spaces_rejected(lib):
    bad = [
        [Param("p", "perm", m=9)],                                   # m > 8
        [Param("p", "perm", m=1)],
        [Param("o", "ord", values=(1, 4, 2))],                       # not ascending
        [Param("o", "ord", log2=True, values=(0, 1, 2))],            # log of 0
        [Param("r", "real", lo=1.0, hi=0.0)],                        # lo > hi
        [Param("r", "real", log2=True, lo=0.0, hi=1.0)],             # log2 with lo = 0
        [Param("i", "int", lo=0.5, hi=3)],                           # non-integer bound
        [Param("c", "cat", levels=0)],
        [Param(f"x{k}", "real") for k in range(65)],                 # d > 64
    ]
    for params in bad:
        sp = gp.Space(params)
        assert lib.gp_fit_workspace_bytes(sp.ref(), 10, 0) == 0, params
    ok = gp.Space([Param("c", "cat", levels=40), Param("p", "perm", m=8, dist="naive"),
                   Param("h", "perm", m=8, dist="hamming"), Param("k", "perm", m=8, dist="kendall")])
    assert lib.gp_fit_workspace_bytes(ok.ref(), 10, 1) > 0


def test_error_paths_without_device(lib):
    sp = space_of("C1")
    out = C.c_void_p()
    ls = np.ones(5)
    reg = gp._Hyper(ls.ctypes.data_as(C.POINTER(C.c_double)), 1.0, 1e-4)
    # NULL out
    assert lib.gp_fit(sp.ref(), None, 10, None, None, C.byref(reg), None, None, 0, None, None) == 1
    # NULL y
    assert lib.gp_fit(sp.ref(), None, 10, None, None, C.byref(reg), None, None, 0, None,
                      C.byref(out)) == 1
    assert b"y is NULL" in lib.gp_last_error()
    # negative noise
    reg2 = gp._Hyper(ls.ctypes.data_as(C.POINTER(C.c_double)), 1.0, -1.0)
    assert lib.gp_fit(sp.ref(), None, 10, C.c_void_p(16), None, C.byref(reg2), None, None, 0, None,
                      C.byref(out)) == 1
    # bad lengthscale
    ls0 = np.zeros(5)
    reg3 = gp._Hyper(ls0.ctypes.data_as(C.POINTER(C.c_double)), 1.0, 1e-4)
    cols = (C.c_void_p * 5)(*([16] * 5))
    assert lib.gp_fit(sp.ref(), cols, 10, C.c_void_p(16), None, C.byref(reg3), None, None, 0, None,
                      C.byref(out)) == 1
    assert b"lengthscale" in lib.gp_last_error()
    # missing workspace
    assert lib.gp_fit(sp.ref(), cols, 10, C.c_void_p(16), None, C.byref(reg), None, None, 0, None,
                      C.byref(out)) == 5
    # misaligned workspace
    assert lib.gp_fit(sp.ref(), cols, 10, C.c_void_p(16), None, C.byref(reg), None,
                      C.c_void_p(1 << 20 | 8), 1 << 30, None, C.byref(out)) == 5
    # fused fit and scoring: argument errors before any device work
    big = C.c_void_p(1 << 20)
    args = lambda M, eps, mu, ws, wsb: (sp.ref(), cols, 10, C.c_void_p(16), None, C.byref(reg),
                                        None, cols, M, None, C.c_float(eps), mu, big, big, None,
                                        big, None, ws, wsb, None, C.byref(out))
    assert lib.gp_fit_score(*args(10, 0.0, big, None, 0)) == 5             # no workspace
    assert lib.gp_fit_score(*args(-1, 0.0, big, big, 1 << 40)) == 1
    assert lib.gp_fit_score(*args(10, 2.0, big, big, 1 << 40)) == 1
    assert b"eps_f" in lib.gp_last_error()
    assert lib.gp_fit_score(*args(10, 0.0, None, big, 1 << 40)) == 1
    assert b"required" in lib.gp_last_error()
    # score without a model
    assert lib.gp_score(None, None, 10, None, 0.0, None, None, None, None, None, None, None, 0,
                        None) == 1
    assert lib.gp_score_workspace_bytes(None, 10) == 0
    # hyperparameter calls: argument errors come before any device work
    P = gp._Prior(1.5, 1.0)
    assert lib.gp_log_posterior(None, None, 10, None, None, None, 1, None, 0.0, None, None,
                                None, 0, None) == 1
    assert lib.gp_log_posterior(sp.ref(), cols, 10, None, None, C.c_void_p(16), 1, None, 0.0,
                                C.c_void_p(16), None, None, 0, None) == 1
    assert b"y is NULL" in lib.gp_last_error()
    bad_prior = gp._Prior(-1.0, 1.0)
    assert lib.gp_log_posterior(sp.ref(), cols, 10, C.c_void_p(16), None, C.c_void_p(16), 1,
                                C.byref(bad_prior), 0.0, C.c_void_p(16), None, None, 0,
                                None) == 1
    assert b"prior" in lib.gp_last_error()
    assert lib.gp_log_posterior(sp.ref(), cols, 10, C.c_void_p(16), None, C.c_void_p(16), 1,
                                C.byref(P), -1.0, C.c_void_p(16), None, None, 0, None) == 1
    assert lib.gp_hyperfit(sp.ref(), cols, 10, C.c_void_p(16), None, C.c_void_p(16), 8, 9,
                           C.byref(P), 1e-6, 10, 1e-5, 0.0, C.c_void_p(16), C.c_void_p(16), None,
                           None, None, None, None, 0, None) == 1
    assert b"n_keep" in lib.gp_last_error()
    assert lib.gp_hyperfit(sp.ref(), cols, 10, C.c_void_p(16), None, C.c_void_p(16), 8, 4,
                           C.byref(P), 1e-6, 10, 1e-5, 0.0, C.c_void_p(16), C.c_void_p(16), None,
                           None, None, None, None, 0, None) == 5      # missing workspace
    # local search without a model
    assert lib.gp_local_search_workspace_bytes(None, 10, 4) == 0
    assert lib.gp_local_search(None, None, 10, None, 0.0, 4, 10, None, None, None, None, None, 0,
                               None) == 1
    info = gp._Info()
    assert lib.gp_model_info(None, C.byref(info)) == 1
    lib.gp_model_free(None)


def test_classifier_lengthscale_must_match(lib):
    sp = space_of("C1")
    out = C.c_void_p()
    ls = np.ones(5)
    ls2 = np.full(5, 2.0)
    reg = gp._Hyper(ls.ctypes.data_as(C.POINTER(C.c_double)), 1.0, 1e-4)
    cls = gp._Hyper(ls2.ctypes.data_as(C.POINTER(C.c_double)), 1.0, 0.0)
    cols = (C.c_void_p * 5)(*([16] * 5))
    assert lib.gp_fit(sp.ref(), cols, 10, C.c_void_p(16), None, C.byref(reg), C.byref(cls), None, 0,
                      None, C.byref(out)) == 4


def test_profile_calls_without_device(lib):
    assert lib.gp_profile_start() == 0
    ms = (C.c_double * 6)()
    calls = C.c_int64(-1)
    assert lib.gp_profile_stop(ms, C.byref(calls)) == 0
    assert calls.value == 0
