"""GPU parity: the HIP library (through its C-ABI) against the CPU fp64 oracle on the
same seeded inputs.

Bars:
  * encodings and per-parameter distance terms: bit-exact;
  * fp32 cross-kernel K*: |dK| <= 4e-6 K + 1e-9 (fp32 arithmetic of r^2, sqrt, exp2);
  * fit (fp64): ||L L^T - K|| / ||K|| <= 1e-10 (max norm), K, alpha, K^-1 and the
    classifier against the oracle at fp64 accuracy scaled by the conditioning;
  * scores (fp32 outputs): relative error <= 1e-4 with floors
      mu:    |d| / max(|mu|, 1)                (y is standardised)
      sigma: |d| / max(sigma, 1e-2 sqrt(s))
      ei:    |d| / max(ei, 1e-3 max ei)
      p:     |d| / max(p, 1e-3)
      acq:   |d| / max(acq, 1e-3 max acq)
"""
import math

import numpy as np
import pytest

from oracle import gp_oracle as go
from workloads import Param, make_workload

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu] {request.node.nodeid}", flush=True)
    yield


def _torch():
    import torch
    return torch


def _gp():
    from paper_2212_11142_amd import gp
    return gp


def dev(a, dtype=None):
    torch = _torch()
    a = np.ascontiguousarray(a if dtype is None else a.astype(dtype))
    return torch.from_numpy(a).cuda()


_MODELS = {}


def fitted(name, M_small):
    """(workload with M_small candidates, gp.Space, device model, oracle model)."""
    key = (name, M_small)
    if key not in _MODELS:
        gp = _gp()
        w = make_workload(name, M_small)
        space = gp.Space(w.space)
        X = gp.to_device_columns(space, w.X)
        y = dev(np.nan_to_num(w.y, nan=0.0))
        feas = dev(w.feasible)
        model = gp.fit(space, X, y, feas, w.lengthscale, w.signal_var, w.noise_var,
                       w.cls_signal_var)
        om = go.fit(w.space, w.X, w.y, w.feasible, w.lengthscale, w.signal_var, w.noise_var,
                    w.cls_signal_var)
        _MODELS[key] = (w, space, model, om)
    return _MODELS[key]


def rel_err(got, ref, floor):
    return np.abs(got - ref) / np.maximum(np.abs(ref), floor)


def check_scores(out, ref, signal_var, has_cls, label, idx=None, with_acq=True):
    g = {k: out[k].double().cpu().numpy() for k in ("mu", "sigma", "ei")}
    g["acq"] = out["acq" if with_acq else "ei"].double().cpu().numpy()
    ref = ref if with_acq else dict(ref, acq=ref["ei"])
    if idx is not None:
        g = {k: v[idx] for k, v in g.items()}
    e_mu = rel_err(g["mu"], ref["mu"], 1.0).max()
    e_sig = rel_err(g["sigma"], ref["sigma"], 1e-2 * math.sqrt(signal_var)).max()
    e_ei = rel_err(g["ei"], ref["ei"], 1e-3 * max(ref["ei"].max(), 1e-300)).max()
    e_acq = rel_err(g["acq"], ref["acq"], 1e-3 * max(ref["acq"].max(), 1e-300)).max()
    msg = f"{label}: mu {e_mu:.2e} sigma {e_sig:.2e} ei {e_ei:.2e} acq {e_acq:.2e}"
    if "p_feas" in out:
        p = out["p_feas"].double().cpu().numpy()
        if idx is not None:
            p = p[idx]
        e_p = rel_err(p, ref["p_feas"], 1e-3).max()
        msg += f" p {e_p:.2e}"
        assert e_p <= TOL, msg
    print(msg, flush=True)
    assert e_mu <= TOL and e_sig <= TOL and e_ei <= TOL and e_acq <= TOL, msg


# ------------------------------------------------------------------ encoding
@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_encode_bit_exact(name):
    gp = _gp()
    w = make_workload(name, 4096)
    space = gp.Space(w.space)
    cols = [np.concatenate([x, c]) for x, c in zip(w.X, w.C)]
    codes, valid = gp.debug_encode(space, gp.to_device_columns(space, cols))
    codes = codes.cpu().numpy()
    assert valid.cpu().numpy().all()
    q = 0
    for p, c in zip(w.space, cols):
        if p.kind in go.NUMERIC:
            ref = go.encode_numeric(p, c)
            np.testing.assert_array_equal(codes[:, q].view(np.uint32), ref.view(np.uint32))
            q += 1
    assert q == codes.shape[1]


def test_encode_edges_and_invalid():
    gp = _gp()
    space_p = [Param("r", "real", lo=-3.0, hi=7.5), Param("lr", "real", log2=True, lo=0.5, hi=64.0),
               Param("i", "int", lo=-5, hi=1000), Param("li", "int", log2=True, lo=1, hi=1024),
               Param("o", "ord", values=(0.5, 1.0, 3.0, 9.0)), Param("c", "cat", levels=5),
               Param("p", "perm", m=6, dist="kendall")]
    space = gp.Space(space_p)
    r = np.array([-3.0, 7.5, 0.1, 2.25, -3.0, 1.0, np.nan, 1.0, 1.0, 1.0, 1.0])
    lr = np.array([0.5, 64.0, 1.0, 8.0, 2.0, 4.0, 1.0, 1.0, 1.0, 1.0, 1.0])
    i = np.array([-5, 1000, 0, 7, 3, 2, 1, 1001, 1, 1, 1], np.int32)
    li = np.array([1, 1024, 2, 512, 64, 8, 1, 1, 1, 1, 1], np.int32)
    o = np.array([0, 3, 1, 2, 0, 1, 1, 1, 4, 1, 1], np.int32)
    c = np.array([0, 4, 1, 2, 3, 0, 1, 1, 1, 5, 1], np.int32)
    perm = np.tile(np.arange(6, dtype=np.int32), (11, 1))
    perm[10] = [0, 1, 2, 3, 3, 5]
    cols = [r, lr, i, li, o, c, perm]
    codes, valid = gp.debug_encode(space, gp.to_device_columns(space, cols))
    valid = valid.cpu().numpy()
    np.testing.assert_array_equal(valid, [1, 1, 1, 1, 1, 1, 0, 0, 0, 0, 0])
    codes = codes.cpu().numpy()
    ok = valid.astype(bool)
    qi = 0
    for p, col in zip(space_p, cols):
        if p.kind in go.NUMERIC:
            got = codes[ok, qi]
            ref = go.encode_numeric(p, col[ok])
            if p.log2 and p.kind != "ord":
                # device log2 vs host log2 of non-powers of two may differ by 1 fp64 ulp
                np.testing.assert_allclose(got, ref, rtol=2 ** -23, atol=0)
            else:
                np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))
            qi += 1
    assert codes[0, 0] == 0.0 and codes[1, 0] == 1.0


# ------------------------------------------------------------------ terms and kernel
@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_terms_bit_exact(name):
    gp = _gp()
    w, space, model, om = fitted(name, 4096)
    order = model.export("FEASIBLE_INDEX").astype(np.int64)
    C = w.candidate_slice(0, 48)
    t = gp.debug_terms(model, gp.to_device_columns(space, C)).cpu().numpy()
    encX = [e[order] for e in go.encode(w.space, w.X)]
    ref = go.terms(w.space, go.encode(w.space, C), encX)
    np.testing.assert_array_equal(t.astype(np.float64), ref)


def test_terms_all_permutation_kinds():
    gp = _gp()
    import itertools
    ps = [Param("k", "perm", m=5, dist="kendall"), Param("s", "perm", m=5, dist="spearman"),
          Param("h", "perm", m=5, dist="hamming"), Param("n", "perm", m=5, dist="naive"),
          Param("c", "cat", levels=40), Param("b", "cat", levels=7)]
    perms = np.array(list(itertools.permutations(range(5))), dtype=np.int32)
    rng = np.random.default_rng(4)
    X = [perms[rng.permutation(120)[:60]] for _ in range(4)] + [rng.integers(0, 40, 60).astype(np.int32),
                                                                 rng.integers(0, 7, 60).astype(np.int32)]
    C = [perms] * 4 + [rng.integers(0, 40, 120).astype(np.int32), rng.integers(0, 7, 120).astype(np.int32)]
    space = gp.Space(ps)
    y = rng.normal(size=60)
    model = gp.fit(space, gp.to_device_columns(space, X), dev(y), None, np.ones(6), 1.0, 1e-2)
    t = gp.debug_terms(model, gp.to_device_columns(space, C)).cpu().numpy()
    ref = go.terms(ps, go.encode(ps, C), go.encode(ps, X))
    np.testing.assert_array_equal(t.astype(np.float64), ref)


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_xkernel(name):
    gp = _gp()
    w, space, model, om = fitted(name, 4096)
    order = model.export("FEASIBLE_INDEX").astype(np.int64)
    C = w.candidate_slice(0, 1000)
    K = gp.debug_xkernel(model, gp.to_device_columns(space, C)).double().cpu().numpy()
    encX = [e[order] for e in go.encode(w.space, w.X)]
    ref = go.kernel(w.space, go.encode(w.space, C), encX, w.lengthscale, w.signal_var)
    err = np.abs(K - ref) - (4e-6 * ref + 1e-9)
    assert err.max() <= 0, f"max excess {err.max():.3e}, max rel {(np.abs(K - ref) / ref).max():.3e}"


def _word_expectation(space, t, masks):
    """Expected integer word sums from the oracle's per-parameter terms t[count, n, d]
    (Sec. 4.1): a categorical one-hot field adds 2 per differing category, a Kendall
    word the discordant pairs, a Spearman entry half the sum of squared position
    changes, an equality word [c != x]; a Hamming permutation's two words together hold
    twice its moved items (checked on their sum)."""
    exp = np.zeros(t.shape[:2] + (len(masks),), np.int64)
    ham_pairs = {}
    for w, mk in enumerate(masks):
        for p, prm in enumerate(space):
            if not (mk >> p) & 1:
                continue
            tp = np.rint(t[:, :, p]).astype(np.int64)
            if prm.kind == "cat":
                exp[:, :, w] += 2 * tp if prm.levels <= 32 else tp
            elif prm.dist == "spearman":
                assert np.all(tp % 2 == 0)
                exp[:, :, w] += tp // 2
            elif prm.dist == "hamming":
                ham_pairs.setdefault(p, []).append(w)
                exp[:, :, w] += 2 * tp      # of the pair's sum (first word only)
            else:                           # kendall, naive
                exp[:, :, w] += tp
    return exp, ham_pairs


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_xkernel_pair_sums(name):
    """The production cross-kernel's own integer semimetric sums (its inspection
    instantiation, not a separate kernel) are bit-exact, and the r^2 it feeds to the
    Matern function agrees with the oracle's fp64 r^2 to fp32 rounding."""
    gp = _gp()
    w, space, model, om = fitted(name, 4096)
    order = model.export("FEASIBLE_INDEX").astype(np.int64)
    C = w.candidate_slice(0, 160)
    r2, cnt, masks = gp.debug_pairs(model, gp.to_device_columns(space, C))
    r2 = r2.double().cpu().numpy()
    cnt = cnt.cpu().numpy().astype(np.int64)
    encC = go.encode(w.space, C)
    encX = [e[order] for e in go.encode(w.space, w.X)]
    t = go.terms(w.space, encC, encX)
    # every non-numeric parameter is behind exactly one word (a Hamming one: two)
    cover = np.zeros(len(w.space), int)
    for mk in masks:
        for p in range(len(w.space)):
            cover[p] += (mk >> p) & 1
    for p, prm in enumerate(w.space):
        want = 0 if prm.kind in go.NUMERIC else (2 if prm.kind == "perm" and prm.dist == "hamming" else 1)
        assert cover[p] == want, (p, prm, cover[p])
    exp, ham = _word_expectation(w.space, t, masks)
    for p, (w0, w1) in ham.items():
        np.testing.assert_array_equal(cnt[:, :, w0] + cnt[:, :, w1], exp[:, :, w0])
        cnt[:, :, w0] += cnt[:, :, w1]
        cnt[:, :, w1] = 0
        exp[:, :, w1] = 0
    for wd in range(len(masks)):
        np.testing.assert_array_equal(cnt[:, :, wd], exp[:, :, wd], err_msg=f"word {wd}")
    ref = go.sqdist(w.space, encC, encX, w.lengthscale)
    mag = ref.copy()
    for p, a, b, l in zip(w.space, encC, encX, w.lengthscale):
        if p.kind in go.NUMERIC:
            mag += (np.abs(a.astype(np.float64))[:, None] + np.abs(b.astype(np.float64))[None, :]) ** 2 / l ** 2
    err = np.abs(r2 - ref) / mag
    print(f"{name}: {len(masks)} integer words, max r2 error {err.max():.2e} of the term magnitude")
    assert err.max() <= 1e-6


# ------------------------------------------------------------------ fit
@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_fit_value_model(name):
    w, space, model, om = fitted(name, 4096)
    inf = model.info()
    assert inf["n"] == len(w.y) and inf["n_feasible"] == int(w.feasible.sum())
    K = model.export("K")
    L = model.export("L")
    np.testing.assert_allclose(K, om.K, rtol=1e-13, atol=1e-15)
    recon = np.abs(L @ L.T - K).max() / np.abs(K).max()
    assert recon <= 1e-10, recon
    assert np.all(np.triu(L, 1) == 0)
    Linv = model.export("LINV")
    assert np.abs(Linv @ L - np.eye(len(L))).max() <= 1e-9 * np.linalg.cond(L)
    Kinv = model.export("KINV")
    assert np.abs(Kinv @ K - np.eye(len(K))).max() <= 1e-12 * np.linalg.cond(K)
    alpha = model.export("ALPHA")
    scale = np.abs(om.alpha).max() * np.linalg.cond(K) * 1e-14
    assert np.abs(alpha - om.alpha).max() <= max(scale, 1e-12)
    assert inf["fstar"] == om.fstar


@pytest.mark.parametrize("name", ["C3", "C4"])
def test_fit_classifier(name):
    w, space, model, om = fitted(name, 4096)
    order = model.export("FEASIBLE_INDEX").astype(np.int64)
    f = model.export("CLS_F")
    np.testing.assert_allclose(f, om.cls_f[order], atol=1e-8, rtol=0)
    np.testing.assert_allclose(model.export("CLS_GRAD"), om.cls_grad[order], atol=1e-8, rtol=0)
    np.testing.assert_allclose(model.export("CLS_SQRTW"), om.cls_sw[order], atol=1e-8, rtol=0)
    Lb = model.export("CLS_L")
    sw = model.export("CLS_SQRTW")
    encX = [e[order] for e in go.encode(w.space, w.X)]
    Kc = go.kernel(w.space, encX, encX, w.lengthscale, w.cls_signal_var)
    B = np.eye(len(sw)) + sw[:, None] * Kc * sw[None, :]
    assert np.abs(Lb @ Lb.T - B).max() / np.abs(B).max() <= 1e-10
    assert abs(model.info()["cls_iterations"] - om.cls_iters) <= 1


def test_fit_not_spd_reported():
    gp = _gp()
    w = make_workload("C1", 64)
    X = [np.concatenate([c[:8], c[:1]]) for c in w.X]    # observation 0 duplicated
    y = np.concatenate([w.y[:8], w.y[:1]])
    space = gp.Space(w.space)
    with pytest.raises(gp.GPError) as ei:
        gp.fit(space, gp.to_device_columns(space, X), dev(y), None, w.lengthscale, 1.0, 0.0)
    assert ei.value.status == 2
    assert "pivot" in str(ei.value)
    # the same data with noise fits
    gp.fit(space, gp.to_device_columns(space, X), dev(y), None, w.lengthscale, 1.0, 1e-4)


def test_fit_rejects_invalid_observation():
    gp = _gp()
    w = make_workload("C2", 64)
    X = [c.copy() for c in w.X]
    X[5][3] = [0, 0, 1, 2, 3]
    space = gp.Space(w.space)
    with pytest.raises(gp.GPError) as ei:
        gp.fit(space, gp.to_device_columns(space, X), dev(w.y), None, w.lengthscale, 1.0, 1e-4)
    assert ei.value.status == 1 and "observation 3" in str(ei.value)


# ------------------------------------------------------------------ scoring
@pytest.mark.parametrize("name,M", [("C1", 4096), ("C2", 8192), ("C3", 8192), ("C4", 8192),
                                    ("C5", 2048)])
def test_score_parity(name, M):
    gp = _gp()
    w, space, model, om = fitted(name, M)
    mask = dev(w.mask) if w.mask is not None else None
    out = gp.score(model, gp.to_device_columns(space, w.C), mask=mask, eps_f=w.eps_f)
    ref = go.score(om, w.C, w.mask, w.eps_f)
    check_scores(out, ref, w.signal_var, w.cls_signal_var is not None, f"{name} M={M}")
    nref = gp.refined_count(model, out["_buffers"])
    print(f"{name}: {nref} of {M} candidates recomputed in fp64", flush=True)


# The fp64 recomputation path on its own: mu, sigma and EI come out of fp64 arithmetic
# rounded once to fp32, so they meet a tighter bar than the fp32 path.
REFINE_TOL = 1e-5


def _fit_fresh(w, space):
    gp = _gp()
    return gp.fit(space, gp.to_device_columns(space, w.X), dev(np.nan_to_num(w.y, nan=0.0)),
                  dev(w.feasible), w.lengthscale, w.signal_var, w.noise_var, w.cls_signal_var)


def _score_all_refined(w, label, pick=None):
    """Every candidate (or, with `pick`, the `pick` candidates of largest oracle EI)
    through the fp64 recomputation."""
    gp = _gp()
    space = gp.Space(w.space)
    model = _fit_fresh(w, space)
    gp.debug_set_refine(model, math.inf, -1.0)
    om = go.fit(w.space, w.X, w.y, w.feasible, w.lengthscale, w.signal_var, w.noise_var,
                w.cls_signal_var)
    C, cmask = w.C, w.mask
    if pick is not None:
        idx = np.sort(np.argsort(-go.score(om, w.C, w.mask, w.eps_f)["ei"], kind="stable")[:pick])
        C = [c[idx] for c in w.C]
        cmask = None if w.mask is None else w.mask[idx]
    M = len(C[0])
    mask = dev(cmask) if cmask is not None else None
    out = gp.score(model, gp.to_device_columns(space, C), mask=mask, eps_f=w.eps_f)
    nref = gp.refined_count(model, out["_buffers"])
    assert nref == M, f"{label}: {nref} of {M} candidates refined"
    ref = go.score(om, C, cmask, w.eps_f)
    g = {k: out[k].double().cpu().numpy() for k in ("mu", "sigma", "ei")}
    e_mu = rel_err(g["mu"], ref["mu"], 1.0).max()
    e_sig = rel_err(g["sigma"], ref["sigma"], 1e-2 * math.sqrt(w.signal_var)).max()
    e_ei = rel_err(g["ei"], ref["ei"], 1e-3 * max(ref["ei"].max(), 1e-300)).max()
    msg = f"{label} (all fp64): mu {e_mu:.2e} sigma {e_sig:.2e} ei {e_ei:.2e}"
    print(msg, flush=True)
    assert e_mu <= REFINE_TOL and e_sig <= REFINE_TOL and e_ei <= REFINE_TOL, msg
    check_scores(out, ref, w.signal_var, w.cls_signal_var is not None, label)


@pytest.mark.parametrize("name,M", [("C2", 1000), ("C3", 777), ("C4", 777), ("C5", 300)])
def test_refine_every_candidate(name, M):
    """Every candidate through the fp64 recomputation (thresholds forced open): ragged
    candidate counts against the per-workgroup group of 8 (n_f <= 1920) or 4 (C5)."""
    _score_all_refined(make_workload(name, M), f"{name} M={M}")


@pytest.mark.parametrize("name,M,n,pick", [("C4", 100, None, None), ("C3", 128, None, None),
                                           ("C2", 1, None, None), ("C5", 50, None, None),
                                           ("C1", 301, 4096, 31)])
def test_refine_split_path(name, M, n, pick):
    """Few flagged candidates (at most 16 groups of the per-workgroup group size): the
    recomputation splits each group's triangular product over 64-column ranges and sums
    them in a second pass; includes the largest count that still takes this path (C3:
    16 x 8) and a group size of 2 (n = 4096: the 31 candidates of largest EI among 301,
    as the first 31 have EI below the fp32 range)."""
    w = make_workload(name, M) if n is None else make_workload(name, M, n=n)
    _score_all_refined(w, f"{name} M={M} n={n}", pick)


@pytest.mark.parametrize("name,M", [("C2", 4097), ("C3", 5000), ("C4", 4500), ("C5", 4200)])
def test_refine_block_path(name, M):
    """Many flagged candidates (more than 4096): the recomputation runs as fp64 MFMA
    products over groups of 64 candidates and 256-column tiles of L_f^-T (one tile at
    C2/C3, two at C4, eight at C5), with ragged last groups (4097 = 64 x 64 + 1)."""
    _score_all_refined(make_workload(name, M), f"{name} M={M}")


@pytest.mark.parametrize("n", [2500, 4096])
def test_refine_large_n(n):
    """Large observation counts (up to the library's maximum, 4096): the fp64
    recomputation stages 4, then 2 candidates per workgroup; the fit runs at full size."""
    _score_all_refined(make_workload("C1", 301, n=n), f"C1 n={n} M=301")


@pytest.mark.parametrize("name", ["C3", "C4", "C5"])
def test_score_full_size_sampled(name):
    """Full candidate count (the benchmark's launch configuration); the oracle scores a
    seeded sample of 1536 candidates one by one."""
    gp = _gp()
    w = make_workload(name)
    space = gp.Space(w.space)
    model = gp.fit(space, gp.to_device_columns(space, w.X), dev(np.nan_to_num(w.y, nan=0.0)),
                   dev(w.feasible), w.lengthscale, w.signal_var, w.noise_var, w.cls_signal_var)
    mask = dev(w.mask) if w.mask is not None else None
    out = gp.score(model, gp.to_device_columns(space, w.C), mask=mask, eps_f=w.eps_f,
                   want_argmax=True)
    idx = np.sort(np.random.default_rng(77).choice(w.M, size=1536, replace=False))
    idx[-1] = w.M - 1   # include the ragged tail
    om = go.fit(w.space, w.X, w.y, w.feasible, w.lengthscale, w.signal_var, w.noise_var,
                w.cls_signal_var)
    ref = go.score(om, [c[idx] for c in w.C], None if w.mask is None else w.mask[idx], w.eps_f)
    check_scores(out, ref, w.signal_var, w.cls_signal_var is not None, f"{name} full M={w.M}", idx)
    acq = out["acq"].cpu().numpy()
    am = int(out["argmax"].item())
    assert acq[am] == acq.max() and am == int(np.argmax(acq))


def test_score_ragged_and_edge_cases():
    gp = _gp()
    torch = _torch()
    w, space, model, om = fitted("C3", 4096)
    # ragged M, not a multiple of the 128-row tile, nor of 64
    for M in (1, 77, 1000, 4095):
        C = w.candidate_slice(0, M)
        mask = dev(w.mask[:M])
        out = gp.score(model, gp.to_device_columns(space, C), mask=mask)
        ref = go.score(om, C, w.mask[:M])
        check_scores(out, ref, w.signal_var, True, f"C3 ragged M={M}")
    # M = 0 is a no-op
    gp.score(model, gp.to_device_columns(space, w.candidate_slice(0, 0)))
    C = w.candidate_slice(0, 512)
    dc = gp.to_device_columns(space, C)
    # everything masked -> acq 0; eps_f = 1 -> acq 0 (no probability exceeds 1)
    out = gp.score(model, dc, mask=dev(np.zeros(512, np.uint8)))
    assert torch.all(out["acq"] == 0)
    out = gp.score(model, dc, eps_f=1.0)
    assert torch.all(out["acq"] == 0)
    # deterministic: bit-identical repeated calls
    a = gp.score(model, dc)
    b = gp.score(model, dc)
    for k in ("mu", "sigma", "ei", "acq", "p_feas"):
        assert torch.equal(a[k], b[k]), k


# The classifier's latent mean is one dense column of the contraction, placed in a spare
# 16-column sub-tile of the last value tile (n_f % 128 in 1..112), else of the last
# classifier tile (n % 128 in 1..112), else in a column tile of its own. Observation
# subsets of C4 (359 feasible, 153 infeasible) that take each placement:
@pytest.mark.parametrize("n_feas,n_infeas,where", [
    (359, 153, "last value tile"), (103, 0, "last value tile, n = n_f"),
    (256, 44, "last classifier tile"), (248, 112, "last classifier tile (value tile full)"),
    (256, 128, "own tile"), (248, 136, "own tile (value tile 120 wide)")])
def test_score_latent_mean_column(n_feas, n_infeas, where):
    gp = _gp()
    w = make_workload("C4", 4096)
    fi = np.nonzero(w.feasible)[0][:n_feas]
    ii = np.nonzero(~w.feasible.astype(bool))[0][:n_infeas]
    assert len(fi) == n_feas and len(ii) == n_infeas
    idx = np.sort(np.concatenate([fi, ii]))
    X = [c[idx] for c in w.X]
    y, feas = w.y[idx], w.feasible[idx]
    space = gp.Space(w.space)
    model = gp.fit(space, gp.to_device_columns(space, X), dev(np.nan_to_num(y, nan=0.0)),
                   dev(feas), w.lengthscale, w.signal_var, w.noise_var, w.cls_signal_var)
    om = go.fit(w.space, X, y, feas, w.lengthscale, w.signal_var, w.noise_var,
                w.cls_signal_var)
    out = gp.score(model, gp.to_device_columns(space, w.C), eps_f=w.eps_f)
    ref = go.score(om, w.C, None, w.eps_f)
    check_scores(out, ref, w.signal_var, True, f"C4 n_f={n_feas} n={len(idx)} ({where})")


def _same(a, b):
    return np.array_equal(a.cpu().numpy(), b.cpu().numpy(), equal_nan=True)


@pytest.mark.parametrize("name,M", [("C3", 8192), ("C4", 8192), ("C4", 1000), ("C1", 777),
                                    ("C5", 2048)])
def test_fit_score_equals_fit_then_score(name, M):
    """gp_fit_score overlaps the fit with the first half of scoring on split streams;
    the model and every output must equal those of gp_fit followed by gp_score."""
    gp = _gp()
    torch = _torch()
    w = make_workload(name, M)
    space = gp.Space(w.space)
    X = gp.to_device_columns(space, w.X)
    Cc = gp.to_device_columns(space, w.C)
    y = dev(np.nan_to_num(w.y, nan=0.0))
    feas = dev(w.feasible)
    mask = dev(w.mask) if w.mask is not None else None
    hyp = (w.lengthscale, w.signal_var, w.noise_var, w.cls_signal_var)
    model = gp.fit(space, X, y, feas, *hyp)
    ref = gp.score(model, Cc, mask=mask, eps_f=w.eps_f, want_argmax=True)
    bufs = gp.FitScoreBuffers(space, len(w.y), M, w.cls_signal_var is not None, True, True)
    for rep in range(2):
        m2 = gp.fit_score_into(space, X, y, feas, *hyp, Cc, bufs, mask, w.eps_f)
        torch.cuda.synchronize()
        out = bufs.result()
        for k in ("mu", "sigma", "ei", "acq", "p_feas", "argmax"):
            assert _same(out[k], ref[k]), f"{name} M={M} call {rep}: {k} differs"
        assert m2.info() == model.info()
        assert gp.refined_count(m2, bufs) == gp.refined_count(model, ref["_buffers"])
        # the returned model scores like the one of gp_fit (after a fused step whose
        # classifier's dense column had a tile of its own, later calls find it in the last
        # value tile, as after gp_fit)
        again = gp.score(m2, Cc, mask=mask, eps_f=w.eps_f, want_argmax=True)
        for k in ("mu", "sigma", "ei", "acq", "p_feas", "argmax"):
            assert _same(again[k], ref[k]), f"{name} M={M} call {rep}: rescoring {k} differs"
        del m2


def check_acq_cut(out, ref, eps_f, label, idx=None):
    """acq at a minimum feasible limit eps_f (Sec. 4.2: only probabilities greater than
    eps_f count). Where the oracle's p lies farther from eps_f than the p tolerance the
    cut decision is unique and acq is compared with the oracle's; inside that band
    either decision is valid, so acq must be 0 or the oracle's EI * p."""
    acq = out["acq"].double().cpu().numpy()
    p = out["p_feas"].double().cpu().numpy()
    if idx is not None:
        acq, p = acq[idx], p[idx]
    floor = 1e-3 * max(ref["acq"].max(), 1e-300)
    band = np.abs(ref["p_feas"] - eps_f) <= TOL * np.maximum(ref["p_feas"], 1e-3)
    e = rel_err(acq[~band], ref["acq"][~band], floor)
    cut = int((ref["p_feas"][~band] <= eps_f).sum())
    assert cut > 0, f"{label}: eps_f {eps_f} cuts nothing"
    assert e.max() <= TOL, f"{label}: acq outside the band {e.max():.2e}"
    inb = np.nonzero(band)[0]
    full = ref["ei"][inb] * ref["p_feas"][inb]
    ok = (acq[inb] == 0) | (rel_err(acq[inb], full, floor) <= TOL)
    assert ok.all(), f"{label}: invalid acq inside the band"
    print(f"{label}: eps_f {eps_f}: {cut} cut, {len(inb)} within the band", flush=True)


def check_argmax(out, ref_acq, label):
    """The device's arg-max is a maximiser of the oracle's acquisition values up to the
    score tolerance (ties within it may go either way; exact ties to the lower index)."""
    am = int(out["argmax"].item())
    o = int(np.argmax(ref_acq))
    top = ref_acq[o]
    assert rel_err(np.array([ref_acq[am]]), np.array([top]), 1e-3 * max(top, 1e-300))[0] <= TOL, \
        f"{label}: device arg-max {am} (oracle acq {ref_acq[am]:.6g}) vs oracle {o} ({top:.6g})"
    acq = out["acq"].cpu().numpy()
    assert acq[am] == acq.max() and am == int(np.argmax(acq))
    print(f"{label}: arg-max device {am} oracle {o}", flush=True)


_ORACLE_FULL = {}


def _oracle_full(w, eps_f, idx=None):
    key = (w.name, w.M, eps_f, None if idx is None else len(idx))
    if key not in _ORACLE_FULL:
        om = go.fit(w.space, w.X, w.y, w.feasible, w.lengthscale, w.signal_var, w.noise_var,
                    w.cls_signal_var)
        C = w.C if idx is None else [c[idx] for c in w.C]
        mask = w.mask if (w.mask is None or idx is None) else w.mask[idx]
        _ORACLE_FULL[key] = go.score(om, C, mask, eps_f)
    return _ORACLE_FULL[key]


# The benchmarked call at the benchmarked size: gp_fit_score on the whole candidate set
# (single-split cross-kernel, contraction in two launches on two streams) against
# gp_fit + gp_score bit for bit, and against the oracle on every candidate (at eps_f =
# 0.1 on C4 on a seeded sample of 1536 candidates, to bound the oracle's time).
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,eps_f", [("C3", 0.0), ("C3", 0.1), ("C4", 0.0), ("C4", 0.1)])
def test_fit_score_full_size(name, eps_f):
    gp = _gp()
    torch = _torch()
    w = make_workload(name)
    space = gp.Space(w.space)
    X = gp.to_device_columns(space, w.X)
    Cc = gp.to_device_columns(space, w.C)
    y = dev(np.nan_to_num(w.y, nan=0.0))
    feas = dev(w.feasible)
    mask = dev(w.mask) if w.mask is not None else None
    hyp = (w.lengthscale, w.signal_var, w.noise_var, w.cls_signal_var)
    bufs = gp.FitScoreBuffers(space, len(w.y), w.M, True, True, True)
    gp.fit_score_into(space, X, y, feas, *hyp, Cc, bufs, mask, eps_f)
    torch.cuda.synchronize()
    out = {k: v.clone() for k, v in bufs.result().items() if k != "_buffers"}
    ref = gp.score(gp.fit(space, X, y, feas, *hyp), Cc, mask=mask, eps_f=eps_f,
                   want_argmax=True)
    for k in ("mu", "sigma", "ei", "acq", "p_feas", "argmax"):
        assert _same(out[k], ref[k]), f"{name}: fused {k} differs from gp_fit + gp_score"
    del bufs, ref
    label = f"{name} full M={w.M} fused"
    if name == "C4" and eps_f > 0:
        idx = np.sort(np.random.default_rng(78).choice(w.M, size=1536, replace=False))
        idx[-1] = w.M - 1
        oref = _oracle_full(w, eps_f, idx)
    else:
        idx = None
        oref = _oracle_full(w, eps_f)
    check_scores(out, oref, w.signal_var, True, label, idx, with_acq=eps_f == 0)
    if eps_f > 0:
        check_acq_cut(out, oref, eps_f, label, idx)
    if idx is None:
        check_argmax(out, oref["acq"], label)


@pytest.mark.parametrize("name,M", [("C3", 8192), ("C4", 8192)])
def test_score_eps_cut(name, M):
    """gp_score at a minimum feasible limit of 0.1 (Sec. 4.2) against the oracle."""
    gp = _gp()
    w, space, model, om = fitted(name, M)
    mask = dev(w.mask) if w.mask is not None else None
    out = gp.score(model, gp.to_device_columns(space, w.C), mask=mask, eps_f=0.1,
                   want_argmax=True)
    ref = go.score(om, w.C, w.mask, 0.1)
    check_acq_cut(out, ref, 0.1, f"{name} M={M}")
    check_argmax(out, ref["acq"], f"{name} M={M} eps_f 0.1")


def test_fit_score_errors_leave_nothing_in_flight():
    gp = _gp()
    torch = _torch()
    w = make_workload("C3", 4096)
    space = gp.Space(w.space)
    Cc = gp.to_device_columns(space, w.C)
    y = dev(np.nan_to_num(w.y, nan=0.0))
    feas = dev(w.feasible)
    hyp = (w.lengthscale, w.signal_var, w.noise_var, w.cls_signal_var)
    bufs = gp.FitScoreBuffers(space, len(w.y), 4096, True, True, True)
    bad = [c.copy() for c in w.X]
    bad[0][5] = 1000                                  # an ordinal index out of range
    with pytest.raises(gp.GPError, match="observation 5"):
        gp.fit_score_into(space, gp.to_device_columns(space, bad), y, feas, *hyp, Cc, bufs)
    with pytest.raises(gp.GPError):                   # buffers made for another M
        gp.fit_score_into(space, gp.to_device_columns(space, w.X), y, feas, *hyp,
                          [c[:100] for c in Cc], bufs)
    X = gp.to_device_columns(space, w.X)
    m = gp.fit_score_into(space, X, y, feas, *hyp, Cc, bufs, dev(w.mask))
    torch.cuda.synchronize()
    ref = gp.score(gp.fit(space, X, y, feas, *hyp), Cc, mask=dev(w.mask), want_argmax=True)
    for k in ("mu", "sigma", "ei", "acq", "p_feas", "argmax"):
        assert _same(bufs.result()[k], ref[k]), k
    assert m.info()["n"] == len(w.y)


def test_score_invalid_candidates():
    gp = _gp()
    w, space, model, om = fitted("C2", 4096)
    C = [c[:256].copy() for c in w.C]
    C[5][10] = [1, 1, 2, 3, 4]          # not a permutation
    C[3][11] = 0                        # threads below 1
    C[2][12] = 3                        # schedule level out of range
    out = gp.score(model, gp.to_device_columns(space, C))
    mu = out["mu"].cpu().numpy()
    acq = out["acq"].cpu().numpy()
    pf = out["p_feas"].cpu().numpy()
    for j in (10, 11, 12):
        assert np.isnan(mu[j]) and acq[j] == 0 and pf[j] == 0
    good = np.ones(256, bool)
    good[[10, 11, 12]] = False
    ref = go.score(om, [c[good] for c in C])
    sub = {k: out[k][torch_index(good)] for k in ("mu", "sigma", "ei", "acq")}
    check_scores(sub, ref, w.signal_var, False, "C2 valid subset")


def torch_index(mask):
    torch = _torch()
    return torch.from_numpy(np.nonzero(mask)[0]).cuda()


def test_single_observation_and_no_classifier():
    gp = _gp()
    w = make_workload("C4", 4096)
    X = [c[:1] for c in w.X]
    y = np.array([0.3])
    space = gp.Space(w.space)
    model = gp.fit(space, gp.to_device_columns(space, X), dev(y), None, w.lengthscale, 1.0, 1e-4)
    out = gp.score(model, gp.to_device_columns(space, w.C))
    om = go.fit(w.space, X, y, np.ones(1, np.uint8), w.lengthscale, 1.0, 1e-4)
    ref = go.score(om, w.C)
    check_scores(out, ref, 1.0, False, "n=1")
    assert np.all(out["p_feas"].cpu().numpy() == 1.0)


def test_profile_stages():
    gp = _gp()
    w, space, model, om = fitted("C4", 8192)
    dc = gp.to_device_columns(space, w.C)
    bufs = gp.ScoreBuffers(model, w.M)
    gp.profile_start()
    for _ in range(3):
        gp.score_into(model, dc, bufs)
    prof = gp.profile_stop()
    assert prof["calls"] == 3
    for s in ("encode", "xkernel", "contract", "epilogue", "refine"):
        assert prof[s] > 0, prof


# ------------------------------------------------------------------ local search
def _ls_rows(w, out):
    cols = [c.cpu().numpy() for c in out["cols"]]
    return go.rows_of(w.space, cols, range(len(out["acq"])))


def _same_row(space, a, b):
    for p, u, v in zip(space, a, b):
        if p.kind == "real":
            if abs(u - v) > 1e-12 * max(abs(u), abs(v)):
                return False
        elif u != v:
            return False
    return True


def _check_local_search(w, om, out, ref, acq0, max_steps, label):
    """Device climb against the oracle climb (Sec. 3.3). Unique results are compared
    exactly; where rounding could reorder a decision, the device result is checked for
    validity: a genuine start, an acquisition value matching the oracle's score of the
    configuration it reports, and a local optimum under the oracle's scores."""
    floor = 1e-3 * max(float(acq0.max()), 1e-300)
    k = len(ref["start_index"])
    start = out["start_index"].cpu().numpy()
    acq = out["acq"].double().cpu().numpy()
    steps = out["steps"].cpu().numpy()
    assert len(start) == k and len(set(start.tolist())) == k, label
    # starts: the k largest acquisition values, up to the score tolerance
    e = rel_err(np.sort(acq0[start])[::-1], acq0[ref["start_index"]], floor)
    assert e.max() <= TOL, f"{label}: start values {e.max():.2e}"
    rows = _ls_rows(w, out)
    fin = go.score(om, go.cols_of(w.space, rows))["acq"]
    e = rel_err(acq, fin, floor)
    assert e.max() <= TOL, f"{label}: final acq vs oracle score {e.max():.2e}"
    assert np.all(steps >= 0) and np.all(steps <= max_steps), label
    assert np.all(fin >= acq0[start] - 2 * TOL * np.maximum(acq0[start], floor)), label
    moves = go.neighbour_moves(w.space)
    for s in range(k):
        if steps[s] == max_steps:
            continue
        nbs = [go.apply_move(w.space, rows[s], mv) for mv in moves]
        ok = [nb for nb in nbs if nb is not None]
        if not ok:
            continue
        nb_acq = go.score(om, go.cols_of(w.space, ok))["acq"]
        slack = 2 * TOL * max(fin[s], floor)
        assert nb_acq.max() <= fin[s] + slack, f"{label}: start {s} is not a local optimum"
    # unambiguous oracle paths are reproduced exactly
    exact = 0
    for s in range(k):
        o = int(np.nonzero(ref["start_index"] == start[s])[0][0]) \
            if start[s] in ref["start_index"] else -1
        if o < 0 or ref["margin"][o] <= 4 * TOL * max(ref["acq"][o], floor):
            continue
        assert steps[s] == ref["steps"][o], f"{label}: start {s} steps {steps[s]} vs {ref['steps'][o]}"
        assert _same_row(w.space, rows[s], ref["rows"][o]), f"{label}: start {s} final config"
        exact += 1
    return exact


# C4 and C5 climb through decisions closer than fp32 scoring resolves (oracle margins
# ~2e-5 and ~1e-8 of the acquisition value): there only the validity checks apply.
@pytest.mark.parametrize("name,M,n_starts,max_steps,min_exact", [
    ("C1", 4096, 8, 200, 1), ("C2", 4096, 8, 200, 1), ("C3", 2048, 4, 200, 1),
    ("C4", 2048, 4, 200, 0), ("C5", 1024, 4, 100, 0)])
def test_local_search(name, M, n_starts, max_steps, min_exact):
    gp = _gp()
    w, space, model, om = fitted(name, M)
    C = gp.to_device_columns(space, w.C)
    out = gp.local_search(model, C, None, 0.0, n_starts, max_steps)
    ref = go.local_search(om, w.C, None, 0.0, n_starts, max_steps)
    acq0 = go.score(om, w.C)["acq"]
    exact = _check_local_search(w, om, out, ref, acq0, max_steps, name)
    print(f"{name}: steps {out['steps'].cpu().numpy()} oracle {ref['steps']} exact {exact}")
    assert exact >= min_exact, f"{name}: no start compared exactly"


@pytest.mark.parametrize("name,M,masked", [("C4", 131072, False), ("C4", 131072, True),
                                           ("C2", 131072, False), ("C3", 65536, False)])
def test_local_search_bounded_starts(name, M, masked):
    """From 65,536 candidates on, the starts are chosen with an upper bound of the
    acquisition value from the cross-kernel's mean (only candidates whose bound reaches
    the n_starts-th best value of the best-bounded ones are scored; C3's dense batch
    leaves too many and scores all). The starts and their values must be the n_starts
    best of a full scoring (lower index first on ties)."""
    gp = _gp()
    w = make_workload(name, M)
    space = gp.Space(w.space)
    X = gp.to_device_columns(space, w.X)
    C = gp.to_device_columns(space, w.C)
    model = gp.fit(space, X, dev(np.nan_to_num(w.y, nan=0.0)), dev(w.feasible), w.lengthscale,
                   w.signal_var, w.noise_var, w.cls_signal_var)
    full = gp.score(model, C, eps_f=w.eps_f)["acq"].cpu().numpy()
    mask = None
    if masked:  # the 16 best never start
        m = np.ones(M, np.uint8)
        m[np.lexsort((np.arange(M), -full))[:16]] = 0
        mask = dev(m)
        full = gp.score(model, C, mask=mask, eps_f=w.eps_f)["acq"].cpu().numpy()
    for ns in (16, 5):
        out = gp.local_search(model, C, mask, w.eps_f, ns, 0)
        want = np.lexsort((np.arange(M), -full))[:ns]
        got = out["start_index"].cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=f"{name} M={M} starts={ns}")
        np.testing.assert_allclose(out["acq"].cpu().numpy(), full[want], rtol=1e-6, atol=0,
                                   err_msg=f"{name} M={M} starts={ns}")


def test_local_search_edges():
    gp = _gp()
    torch = _torch()
    w, space, model, om = fitted("C2", 1000)
    C = gp.to_device_columns(space, w.C)
    acq0 = go.score(om, w.C)["acq"]
    # no steps: the starts themselves
    out = gp.local_search(model, C, None, 0.0, 5, 0)
    ref = go.local_search(om, w.C, None, 0.0, 5, 0)
    _check_local_search(w, om, out, ref, acq0, 0, "max_steps=0")
    assert np.all(out["steps"].cpu().numpy() == 0)
    # more starts than candidates, single candidate, a step budget that runs out
    for M, ns, ms in [(3, 8, 50), (1, 4, 50), (200, 6, 2)]:
        Cs = [c[:M] for c in C]
        ws = go.cols_of(w.space, go.rows_of(w.space, w.C, range(M)))
        out = gp.local_search(model, Cs, None, 0.0, ns, ms)
        ref = go.local_search(om, ws, None, 0.0, ns, ms)
        _check_local_search(w, om, out, ref, go.score(om, ws)["acq"], ms, f"M={M}")
        assert len(out["acq"]) == min(ns, M)
    # masked candidates never start: mask out the 16 best
    top = np.lexsort((np.arange(len(acq0)), -acq0))[:16]
    mask = np.ones(len(acq0), np.uint8)
    mask[top] = 0
    out = gp.local_search(model, C, dev(mask), 0.0, 8, 50)
    ref = go.local_search(om, w.C, mask, 0.0, 8, 50)
    assert not set(out["start_index"].cpu().numpy().tolist()) & set(top.tolist())
    acq0m = go.score(om, w.C, mask)["acq"]
    _check_local_search(w, om, out, ref, acq0m, 50, "masked")
    # rejected arguments
    for ns in (0, 65):
        with pytest.raises(gp.GPError):
            gp.local_search(model, C, None, 0.0, ns, 10)
    with pytest.raises(gp.GPError):
        gp.local_search(model, C, None, 0.0, 4, -1)
    torch.cuda.synchronize()
