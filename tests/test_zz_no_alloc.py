"""gp_score_noalloc (scoring with the library's fixed device scratch array instead of a
caller workspace) against gp_score, through the C-ABI: two calls in a row, the second
with fewer candidates, each bit-identical to gp_score and within the oracle tolerance on
a sample; the size limit is enforced with a clear error."""
import math

import numpy as np
import pytest

from oracle import gp_oracle as go
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _same(a, b):
    return np.array_equal(a.cpu().numpy(), b.cpu().numpy(), equal_nan=True)


def test_score_noalloc_matches_gp_score():
    import torch
    from paper_2212_11142_amd import gp
    w = make_workload("C4", 24000)
    space = gp.Space(w.space)
    model = gp.fit(space, gp.to_device_columns(space, w.X),
                   torch.from_numpy(np.nan_to_num(w.y, nan=0.0)).cuda(),
                   torch.from_numpy(w.feasible).cuda(), w.lengthscale, w.signal_var,
                   w.noise_var, w.cls_signal_var)
    cap = gp.score_noalloc_max(model)
    assert 24000 <= cap < 10 ** 6, cap
    om = go.fit(w.space, w.X, w.y, w.feasible, w.lengthscale, w.signal_var, w.noise_var,
                w.cls_signal_var)
    for M in (24000, 3001):                 # the second call is smaller: stale scratch
        C = w.candidate_slice(0, M)
        dc = gp.to_device_columns(space, C)
        got = gp.score_noalloc(model, dc, eps_f=0.1, want_argmax=True)
        ref = gp.score(model, dc, eps_f=0.1, want_argmax=True)
        torch.cuda.synchronize()
        for k in ("mu", "sigma", "ei", "p_feas", "acq", "argmax"):
            assert _same(got[k], ref[k]), f"M={M}: {k} differs from gp_score"
        idx = np.sort(np.random.default_rng(M).choice(M, size=256, replace=False))
        oref = go.score(om, [c[idx] for c in C], None, 0.1)
        for k, floor in (("mu", 1.0), ("sigma", 1e-2 * math.sqrt(w.signal_var)),
                         ("ei", 1e-3 * oref["ei"].max()), ("p_feas", 1e-3)):
            g = got[k].double().cpu().numpy()[idx]
            e = np.max(np.abs(g - oref[k]) / np.maximum(np.abs(oref[k]), floor))
            assert e <= 1e-4, (M, k, e)
    # one candidate more than the array holds is rejected before any device work
    one = gp.to_device_columns(space, w.candidate_slice(0, 1))
    big = [torch.zeros((cap + 1,) + tuple(c.shape[1:]), dtype=c.dtype, device="cuda") for c in one]
    with pytest.raises(gp.GPError) as ei:
        gp.score_noalloc(model, big)
    assert ei.value.status == 5 and "scratch" in str(ei.value)
