"""The parity checker itself (CPU): it must reject a result with one wrong point even where
the normwise error stays far inside the tolerance, and the pair-parallel oracle driver must
reproduce the plain oracle call bit for bit."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from paritycheck import ELEM_TOL, KAPPA, TOL, Checker, measures, oracle_pairs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_checker_rejects_one_perturbed_point(dtype):
    rng = np.random.default_rng(11)
    B, N, H, V = 1, 1 << 16, 8, 32
    ref = rng.standard_normal((B, N, H, V))
    tol, etol, kappa = TOL[dtype], ELEM_TOL[dtype], KAPPA[dtype]
    # a correct result: relative noise well inside the tolerance everywhere
    good = ref * (1 + 0.1 * tol * rng.uniform(-1, 1, ref.shape))
    n0, e0 = measures(good, ref, kappa)
    assert n0 <= tol and e0 <= etol
    p = int(np.argmax(np.abs(ref[0, :, 3, :]).max(axis=1) > 1.5))   # a point with a value above 1.5 rms
    for planted in ("zero row", "sign flip", "swapped heads"):
        bad = good.copy()
        if planted == "zero row":
            bad[0, p, 3, :] = 0.0
        elif planted == "sign flip":
            v = int(np.argmax(np.abs(ref[0, p, 3, :])))
            bad[0, p, 3, v] = -bad[0, p, 3, v]
        else:
            bad[0, p, [2, 3], :] = bad[0, p, [3, 2], :]
        n, e = measures(bad, ref, kappa)
        if dtype == "bf16":
            assert n <= tol, (planted, n)      # invisible to the normwise measure ...
        assert e > etol, (planted, e)          # ... but not to the element-wise one
        c = Checker("plant", dtype)
        c.add("out", bad, ref)
        with pytest.raises(AssertionError):
            c.finish()


def test_checker_reports_non_finite():
    ref = np.ones(100)
    got = ref.copy()
    got[5] = np.nan
    assert measures(got, ref, 1.0) == (float("inf"), float("inf"))


def test_oracle_pairs_matches_plain_call():
    for w in (W.Workload("pp_lin", 901, "f32", 2, 300, 3, 16, 16, 32, O.MIX_LINEAR_G,
                         ws_per_head=True, a_per_head=True),
              W.Workload("pp_attn", 902, "bf16", 2, 257, 2, 32, 32, 64, O.MIX_ATTN)):
        inp = W.make_inputs(w)
        f0, b0 = O.run_inputs(inp, w.mix, w.eps)
        f1, b1 = oracle_pairs(O, inp, w.mix, w.eps)
        for k, v in f0.items():
            if v is not None:
                assert np.array_equal(v, f1[k]), (w.name, k)
        for k, v in b0.items():
            assert np.array_equal(v, b1[k]), (w.name, k)
