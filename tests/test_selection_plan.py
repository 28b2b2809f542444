"""The fused top-k selection's plan (host only, no GPU): for every workload,
the pivot rank and list cap the library chooses keep each way a row's
candidate list can miss at or below 1e-9 per row, evaluated independently
with scipy's hypergeometric law.

Model (the same the library states): a row's scores are exchangeable over
token positions, so the ns evenly spaced sampled keys are a uniform random
ns-subset of the N tokens. The list (tokens scoring >= the r-th largest
sample) is shorter than k only if at least r samples fall among the row's
first k - 1 tokens, and longer than cap only if fewer than r samples fall
among its first cap tokens."""
import os

import pytest
from scipy.stats import hypergeom

from paper_2602_01219_amd import mita, synth

EPS = 1e-9


def _plan(wl):
    if not os.path.exists(mita.LIB_PATH):
        pytest.skip("libmita.so not built")
    return mita.select_plan(mita.Config.from_workload(wl))


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER + synth.OPERATING_ORDER)
def test_overflow_bounds_per_row(name):
    wl = synth.WORKLOADS[name]
    p = _plan(wl)
    N, k = wl.N, wl.k
    if not p["fused"]:
        # only the dense-equivalence mode (k = N beyond the sample) stores S
        assert k > N // 2, (name, p)
        return
    ns, r, cap = p["ns"], p["rank"], p["cap"]
    if ns == N:  # the sample is the row: the pivot is the k-th score itself
        assert r == k and cap >= N
        return
    short = hypergeom(N, k - 1, ns).sf(r - 1)              # P(X >= r)
    long_ = 0.0 if cap >= N else hypergeom(N, cap, ns).cdf(r - 1)  # P(Y < r)
    print(f"{name}: ns {ns} rank {r} cap {cap}: P(short) {short:.2e}, P(long) {long_:.2e}")
    assert short <= EPS and long_ <= EPS
    # the rank is the smallest meeting the bound (no needless candidates)
    assert hypergeom(N, k - 1, ns).sf(r - 2) > EPS


def test_headline_plan():
    p = _plan(synth.WORKLOADS["dense_pred_bf16"])
    assert p == {"fused": 1, "ns": 1024, "rank": 69, "cap": 2048}


def test_long_sequence_cap_meets_its_bound():
    # the cap the earlier fixed rule clamped at 4096 (below its own bound)
    p = _plan(synth.WORKLOADS["long_bf16"])
    assert p["fused"] and p["cap"] == 8192
    assert hypergeom(65536, 4096, 1024).cdf(p["rank"] - 1) > EPS      # 4096 would not do
    assert hypergeom(65536, 8192, 1024).cdf(p["rank"] - 1) <= EPS
