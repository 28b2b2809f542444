"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each pin compares the oracle with something other than itself: hand-derived
fixtures, brute-force enumeration, library routines (torch's adaptive pooling
and scaled-dot-product attention, heapq), closed forms and invariants. The
degenerate cases come from Sec. 3.2 and Tab. A1 (compress-only, route-only) and
from the definition of Eq. mita (with k = N every expert holds every key).
"""
import heapq
import itertools
import json
import os

import numpy as np
import pytest
import torch

from oracle import mita_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(s=0):
    return np.random.default_rng(s)


def _sdpa(q, K, V, scale):
    """torch scaled_dot_product_attention in float64 on the CPU (library routine)."""
    tq = torch.from_numpy(np.atleast_2d(q))[None]
    tk = torch.from_numpy(K)[None]
    tv = torch.from_numpy(V)[None]
    return torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale)[0].numpy()


def _clustered(N, d, C=4, s=1):
    r = _rng(s)
    cen = r.standard_normal((C, d))
    z = r.integers(0, C, N)
    q = (cen[z] + 0.5 * r.standard_normal((N, d))) / np.sqrt(d)
    k = (cen[z] + 0.5 * r.standard_normal((N, d))) / np.sqrt(d)
    v = r.standard_normal((N, d))
    return q, k, v


# ---------------------------------------------------------------- pooling
def test_pool_windows_hand_fixture():
    cases = json.load(open(os.path.join(GOLDEN, "pool_windows_hand.json")))["cases"]
    for c in cases:
        w = O.pool_windows(c["G"], c["g"])
        if "expect" in c:
            assert [list(x) for x in w] == c["expect"], c
        else:
            u = c["expect_uniform"]
            assert w == [(i * u, (i + 1) * u) for i in range(c["g"])], c


def test_landmarks_divisible_equals_block_mean():
    gh, gw, lh, lw, d = 8, 12, 4, 3, 5
    q = _rng(1).standard_normal((gh * gw, d))
    got = O.landmarks(q, gh, gw, lh, lw)
    blocks = q.reshape(lh, gh // lh, lw, gw // lw, d).mean(axis=(1, 3)).reshape(lh * lw, d)
    np.testing.assert_allclose(got, blocks, rtol=0, atol=1e-14)


@pytest.mark.parametrize("gh,gw,lh,lw", [(14, 14, 4, 4), (14, 14, 5, 5), (32, 32, 7, 7),
                                         (64, 64, 8, 8), (128, 128, 8, 16), (9, 5, 4, 3)])
def test_landmarks_vs_torch_adaptive_avg_pool2d(gh, gw, lh, lw):
    d = 6
    q = _rng(2).standard_normal((gh * gw, d))
    got = O.landmarks(q, gh, gw, lh, lw)
    img = torch.from_numpy(q.T.reshape(d, gh, gw).copy())[None]
    ref = torch.nn.functional.adaptive_avg_pool2d(img, (lh, lw))[0].reshape(d, -1).T.numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("N,M", [(196, 16), (197, 25), (100, 7)])
def test_landmarks_1d_vs_torch_adaptive_avg_pool1d(N, M):
    d = 4
    q = _rng(3).standard_normal((N, d))
    got = O.landmarks(q, 1, N, 1, M)
    ref = torch.nn.functional.adaptive_avg_pool1d(torch.from_numpy(q.T.copy())[None], M)[0].T.numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-13)


def test_single_landmark_is_global_mean():
    q = _rng(4).standard_normal((35, 3))
    np.testing.assert_allclose(O.landmarks(q, 5, 7, 1, 1)[0], q.sum(0) / 35, atol=1e-14)


# ---------------------------------------------------------------- scores
def test_scores_elementwise_dot():
    r = _rng(5)
    ql, k = r.standard_normal((3, 4)), r.standard_normal((6, 4))
    S = O.scores(ql, k, 0.5)
    for i in range(3):
        for n in range(6):
            acc = 0.0
            for j in range(4):
                acc += ql[i, j] * k[n, j]
            assert abs(S[i, n] - 0.5 * acc) < 1e-14


# ---------------------------------------------------------------- top-k
def _precedes(s, a, b):
    """a comes before b in the (larger score, then lower index) order."""
    return s[a] > s[b] or (s[a] == s[b] and a < b)


def _topk_bruteforce(s, k):
    N = len(s)
    winners = []
    for sub in itertools.combinations(range(N), k):
        inside = set(sub)
        if all(_precedes(s, a, b) for a in inside for b in range(N) if b not in inside):
            winners.append(sub)
    assert len(winners) == 1       # the total order makes the set unique
    return list(winners[0])


@pytest.mark.parametrize("seed", range(12))
def test_topk_bruteforce_all_subsets(seed):
    r = _rng(100 + seed)
    N = int(r.integers(1, 11))
    M = 3
    if seed % 3 == 0:
        S = r.integers(-2, 3, size=(M, N)).astype(np.float64)       # many ties
    elif seed % 3 == 1:
        S = r.choice([-0.0, 0.0, 1.0, -np.inf, np.inf, 5e-324], size=(M, N))
    else:
        S = r.standard_normal((M, N))
    for k in range(1, N + 1):
        got = O.topk_indices(S, k)
        for i in range(M):
            assert list(got[i]) == _topk_bruteforce(S[i], k), (S[i], k)


def test_topk_hand_fixture():
    cases = json.load(open(os.path.join(GOLDEN, "topk_hand.json")))["cases"]
    for c in cases:
        s = np.array([float(x) for x in c["scores"]])[None]
        assert list(O.topk_indices(s, c["k"])[0]) == c["expect"], c


@pytest.mark.parametrize("seed", range(4))
def test_topk_vs_heapq(seed):
    r = _rng(200 + seed)
    N = 300
    S = np.round(r.standard_normal((4, N)) * 3) / 3          # quantised: many ties
    S[:, ::17] = -0.0
    for k in (1, 7, 64, N):
        got = O.topk_indices(S, k)
        for i in range(4):
            # (score, -index) tuples: the largest come first by score, then by lower index
            best = heapq.nlargest(k, ((S[i, n] + 0.0, -n) for n in range(N)))
            assert list(got[i]) == sorted(-m for _, m in best)


def test_topk_k1_is_first_argmax_and_kN_is_all():
    S = _rng(6).integers(0, 4, size=(5, 40)).astype(np.float64)
    assert (O.topk_indices(S, 1)[:, 0] == np.argmax(S, axis=1)).all()
    assert (O.topk_indices(S, 40) == np.arange(40)).all()


# ---------------------------------------------------------------- landmark values
def test_landmark_values_equal_sdpa_of_landmark_query():
    q, k, v = _clustered(50, 8)
    ql = O.landmarks(q, 5, 10, 2, 3)
    sc = 1 / np.sqrt(8)
    got = O.landmark_values(O.scores(ql, k, sc), v)
    for i in range(ql.shape[0]):
        np.testing.assert_allclose(got[i], _sdpa(ql[i], k, v, sc)[0], atol=1e-13)


def test_landmark_weights_are_a_distribution():
    S = _rng(7).standard_normal((4, 30)) * 10
    w = O.softmax_rows(S)
    assert (w >= 0).all()
    np.testing.assert_allclose(w.sum(1), 1, atol=1e-14)


# ---------------------------------------------------------------- routing
@pytest.mark.parametrize("seed", range(3))
def test_routing_bruteforce(seed):
    r = _rng(300 + seed)
    N, M, d = 60, 7, 3
    q = r.integers(-2, 3, size=(N, d)).astype(np.float64)        # integer logits: ties
    ql = r.integers(-2, 3, size=(M, d)).astype(np.float64)
    ql[3] = ql[1]                                                 # a duplicated landmark
    rt = O.route(q, ql, 0.5)
    for n in range(N):
        best, arg = None, None
        for i in range(M):
            z = 0.5 * sum(q[n, j] * ql[i, j] for j in range(d))
            if best is None or z > best:
                best, arg = z, i
        assert rt.expert[n] == arg
    assert rt.offsets[0] == 0 and rt.offsets[-1] == N
    assert sorted(rt.perm.tolist()) == list(range(N))
    for i in range(M):
        grp = rt.perm[rt.offsets[i]:rt.offsets[i + 1]]
        assert (rt.expert[grp] == i).all()
        assert (np.diff(grp) > 0).all()


def test_single_landmark_routes_everything_to_it():
    q = _rng(8).standard_normal((20, 4))
    rt = O.route(q, q.mean(0, keepdims=True), 0.5)
    assert (rt.expert == 0).all() and (rt.perm == np.arange(20)).all()


# ---------------------------------------------------------------- outputs
def _slice(N=48, d=8, gh=6, gw=8, lh=2, lw=3, k=10, seed=9, **kw):
    q, kk, v = _clustered(N, d, s=seed)
    return q, kk, v, O.forward_slice(q, kk, v, gh, gw, lh, lw, k, **kw)


@pytest.mark.parametrize("lh,lw", [(1, 1), (2, 3)])
def test_route_only_with_k_eq_N_is_full_attention(lh, lw):
    q, k, v, r = _slice(k=48, lh=lh, lw=lw, use_shared=0)
    np.testing.assert_allclose(r.o, _sdpa(q, k, v, 1 / np.sqrt(8)), atol=1e-12)


def test_compress_and_route_with_k_eq_N_is_attention_over_augmented_keys():
    q, k, v, r = _slice(k=48)
    ref = _sdpa(q, np.concatenate([r.q_lm, k]), np.concatenate([r.v_lm, v]), 1 / np.sqrt(8))
    np.testing.assert_allclose(r.o, ref, atol=1e-12)


def test_compress_only_is_agent_form():
    q, k, v, r = _slice(use_routed=0)
    sc = 1 / np.sqrt(8)
    v_lm = _sdpa(r.q_lm, k, v, sc)
    np.testing.assert_allclose(r.o, _sdpa(q, r.q_lm, v_lm, sc), atol=1e-12)


def test_output_is_sdpa_over_shared_plus_routed_keys():
    q, k, v, r = _slice()
    sc = 1 / np.sqrt(8)
    for n in range(q.shape[0]):
        I = r.idx[r.routing.expert[n]]
        ref = _sdpa(q[n], np.concatenate([r.q_lm, k[I]]), np.concatenate([r.v_lm, v[I]]), sc)[0]
        np.testing.assert_allclose(r.o[n], ref, atol=1e-12)


@pytest.mark.parametrize("flags", [(1, 1), (0, 1), (1, 0)])
def test_per_query_form_equals_grouped_lse_form(flags):
    q, k, v, r = _slice(N=96, gh=8, gw=12, lh=2, lw=3, k=13, seed=11,
                        use_shared=flags[0], use_routed=flags[1])
    kx, vx = O.gather(k, v, r.idx)
    g = O.output_grouped(q, r.q_lm, r.v_lm, kx, vx, r.routing, 1 / np.sqrt(8), *flags)
    np.testing.assert_allclose(r.o, g, atol=1e-12)


def test_convexity_and_effective_weights():
    q, k, v, r = _slice()
    W = O.effective_weights(q, k, r.q_lm, r.S, r.idx, r.routing.expert, 1 / np.sqrt(8))
    assert (W >= 0).all()
    np.testing.assert_allclose(W.sum(1), 1, atol=1e-13)
    np.testing.assert_allclose(W @ v, r.o, atol=1e-12)
    assert (r.o <= v.max(0) + 1e-12).all() and (r.o >= v.min(0) - 1e-12).all()


def test_affine_equivariance_in_v():
    q, k, v, r = _slice()
    b = _rng(12).standard_normal(8)
    r2 = O.forward_slice(q, k, 2.5 * v + b, 6, 8, 2, 3, 10)
    np.testing.assert_allclose(r2.o, 2.5 * r.o + b, atol=1e-12)
    assert (r2.idx == r.idx).all()


def test_slices_are_independent():
    r = _rng(13)
    q, k, v = (r.standard_normal((2, 3, 24, 4)) for _ in range(3))
    o, _ = O.forward(q, k, v, 4, 6, 2, 2, 5)
    o1 = O.forward_slice(q[1, 2], k[1, 2], v[1, 2], 4, 6, 2, 2, 5).o
    np.testing.assert_array_equal(o[1, 2], o1)


def test_forced_selection_reproduces_own_selection():
    q, k, v, r = _slice()
    r2 = O.forward_slice(q, k, v, 6, 8, 2, 3, 10, force_idx=r.idx, force_expert=r.routing.expert)
    np.testing.assert_array_equal(r.o, r2.o)


def test_rows_subset_matches_full():
    q, k, v, r = _slice()
    rows = [0, 5, 47]
    r2 = O.forward_slice(q, k, v, 6, 8, 2, 3, 10, rows=rows)
    np.testing.assert_array_equal(r2.o, r.o[rows])
