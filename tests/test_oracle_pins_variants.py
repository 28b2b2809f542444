"""Pins of the oracle's s > 1 routing and random-selection landmarks.

s > 1 (Sec. 3.2, Eq. mita): e_j(q) is the rank-j expert under the routing
logits, and K* = [Q_lm, K^(e_1), ..., K^(e_s)] has m + k s columns, so a key
that two of the query's experts select enters the softmax twice. Each pin
compares the oracle with something other than itself: brute-force ranking,
hand-derived tie fixtures with exactly representable logits, and torch's
scaled-dot-product attention with an additive log-multiplicity bias (a key
present c times weighs c exp(z), i.e. exp(z + log c)).

Random selection (Tab. A1, landmark extraction): landmark i is the query of
token sel[i].
"""
import numpy as np
import pytest
import torch

from oracle import mita_oracle as O


def _rng(s=0):
    return np.random.default_rng(s)


def _sdpa_bias(q, K, V, scale, bias):
    """torch SDPA in float64 on the CPU with an additive per-key bias."""
    tq = torch.from_numpy(np.atleast_2d(q))[None]
    tk = torch.from_numpy(K)[None]
    tv = torch.from_numpy(V)[None]
    tb = torch.from_numpy(np.broadcast_to(bias, (tq.shape[1], K.shape[0])).copy())[None]
    return torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=tb, scale=scale)[0].numpy()


def _clustered(N, d, C=4, s=1):
    r = _rng(s)
    cen = r.standard_normal((C, d))
    z = r.integers(0, C, N)
    q = (cen[z] + 0.5 * r.standard_normal((N, d))) / np.sqrt(d)
    k = (cen[z] + 0.5 * r.standard_normal((N, d))) / np.sqrt(d)
    v = r.standard_normal((N, d))
    return q, k, v


# ---------------------------------------------------------------- top-s routing
@pytest.mark.parametrize("seed,s", [(0, 2), (1, 3), (2, 4), (3, 6)])
def test_route_top_bruteforce(seed, s):
    r = _rng(seed)
    q = r.standard_normal((30, 5))
    q_lm = r.standard_normal((7, 5))
    ex = O.route_top(q, q_lm, 0.7, s)
    for n in range(30):
        z = [float(q[n] @ q_lm[i]) * 0.7 for i in range(7)]
        ranked = sorted(range(7), key=lambda i: (-z[i], i))
        assert list(ex[n]) == ranked[:s]


def test_route_top_ties_go_to_the_lower_landmark():
    # integer vectors: every logit is an exact small integer, so ties are exact
    q_lm = np.array([[1, 0], [2, 0], [1, 0], [2, 0], [0, 3]], dtype=np.float64)
    q = np.array([[1, 0], [0, 1], [-1, 0]], dtype=np.float64)
    ex = O.route_top(q, q_lm, 1.0, 4)
    # token 0: logits [1, 2, 1, 2, 0] -> 1, 3, 0, 2
    # token 1: logits [0, 0, 0, 0, 3] -> 4, 0, 1, 2
    # token 2: logits [-1, -2, -1, -2, 0] -> 4, 0, 2, 1
    assert ex.tolist() == [[1, 3, 0, 2], [4, 0, 1, 2], [4, 0, 2, 1]]


def test_route_top_one_is_the_argmax_routing():
    q, _, _ = _clustered(64, 8, s=3)
    q_lm = O.landmarks(q, 8, 8, 2, 2)
    np.testing.assert_array_equal(O.route_top(q, q_lm, 0.3, 1)[:, 0], O.route(q, q_lm, 0.3).expert)


def test_pair_grouping_hand_fixture():
    # N = 3 queries, s = 2, M = 3: pairs p = 2 n + j
    ex = np.array([[2, 0], [0, 2], [2, 1]])
    g = O.pair_grouping(ex, 3)
    # groups: p0 -> 2, p1 -> 3 + 0, p2 -> 0, p3 -> 3 + 2, p4 -> 2, p5 -> 3 + 1
    assert g.expert.tolist() == [2, 3, 0, 5, 2, 4]
    assert g.perm.tolist() == [2, 0, 4, 1, 5, 3]
    assert g.offsets.tolist() == [0, 1, 1, 3, 4, 5, 6]


# ---------------------------------------------------------------- s > 1 outputs
def _slice(N=48, d=8, gh=6, gw=8, lh=2, lw=3, k=10, seed=9, **kw):
    q, kk, v = _clustered(N, d, s=seed)
    return q, kk, v, O.forward_slice(q, kk, v, gh, gw, lh, lw, k, **kw)


@pytest.mark.parametrize("s", [2, 3, 6])
def test_route_only_k_eq_N_any_s_is_full_attention(s):
    # every expert holds every key: each key enters s times, which cancels
    q, k, v, r = _slice(k=48, use_shared=0, s=s)
    np.testing.assert_allclose(r.o, _sdpa_bias(q, k, v, 1 / np.sqrt(8), 0.0), atol=1e-12)


@pytest.mark.parametrize("s", [2, 5])
def test_shared_and_routed_k_eq_N_weighs_keys_s_times(s):
    q, k, v, r = _slice(k=48, s=s)
    bias = np.concatenate([np.zeros(6), np.full(48, np.log(s))])
    ref = _sdpa_bias(q, np.concatenate([r.q_lm, k]), np.concatenate([r.v_lm, v]), 1 / np.sqrt(8), bias)
    np.testing.assert_allclose(r.o, ref, atol=1e-12)


@pytest.mark.parametrize("s", [2, 3])
def test_duplicate_keys_count_once_per_expert(s):
    # experts overlap (clustered data, k = 20 of 48): per query, attention over
    # the distinct keys with bias log(multiplicity)
    q, k, v, r = _slice(k=20, s=s, seed=4)
    sc = 1 / np.sqrt(8)
    overlaps = 0
    for n in range(q.shape[0]):
        sel = np.concatenate([r.idx[e] for e in r.experts[n]])
        keys, mult = np.unique(sel, return_counts=True)
        overlaps += int((mult > 1).sum())
        bias = np.concatenate([np.zeros(6), np.log(mult)])
        ref = _sdpa_bias(q[n], np.concatenate([r.q_lm, k[keys]]), np.concatenate([r.v_lm, v[keys]]), sc, bias)[0]
        np.testing.assert_allclose(r.o[n], ref, atol=1e-12)
    assert overlaps > 0  # the case the pin is about does occur


@pytest.mark.parametrize("flags,s", [((1, 1), 2), ((0, 1), 3), ((1, 1), 4), ((1, 0), 2)])
def test_pair_form_equals_per_query_form(flags, s):
    q, k, v, r = _slice(N=96, gh=8, gw=12, lh=2, lw=3, k=13, seed=11, s=s,
                        use_shared=flags[0], use_routed=flags[1])
    kx, vx = O.gather(k, v, r.idx)
    g = O.output_pairs(q, r.q_lm, r.v_lm, kx, vx, r.experts, 1 / np.sqrt(8), *flags)
    np.testing.assert_allclose(r.o, g, atol=1e-12)


def test_s_effective_weights_reproduce_the_output():
    q, k, v, r = _slice(s=3)
    W = O.effective_weights(q, k, r.q_lm, r.S, r.idx, r.experts, 1 / np.sqrt(8))
    assert (W >= 0).all()
    np.testing.assert_allclose(W.sum(1), 1, atol=1e-13)
    np.testing.assert_allclose(W @ v, r.o, atol=1e-12)


def test_s_one_matches_the_default_path():
    q, k, v, r1 = _slice()
    r2 = O.forward_slice(q, k, v, 6, 8, 2, 3, 10, s=1)
    np.testing.assert_array_equal(r1.o, r2.o)
    assert r2.experts.shape == (48, 1)


# ---------------------------------------------------------------- random selection
def test_random_selection_picks_the_drawn_queries():
    q = _rng(5).standard_normal((40, 6))
    sel = np.array([17, 3, 39, 0])
    q_lm = O.landmarks_random(q, sel)
    for i, t in enumerate(sel):
        np.testing.assert_array_equal(q_lm[i], q[t])


def test_random_selection_of_every_token_equals_unit_window_pooling():
    q = _rng(6).standard_normal((24, 5))
    np.testing.assert_array_equal(O.landmarks_random(q, np.arange(24)), O.landmarks(q, 4, 6, 4, 6))


def test_random_landmarks_forward_is_sdpa_over_shared_plus_routed_keys():
    q, k, v = _clustered(48, 8, s=7)
    sel = _rng(7).permutation(48)[:6]
    r = O.forward_slice(q, k, v, 6, 8, 2, 3, 10, lm_sel=sel)
    np.testing.assert_array_equal(r.q_lm, q[sel])
    sc = 1 / np.sqrt(8)
    v_lm = np.stack([_sdpa_bias(q[t], k, v, sc, 0.0)[0] for t in sel])
    np.testing.assert_allclose(r.v_lm, v_lm, atol=1e-12)
    for n in range(48):
        I = r.idx[r.experts[n, 0]]
        ref = _sdpa_bias(q[n], np.concatenate([r.q_lm, k[I]]), np.concatenate([v_lm, v[I]]), sc, 0.0)[0]
        np.testing.assert_allclose(r.o[n], ref, atol=1e-12)


# ---------------------------------------------------------------- token merging (ToMe)
def test_tome_merges_by_cosine_not_dot():
    # positions 0 (A), 1 (B), 2 (A), 3 (B); M = 3: one edge merges.
    # A0 = (1, 0): cosine 0.707 with B1 = (10, 10), 0.994 with B3 = (0.9, 0.1)
    # (a dot product would prefer B1); A2 = (0, 1): 0.707 with B1, 0.110 with B3.
    # Edge scores 0.994 (A0) > 0.707 (A2): A0 joins B3.
    q = np.array([[1, 0], [10, 10], [0, 1], [0.9, 0.1]], dtype=np.float64)
    r = O.landmarks_tome(q, 3)
    np.testing.assert_allclose(r.q_lm, [[10, 10], [0, 1], [0.95, 0.05]], atol=1e-15)
    assert r.assign.tolist() == [2, 0, 1, 2]


def test_tome_ties_go_to_the_lower_position():
    # A0 = (1, 0) has cosine 1 with both B1 = (2, 0) and B3 = (3, 0): B1 (lower).
    # A2 = (0, 1) has cosine 0 with both: B1. Edge scores 1 (A0), 0 (A2).
    q = np.array([[1, 0], [2, 0], [0, 1], [3, 0]], dtype=np.float64)
    r3 = O.landmarks_tome(q, 3)                 # one edge: A0 -> B1
    np.testing.assert_allclose(r3.q_lm, [[1.5, 0], [0, 1], [3, 0]], atol=1e-15)
    r2 = O.landmarks_tome(q, 2)                 # both edges: A0, A2 -> B1
    np.testing.assert_allclose(r2.q_lm, [[1, 1 / 3], [3, 0]], atol=1e-15)
    assert r2.assign.tolist() == [0, 0, 0, 1]


def test_tome_twins_merge_with_each_other():
    # tokens in identical pairs at (2i, 2i + 1), pairs far apart: one round
    # with M = N / 2 merges every A token into its twin
    r = _rng(31)
    base = r.standard_normal((12, 16))
    q = np.repeat(base, 2, axis=0)
    t = O.landmarks_tome(q, 12)
    np.testing.assert_allclose(t.q_lm, base, atol=1e-14)
    assert t.assign.tolist() == [i // 2 for i in range(24)]


def test_tome_with_M_eq_N_merges_nothing():
    q = _rng(32).standard_normal((20, 5))
    t = O.landmarks_tome(q, 20)
    np.testing.assert_array_equal(t.q_lm, q)
    assert t.assign.tolist() == list(range(20))


@pytest.mark.parametrize("N,M", [(196, 25), (196, 16), (100, 7), (64, 63), (33, 1)])
def test_tome_landmarks_are_means_of_a_partition(N, M):
    q = _rng(N + M).standard_normal((N, 6))
    t = O.landmarks_tome(q, M)
    assert t.assign.min() == 0 and t.assign.max() == M - 1
    assert (np.bincount(t.assign, minlength=M) > 0).all()
    for i in range(M):
        np.testing.assert_allclose(t.q_lm[i], q[t.assign == i].mean(axis=0), atol=1e-13)


def test_tome_is_invariant_to_a_positive_scale():
    q = _rng(33).standard_normal((64, 8))
    a, b = O.landmarks_tome(q, 10), O.landmarks_tome(3.5 * q, 10)
    np.testing.assert_array_equal(a.assign, b.assign)
    np.testing.assert_allclose(b.q_lm, 3.5 * a.q_lm, atol=1e-13)
