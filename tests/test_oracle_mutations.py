"""Planted mistakes in the oracle (CPU only) must each fail at least one pin.

Each mutant is a plausible slip (a wrong tie rule, a dropped term, a wrong
softmax axis, a wrong index or sign); the test swaps it into the oracle module
for the duration of one pin and asserts that pin fails.
"""
import numpy as np
import pytest

from oracle import mita_oracle as O
from tests import test_oracle_pins as P


def _topk_ties_high(S, topk):
    M, N = S.shape
    out = np.empty((M, topk), dtype=np.int64)
    for i in range(M):
        order = np.lexsort((-np.arange(N), -S[i]))
        out[i] = np.sort(order[:topk])
    return out


def _topk_smallest(S, topk):
    return np.sort(np.argsort(S, axis=1, kind="stable")[:, :topk], axis=1)


def _lmv_wrong_axis(S, v):
    w = np.exp(S - S.max(axis=0, keepdims=True))
    return (w / w.sum(axis=0, keepdims=True)) @ v


def _windows_floor_end(G, g):
    return [((i * G) // g, ((i + 1) * G) // g) for i in range(g)]


def _route_argmin(q, q_lm, scale):
    return O.routing_from_expert(np.argmin((q @ q_lm.T) * scale, axis=1), q_lm.shape[0])


def _route_last_max(q, q_lm, scale):
    z = (q @ q_lm.T) * scale
    return O.routing_from_expert(z.shape[1] - 1 - np.argmax(z[:, ::-1], axis=1), q_lm.shape[0])


_orig_out = O.output_per_query


def _out_drop_shared(q, q_lm, v_lm, kx, vx, expert, scale, use_shared=1, use_routed=1):
    return _orig_out(q, q_lm, v_lm, kx, vx, expert, scale, 0, use_routed)


def _out_no_scale(q, q_lm, v_lm, kx, vx, expert, scale, use_shared=1, use_routed=1):
    return _orig_out(q, q_lm, v_lm, kx, vx, expert, 1.0, use_shared, use_routed)


def _out_shared_values_swapped(q, q_lm, v_lm, kx, vx, expert, scale, use_shared=1, use_routed=1):
    return _orig_out(q, q_lm, q_lm, kx, vx, expert, scale, use_shared, use_routed)


MUTANTS = [
    ("topk_indices", _topk_ties_high, lambda: P.test_topk_hand_fixture()),
    ("topk_indices", _topk_smallest, lambda: P.test_topk_bruteforce_all_subsets(2)),
    ("landmark_values", _lmv_wrong_axis, lambda: P.test_landmark_values_equal_sdpa_of_landmark_query()),
    ("pool_windows", _windows_floor_end, lambda: P.test_landmarks_vs_torch_adaptive_avg_pool2d(14, 14, 4, 4)),
    ("route", _route_argmin, lambda: P.test_routing_bruteforce(0)),
    ("route", _route_last_max, lambda: P.test_routing_bruteforce(0)),
    ("output_per_query", _out_drop_shared,
     lambda: P.test_compress_and_route_with_k_eq_N_is_attention_over_augmented_keys()),
    ("output_per_query", _out_no_scale, lambda: P.test_route_only_with_k_eq_N_is_full_attention(2, 3)),
    ("output_per_query", _out_shared_values_swapped, lambda: P.test_compress_only_is_agent_form()),
]


@pytest.mark.parametrize("name,mutant,pin", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_planted_mistake_is_caught(monkeypatch, name, mutant, pin):
    pin()                                    # the pin passes on the real oracle
    monkeypatch.setattr(O, name, mutant)
    with pytest.raises(AssertionError):
        pin()


# ---------------------------------------------------------------- s > 1 and random landmarks
from tests import test_oracle_pins_variants as PV  # noqa: E402


def _route_top_ties_high(q, q_lm, scale, s):
    z = (q @ q_lm.T) * scale
    M = z.shape[1]
    return np.stack([np.lexsort((-np.arange(M), -z[n]))[:s] for n in range(z.shape[0])])


def _route_top_smallest(q, q_lm, scale, s):
    z = (q @ q_lm.T) * scale
    return np.argsort(z, axis=1, kind="stable")[:, :s]


def _out_union_of_experts(q, q_lm, v_lm, kx, vx, expert, scale, use_shared=1, use_routed=1):
    # a plausible misreading: the union of the experts' keys, duplicates dropped
    e = np.asarray(expert)
    if e.ndim == 1:
        return _orig_out(q, q_lm, v_lm, kx, vx, expert, scale, use_shared, use_routed)
    o = np.empty_like(q)
    flat_k = kx.reshape(-1, kx.shape[-1])
    for n in range(q.shape[0]):
        rows = np.unique(np.concatenate([np.arange(kx.shape[1]) + kx.shape[1] * x for x in e[n]]))
        keys = [q_lm] if use_shared else []
        vals = [v_lm] if use_shared else []
        kk = flat_k[rows]
        keys.append(kk)
        vals.append(vx.reshape(-1, vx.shape[-1])[rows])
        # drop rows whose key vector repeats an earlier one
        Ks = np.concatenate(keys)
        _, first = np.unique(Ks, axis=0, return_index=True)
        first = np.sort(first)
        z = (Ks[first] @ q[n]) * scale
        p = np.exp(z - z.max())
        o[n] = (p / p.sum()) @ np.concatenate(vals)[first]
    return o


def _out_first_expert_only(q, q_lm, v_lm, kx, vx, expert, scale, use_shared=1, use_routed=1):
    e = np.asarray(expert)
    return _orig_out(q, q_lm, v_lm, kx, vx, e if e.ndim == 1 else e[:, 0], scale, use_shared, use_routed)


def _landmarks_random_sorted(q, sel):
    return q[np.sort(np.asarray(sel))].copy()


MUTANTS_VARIANTS = [
    ("route_top", _route_top_ties_high, lambda: PV.test_route_top_ties_go_to_the_lower_landmark()),
    ("route_top", _route_top_smallest, lambda: PV.test_route_top_bruteforce(0, 2)),
    ("output_per_query", _out_union_of_experts, lambda: PV.test_duplicate_keys_count_once_per_expert(2)),
    ("output_per_query", _out_first_expert_only, lambda: PV.test_shared_and_routed_k_eq_N_weighs_keys_s_times(2)),
    ("landmarks_random", _landmarks_random_sorted, lambda: PV.test_random_selection_picks_the_drawn_queries()),
]


@pytest.mark.parametrize("name,mutant,pin", MUTANTS_VARIANTS, ids=[m[1].__name__ for m in MUTANTS_VARIANTS])
def test_planted_mistake_in_a_variant_is_caught(monkeypatch, name, mutant, pin):
    pin()
    monkeypatch.setattr(O, name, mutant)
    with pytest.raises(AssertionError):
        pin()


# ---------------------------------------------------------------- backward
from tests import test_oracle_pins_backward as PB  # noqa: E402

_orig_lvb = O.landmark_values_backward
_orig_pb = O.pooling_backward
_orig_ab = O.attention_backward


def _lvb_uncentred(S, q_lm, k, v, dv_lm, scale):
    A = O.softmax_rows(S)
    dS = A * (dv_lm @ v.T)                      # softmax backward without the centring term
    return scale * (dS @ k), scale * (dS.T @ q_lm), A.T @ dv_lm


def _lvb_dk_unscaled(S, q_lm, k, v, dv_lm, scale):
    a, b, c = _orig_lvb(S, q_lm, k, v, dv_lm, scale)
    return a, b / scale, c


def _pb_not_averaged(dq_lm, grid_h, grid_w, lm_h, lm_w):
    rows, cols = O.pool_windows(grid_h, lm_h), O.pool_windows(grid_w, lm_w)
    out = np.zeros((grid_h * grid_w, dq_lm.shape[1]))
    for a, (r0, r1) in enumerate(rows):
        for b, (c0, c1) in enumerate(cols):
            for rr in range(r0, r1):
                out[rr * grid_w + c0: rr * grid_w + c1] += dq_lm[a * lm_w + b]
    return out


def _ab_no_dv_lm(q, dO, q_lm, v_lm, k, v, idx, experts, scale, use_shared=1, use_routed=1):
    dq, dk, dv, dq_lm, dv_lm = _orig_ab(q, dO, q_lm, v_lm, k, v, idx, experts, scale, use_shared, use_routed)
    return dq, dk, dv, dq_lm, 0 * dv_lm         # the shared values' gradient dropped


MUTANTS_BACKWARD = [
    ("landmark_values_backward", _lvb_uncentred, lambda: PB.test_backward_matches_torch_autograd((1, 1), 1)),
    ("landmark_values_backward", _lvb_dk_unscaled, lambda: PB.test_backward_matches_torch_autograd((1, 1), 1)),
    ("pooling_backward", _pb_not_averaged, lambda: PB.test_pooling_backward_is_the_adjoint_of_pooling()),
    ("attention_backward", _ab_no_dv_lm, lambda: PB.test_backward_matches_torch_autograd((1, 0), 1)),
]


@pytest.mark.parametrize("name,mutant,pin", MUTANTS_BACKWARD, ids=[m[1].__name__ for m in MUTANTS_BACKWARD])
def test_planted_mistake_in_the_backward_is_caught(monkeypatch, name, mutant, pin):
    pin()
    monkeypatch.setattr(O, name, mutant)
    with pytest.raises(AssertionError):
        pin()


# ---------------------------------------------------------------- token merging
_orig_tome = O.landmarks_tome


def _tome_sim_dot(XA, XB):
    return XA @ XB.T                            # dot products instead of cosines


def _tome_odd_as_A(q, M):
    # A and B swapped (A = odd positions): emulated by reversing the order of pairs
    N = q.shape[0]
    perm = np.arange(N)
    perm[0:N - N % 2:2], perm[1:N - N % 2:2] = np.arange(1, N - N % 2, 2), np.arange(0, N - N % 2, 2)
    r = _orig_tome(q[perm], M)
    assign = np.empty(N, dtype=np.int64)
    assign[perm] = r.assign
    means = np.stack([q[assign == i].mean(axis=0) for i in range(M)])
    return O.TomeResult(means, assign, r.margins)


MUTANTS_TOME = [
    ("tome_similarity", _tome_sim_dot, lambda: PV.test_tome_merges_by_cosine_not_dot()),
    ("landmarks_tome", _tome_odd_as_A, lambda: PV.test_tome_ties_go_to_the_lower_position()),
]


@pytest.mark.parametrize("name,mutant,pin", MUTANTS_TOME, ids=[m[1].__name__ for m in MUTANTS_TOME])
def test_planted_mistake_in_token_merging_is_caught(monkeypatch, name, mutant, pin):
    pin()
    monkeypatch.setattr(O, name, mutant)
    with pytest.raises(AssertionError):
        pin()
