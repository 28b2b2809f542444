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
