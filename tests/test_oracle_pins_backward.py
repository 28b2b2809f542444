"""Pins of the oracle's backward pass (gradients of Eq. mita's output with the
top-k sets and routing held fixed).

Two independent references: central finite differences of the (pinned)
forward with the discrete choices frozen, and torch autograd in float64
through library operations (adaptive average pooling, scaled-dot-product
attention, gathers) that compute the same forward. Degenerate cases reduce to
dense attention's gradients.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import mita_oracle as O


def _rng(s=0):
    return np.random.default_rng(s)


def _inputs(N, d, seed):
    r = _rng(seed)
    return (r.standard_normal((N, d)), r.standard_normal((N, d)), r.standard_normal((N, d)),
            r.standard_normal((N, d)))


def _loss(q, k, v, dO, gh, gw, lh, lw, topk, fi, fe, flags, s, sel):
    r = O.forward_slice(q, k, v, gh, gw, lh, lw, topk, None, *flags, force_idx=fi, force_expert=fe, s=s,
                        lm_sel=sel)
    return float((r.o * dO).sum())


CASES = [  # grid, landmark grid, k, flags, s, random selection
    ((3, 4), (2, 2), 5, (1, 1), 1, False),
    ((3, 4), (2, 2), 5, (0, 1), 1, False),
    ((3, 4), (2, 2), 5, (1, 0), 1, False),
    ((3, 5), (2, 3), 4, (1, 1), 2, False),
    ((1, 10), (1, 3), 4, (1, 1), 1, False),
    ((3, 4), (2, 2), 5, (1, 1), 1, True),
]


@pytest.mark.parametrize("case", CASES, ids=[f"g{c[0]}_l{c[1]}_k{c[2]}_f{c[3]}_s{c[4]}_r{int(c[5])}" for c in CASES])
def test_backward_matches_central_differences(case):
    (gh, gw), (lh, lw), topk, flags, s, rnd = case
    N, d = gh * gw, 3
    q, k, v, dO = _inputs(N, d, seed=N + topk + s)
    sel = _rng(3).permutation(N)[:lh * lw] if rnd else None
    base = O.forward_slice(q, k, v, gh, gw, lh, lw, topk, None, *flags, s=s, lm_sel=sel)
    fi, fe = base.idx, base.experts
    g = O.backward_slice(q, k, v, dO, gh, gw, lh, lw, topk, None, *flags, force_idx=fi, force_expert=fe, s=s,
                         lm_sel=sel)
    h = 1e-6
    for name, x, gx in (("q", q, g.dq), ("k", k, g.dk), ("v", v, g.dv)):
        num = np.zeros_like(x)
        for i in range(N):
            for j in range(d):
                xp, xm = x.copy(), x.copy()
                xp[i, j] += h
                xm[i, j] -= h
                args = {"q": q, "k": k, "v": v}
                args[name] = xp
                fp = _loss(args["q"], args["k"], args["v"], dO, gh, gw, lh, lw, topk, fi, fe, flags, s, sel)
                args[name] = xm
                fm = _loss(args["q"], args["k"], args["v"], dO, gh, gw, lh, lw, topk, fi, fe, flags, s, sel)
                num[i, j] = (fp - fm) / (2 * h)
        np.testing.assert_allclose(gx, num, atol=1e-7, rtol=1e-6, err_msg=f"d{name}")


def _torch_forward(q, k, v, gh, gw, lh, lw, idx, ex, scale, flags):
    """The same forward from library ops: adaptive_avg_pool2d for the
    landmarks, SDPA for Eq. landmark-value and for each query's attention
    over [landmarks ; gathered keys] (indices fixed)."""
    N, d = q.shape
    sh, rt = flags
    q_lm = F.adaptive_avg_pool2d(q.T.reshape(1, d, gh, gw), (lh, lw)).reshape(d, -1).T
    v_lm = F.scaled_dot_product_attention(q_lm[None], k[None], v[None], scale=scale)[0]
    keys, vals = [], []
    if sh:
        keys.append(q_lm[None].expand(N, -1, -1))
        vals.append(v_lm[None].expand(N, -1, -1))
    if rt:
        for j in range(ex.shape[1]):
            I = torch.from_numpy(idx[ex[:, j]])              # [N, k]
            keys.append(k[I])
            vals.append(v[I])
    Ks, Vs = torch.cat(keys, 1), torch.cat(vals, 1)
    return F.scaled_dot_product_attention(q[:, None, :], Ks, Vs, scale=scale)[:, 0]


@pytest.mark.parametrize("flags,s", [((1, 1), 1), ((0, 1), 1), ((1, 0), 1), ((1, 1), 2), ((0, 1), 3)])
def test_backward_matches_torch_autograd(flags, s):
    gh, gw, lh, lw, topk, d = 6, 8, 2, 3, 10, 8
    N = gh * gw
    q, k, v, dO = _inputs(N, d, seed=21 + s)
    sc = 1 / np.sqrt(d)
    base = O.forward_slice(q, k, v, gh, gw, lh, lw, topk, None, *flags, s=s)
    g = O.backward_slice(q, k, v, dO, gh, gw, lh, lw, topk, None, *flags, s=s)
    tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
    o = _torch_forward(tq, tk, tv, gh, gw, lh, lw, base.idx, base.experts, sc, flags)
    np.testing.assert_allclose(o.detach().numpy(), base.o, atol=1e-12)
    (o * torch.from_numpy(dO)).sum().backward()
    np.testing.assert_allclose(g.dq, tq.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(g.dk, tk.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(g.dv, tv.grad.numpy(), atol=1e-11)


def test_route_only_k_eq_N_gradients_are_dense_attention_gradients():
    N, d = 20, 4
    q, k, v, dO = _inputs(N, d, seed=5)
    g = O.backward_slice(q, k, v, dO, 4, 5, 1, 1, N, None, 0, 1)
    tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
    o = F.scaled_dot_product_attention(tq[None], tk[None], tv[None])[0]
    (o * torch.from_numpy(dO)).sum().backward()
    for a, b in ((g.dq, tq.grad), (g.dk, tk.grad), (g.dv, tv.grad)):
        np.testing.assert_allclose(a, b.numpy(), atol=1e-12)


def test_pooling_backward_is_the_adjoint_of_pooling():
    # <pool(x), y> == <x, pool^T(y)> for the 14 -> 5 overlapping windows
    r = _rng(9)
    x = r.standard_normal((14 * 14, 3))
    y = r.standard_normal((25, 3))
    lhs = float((O.landmarks(x, 14, 14, 5, 5) * y).sum())
    rhs = float((x * O.pooling_backward(y, 14, 14, 5, 5)).sum())
    assert abs(lhs - rhs) < 1e-12
