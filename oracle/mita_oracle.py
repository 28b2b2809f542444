"""CPU oracle for the MiTA forward pass (Mixture-of-Top-k Attention, arXiv 2602.01219).

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or run
this module: only the tests, the smoke check and the benchmark's CPU-baseline
leg use it. It shares no code with the HIP library (no kernels, headers,
tables or helpers) and it never imports the package.

Plain, slow and written to be checked by eye against the paper. Arithmetic is
numpy float64 on the exact input values (bf16/fp32 inputs widened exactly);
given float32 arrays it computes in float32 instead (the CPU timing baseline).
Everything is per (batch, head) slice; nothing is shared across slices.

Notation follows Sec. 3.2 with tokens as rows: q, k, v are [N, d] (the paper's
Q, K, V in R^{d x N} have tokens as columns), landmarks q_lm, v_lm are [M, d]
(the paper's m is M here), the expert width is k (here `topk`).

Steps, in the order of Algorithm 1 (Appendix B):
  1. landmark queries by adaptive average pooling over the token grid
     (Sec. 3.2, landmark queries; Tab. A1: 2-D pooling is the default)
  2. scores S = K^T q_lm / sqrt(d)                 (Eq. top-k; Algorithm 1)
  3. I_i = Top_k(S[i, :])                           (Eq. top-k)
  4. K^(i) = K[:, I_i], V^(i) = V[:, I_i]           (Eq. gather)
  5. v_lm_i = Atten(q_lm_i, K, V)                   (Eq. landmark-value)
  6. e(q) = argmax_i q . q_lm_i (routing logits Q^T Q_lm, Sec. 3.2)
  7. MiTA(q) = V* softmax(K*^T q / sqrt(d)),  K* = [Q_lm, K^(e_1(q)), ...,
     K^(e_s(q))], V* likewise                       (Eq. mita)
A second formulation (Algorithm 1's grouped form: shared-expert attention,
varlen attention over queries grouped by expert, log-sum-exp combine; for
s > 1 the expert-wise form with one partial per (query, expert) pair that
Sec. 3.2 allows) is provided for cross-checking step 7.
Landmark queries may also come from random selection of M tokens (Tab. A1),
the draw being an input.
The backward pass (backward_slice) gives the gradients of the output with
respect to q, k and v by the chain rule through Eq. mita, Eq. landmark-value
and the pooling, the top-k sets and the routing held fixed (they are
piecewise constant in the inputs and take no gradient).

Readings where the paper is silent or ambiguous:
  * pooling windows: start = floor(i*G/g), end = ceil((i+1)*G/g) per axis
    (the adaptive-average-pool rule Algorithm 1 names); 1-D pooling when
    grid_h == 1.
  * top-k order: larger score first, equal scores by lower token index;
    -0 == +0; the index set is returned ascending.
  * selection uses the scaled scores S (Algorithm 1), which Eq. landmark-value's
    softmax also uses.
  * routing: e(q) is the lowest landmark index attaining the maximum of
    (q . q_lm_i) / sqrt(d); counts are the bincount of e (minlength M),
    offsets = [0, cumsum(counts)], grouping is stable.
  * s > 1: e_j(q) is the j-th landmark in the order (larger logit first,
    equal logits by lower landmark index); K* concatenates the s experts' key
    sets as Eq. mita writes them (m + k s columns), so a key selected by two
    of the query's experts enters the softmax twice.
  * random selection: landmark i is the query of token sel[i], sel being M
    distinct token indices supplied by the caller.
  * token merging (ToMe) as landmark extraction (Tab. A1 names it; bipartite
    soft matching, applied repeatedly): see landmarks_tome.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np


# ----------------------------------------------------------------------------
# Step 1: landmark queries (Sec. 3.2, average pooling over uniformly spaced
# windows; Algorithm 1's AdaptiveAvgPool; Tab. A1 default is 2-D pooling).
# ----------------------------------------------------------------------------
def pool_windows(G: int, g: int) -> list[tuple[int, int]]:
    """Adaptive pooling windows splitting G positions into g windows:
    window i covers [floor(i*G/g), ceil((i+1)*G/g))."""
    return [((i * G) // g, -((-(i + 1) * G) // g)) for i in range(g)]


def landmarks(q: np.ndarray, grid_h: int, grid_w: int, lm_h: int, lm_w: int) -> np.ndarray:
    """q: [N, d] with token t at grid position (t // grid_w, t % grid_w).
    Returns q_lm [M, d], M = lm_h * lm_w, landmark i at (i // lm_w, i % lm_w)
    is the arithmetic mean of q over its 2-D window."""
    N, d = q.shape
    assert N == grid_h * grid_w
    grid = q.reshape(grid_h, grid_w, d)
    rows = pool_windows(grid_h, lm_h)
    cols = pool_windows(grid_w, lm_w)
    out = np.empty((lm_h * lm_w, d), dtype=q.dtype)
    for a, (r0, r1) in enumerate(rows):
        for b, (c0, c1) in enumerate(cols):
            out[a * lm_w + b] = grid[r0:r1, c0:c1, :].reshape(-1, d).mean(axis=0)
    return out


def landmarks_random(q: np.ndarray, sel) -> np.ndarray:
    """Random selection (Tab. A1, landmark extraction): landmark i is the
    query of token sel[i]; sel [M] holds distinct token indices drawn by the
    caller. Returns q_lm [M, d]."""
    sel = np.asarray(sel, dtype=np.int64)
    assert sel.ndim == 1 and len(np.unique(sel)) == len(sel)
    assert sel.min() >= 0 and sel.max() < q.shape[0]
    return q[sel].copy()


@dataclass
class TomeResult:
    q_lm: np.ndarray       # [M, d] landmark queries (means of their members)
    assign: np.ndarray     # [N] landmark of every token
    margins: list          # per round: (smallest gap between an A token's best and second-best
                           # similarity, gap between the r-th and (r+1)-th edge), for parity budgets


def tome_similarity(XA: np.ndarray, XB: np.ndarray) -> np.ndarray:
    """Cosine similarity of every A token with every B token (rows: merged
    queries)."""
    na = XA / np.linalg.norm(XA, axis=1, keepdims=True)
    nb = XB / np.linalg.norm(XB, axis=1, keepdims=True)
    return na @ nb.T


def landmarks_tome(q: np.ndarray, M: int) -> TomeResult:
    """Token merging as landmark extraction (Tab. A1; bipartite soft matching
    applied in rounds until M tokens remain). A round over the current
    sequence of n merged tokens (each the mean of its original members, in
    sequence order):
      1. A = the tokens at even positions, B = those at odd positions;
      2. each A token's match is the B token of largest cosine similarity of
         the merged queries (ties: lower B position), its edge score that
         similarity;
      3. the r = min(n - M, |A|) edges of largest score (ties: lower A
         position) merge: each of those A tokens joins its match;
      4. the survivors (unmerged A tokens and all B tokens) keep their order.
    The landmarks are the final tokens' means, in sequence order."""
    N, d = q.shape
    assert 1 <= M <= N
    groups = [[t] for t in range(N)]            # members of each current token, in sequence order
    margins = []
    while len(groups) > M:
        n = len(groups)
        X = np.stack([q[g].mean(axis=0) for g in groups])
        A = list(range(0, n, 2))
        B = list(range(1, n, 2))
        sim = tome_similarity(X[A], X[B])        # [|A|, |B|]
        match = np.empty(len(A), dtype=np.int64)
        score = np.empty(len(A))
        gap_best = np.inf
        for i in range(len(A)):
            order = np.lexsort((np.arange(len(B)), -sim[i]))
            match[i] = order[0]
            score[i] = sim[i, order[0]]
            if len(B) > 1:
                gap_best = min(gap_best, sim[i, order[0]] - sim[i, order[1]])
        r = min(n - M, len(A))
        eorder = np.lexsort((np.arange(len(A)), -score))
        merged = set(eorder[:r].tolist())
        gap_edge = score[eorder[r - 1]] - score[eorder[r]] if r < len(A) else np.inf
        margins.append((gap_best, gap_edge))
        new_groups = {}
        for i in sorted(merged):                 # A tokens join their matches, in A order
            new_groups.setdefault(match[i], []).extend(groups[A[i]])
        out = []
        for j in range(n):
            if j % 2 == 0:
                if j // 2 not in merged:
                    out.append(groups[j])
            else:
                out.append(groups[j] + new_groups.get(j // 2, []))
        groups = out
    assign = np.empty(N, dtype=np.int64)
    for i, g in enumerate(groups):
        assign[g] = i
    q_lm = np.stack([q[g].mean(axis=0) for g in groups])
    return TomeResult(q_lm, assign, margins)


# ----------------------------------------------------------------------------
# Step 2: landmark-key scores (Eq. top-k; Algorithm 1 scales by 1/sqrt(d)).
# ----------------------------------------------------------------------------
def scores(q_lm: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """S[i, n] = (q_lm_i . k_n) * scale, shape [M, N]."""
    return (q_lm @ k.T) * scale


# ----------------------------------------------------------------------------
# Step 3: top-k selection per landmark (Eq. top-k).
# ----------------------------------------------------------------------------
def topk_indices(S: np.ndarray, topk: int) -> np.ndarray:
    """For each row of S [M, N], the topk token indices that come first in the
    order (larger score first, then lower index), returned ascending.
    Returns int64 [M, topk]."""
    M, N = S.shape
    assert 1 <= topk <= N
    idx = np.empty((M, topk), dtype=np.int64)
    n = np.arange(N)
    for i in range(M):
        order = np.lexsort((n, -S[i]))      # primary: -S ascending; secondary: n ascending
        idx[i] = np.sort(order[:topk])
    return idx


# ----------------------------------------------------------------------------
# Step 4: gather (Eq. gather).
# ----------------------------------------------------------------------------
def gather(k: np.ndarray, v: np.ndarray, idx: np.ndarray):
    """Expert tiles K^(i) = K[I_i], V^(i) = V[I_i]: [M, topk, d] each."""
    return k[idx], v[idx]


# ----------------------------------------------------------------------------
# Step 5: landmark values (Eq. landmark-value): v_lm_i = Atten(q_lm_i, K, V),
# the softmax running over the N keys of landmark i.
# ----------------------------------------------------------------------------
def softmax_rows(z: np.ndarray) -> np.ndarray:
    w = np.exp(z - z.max(axis=-1, keepdims=True))
    return w / w.sum(axis=-1, keepdims=True)


def landmark_values(S: np.ndarray, v: np.ndarray) -> np.ndarray:
    return softmax_rows(S) @ v


# ----------------------------------------------------------------------------
# Step 6: routing (Sec. 3.2: logits Q^T Q_lm; rank-1 expert e_1(q); Algorithm 1
# ArgMax / ArgSort / BinCount / CumSum).
# ----------------------------------------------------------------------------
@dataclass
class Routing:
    expert: np.ndarray     # [N] int64, e(q) in [0, M)
    counts: np.ndarray     # [M] int64
    offsets: np.ndarray    # [M+1] int64, offsets[0] = 0, offsets[M] = N
    perm: np.ndarray       # [N] int64, tokens grouped by expert, ascending within a group


def route(q: np.ndarray, q_lm: np.ndarray, scale: float) -> Routing:
    logits = (q @ q_lm.T) * scale               # [N, M]
    expert = np.argmax(logits, axis=1)          # first maximum = lowest landmark index
    return routing_from_expert(expert, q_lm.shape[0])


def route_top(q: np.ndarray, q_lm: np.ndarray, scale: float, s: int) -> np.ndarray:
    """The s experts of every query (Sec. 3.2: e_j(q) is the rank-j expert
    under the logits Q^T Q_lm): landmarks ordered by larger logit first, equal
    logits by lower landmark index. Returns int64 [N, s], rank order."""
    logits = (q @ q_lm.T) * scale               # [N, M]
    N, M = logits.shape
    assert 1 <= s <= M
    out = np.empty((N, s), dtype=np.int64)
    lm = np.arange(M)
    for n in range(N):
        order = np.lexsort((lm, -logits[n]))    # primary: -logit; secondary: landmark index
        out[n] = order[:s]
    return out


def pair_grouping(experts: np.ndarray, M: int) -> Routing:
    """Grouping of the (query, rank) pairs of s > 1 routing for the
    expert-wise computation: pair p = n * s + j goes to group e_j(n) when
    j = 0 (the pairs that also carry the shared expert) and to group
    M + e_j(n) otherwise; groups are stable in the pair id. Returns a Routing
    over the 2 M groups whose expert field holds the group of each pair."""
    experts = np.asarray(experts, dtype=np.int64)
    N, s = experts.shape
    group = experts + M * (np.arange(s)[None, :] > 0)
    return routing_from_expert(group.reshape(-1), 2 * M)


def routing_from_expert(expert: np.ndarray, M: int) -> Routing:
    expert = np.asarray(expert, dtype=np.int64)
    counts = np.bincount(expert, minlength=M)
    offsets = np.concatenate([[0], np.cumsum(counts)])
    perm = np.argsort(expert, kind="stable")
    return Routing(expert, counts, offsets, perm)


# ----------------------------------------------------------------------------
# Step 7: the MiTA output (Eq. mita), per query.
# ----------------------------------------------------------------------------
def _experts_2d(expert) -> np.ndarray:
    e = np.asarray(expert, dtype=np.int64)
    return e[:, None] if e.ndim == 1 else e


def output_per_query(q, q_lm, v_lm, kx, vx, expert, scale, use_shared=1, use_routed=1):
    """o_n = V* softmax(K*^T q_n * scale) with K* = [q_lm ; kx[e_1(n)] ; ... ;
    kx[e_s(n)]] and V* likewise (either part dropped by its flag); expert is
    [N] (s = 1) or [N, s] in rank order."""
    N, d = q.shape
    ex = _experts_2d(expert)
    o = np.empty((N, d), dtype=q.dtype)
    for n in range(N):
        keys, vals = [], []
        if use_shared:
            keys.append(q_lm)
            vals.append(v_lm)
        if use_routed:
            for e in ex[n]:
                keys.append(kx[e])
                vals.append(vx[e])
        Ks = np.concatenate(keys, axis=0)
        Vs = np.concatenate(vals, axis=0)
        p = softmax_rows((Ks @ q[n]) * scale)
        o[n] = p @ Vs
    return o


def output_grouped(q, q_lm, v_lm, kx, vx, routing: Routing, scale, use_shared=1, use_routed=1):
    """Algorithm 1's form: shared-expert attention and per-expert (varlen)
    attention over queries grouped by expert, each with its log-sum-exp,
    combined by online-softmax weights (Sec. 3.2, computing expert-wise and
    combining). Returns o [N, d]."""
    N, d = q.shape
    parts = []
    if use_shared:
        z = (q @ q_lm.T) * scale                      # [N, M]
        mx = z.max(axis=1, keepdims=True)
        w = np.exp(z - mx)
        s = w.sum(axis=1, keepdims=True)
        parts.append(((w @ v_lm) / s, (mx + np.log(s))[:, 0]))
    if use_routed:
        o_e = np.empty((N, d))
        lse_e = np.empty(N)
        qs = q[routing.perm]
        for i in range(q_lm.shape[0]):
            a, b = routing.offsets[i], routing.offsets[i + 1]
            if a == b:
                continue
            z = (qs[a:b] @ kx[i].T) * scale
            mx = z.max(axis=1, keepdims=True)
            w = np.exp(z - mx)
            s = w.sum(axis=1, keepdims=True)
            rows = routing.perm[a:b]                   # scatter back to token order
            o_e[rows] = (w @ vx[i]) / s
            lse_e[rows] = (mx + np.log(s))[:, 0]
        parts.append((o_e, lse_e))
    if len(parts) == 1:
        return parts[0][0]
    (o1, l1), (o2, l2) = parts
    mx = np.maximum(l1, l2)
    w1 = np.exp(l1 - mx)[:, None]
    w2 = np.exp(l2 - mx)[:, None]
    return (w1 * o1 + w2 * o2) / (w1 + w2)


def output_pairs(q, q_lm, v_lm, kx, vx, experts, scale, use_shared=1, use_routed=1):
    """The expert-wise form of Eq. mita for s >= 1 (Sec. 3.2: attention
    computed per expert and combined by online softmax): for every expert,
    attention of the (query, rank) pairs routed to it over its k keys, each
    pair keeping its log-sum-exp; the shared-expert attention of every query
    likewise; each query's s + 1 partials combined with weights
    exp(lse - max lse). Returns o [N, d]."""
    N, d = q.shape
    ex = _experts_2d(experts)
    s = ex.shape[1]
    outs, lses = [], []
    if use_shared:
        z = (q @ q_lm.T) * scale
        mx = z.max(axis=1, keepdims=True)
        w = np.exp(z - mx)
        sm = w.sum(axis=1, keepdims=True)
        outs.append((w @ v_lm) / sm)
        lses.append((mx + np.log(sm))[:, 0])
    if use_routed:
        for j in range(s):
            o_j = np.empty((N, d))
            l_j = np.empty(N)
            for e in range(q_lm.shape[0]):
                rows = np.nonzero(ex[:, j] == e)[0]
                if len(rows) == 0:
                    continue
                z = (q[rows] @ kx[e].T) * scale
                mx = z.max(axis=1, keepdims=True)
                w = np.exp(z - mx)
                sm = w.sum(axis=1, keepdims=True)
                o_j[rows] = (w @ vx[e]) / sm
                l_j[rows] = (mx + np.log(sm))[:, 0]
            outs.append(o_j)
            lses.append(l_j)
    L = np.stack(lses, axis=1)                          # [N, parts]
    wts = np.exp(L - L.max(axis=1, keepdims=True))
    num = sum(wts[:, i:i + 1] * outs[i] for i in range(len(outs)))
    return num / wts.sum(axis=1, keepdims=True)


def effective_weights(q, k, q_lm, S, idx, expert, scale, use_shared=1, use_routed=1):
    """W [N, N] with o = W v: the shared part spreads landmark j's weight over
    the keys through softmax(S[j, :]) (Eq. landmark-value), the routed part puts
    its weights on the selected keys. Tiny inputs only."""
    N = q.shape[0]
    A = softmax_rows(S)
    W = np.zeros((N, N))
    M = q_lm.shape[0]
    ex = _experts_2d(expert)
    for n in range(N):
        z = []
        if use_shared:
            z.append((q_lm @ q[n]) * scale)
        if use_routed:
            for e in ex[n]:
                z.append((k[idx[e]] @ q[n]) * scale)
        p = softmax_rows(np.concatenate(z))
        j = 0
        if use_shared:
            W[n] += p[:M] @ A
            j = M
        if use_routed:
            for e in ex[n]:                              # repeated keys add up
                np.add.at(W[n], idx[e], p[j:j + idx.shape[1]])
                j += idx.shape[1]
    return W


# ----------------------------------------------------------------------------
# The whole forward over [B, H, N, d] inputs.
# ----------------------------------------------------------------------------
@dataclass
class SliceResult:
    q_lm: np.ndarray
    S: np.ndarray
    idx: np.ndarray
    v_lm: np.ndarray
    routing: Routing        # grouping by the rank-1 expert
    o: np.ndarray
    experts: np.ndarray     # [N, s] routed experts in rank order


def forward_slice(q, k, v, grid_h, grid_w, lm_h, lm_w, topk, scale=None,
                  use_shared=1, use_routed=1, force_idx=None, force_expert=None,
                  rows=None, s=1, lm_sel=None, q_lm=None) -> SliceResult:
    """One (b, h) slice of the forward. force_idx / force_expert replace the
    oracle's own selection / routing (to compare outputs given another
    implementation's discrete choices; force_expert is [N] or [N, s]). rows:
    compute o only for these tokens (o is then [len(rows), d]). s: routed
    experts per query. Landmarks come from pooling, or from random selection
    when lm_sel (the M drawn token indices) is given, or are q_lm when given."""
    N, d = q.shape
    if scale is None:
        scale = float(1.0 / np.sqrt(d))
    if q_lm is None:
        q_lm = landmarks(q, grid_h, grid_w, lm_h, lm_w) if lm_sel is None else landmarks_random(q, lm_sel)
    S = scores(q_lm, k, scale)
    idx = topk_indices(S, topk) if force_idx is None else np.asarray(force_idx, dtype=np.int64)
    v_lm = landmark_values(S, v)
    if force_expert is None:
        experts = route(q, q_lm, scale).expert[:, None] if s == 1 else route_top(q, q_lm, scale, s)
    else:
        experts = _experts_2d(force_expert)
    routing = routing_from_expert(experts[:, 0], q_lm.shape[0])
    kx, vx = gather(k, v, idx)
    if rows is None:
        o = output_per_query(q, q_lm, v_lm, kx, vx, experts, scale, use_shared, use_routed)
    else:
        rows = np.asarray(rows)
        o = output_per_query(q[rows], q_lm, v_lm, kx, vx, experts[rows], scale,
                             use_shared, use_routed)
    return SliceResult(q_lm, S, idx, v_lm, routing, o, experts)


def forward(q, k, v, grid_h, grid_w, lm_h, lm_w, topk, scale=None, use_shared=1,
            use_routed=1, s=1, lm_sel=None):
    """q, k, v: [B, H, N, d] float64; lm_sel: [B, H, M] random-selection
    draws or None (pooling). Returns o [B, H, N, d] and the per-slice results
    (a list in (b, h) order)."""
    B, H, N, d = q.shape
    o = np.empty((B, H, N, d))
    res = []
    for b in range(B):
        for h in range(H):
            r = forward_slice(q[b, h], k[b, h], v[b, h], grid_h, grid_w, lm_h, lm_w,
                              topk, scale, use_shared, use_routed, s=s,
                              lm_sel=None if lm_sel is None else lm_sel[b, h])
            o[b, h] = r.o
            res.append(r)
    return o, res


# ----------------------------------------------------------------------------
# Backward pass: gradients of o with respect to q, k, v for an upstream
# gradient dO, by the chain rule through step 7 (Eq. mita), step 5 (Eq.
# landmark-value) and step 1 (pooling). The top-k sets I_i and the experts
# e_j(q) are held fixed: they change only where a score or logit crosses
# another, so the output is differentiable with them constant.
# ----------------------------------------------------------------------------
@dataclass
class Grads:
    dq: np.ndarray
    dk: np.ndarray
    dv: np.ndarray
    dq_lm: np.ndarray      # gradient reaching the landmark queries (before pooling)
    dv_lm: np.ndarray      # gradient reaching the landmark values


def attention_backward(q, dO, q_lm, v_lm, k, v, idx, experts, scale, use_shared=1, use_routed=1):
    """Step 7 backward, per query: z = K*^T q * scale, p = softmax(z),
    o = V* p. Returns (dq [N, d], dk [N, d], dv [N, d], dq_lm [M, d],
    dv_lm [M, d]): the routed keys' gradients land on their token rows, the
    shared keys' on the landmark rows."""
    N, d = q.shape
    M = q_lm.shape[0]
    dq, dk, dv = np.zeros((N, d)), np.zeros((N, d)), np.zeros((N, d))
    dq_lm, dv_lm = np.zeros((M, d)), np.zeros((M, d))
    for n in range(N):
        keys, vals = [], []
        if use_shared:
            keys.append(q_lm)
            vals.append(v_lm)
        if use_routed:
            for e in experts[n]:
                keys.append(k[idx[e]])
                vals.append(v[idx[e]])
        Ks = np.concatenate(keys)
        Vs = np.concatenate(vals)
        p = softmax_rows((Ks @ q[n]) * scale)
        dp = Vs @ dO[n]                         # dL/dp_j = dO . v*_j
        dz = p * (dp - p @ dp)                  # softmax backward
        dq[n] += scale * (dz @ Ks)
        j = 0
        if use_shared:
            dq_lm += scale * np.outer(dz[:M], q[n])
            dv_lm += np.outer(p[:M], dO[n])
            j = M
        if use_routed:
            for e in experts[n]:
                I = idx[e]
                np.add.at(dk, I, scale * np.outer(dz[j:j + len(I)], q[n]))
                np.add.at(dv, I, np.outer(p[j:j + len(I)], dO[n]))
                j += len(I)
    return dq, dk, dv, dq_lm, dv_lm


def landmark_values_backward(S, q_lm, k, v, dv_lm, scale):
    """Step 5 backward: v_lm = A v with A = softmax(S) over the N keys and
    S = q_lm k^T * scale. Returns (dq_lm, dk, dv) contributions."""
    A = softmax_rows(S)
    dA = dv_lm @ v.T
    dS = A * (dA - (A * dA).sum(axis=1, keepdims=True))
    return scale * (dS @ k), scale * (dS.T @ q_lm), A.T @ dv_lm


def pooling_backward(dq_lm, grid_h, grid_w, lm_h, lm_w):
    """Step 1 backward: q_lm_i is the mean of q over window W_i, so each token
    of W_i receives dq_lm_i / |W_i|. Returns dq [N, d]."""
    M, d = dq_lm.shape
    dq = np.zeros((grid_h * grid_w, d))
    rows = pool_windows(grid_h, lm_h)
    cols = pool_windows(grid_w, lm_w)
    for a, (r0, r1) in enumerate(rows):
        for b, (c0, c1) in enumerate(cols):
            cnt = (r1 - r0) * (c1 - c0)
            for rr in range(r0, r1):
                dq[rr * grid_w + c0: rr * grid_w + c1] += dq_lm[a * lm_w + b] / cnt
    return dq


def backward_slice(q, k, v, dO, grid_h, grid_w, lm_h, lm_w, topk, scale=None,
                   use_shared=1, use_routed=1, force_idx=None, force_expert=None,
                   s=1, lm_sel=None) -> Grads:
    """One (b, h) slice: dq, dk, dv [N, d] for upstream gradient dO [N, d]."""
    N, d = q.shape
    if scale is None:
        scale = float(1.0 / np.sqrt(d))
    r = forward_slice(q, k, v, grid_h, grid_w, lm_h, lm_w, topk, scale, use_shared, use_routed,
                      force_idx, force_expert, s=s, lm_sel=lm_sel)
    dq, dk, dv, dq_lm, dv_lm = attention_backward(q, dO, r.q_lm, r.v_lm, k, v, r.idx, r.experts, scale,
                                                  use_shared, use_routed)
    if use_shared:
        a, b, c = landmark_values_backward(r.S, r.q_lm, k, v, dv_lm, scale)
        dq_lm = dq_lm + a
        dk = dk + b
        dv = dv + c
    if lm_sel is not None:                      # random selection: q_lm_i = q[sel_i]
        np.add.at(dq, np.asarray(lm_sel, dtype=np.int64), dq_lm)
    else:
        dq = dq + pooling_backward(dq_lm, grid_h, grid_w, lm_h, lm_w)
    return Grads(dq, dk, dv, dq_lm, dv_lm)
