"""CPU oracle of the token-condensation MoE layer (Luffy, arXiv 2411.15419).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
and the CPU-baseline leg of the benchmark may import it.  It shares no code
with the HIP path; both consume the arrays drawn by ``luffy_gen``.

It is a plain, slow, fp64 statement of what the layer computes, one function
per step, in the paper's order:

  gate      Sec. 2.1: the gate network picks experts for every token
            (top-2 in the paper's setup, Sec. 2.2 and Sec. 7.1; top-1 also
            supported).
  dispatch  Sec. 2.1: tokens are grouped by the expert that will run them.
  cosine    Sec. 2.2: token similarity is the cosine of the embeddings.
  adjacency Sec. 5.1 step 1 (pairs routed to different experts are never
            similar -> similarity only inside a bucket) and step 3 (true
            cosine for the remaining pairs); Sec. 5.2: edges whose weight is
            below the threshold are deleted.
  historical_weights, historical_record
            Sec. 5.1 step 2 (a NEXT piece with no GPU path): pairs whose
            previous-block similarity is above S1 / below S2 take weight
            1 / 0 without a cosine; condense(history=...) uses them.
  greedy    Sec. 5.2: in the thresholded graph keep the highest-degree token,
            condense its neighbours, repeat until every token is decided.
  ffn       Sec. 2.1: an expert is an FFN; Sec. 3: only the kept token of a
            similar group goes through the expert.
  combine   Sec. 2.1: expert outputs are brought back into sequence order;
            Sec. 6: a condensed token takes the expert output of the token
            that replaced it (token_to_token(i) = j).

Readings of points the paper leaves open (each is a keyword so tests can show
the alternatives):
  * similarity: the raw cosine, edge iff cos >= h (sim_mode="raw");
    "clamp" = max(0, cos) and "affine" = (1 + cos)/2 are the two readings of
    the "normalized cosine in [0,1]" of Sec. 2.2.
  * a zero-norm token has cosine 0 with everything.
  * degree: counted once in the full thresholded bucket graph
    (degree_mode="static"); "dynamic" recounts in the residual graph after
    every pick.
  * ties in degree go to the lower bucket position; a token next to several
    kept tokens joins the first one picked (the one of highest priority).
  * a group is a star: the kept token absorbs only its direct neighbours.
  * gates: softmax over all experts; top-1 uses the probability itself,
    top-2 renormalises over the two chosen experts; every slot keeps its own
    gate, only the expert output is shared.
  * bucket order is stable over slot id s = j*T + t (all first choices,
    then all second choices); with a capacity C the first C slots of a
    bucket are kept and the rest dropped before condensation; a dropped slot
    contributes nothing and tokens with no kept slot get a zero output.
  * FFN: two matrices, no bias, act = exact (erf) GELU or SiLU.
"""
from __future__ import annotations

import math
from types import SimpleNamespace

import numpy as np
from scipy.special import erf as _erf

__all__ = [
    "gate", "dispatch", "cosine", "adjacency", "greedy", "condense",
    "activation", "expert_ffn", "combine", "moe_layer", "capacity_of",
    "adaptive_threshold", "activation_grad", "combine_backward", "expert_ffn_backward",
]


# --------------------------------------------------------------------------
# 1. Gate (Sec. 2.1)
# --------------------------------------------------------------------------
def gate(x, w_g, b_g, k):
    """Gate network: logits = x W_g^T + b_g, p = softmax(logits), the top-k
    experts by descending logit (ties: lower expert id first).

    Returns (topk_idx int32 [T,k], topk_gate float64 [T,k], logits [T,E]).
    """
    x = np.asarray(x, np.float64)
    w = np.asarray(w_g, np.float64)
    logits = x @ w.T
    if b_g is not None:
        logits = logits + np.asarray(b_g, np.float64)[None, :]
    m = logits.max(axis=1, keepdims=True)
    ex = np.exp(logits - m)
    p = ex / ex.sum(axis=1, keepdims=True)
    order = np.argsort(-logits, axis=1, kind="stable")
    topk_idx = order[:, :k].astype(np.int32)
    chosen = np.take_along_axis(p, topk_idx.astype(np.int64), axis=1)
    if k == 1:
        topk_gate = chosen
    else:
        topk_gate = chosen / chosen.sum(axis=1, keepdims=True)
    return topk_idx, topk_gate, logits


def capacity_of(T, k, E, cf):
    """Capacity per expert, ceil(cf*k*T/E) slots; 0 = unlimited."""
    if cf is None or cf <= 0:
        return 0
    return int(math.ceil(cf * k * T / E - 1e-9))


# --------------------------------------------------------------------------
# 2. Dispatch order (Sec. 2.1)
# --------------------------------------------------------------------------
def dispatch(topk_idx, E, capacity=0):
    """Group slots by expert.

    A slot is (token t, choice j); its id is s = j*T + t.  Bucket e lists the
    slots routed to e in ascending slot id; with capacity C > 0 only the first
    C stay.  Buckets are laid out one after another in expert order.

    Returns offsets int32 [E+1], perm_token int32 [S] (token of each bucket
    position), slot_pos int32 [T,k] (bucket position of each slot, -1 when
    dropped).
    """
    topk_idx = np.asarray(topk_idx)
    T, k = topk_idx.shape
    buckets = [[] for _ in range(E)]
    for s in range(k * T):
        t, j = s % T, s // T
        e = int(topk_idx[t, j])
        if capacity > 0 and len(buckets[e]) >= capacity:
            continue
        buckets[e].append(s)
    offsets = np.zeros(E + 1, np.int32)
    perm_token = []
    slot_pos = np.full((T, k), -1, np.int32)
    pos = 0
    for e in range(E):
        offsets[e] = pos
        for s in buckets[e]:
            t, j = s % T, s // T
            slot_pos[t, j] = pos
            perm_token.append(t)
            pos += 1
    offsets[E] = pos
    return offsets, np.asarray(perm_token, np.int32), slot_pos


# --------------------------------------------------------------------------
# 3. Similarity and threshold graph (Sec. 2.2, Sec. 5.1, Sec. 5.2)
# --------------------------------------------------------------------------
def cosine(xb, sim_mode="raw"):
    """Pairwise similarity of the rows of xb (fp64).

    raw    : <a,b> / (|a||b|), 0 when a norm is 0
    clamp  : max(0, raw)
    affine : (1 + raw) / 2
    """
    xb = np.asarray(xb, np.float64)
    g = xb @ xb.T
    n = np.sqrt(np.diag(g))
    den = np.outer(n, n)
    with np.errstate(invalid="ignore", divide="ignore"):
        c = np.where(den > 0, g / np.where(den > 0, den, 1.0), 0.0)
    if sim_mode == "raw":
        return c
    if sim_mode == "clamp":
        return np.maximum(c, 0.0)
    if sim_mode == "affine":
        return np.where(den > 0, (1.0 + c) / 2.0, 0.0)
    raise ValueError(sim_mode)


def adjacency(xb, h, sim_mode="raw"):
    """Thresholded token graph of one bucket: edge a-b (a != b) iff
    similarity >= h.  Pairs in different buckets are never built."""
    c = cosine(xb, sim_mode)
    adj = c >= h
    np.fill_diagonal(adj, False)
    return adj


# --------------------------------------------------------------------------
# 4. Representative selection (Sec. 5.2)
# --------------------------------------------------------------------------
def greedy(adj, degree_mode="static"):
    """Walk the thresholded graph: the undecided token of highest degree
    (lower position first on ties) is kept and every undecided neighbour is
    condensed onto it; repeat until all tokens are decided.

    Returns (rep int64 [n]: position of the kept token each position maps to,
    degree int64 [n] in the full graph).
    """
    adj = np.asarray(adj, bool)
    n = adj.shape[0]
    deg = adj.sum(axis=1).astype(np.int64)
    rep = np.full(n, -1, np.int64)
    if degree_mode == "static":
        order = sorted(range(n), key=lambda a: (-deg[a], a))
        for a in order:
            if rep[a] >= 0:
                continue
            rep[a] = a
            take = adj[a] & (rep < 0)
            rep[take] = a
    elif degree_mode == "dynamic":
        while True:
            free = rep < 0
            if not free.any():
                break
            rdeg = (adj & free[None, :]).sum(axis=1)
            cand = np.flatnonzero(free)
            best = max(cand, key=lambda a: (rdeg[a], -a))
            rep[best] = best
            take = adj[best] & free
            rep[take] = best
    else:
        raise ValueError(degree_mode)
    return rep, deg


def historical_weights(x, tokens, prev_sim, S1, S2, sim_mode="raw"):
    """Edge weights of one bucket under the fast similarity measurement of
    Sec. 5.1 (NEXT piece; no GPU path).  Step 1 is the bucketing itself
    (tokens of different experts get weight 0, so only a bucket's pairs
    exist); step 2: a pair whose similarity in the previous block exceeds S1
    gets weight 1, one below S2 gets weight 0, neither computed; step 3: the
    remaining pairs (no previous value, NaN, or one in [S2, S1]) get their
    cosine.  prev_sim is a [T, T] record indexed by token id.

    Returns (weights [n, n], computed bool [n, n]); the diagonal is not a
    pair (computed False)."""
    tokens = np.asarray(tokens, np.int64)
    prev = np.asarray(prev_sim, np.float64)[np.ix_(tokens, tokens)]
    with np.errstate(invalid="ignore"):
        one, zero = prev > S1, prev < S2
    computed = ~(one | zero)
    np.fill_diagonal(computed, False)
    w = np.where(one, 1.0, np.where(zero, 0.0, cosine(np.asarray(x, np.float64)[tokens], sim_mode)))
    return w, computed


def historical_record(x, perm_token, offsets, prev_sim, S1, S2, sim_mode="raw"):
    """The similarity record this block leaves for the next one: the weight
    of every pair that shares a bucket (decided or computed), NaN for every
    other pair and the diagonal; and the number of distinct pairs (a < b)
    whose cosine was computed, the cost Sec. 7 reports against S1 and S2.
    Reading: a pair decided by history passes on its weight (1 or 0)."""
    T = np.asarray(prev_sim).shape[0]
    rec = np.full((T, T), np.nan)
    done = np.zeros((T, T), bool)
    for e in range(len(offsets) - 1):
        tok = np.asarray(perm_token[offsets[e]:offsets[e + 1]], np.int64)
        if tok.size == 0:
            continue
        w, comp = historical_weights(x, tok, prev_sim, S1, S2, sim_mode)
        rec[np.ix_(tok, tok)] = w
        done[np.ix_(tok, tok)] |= comp
    np.fill_diagonal(rec, np.nan)
    return rec, int(np.triu(done, 1).sum())


def condense(x, perm_token, offsets, h, sim_mode="raw", degree_mode="static", history=None):
    """Per-bucket similarity + greedy, then compaction of the kept tokens.
    history = (prev_sim, S1, S2) takes the edge weights of
    historical_weights (Sec. 5.1 step 2) instead of the cosine of every pair.

    Returns a namespace with
      rep_of_pos  int32 [S]  bucket position of the representative of each
                             position (a representative maps to itself)
      degree      int32 [S]
      is_rep      bool  [S]
      rep_row     int32 [S]  row of the representative in the compacted
                             representative list (representatives in
                             ascending position, i.e. bucket by bucket)
      rep_offsets int32 [E+1]
      rep_token   int32 [R]  token id of each representative row
    """
    x = np.asarray(x, np.float64)
    E = len(offsets) - 1
    S = int(offsets[E])
    rep_of_pos = np.zeros(S, np.int32)
    degree = np.zeros(S, np.int32)
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        if history is None:
            adj = adjacency(x[perm_token[lo:hi]], h, sim_mode)
        else:                          # (prev_sim, S1, S2): Sec. 5.1 step 2
            w, _ = historical_weights(x, perm_token[lo:hi], *history, sim_mode=sim_mode)
            adj = w >= h
            np.fill_diagonal(adj, False)
        rep, deg = greedy(adj, degree_mode)
        rep_of_pos[lo:hi] = rep + lo
        degree[lo:hi] = deg
    is_rep = rep_of_pos == np.arange(S)
    row_of_rep = np.full(S, -1, np.int64)
    rep_positions = np.flatnonzero(is_rep)
    row_of_rep[rep_positions] = np.arange(rep_positions.size)
    rep_row = row_of_rep[rep_of_pos].astype(np.int32)
    rep_offsets = np.zeros(E + 1, np.int32)
    for e in range(E):
        rep_offsets[e + 1] = rep_offsets[e] + int(
            is_rep[offsets[e]:offsets[e + 1]].sum())
    rep_token = np.asarray(perm_token, np.int32)[rep_positions]
    return SimpleNamespace(rep_of_pos=rep_of_pos, degree=degree, is_rep=is_rep,
                           rep_row=rep_row, rep_offsets=rep_offsets,
                           rep_token=rep_token)


# --------------------------------------------------------------------------
# 5. Expert FFN on representatives (Sec. 2.1, Sec. 3)
# --------------------------------------------------------------------------
def activation(z, act):
    """Exact GELU 0.5 z (1 + erf(z / sqrt 2)) or SiLU z / (1 + exp(-z))."""
    z = np.asarray(z, np.float64)
    if act == "gelu":
        return 0.5 * z * (1.0 + _erf(z / math.sqrt(2.0)))
    if act == "silu":
        return z / (1.0 + np.exp(-z))
    raise ValueError(act)


def expert_ffn(x_rep, rep_offsets, w1, w2, act):
    """Y_rep[r] = W2_e act(W1_e x_r) for every representative r of expert e
    (two weight matrices, no biases)."""
    x_rep = np.asarray(x_rep, np.float64)
    E = len(rep_offsets) - 1
    d = w2.shape[1]
    y = np.zeros((x_rep.shape[0], d), np.float64)
    for e in range(E):
        lo, hi = int(rep_offsets[e]), int(rep_offsets[e + 1])
        if hi == lo:
            continue
        hid = activation(x_rep[lo:hi] @ np.asarray(w1[e], np.float64).T, act)
        y[lo:hi] = hid @ np.asarray(w2[e], np.float64).T
    return y


# --------------------------------------------------------------------------
# 6. Combine (Sec. 2.1, Sec. 6)
# --------------------------------------------------------------------------
def combine(y_rep, rep_row, slot_pos, topk_gate):
    """y_t = sum over kept slots j of gate[t,j] * Y_rep[rep_row[slot_pos[t,j]]];
    a token with no kept slot gets zeros."""
    y_rep = np.asarray(y_rep, np.float64)
    T, k = slot_pos.shape
    y = np.zeros((T, y_rep.shape[1]), np.float64)
    for j in range(k):
        kept = slot_pos[:, j] >= 0
        rows = rep_row[slot_pos[kept, j]]
        y[kept] += np.asarray(topk_gate, np.float64)[kept, j, None] * y_rep[rows]
    return y


# --------------------------------------------------------------------------
# The whole layer
# --------------------------------------------------------------------------
def moe_layer(x, w_g, b_g, w1, w2, *, k, h, act, capacity_factor=0.0,
              sim_mode="raw", degree_mode="static", with_ffn=True):
    """All steps in order; returns a namespace with every intermediate."""
    T = x.shape[0]
    E = w_g.shape[0]
    topk_idx, topk_gate, logits = gate(x, w_g, b_g, k)
    C = capacity_of(T, k, E, capacity_factor)
    offsets, perm_token, slot_pos = dispatch(topk_idx, E, C)
    cz = condense(x, perm_token, offsets, h, sim_mode, degree_mode)
    out = SimpleNamespace(topk_idx=topk_idx, topk_gate=topk_gate,
                          logits=logits, capacity=C, offsets=offsets,
                          perm_token=perm_token, slot_pos=slot_pos,
                          **vars(cz))
    if with_ffn:
        x_rep = np.asarray(x, np.float64)[cz.rep_token]
        out.y_rep = expert_ffn(x_rep, cz.rep_offsets, w1, w2, act)
        out.y = combine(out.y_rep, cz.rep_row, slot_pos, topk_gate)
    return out


# --------------------------------------------------------------------------
# Adaptive threshold (Sec. 5.2, Eq. 2)
# --------------------------------------------------------------------------
def adaptive_threshold(l_ini, l_prev):
    """Sec. 5.2 Eq. 2, as printed: the loss decrease since the first
    iteration, normalised by the first loss, through 1/(1 + e^x).

    l_norm = (l_ini - l_prev) / l_ini;  h_t = 1 / (1 + exp(l_norm)).
    The first iteration has no previous loss and takes l_prev = l_ini
    (h = 1/2)."""
    l_ini = float(l_ini)
    l_prev = float(l_prev)
    if not math.isfinite(l_ini) or l_ini == 0.0 or not math.isfinite(l_prev):
        raise ValueError("l_ini must be finite and non-zero, l_prev finite")
    l_norm = (l_ini - l_prev) / l_ini
    return 1.0 / (1.0 + math.exp(l_norm))


# --------------------------------------------------------------------------
# Backward of the condensed layer (training, Sec. 3 and Sec. 7: the layer is
# trained).  The paper does not say how gradients pass a condensed token.
# Reading: the gradient of the function the forward computes, with every
# discrete decision (routing, capacity, graph, representatives) held fixed:
# a condensed slot's output is its representative's expert output, so its
# gradient flows into that representative's row, and its own embedding
# receives none through the expert.
# --------------------------------------------------------------------------
def combine_backward(dy, y_rep, rep_row, slot_pos, topk_gate):
    """Transpose of combine for a given dy = dL/dy [T, d]:

    dgate[t, j]  = <dy[t], Y_rep[rep_row[slot_pos[t, j]]]>  (0 for a dropped slot)
    dy_rep[r]    = sum over kept slots (t, j) with rep_row[slot_pos[t, j]] = r
                   of gate[t, j] * dy[t]
    (every slot of a condensed group adds its own gate-weighted gradient to
    the group's representative row)."""
    dy = np.asarray(dy, np.float64)
    y_rep = np.asarray(y_rep, np.float64)
    T, k = slot_pos.shape
    dy_rep = np.zeros_like(y_rep)
    dgate = np.zeros((T, k), np.float64)
    for t in range(T):
        for j in range(k):
            p = int(slot_pos[t, j])
            if p < 0:
                continue
            r = int(rep_row[p])
            dgate[t, j] = float(dy[t] @ y_rep[r])
            dy_rep[r] += float(topk_gate[t, j]) * dy[t]
    return dy_rep, dgate


def activation_grad(z, act):
    """Derivative of the expert activation: GELU'(z) = Phi(z) + z phi(z)
    (Phi, phi: the standard normal CDF and density), SiLU'(z) =
    s(z) (1 + z (1 - s(z))) with s the logistic function."""
    z = np.asarray(z, np.float64)
    if act == "gelu":
        return 0.5 * (1.0 + _erf(z / math.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / math.sqrt(2.0 * math.pi)
    if act == "silu":
        sg = 1.0 / (1.0 + np.exp(-z))
        return sg * (1.0 + z * (1.0 - sg))
    raise ValueError(act)


def expert_ffn_backward(x_rep, rep_offsets, w1, w2, act, dy_rep):
    """Gradients of Y_rep[r] = W2_e act(W1_e x_r) for dy_rep = dL/dY_rep:
    with Z = X_e W1_e^T, A = act(Z), dA = dY_e W2_e, dZ = dA * act'(Z):
    dx_rep = dZ W1_e, dW1_e = dZ^T X_e, dW2_e = dY_e^T A (zero for an
    expert without representatives)."""
    x_rep = np.asarray(x_rep, np.float64)
    dy_rep = np.asarray(dy_rep, np.float64)
    E = len(rep_offsets) - 1
    dx = np.zeros_like(x_rep)
    dw1 = np.zeros(np.shape(w1), np.float64)
    dw2 = np.zeros(np.shape(w2), np.float64)
    for e in range(E):
        lo, hi = int(rep_offsets[e]), int(rep_offsets[e + 1])
        if hi == lo:
            continue
        W1 = np.asarray(w1[e], np.float64)
        W2 = np.asarray(w2[e], np.float64)
        z = x_rep[lo:hi] @ W1.T
        a = activation(z, act)
        dz = (dy_rep[lo:hi] @ W2) * activation_grad(z, act)
        dx[lo:hi] = dz @ W1
        dw1[e] = dz.T @ x_rep[lo:hi]
        dw2[e] = dy_rep[lo:hi].T @ a
    return dx, dw1, dw2

