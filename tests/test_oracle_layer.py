"""Pins for the oracle's FFN, combine and whole-layer behaviour (CPU only):
textbook constants of the activations, closed forms with one-hot weights, the
dense-MoE reduction when nothing condenses, the clique-union closed form on
the generator's clustered tokens, and the method's invariants."""
import math

import numpy as np
import pytest

import luffy_gen as G
from oracle import luffy_oracle as O


def test_activation_textbook_values():
    # GELU(z) = z * Phi(z); Phi(1) = 0.8413447460685429, Phi(-1) = 1 - Phi(1)
    assert O.activation(1.0, "gelu") == pytest.approx(0.8413447460685429, abs=1e-15)
    assert O.activation(-1.0, "gelu") == pytest.approx(-(1 - 0.8413447460685429), abs=1e-15)
    assert O.activation(0.0, "gelu") == 0.0
    # Phi(2) = 0.9772498680518208
    assert O.activation(2.0, "gelu") == pytest.approx(2 * 0.9772498680518208, abs=1e-15)
    # SiLU(z) = z * sigmoid(z); sigmoid(1) = 0.7310585786300049
    assert O.activation(1.0, "silu") == pytest.approx(0.7310585786300049, abs=1e-15)
    z = np.linspace(-6, 6, 101)
    for act in ("gelu", "silu"):
        # both are z * (symmetric CDF): f(z) - f(-z) = z
        assert np.allclose(O.activation(z, act) - O.activation(-z, act), z, atol=1e-14)


def test_ffn_one_hot_weights_closed_form():
    # W1 picks coordinate (2*j) % d into hidden unit j; W2 picks hidden unit
    # (i + 1) % dff into output i, so y_i = act(x[(2*((i+1) % dff)) % d]).
    d, dff, E = 5, 7, 2
    w1 = np.zeros((E, dff, d))
    w2 = np.zeros((E, d, dff))
    for j in range(dff):
        w1[0, j, (2 * j) % d] = 1.0
        w1[1, j, (3 * j) % d] = 2.0          # expert 1: scaled, other pattern
    for i in range(d):
        w2[0, i, (i + 1) % dff] = 1.0
        w2[1, i, (2 * i) % dff] = -1.0
    x = np.array([[0.3, -1.2, 2.0, 0.7, -0.1], [1.0, 2.0, -3.0, 0.5, 0.25]])
    ro = np.array([0, 1, 2])
    y = O.expert_ffn(x, ro, w1, w2, "gelu")
    g = lambda v: v * 0.5 * (1 + math.erf(v / math.sqrt(2)))
    for i in range(d):
        assert y[0, i] == pytest.approx(g(x[0, (2 * ((i + 1) % dff)) % d]), abs=1e-15)
        assert y[1, i] == pytest.approx(-g(2 * x[1, (3 * ((2 * i) % dff)) % d]), abs=1e-15)


def test_combine_gates_and_drops():
    y_rep = np.array([[1.0, 2.0], [10.0, 20.0]])
    rep_row = np.array([0, 1, 1], np.int32)
    slot_pos = np.array([[0, 2], [-1, -1], [1, -1]], np.int32)
    g = np.array([[0.25, 0.75], [0.5, 0.5], [1.0, 0.0]])
    y = O.combine(y_rep, rep_row, slot_pos, g)
    assert y.tolist() == [[0.25 * 1 + 0.75 * 10, 0.25 * 2 + 0.75 * 20], [0, 0], [10, 20]]


def dense_moe_textbook(x, w_g, b_g, w1, w2, k, act, cf):
    """Per-token MoE with no condensation: y_t = sum_j g_tj FFN_{e_tj}(x_t),
    slots over capacity dropped in slot-id order.  Written token by token,
    independently of the oracle's per-expert structure."""
    T, E = x.shape[0], w_g.shape[0]
    logits = x @ w_g.T + b_g
    C = math.ceil(cf * k * T / E - 1e-9) if cf > 0 else 0
    used = [0] * E
    kept = {}
    choice = []
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-logits[t, e], e))[:k]
        choice.append(order)
    for j in range(k):
        for t in range(T):
            e = choice[t][j]
            used[e] += 1
            kept[(t, j)] = (C == 0 or used[e] <= C)
    y = np.zeros((T, w2.shape[1]))
    for t in range(T):
        p = np.exp(logits[t] - logits[t].max())
        p /= p.sum()
        sel = [p[e] for e in choice[t]]
        gates = sel if k == 1 else [s / sum(sel) for s in sel]
        for j, e in enumerate(choice[t]):
            if kept[(t, j)]:
                hdn = O.activation(w1[e] @ x[t], act)
                y[t] += gates[j] * (w2[e] @ hdn)
    return y


@pytest.mark.parametrize("name,k,cf", [("c1", 1, 0.0), ("c2", 2, 1.25), ("c5", 1, 1.0)])
def test_no_condensation_equals_dense_moe(name, k, cf):
    inp = G.make_inputs(name, seed=1, T=96, d=32, d_ff=48, E=4, n_centres=8,
                        k=k, capacity_factor=cf, w_scale=0.3)
    x = inp.x.astype(np.float64)
    out = O.moe_layer(x, inp.w_g, inp.b_g, inp.w1, inp.w2, k=k, h=2.0,
                      act=inp.cfg.act, capacity_factor=cf)
    assert out.rep_offsets[-1] == out.offsets[-1]          # R == S
    ref = dense_moe_textbook(x, inp.w_g.astype(np.float64), inp.b_g.astype(np.float64),
                             inp.w1.astype(np.float64), inp.w2.astype(np.float64),
                             k, inp.cfg.act, cf)
    assert np.allclose(out.y, ref, rtol=1e-12, atol=1e-13)
    if cf > 0:
        assert (out.slot_pos < 0).any(), "test should exercise drops"
        dropped_all = (out.slot_pos < 0).all(axis=1)
        assert np.all(out.y[dropped_all] == 0)


def check_invariants(out):
    S = int(out.offsets[-1])
    E = len(out.offsets) - 1
    pos = np.arange(S)
    bucket = np.searchsorted(out.offsets, pos, side="right") - 1
    rep = out.rep_of_pos
    # every position maps to one representative in its own bucket, which maps to itself
    assert np.all(bucket[rep] == bucket)
    assert np.all(rep[rep] == rep)
    # a duplicate is adjacent (cos >= h) to its representative: checked by caller
    # rep_row indexes the compacted list and rep_token holds the rep's token
    assert np.all(out.rep_token[out.rep_row] == out.perm_token[rep])
    assert out.rep_offsets[-1] == out.is_rep.sum()
    for e in range(E):
        lo, hi = out.offsets[e], out.offsets[e + 1]
        assert out.rep_offsets[e + 1] - out.rep_offsets[e] == out.is_rep[lo:hi].sum()


def clique_union_reps(out, centre_id):
    """Closed form for clustered tokens whose threshold graph is a union of
    cliques (one per centre per bucket): every position maps to the first
    position of its bucket holding the same centre."""
    S = int(out.offsets[-1])
    E = len(out.offsets) - 1
    rep = np.empty(S, np.int64)
    for e in range(E):
        first = {}
        for p in range(out.offsets[e], out.offsets[e + 1]):
            c = int(centre_id[out.perm_token[p]])
            first.setdefault(c, p)
            rep[p] = first[c]
    return rep


def within_bucket_margin(x, out, centre_id, h):
    """Smallest |cos - h| over within-bucket pairs, and whether the clique
    structure holds (same centre >= h, different centre < h)."""
    worst = np.inf
    clique = True
    E = len(out.offsets) - 1
    for e in range(E):
        lo, hi = out.offsets[e], out.offsets[e + 1]
        if hi - lo < 2:
            continue
        c = O.cosine(x[out.perm_token[lo:hi]])
        iu = np.triu_indices(hi - lo, 1)
        v = c[iu]
        worst = min(worst, float(np.abs(v - h).min()))
        if centre_id is not None:
            cid = centre_id[out.perm_token[lo:hi]]
            same = (cid[:, None] == cid[None, :])[iu]
            clique &= bool(np.all(v[same] >= h) and np.all(v[~same] < h))
    return worst, clique


@pytest.mark.parametrize("name,overrides", [
    ("c1", {}),
    ("c2", dict(T=2048, d=256)),
    ("c3", dict(T=2048, d=256, n_centres=256)),
    ("c5", dict(T=4096, d=256, n_centres=512)),
])
def test_clique_union_closed_form_on_generator_data(name, overrides):
    inp = G.make_inputs(name, seed=0, weights=False, **overrides)
    cfg = inp.cfg
    x = inp.x.astype(np.float64)
    out = O.moe_layer(x, inp.w_g, inp.b_g, None, None, k=cfg.k, h=cfg.h,
                      act=cfg.act, capacity_factor=cfg.capacity_factor,
                      with_ffn=False)
    check_invariants(out)
    margin, clique = within_bucket_margin(x, out, inp.centre_id, cfg.h)
    assert margin >= 0.01 and clique
    assert np.array_equal(out.rep_of_pos, clique_union_reps(out, inp.centre_id))
    # R_e = number of distinct centres in bucket e
    for e in range(cfg.E):
        lo, hi = out.offsets[e], out.offsets[e + 1]
        n_c = len(set(inp.centre_id[out.perm_token[lo:hi]].tolist()))
        assert out.rep_offsets[e + 1] - out.rep_offsets[e] == n_c
    # static and dynamic degree give the same groups on a union of cliques
    out_dyn = O.moe_layer(x, inp.w_g, inp.b_g, None, None, k=cfg.k, h=cfg.h,
                          act=cfg.act, capacity_factor=cfg.capacity_factor,
                          degree_mode="dynamic", with_ffn=False)
    assert np.array_equal(out.rep_of_pos, out_dyn.rep_of_pos)


def test_iid_tokens_never_merge():
    inp = G.make_inputs("c4", seed=0, weights=False, T=1024, d=512)
    x = inp.x.astype(np.float64)
    for h in inp.cfg.thresholds:
        out = O.moe_layer(x, inp.w_g, inp.b_g, None, None, k=1, h=h,
                          act="silu", with_ffn=False)
        assert out.is_rep.all() and out.degree.sum() == 0


def test_planted_duplicates_always_merge():
    for h in (0.5, 0.9, 0.99):
        inp = G.make_inputs("c4", seed=3, weights=False, T=512, d=128,
                            planted_duplicates=20)
        x = inp.x.astype(np.float64)
        out = O.moe_layer(x, inp.w_g, inp.b_g, None, None, k=1, h=h,
                          act="silu", with_ffn=False)
        check_invariants(out)
        for src, cp in inp.planted:
            ps = out.slot_pos[src, 0]
            pc = out.slot_pos[cp, 0]
            assert ps >= 0 and pc >= 0
            assert out.rep_of_pos[ps] == out.rep_of_pos[pc]


def test_similarity_readings_agree_on_generator_data():
    # the raw, clamped and affine readings group the clustered tokens alike
    inp = G.make_inputs("c2", seed=0, weights=False, T=1024, d=256)
    x = inp.x.astype(np.float64)
    kw = dict(k=2, act="gelu", capacity_factor=1.25, with_ffn=False)
    raw = O.moe_layer(x, inp.w_g, inp.b_g, None, None, h=0.95, **kw)
    clamp = O.moe_layer(x, inp.w_g, inp.b_g, None, None, h=0.95, sim_mode="clamp", **kw)
    aff = O.moe_layer(x, inp.w_g, inp.b_g, None, None, h=(1 + 0.95) / 2, sim_mode="affine", **kw)
    assert np.array_equal(raw.rep_of_pos, clamp.rep_of_pos)
    assert np.array_equal(raw.rep_of_pos, aff.rep_of_pos)


def test_condensed_layer_shares_expert_output():
    inp = G.make_inputs("c1", seed=0)
    cfg = inp.cfg
    x = inp.x.astype(np.float64)
    out = O.moe_layer(x, inp.w_g, inp.b_g, inp.w1, inp.w2, k=1, h=cfg.h, act="gelu")
    check_invariants(out)
    assert out.rep_offsets[-1] < out.offsets[-1]          # something condensed
    # a condensed token's output is its gate times its representative's FFN output
    for t in range(cfg.T):
        p = out.slot_pos[t, 0]
        r = out.rep_of_pos[p]
        tr = out.perm_token[r]
        e = out.topk_idx[t, 0]
        f = inp.w2[e].astype(np.float64) @ O.activation(inp.w1[e].astype(np.float64) @ x[tr], "gelu")
        assert np.allclose(out.y[t], out.topk_gate[t, 0] * f, rtol=1e-12, atol=1e-14)
