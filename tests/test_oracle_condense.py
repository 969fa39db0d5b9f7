"""Pins for the oracle's similarity, threshold graph and representative
selection (CPU only)."""
import itertools
import math
import os

import numpy as np
import pytest

from oracle import luffy_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "greedy_hand_cases.txt")


def load_hand_cases():
    cases = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, n, edges, rs, rd, _ = [f.strip() for f in line.split("|")]
        n = int(n)
        adj = np.zeros((n, n), bool)
        for e in filter(None, edges.split(",")):
            a, b = map(int, e.split("-"))
            adj[a, b] = adj[b, a] = True
        cases.append((name, adj, [int(v) for v in rs.split(",")],
                      [int(v) for v in rd.split(",")]))
    return cases


@pytest.mark.parametrize("case", load_hand_cases(), ids=lambda c: c[0])
def test_greedy_hand_cases(case):
    name, adj, rep_static, rep_dynamic = case
    rep, deg = O.greedy(adj, "static")
    assert rep.tolist() == rep_static
    assert deg.tolist() == adj.sum(1).tolist()
    rep, _ = O.greedy(adj, "dynamic")
    assert rep.tolist() == rep_dynamic


def priority_key(deg, a):
    return (-int(deg[a]), a)


def brute_force_representatives(adj):
    """All subsets S with: a in S iff no neighbour of higher priority is in S.
    For a total priority order exactly one subset qualifies (induction along
    the order); it is the set the sequential walk keeps."""
    n = adj.shape[0]
    deg = adj.sum(1)
    sols = []
    for mask in range(1 << n):
        S = [(mask >> a) & 1 for a in range(n)]
        ok = True
        for a in range(n):
            higher_in = any(S[b] and adj[a, b] and priority_key(deg, b) < priority_key(deg, a)
                            for b in range(n))
            if bool(S[a]) == higher_in:
                ok = False
                break
        if ok:
            sols.append(S)
    return sols


def test_greedy_brute_force_small_graphs():
    rng = np.random.default_rng(11)
    for trial in range(60):
        n = int(rng.integers(1, 11))
        p = rng.uniform(0.1, 0.7)
        upper = np.triu(rng.uniform(size=(n, n)) < p, 1)
        adj = upper | upper.T
        sols = brute_force_representatives(adj)
        assert len(sols) == 1
        S = sols[0]
        rep, deg = O.greedy(adj, "static")
        assert [int(rep[a] == a) for a in range(n)] == S
        for b in range(n):
            if S[b]:
                continue
            # joins the adjacent representative of highest priority
            cand = [a for a in range(n) if S[a] and adj[a, b]]
            assert cand, "representatives must dominate"
            assert rep[b] == min(cand, key=lambda a: priority_key(deg, a))
        reps = [a for a in range(n) if S[a]]
        for a, b in itertools.combinations(reps, 2):
            assert not adj[a, b], "representatives must be independent"


def test_cosine_hand_vectors():
    # a=(1,0,0) b=(2,0,0) c=(1,1,0) d=(0,0,5) e=(-1,0,0) z=0
    X = np.array([[1, 0, 0], [2, 0, 0], [1, 1, 0], [0, 0, 5], [-1, 0, 0], [0, 0, 0]], float)
    c = O.cosine(X)
    assert c[0, 1] == pytest.approx(1.0)
    assert c[0, 2] == pytest.approx(1 / math.sqrt(2))
    assert c[0, 3] == 0.0
    assert c[0, 4] == pytest.approx(-1.0)
    assert np.all(c[5] == 0) and np.all(c[:, 5] == 0)
    # h = 0.70 keeps a-b, a-c, b-c (cos 1, 0.7071, 0.7071): one group kept at a
    rep, _ = O.greedy(O.adjacency(X, 0.70))
    assert rep.tolist() == [0, 0, 0, 3, 4, 5]
    # h = 0.75 keeps only a-b
    rep, _ = O.greedy(O.adjacency(X, 0.75))
    assert rep.tolist() == [0, 0, 2, 3, 4, 5]
    # affine reading (1+cos)/2 >= 0.85 is raw cos >= 0.7
    assert np.array_equal(O.adjacency(X, 0.85, "affine"), O.adjacency(X, 0.70, "raw"))
    # clamp reading equals raw for positive thresholds
    assert np.array_equal(O.adjacency(X, 0.3, "clamp"), O.adjacency(X, 0.3, "raw"))


def test_cosine_scale_invariance():
    rng = np.random.default_rng(5)
    X = rng.normal(size=(7, 16))
    Y = X * rng.uniform(0.1, 10, size=(7, 1))
    assert np.allclose(O.cosine(X), O.cosine(Y), atol=1e-14)


def test_threshold_above_one_keeps_everyone():
    rng = np.random.default_rng(2)
    X = rng.normal(size=(9, 4))
    X[3] = X[0]                       # exact duplicate
    rep, deg = O.greedy(O.adjacency(X, 2.0))
    assert rep.tolist() == list(range(9))
    assert deg.sum() == 0


def test_condense_bucket_layout_and_compaction():
    # two buckets over hand vectors; bucket 1 holds a duplicate pair
    X = np.array([[1, 0], [0, 1], [1, 0.01], [3, 3], [3, 3.0]], float)
    perm = np.array([0, 1, 2, 3, 4], np.int32)
    off = np.array([0, 3, 5], np.int32)
    cz = O.condense(X, perm, off, 0.99)
    # bucket 0: 0~2 (cos 0.99995), 1 alone -> reps at 0, 1; bucket 1: 3~4 -> rep 3
    assert cz.rep_of_pos.tolist() == [0, 1, 0, 3, 3]
    assert cz.is_rep.tolist() == [True, True, False, True, False]
    assert cz.rep_offsets.tolist() == [0, 2, 3]
    assert cz.rep_token.tolist() == [0, 1, 3]
    assert cz.rep_row.tolist() == [0, 1, 0, 2, 2]
    assert cz.degree.tolist() == [1, 0, 1, 1, 1]
