"""Pins for the oracle's gate and dispatch steps (CPU only).

The expected values come from hand derivation, brute force over tiny inputs
and closed forms, never from the oracle itself or from the HIP path.
"""
import itertools
import math

import numpy as np
import pytest

from oracle import luffy_oracle as O


# A 4-token, 3-expert, d=2 example worked by hand (Sec. 2.1 gate, top-2).
# W_g rows e0=(1,0), e1=(0,1), e2=(-1,0), no bias, so logit_e = <x, w_e>.
#   t0=( 2, 1): logits ( 2, 1,-2) -> top-2 (0,1)
#   t1=( 0, 3): logits ( 0, 3, 0) -> 1 first, then 0 and 2 tie -> lower id 0
#   t2=(-1,-2): logits (-1,-2, 1) -> (2,0)
#   t3=( 1, 4): logits ( 1, 4,-1) -> (1,0)
HAND_X = np.array([[2, 1], [0, 3], [-1, -2], [1, 4]], np.float64)
HAND_W = np.array([[1, 0], [0, 1], [-1, 0]], np.float64)
HAND_TOP2 = np.array([[0, 1], [1, 0], [2, 0], [1, 0]])


def sigmoid(z):
    return 1.0 / (1.0 + math.exp(-z))


def test_gate_hand_example_top2():
    idx, g, logits = O.gate(HAND_X, HAND_W, None, 2)
    assert np.array_equal(idx, HAND_TOP2)
    # renormalised over the two chosen experts: g0 = sigmoid(l0 - l1)
    gaps = [2 - 1, 3 - 0, 1 - (-1), 4 - 1]
    for t, gap in enumerate(gaps):
        assert g[t, 0] == pytest.approx(sigmoid(gap), abs=1e-15)
        assert g[t, 1] == pytest.approx(1 - sigmoid(gap), abs=1e-15)


def test_gate_hand_example_top1():
    idx, g, _ = O.gate(HAND_X, HAND_W, None, 1)
    assert np.array_equal(idx[:, 0], HAND_TOP2[:, 0])
    # top-1 gate is the softmax probability over all three experts
    l0 = [(2, 1, -2), (0, 3, 0), (-1, -2, 1), (1, 4, -1)]
    for t, ls in enumerate(l0):
        den = sum(math.exp(v) for v in ls)
        assert g[t, 0] == pytest.approx(math.exp(max(ls)) / den, rel=1e-14)


def test_gate_bias_shifts_choice():
    # a large bias on expert 2 makes it everyone's first choice
    idx, _, _ = O.gate(HAND_X, HAND_W, np.array([0, 0, 100.0]), 1)
    assert np.all(idx[:, 0] == 2)


def test_gate_all_equal_logits():
    # identical logits: ties go to the lower ids, gates are uniform
    x = np.zeros((3, 4))
    w = np.ones((5, 4))
    idx, g, _ = O.gate(x, w, None, 2)
    assert np.array_equal(idx, [[0, 1]] * 3)
    assert np.allclose(g, 0.5)
    idx, g, _ = O.gate(x, w, None, 1)
    assert np.array_equal(idx[:, 0], [0, 0, 0])
    assert np.allclose(g, 1 / 5)


def test_gate_topk_brute_force():
    rng = np.random.default_rng(7)
    for _ in range(20):
        T, E, d = 6, 5, 3
        x, w, b = rng.normal(size=(T, d)), rng.normal(size=(E, d)), rng.normal(size=E)
        idx, g, logits = O.gate(x, w, b, 2)
        for t in range(T):
            l = [sum(x[t, i] * w[e, i] for i in range(d)) + b[e] for e in range(E)]
            best = max(itertools.permutations(range(E), 2),
                       key=lambda p: (l[p[0]], l[p[1]], -p[0], -p[1]))
            assert tuple(idx[t]) == best
            assert g[t].sum() == pytest.approx(1.0, abs=1e-14)
            assert g[t, 0] / g[t, 1] == pytest.approx(math.exp(l[best[0]] - l[best[1]]), rel=1e-12)


def test_dispatch_hand_example_no_capacity():
    # slots s = j*T + t, T=4: s0..s3 first choices (experts 0,1,2,1),
    # s4..s7 second choices (experts 1,0,0,0).
    # bucket 0: s0(t0) s5(t1) s6(t2) s7(t3); bucket 1: s1(t1) s3(t3) s4(t0); bucket 2: s2(t2)
    off, perm, sp = O.dispatch(HAND_TOP2, 3, 0)
    assert list(off) == [0, 4, 7, 8]
    assert list(perm) == [0, 1, 2, 3, 1, 3, 0, 2]
    assert sp.tolist() == [[0, 6], [4, 1], [7, 2], [5, 3]]


def test_dispatch_hand_example_capacity():
    # capacity 2: bucket 0 keeps s0,s5 (drops s6,s7); bucket 1 keeps s1,s3 (drops s4)
    assert O.capacity_of(4, 2, 3, 0.75) == 2
    off, perm, sp = O.dispatch(HAND_TOP2, 3, 2)
    assert list(off) == [0, 2, 4, 5]
    assert list(perm) == [0, 1, 1, 3, 2]
    assert sp.tolist() == [[0, -1], [2, 1], [4, -1], [3, -1]]


def test_dispatch_against_sorting():
    # an independent construction: sort kept slots by (expert, slot id)
    rng = np.random.default_rng(3)
    for trial in range(30):
        T, E = int(rng.integers(1, 16)), int(rng.integers(1, 5))
        k = 1 if E == 1 else int(rng.integers(1, 3))
        topk = np.stack([rng.permutation(E)[:k] for _ in range(T)])
        cap = int(rng.integers(0, 6))
        off, perm, sp = O.dispatch(topk, E, cap)
        slots = sorted(((int(topk[t, j]), j * T + t) for t in range(T) for j in range(k)))
        kept, count = [], {}
        for e, s in slots:
            count[e] = count.get(e, 0) + 1
            if cap == 0 or count[e] <= cap:
                kept.append((e, s))
        assert list(perm) == [s % T for _, s in kept]
        for p, (e, s) in enumerate(kept):
            assert sp[s % T, s // T] == p
            assert off[e] <= p < off[e + 1]
        assert (sp >= 0).sum() == len(kept) == off[E]
        for e in range(E):
            n_e = sum(1 for (ee, _) in kept if ee == e)
            assert off[e + 1] - off[e] == n_e


def test_capacity_values_of_listed_configs():
    assert O.capacity_of(8192, 2, 16, 1.25) == 1280
    assert O.capacity_of(65536, 1, 64, 1.0) == 1024
    assert O.capacity_of(512, 1, 4, 0.0) == 0
