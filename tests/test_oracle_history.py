"""Pins of the oracle's fast similarity measurement with historical
similarity (Sec. 5.1 step 2, a NEXT piece with no GPU path): without
history it is the plain condensation; history-decided pairs take weight 1
or 0 whatever their cosine; exactly the undecided pairs are computed,
counted by brute force over pairs."""
import itertools

import numpy as np

from oracle import luffy_oracle as O


def _case(rng, T=60, d=16, E=3, centres=8):
    c = rng.standard_normal((centres, d))
    x = c[rng.integers(0, centres, T)] + 0.05 * rng.standard_normal((T, d))
    idx = rng.integers(0, E, (T, 1)).astype(np.int32)
    offsets, perm, _ = O.dispatch(idx, E)
    return x, perm, offsets


def _same(a, b):
    for f in ("rep_of_pos", "degree", "is_rep", "rep_row", "rep_offsets", "rep_token"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f


def test_no_history_is_the_plain_condensation():
    rng = np.random.default_rng(1)
    x, perm, off = _case(rng)
    T = x.shape[0]
    plain = O.condense(x, perm, off, 0.95)
    nan = np.full((T, T), np.nan)
    _same(O.condense(x, perm, off, 0.95, history=(nan, 0.8, 0.2)), plain)
    rnd = rng.uniform(-1, 1, (T, T))
    _same(O.condense(x, perm, off, 0.95, history=(rnd, np.inf, -np.inf)), plain)   # nothing decided
    rec, n = O.historical_record(x, perm, off, nan, 0.8, 0.2)
    sizes = np.diff(off)
    assert n == int((sizes * (sizes - 1) // 2).sum())                    # every bucket pair computed


def test_hand_case_history_overrides_cosine():
    # one bucket of three tokens: cos(0,1) = 1 (copies), cos(0,2) = cos(1,2) = 0
    x = np.array([[1.0, 0.0], [2.0, 0.0], [0.0, 3.0]])
    perm, off = np.array([0, 1, 2]), np.array([0, 3])
    prev = np.full((3, 3), np.nan)
    prev[0, 1] = prev[1, 0] = 0.1        # was dissimilar: weight 0 although the copies' cosine is 1
    prev[0, 2] = prev[2, 0] = 0.9        # was similar: weight 1 although the cosine is 0
    w, comp = O.historical_weights(x, [0, 1, 2], prev, 0.8, 0.2)
    assert w[0, 1] == 0.0 and w[0, 2] == 1.0 and w[1, 2] == 0.0
    assert comp[1, 2] and not comp[0, 1] and not comp[0, 2]
    r = O.condense(x, perm, off, 0.95, history=(prev, 0.8, 0.2))
    # edges: only 0-2; degrees 1, 0, 1; token 0 keeps and absorbs 2, token 1 stays alone
    assert r.degree.tolist() == [1, 0, 1] and r.rep_of_pos.tolist() == [0, 1, 0]
    assert O.condense(x, perm, off, 0.95).rep_of_pos.tolist() == [0, 0, 2]    # without history


def test_computed_pairs_by_brute_force():
    rng = np.random.default_rng(2)
    for _ in range(3):
        x, perm, off = _case(rng, T=40)
        T = x.shape[0]
        prev = rng.uniform(-1, 1, (T, T))
        prev = (prev + prev.T) / 2
        prev[rng.random((T, T)) < 0.3] = np.nan
        S1, S2 = 0.5, -0.2
        rec, n = O.historical_record(x, perm, off, prev, S1, S2)
        cos = O.cosine(x)
        bucket = np.empty(T, np.int64)
        for e in range(len(off) - 1):
            bucket[perm[off[e]:off[e + 1]]] = e
        want_n = 0
        for a, b in itertools.combinations(range(T), 2):
            p = prev[a, b]
            if bucket[a] != bucket[b]:
                assert np.isnan(rec[a, b])
                continue
            if p > S1:
                assert rec[a, b] == 1.0
            elif p < S2:
                assert rec[a, b] == 0.0
            else:
                want_n += 1
                assert abs(rec[a, b] - cos[a, b]) < 1e-12
        assert n == want_n


def test_record_feeds_the_next_block():
    # block b leaves its weights; with the same tokens and S1 = S2 = the
    # threshold band collapsed, block b+1 decides every pair from the record
    # and computes none, and its graph equals block b's thresholded graph
    rng = np.random.default_rng(3)
    x, perm, off = _case(rng)
    T = x.shape[0]
    rec, _ = O.historical_record(x, perm, off, np.full((T, T), np.nan), 0.8, 0.2)
    rec2, n2 = O.historical_record(x, perm, off, np.where(rec >= 0.95, 1.0, 0.0), 0.5, 0.5)
    assert n2 == 0
    _same(O.condense(x, perm, off, 0.95, history=(np.where(rec >= 0.95, 1.0, 0.0), 0.5, 0.5)),
          O.condense(x, perm, off, 0.95))
