"""A host model of the parallel rule by which luffy_condense decides the
highest-degree-first walk of Sec. 5.2, run under arbitrary schedules.

The device passes visit positions in any order and may read a neighbour's
state late (a plain load can return "undecided" after another XCD decided
it).  A visit of p keeps p when no neighbour is seen kept and no neighbour of
higher priority is seen undecided, and absorbs p when a neighbour is seen
kept; a visit that keeps p at once marks every neighbour absorbed and
offers p's key (degree, ~position) to it with an atomic maximum.  The model
below plays such visits in random order with random stale reads, asserts
that no visit ever writes a decision that contradicts an earlier one (kept
over absorbed or the reverse), and checks that the final states and claims
give exactly the representatives of the oracle's sequential walk, whatever
the schedule.  It pins the argument that makes claims order-independent; the
GPU tests check the kernels themselves."""
import numpy as np
import pytest

from oracle import luffy_oracle as O

UND, KEPT, ABS = 0, 1, 2


def _parallel_walk(adj, rng, stale):
    n = adj.shape[0]
    deg = adj.sum(axis=1)
    nbrs = [np.flatnonzero(adj[p]) for p in range(n)]
    state = np.zeros(n, np.int64)
    claim = np.full(n, -1, np.int64)          # key = deg * n + (n - 1 - q): larger is earlier in the walk

    def higher(q, p):
        return deg[q] > deg[p] or (deg[q] == deg[p] and q < p)

    def visit(p, s):
        seen = [UND if (state[q] != UND and rng.random() < s) else state[q] for q in nbrs[p]]
        if any(v == KEPT for v in seen):
            assert state[p] != KEPT, "a kept position was absorbed"
            state[p] = ABS
            return
        if any(v == UND and higher(q, p) for q, v in zip(nbrs[p], seen)):
            return
        assert state[p] != ABS, "an absorbed position was kept"
        state[p] = KEPT
        key = deg[p] * n + (n - 1 - p)
        for b in nbrs[p]:
            assert state[b] != KEPT, "two adjacent positions kept"
            state[b] = ABS
            claim[b] = max(claim[b], key)

    # grid rounds: every position visited once, in a random order, reads stale
    for p in rng.permutation(n):
        visit(p, stale)
    # later passes: undecided positions revisited until none is left; a few
    # sweeps may still read late, then the coherent passes read fresh states,
    # so each sweep decides at least the highest-priority undecided position
    rounds = 0
    while (state == UND).any():
        rounds += 1
        assert rounds <= n + 3
        for p in rng.permutation(np.flatnonzero(state == UND)):
            visit(p, stale if rounds <= 3 else 0.0)
    rep = np.arange(n)
    for p in range(n):
        if state[p] == ABS:
            assert claim[p] >= 0, "absorbed without a claim"
            rep[p] = n - 1 - claim[p] % n
    return rep


def _graphs(rng):
    out = []
    # union of cliques, positions shuffled
    sizes = rng.integers(1, 9, size=12)
    n = int(sizes.sum())
    lab = np.repeat(np.arange(len(sizes)), sizes)[rng.permutation(n)]
    out.append(("cliques", lab[:, None] == lab[None, :]))
    # sparse random graphs
    for pe in (0.05, 0.15, 0.4):
        a = rng.random((40, 40)) < pe
        out.append((f"gnp{pe}", a | a.T))
    # a path, in order and shuffled (a decision chain as long as the graph)
    m = 30
    a = np.zeros((m, m), bool)
    a[np.arange(m - 1), np.arange(1, m)] = True
    a |= a.T
    out.append(("path", a))
    perm = rng.permutation(m)
    out.append(("path_shuffled", a[np.ix_(perm, perm)]))
    # stars of chains: a hub with several paths hanging off it
    m = 31
    a = np.zeros((m, m), bool)
    for arm in range(5):
        nodes = [0] + list(range(1 + 6 * arm, 7 + 6 * arm))
        for u, v in zip(nodes[:-1], nodes[1:]):
            a[u, v] = a[v, u] = True
    out.append(("star_of_chains", a))
    out.append(("empty", np.zeros((20, 20), bool)))
    out.append(("complete", np.ones((15, 15), bool)))
    for _, g in out:
        np.fill_diagonal(g, False)
    return out


@pytest.mark.parametrize("seed", range(4))
def test_any_schedule_gives_the_sequential_walk(seed):
    rng = np.random.default_rng(seed)
    for name, adj in _graphs(rng):
        want, _ = O.greedy(adj)
        for trial in range(25):
            stale = (0.0, 0.3, 0.8)[trial % 3]
            got = _parallel_walk(adj, rng, stale)
            assert np.array_equal(got, want), (name, trial, stale)


def test_model_detects_an_order_dependent_claim():
    """The check has teeth: keeping the first offer instead of the largest
    (an order-dependent rule) disagrees with the walk on some schedule."""
    rng = np.random.default_rng(5)
    n = 7
    adj = np.zeros((n, n), bool)
    # the walk keeps 1, then 5, then 3; 2 (next to 1 and 3) and 4 (next to 1
    # and 5) belong to 1, the earlier of their kept neighbours, which a
    # first-offer rule misses when 3 or 5 offers first
    for u, v in ((0, 1), (1, 2), (2, 3), (1, 4), (4, 5), (5, 6)):
        adj[u, v] = adj[v, u] = True
    want, _ = O.greedy(adj)
    deg = adj.sum(axis=1)
    order = sorted(range(n), key=lambda a: (-deg[a], a))
    kept = [p for p in range(n) if want[p] == p]
    differs = False
    for _ in range(50):
        first = {}
        for p in rng.permutation(kept):
            for b in np.flatnonzero(adj[p]):
                first.setdefault(int(b), int(p))
        rep = np.array([first.get(p, p) if want[p] != p else p for p in range(n)])
        differs |= not np.array_equal(rep, want)
    assert differs and order[0] in kept
