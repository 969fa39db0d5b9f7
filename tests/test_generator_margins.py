"""The generated workloads keep every decision that floating point takes
away from its boundary, at the full sizes of the benchmarked workloads
(the oracle's routing and bucketing; cosines per bucket).

* Similarity: every pair of positions in one bucket has |cos - h| >= 0.01
  for each threshold of the workload (the margin the measurement plan
  asks of the generator), so the float32 Gram on the GPU and the float64
  oracle draw the same edges.
* Routing: the float64 gaps that decide the top-k (between the k-th and
  (k+1)-th logit, and for k = 2 between the first two) are never zero and
  stay far above float64 rounding (>= 1e-9), so the GPU's float64
  re-decision of close calls and the oracle's float64 argsort agree.  The
  smallest gap is printed: it is below 1e-3 on some workloads, which is why
  the GPU re-decides close calls in float64 rather than relying on a
  routing margin.

The minima found are printed (``-s``) and recorded beside the generator's
recipe in the design notes."""
import numpy as np
import pytest

import luffy_gen as G
from oracle import luffy_oracle as O

pytestmark = pytest.mark.slow


# Cosines are taken in float32 (the full c3 buckets need 2.5 TFLOP): with
# unit rows of d <= 4096 elements the float32 dot product is within
# d * 2^-24 < 2.5e-4 of the exact cosine, so the margins are asserted with
# that slack added.
F32_SLACK = 2.5e-4


def bucket_cos_margin(x, perm_token, offsets, thresholds, chunk=2048):
    """min over pairs a != b of one bucket of |cos(x_a, x_b) - h|, per h."""
    best = {h: np.inf for h in thresholds}
    for e in range(len(offsets) - 1):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi - lo < 2:
            continue
        xb = x[perm_token[lo:hi]].astype(np.float64)
        nrm = np.linalg.norm(xb, axis=1)
        assert np.all(nrm > 0)
        xb = (xb / nrm[:, None]).astype(np.float32)
        n = hi - lo
        for r0 in range(0, n, chunk):
            c = xb[r0:r0 + chunk] @ xb.T
            idx = np.arange(r0, min(r0 + chunk, n))
            c[idx - r0, idx] = np.nan            # a position with itself is not a pair
            for h in thresholds:
                best[h] = min(best[h], float(np.nanmin(np.abs(c - h))))
    return best


def routing_gap(logits, k):
    s = -np.sort(-logits, axis=1)
    gaps = [s[:, k - 1] - s[:, k]]
    if k == 2:
        gaps.append(s[:, 0] - s[:, 1])
    return float(np.min(np.stack(gaps)))


def check_margins(inp, logits, perm_token, offsets):
    """Asserts both margins for one workload from the oracle's logits and
    buckets; returns (smallest routing gap, {h: smallest |cos - h|})."""
    cfg = inp.cfg
    gap = routing_gap(logits, cfg.k)
    margin = bucket_cos_margin(inp.x, perm_token, offsets, cfg.thresholds)
    print(f"[margins] {cfg.name} T={cfg.T}: smallest routing gap {gap:.3e}; smallest |cos - h| "
          + ", ".join(f"h={h}: {m:.4f}" for h, m in margin.items()), flush=True)
    assert gap >= 1e-9, f"{cfg.name}: routing gap {gap:.3e}"
    for h, m in margin.items():
        assert m >= 0.01 + F32_SLACK, f"{cfg.name} h={h}: |cos - h| = {m:.4f} < 0.01"
    return gap, margin


# The full c2 batch here; the full c3, c4 and c5 batches are checked by the
# full-size GPU tests on the same oracle buckets they compare against (their
# inputs take minutes to draw and route on a small host).
@pytest.mark.timeout(600)
def test_full_size_margins_c2():
    inp = G.make_inputs("c2", seed=0, weights=False)
    cfg = inp.cfg
    idx, _, logits = O.gate(inp.x.astype(np.float64), inp.w_g, inp.b_g, cfg.k)
    offsets, perm_token, _ = O.dispatch(idx, cfg.E, O.capacity_of(cfg.T, cfg.k, cfg.E, cfg.capacity_factor))
    check_margins(inp, logits, perm_token, offsets)
