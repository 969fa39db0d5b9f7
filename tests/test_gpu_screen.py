"""GPU parity of the fp8 similarity screen of luffy_condense.

The screen estimates every cosine of a 256 x 256 tile on fp8 copies of the
rows and decides the tile from the estimates only when none lies within the
rows' quantisation bound of the threshold; other tiles go back to the bf16
pass.  So a screened call must give exactly the outputs of the all-bf16 call:
checked on the generator's clustered tokens at d = 2048 and 4096 (also
against the oracle) and on tokens built so that many pairs have cosines
near the threshold, where most tiles must be handed back."""
import numpy as np
import pytest

import luffy_gen as G
from tests.layer_runner import assert_condense_equal, assert_route_equal, run_gpu, run_oracle, upload

pytestmark = pytest.mark.gpu

KEYS = ("offsets", "perm_token", "rep_of_pos", "rep_row", "rep_offsets", "rep_token", "degree")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_15419_amd as L
    L.load_library()


def _run(inp, screen, h=None, dev=None, norms_from_route=True):
    import paper_2411_15419_amd as L
    prev = L.set_similarity_screen(screen)
    try:
        cfg = inp.cfg
        assert L.similarity_screen_applies(cfg.T, cfg.d, cfg.E, cfg.k) == screen
        return run_gpu(inp, h=h, with_ffn=False, dev=dev, norms_from_route=norms_from_route)
    finally:
        L.set_similarity_screen(prev)


def _assert_same(a, b):
    for key in KEYS:
        bad = np.flatnonzero(a[key] != b[key])
        assert bad.size == 0, f"{key} differs at {bad[:10]}"


@pytest.mark.parametrize("name,over", [
    ("c3", dict(T=4096, E=4, n_centres=512)),            # d = 2048, k = 2
    ("c3", dict(T=3000, E=4, n_centres=300)),            # ragged buckets
    ("c4", dict(T=4096, E=4)),                           # d = 4096, i.i.d. tokens
])
def test_screen_generator_tokens(name, over):
    inp = G.make_inputs(name, seed=1, weights=False, **over)
    print(f"[case] {name} {over}", flush=True)
    dev = upload(inp)
    for h in inp.cfg.thresholds[:2]:
        on = _run(inp, True, h=h, dev=dev)
        off = _run(inp, False, h=h, dev=dev)
        _assert_same(on, off)
        o = run_oracle(inp, h=h, with_ffn=False)
        assert_route_equal(on, o)
        assert_condense_equal(on, o)


def _near_threshold_inputs(T, d, h, seed):
    """Tokens 0..T/2-1: x = u + s g with s spread so that their pairwise
    cosines, about 1 / sqrt((1 + s_a^2)(1 + s_b^2)), cover h - 0.13 .. h + 0.08
    (the screen cannot decide those tiles); tokens T/2..: tight clusters
    along other directions (cosines near 1 among themselves, near 0 to the
    first half: tiles the screen decides)."""
    inp = G.make_inputs("c3", seed=seed, weights=False, T=T, E=2, k=1, n_centres=64)
    rng = np.random.default_rng(seed)
    half = T // 2
    u = rng.standard_normal(d).astype(np.float32)
    s = rng.uniform(0.15, 0.55, size=(half, 1)).astype(np.float32)
    x = np.empty((T, d), np.float32)
    x[:half] = u + s * rng.standard_normal((half, d)).astype(np.float32)
    centres = rng.standard_normal((16, d)).astype(np.float32)
    x[half:] = centres[rng.integers(0, 16, T - half)] + 0.05 * rng.standard_normal((T - half, d)).astype(np.float32)
    inp.x = G.round_bf16(x)
    return inp


@pytest.mark.parametrize("T,seed", [(4096, 0), (2500, 1)])
def test_screen_hands_back_close_tiles(T, seed):
    h = 0.9
    inp = _near_threshold_inputs(T, 2048, h, seed)
    print(f"[case] near-threshold T={T} seed={seed}", flush=True)
    dev = upload(inp)
    on = _run(inp, True, h=h, dev=dev)
    off = _run(inp, False, h=h, dev=dev)
    _assert_same(on, off)
    assert on["degree"].max() > 0 and (on["rep_offsets"][-1] < on["offsets"][-1])


def test_screen_repeat_calls_identical():
    """The screen's counters are reset by every call: two calls in a row,
    the second on a smaller batch, match their all-bf16 runs."""
    for T in (4096, 2048):
        inp = _near_threshold_inputs(T, 2048, 0.9, 7)
        dev = upload(inp)
        _assert_same(_run(inp, True, h=0.9, dev=dev), _run(inp, False, h=0.9, dev=dev))


def test_screen_norms_computed_by_condense():
    """The screen's fp8 rows written by the norm pass that also computes the
    norms (no norms from the route call)."""
    inp = _near_threshold_inputs(3000, 2048, 0.9, 3)
    dev = upload(inp)
    on = _run(inp, True, h=0.9, dev=dev, norms_from_route=False)
    off = _run(inp, False, h=0.9, dev=dev, norms_from_route=False)
    _assert_same(on, off)


@pytest.mark.parametrize("h", [0.02, 0.999])
def test_screen_extreme_thresholds(h):
    """Thresholds at the ends of the range: near 0 the rows past a bucket
    (zero products) and many cross-centre cosines fall inside the band, near
    1 the same-centre cosines (about 0.9996) do, so many tiles go back to the
    bf16 pass; the outputs still equal the all-bf16 call bit for bit.  (The
    oracle is not compared here: at these thresholds some float64 cosines
    lie within float32 rounding of h, which is the all-bf16 path's own
    precision, not the screen's.)"""
    inp = G.make_inputs("c3", seed=4, weights=False, T=3000, E=4, n_centres=300)
    print(f"[case] extreme threshold h={h}", flush=True)
    dev = upload(inp)
    on = _run(inp, True, h=h, dev=dev)
    off = _run(inp, False, h=h, dev=dev)
    _assert_same(on, off)
    assert on["degree"].max() > 0
