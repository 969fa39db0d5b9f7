"""GPU parity: the HIP layer, called through the C ABI, against the CPU oracle
on the same seeded inputs.  Indices bit-exact; outputs within the per-token
relative tolerance (2e-2 bf16, 1e-5 fp32)."""
import numpy as np
import pytest

import luffy_gen as G
from oracle import luffy_oracle as O
from tests.layer_runner import (assert_condense_equal, assert_output_close,
                                assert_route_equal, run_gpu, run_oracle)

pytestmark = pytest.mark.gpu

# Reduced shapes of the five workloads: several 128-row tiles per bucket and
# ragged tails, small enough for the fp64 oracle to finish in seconds.
REDUCED = {
    "c1": dict(),
    "c2": dict(T=4096, d=512, d_ff=1024, n_centres=1024),
    "c3": dict(T=4096, d=512, d_ff=1024, n_centres=512),
    "c4": dict(T=2048, d=1024, d_ff=1408),          # d_ff not a multiple of 128
    "c5": dict(T=8192, d=512, d_ff=1024, n_centres=1024),
}


def print_case(name, **kw):
    print(f"[case] {name} {kw}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_15419_amd as L
    L.load_library()     # raises if the library is not built


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c5"])
def test_layer_reduced(name):
    inp = G.make_inputs(name, seed=0, **REDUCED[name])
    print_case(name, **REDUCED[name])
    g = run_gpu(inp)
    o = run_oracle(inp)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    assert_output_close(g, o, inp.cfg.dtype)
    assert o.rep_offsets[-1] < o.offsets[-1], "workload should condense"


def test_c4_threshold_sweep_reduced():
    inp = G.make_inputs("c4", seed=0, **REDUCED["c4"])
    from tests.layer_runner import upload
    dev = upload(inp)
    for h in inp.cfg.thresholds:
        print_case("c4", h=h, **REDUCED["c4"])
        g = run_gpu(inp, h=h, dev=dev)
        o = run_oracle(inp, h=h)
        assert_route_equal(g, o)
        assert_condense_equal(g, o)
        assert_output_close(g, o, "bf16")


def test_no_condensation_above_one():
    inp = G.make_inputs("c2", seed=1, **REDUCED["c2"])
    g = run_gpu(inp, h=2.0)
    o = run_oracle(inp, h=2.0)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    assert g["rep_offsets"][-1] == g["offsets"][-1]
    assert np.array_equal(g["rep_of_pos"], np.arange(g["offsets"][-1]))
    assert_output_close(g, o, "bf16")


def test_planted_duplicates_merge():
    inp = G.make_inputs("c4", seed=5, T=1024, d=256, d_ff=256, planted_duplicates=64)
    g = run_gpu(inp, h=0.99)
    o = run_oracle(inp, h=0.99)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    for src, cp in inp.planted:
        assert g["rep_of_pos"][g["slot_pos"][src, 0]] == g["rep_of_pos"][g["slot_pos"][cp, 0]]
    # slots that share a representative receive bit-identical expert rows
    rows = g["rep_row"][g["slot_pos"][inp.planted[:, 0], 0]]
    assert np.all(rows == g["rep_row"][g["slot_pos"][inp.planted[:, 1], 0]])
    assert_output_close(g, o, "bf16")


def test_ragged_token_count_and_single_token():
    for T in (1, 63, 1000):
        inp = G.make_inputs("c2", seed=2, T=T, d=256, d_ff=512, n_centres=max(T // 8, 1))
        print_case("c2", T=T)
        g = run_gpu(inp)
        o = run_oracle(inp)
        assert_route_equal(g, o)
        assert_condense_equal(g, o)
        assert_output_close(g, o, "bf16")


def test_empty_buckets_and_full_drop():
    # a large bias sends every token to experts 0..2; capacity drops most
    cfg = G.config("c2", T=512, d=256, d_ff=256, n_centres=32, capacity_factor=0.5)
    inp = G.make_inputs(cfg, seed=3)
    inp.b_g[:] = 0.0
    inp.b_g[:3] = 50.0
    g = run_gpu(inp)
    o = run_oracle(inp)
    assert_route_equal(g, o)
    sizes = np.diff(g["offsets"])
    assert (sizes == 0).sum() >= 10 and (g["slot_pos"] < 0).all(axis=1).any()
    assert_condense_equal(g, o)
    assert_output_close(g, o, "bf16")


def test_decimal_capacity_factor():
    """cf = 1.1 with k*T/E = 500: the capacity is exactly 550 on both sides
    (a float32 factor made it 551 on the device); the four hot buckets are
    larger, so each keeps exactly its first 550 slots, and the layer's
    max_bucket (sized from the same capacity) holds every bucket, so
    condensation still runs."""
    cfg = G.config("c2", T=2000, d=256, d_ff=256, E=8, n_centres=64, capacity_factor=1.1)
    inp = G.make_inputs(cfg, seed=4)
    assert O.capacity_of(2000, 2, 8, 1.1) == 550
    inp.b_g[:] = 0.0
    inp.b_g[:4] = 3.0          # four hot experts overflow the capacity
    print_case("capacity 1.1", T=2000, E=8, k=2)
    g = run_gpu(inp)
    o = run_oracle(inp)
    assert_route_equal(g, o)
    assert np.diff(g["offsets"]).max() == 550
    assert_condense_equal(g, o)
    assert g["rep_offsets"][-1] < g["offsets"][-1]
    assert_output_close(g, o, "bf16")


def test_identical_tokens_one_group():
    # every token identical: one clique per bucket, dense adjacency words
    inp = G.make_inputs("c2", seed=4, T=2048, d=256, d_ff=256, n_centres=1,
                        capacity_factor=0.0)
    inp.x[:] = inp.x[0]
    g = run_gpu(inp)
    o = run_oracle(inp)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    assert g["rep_offsets"][-1] == (np.diff(g["offsets"]) > 0).sum()
    assert_output_close(g, o, "bf16")


def _path_inputs(n_tokens, d, shuffle, seed):
    # x_i = e_i + e_{i+1}: cos 1/2 between path neighbours, 0 otherwise, so
    # the threshold graph at h = 0.25 is a path (bf16-exact values).
    cfg = G.config("c2", T=n_tokens, d=d, d_ff=128, E=1, k=1, n_centres=1,
                   capacity_factor=0.0, thresholds=(0.25,))
    inp = G.make_inputs(cfg, seed=seed)
    x = np.zeros((n_tokens, d), np.float32)
    idx = np.arange(n_tokens)
    x[idx, idx] = 1.0
    x[idx, idx + 1] = 1.0
    if shuffle:
        x = x[np.random.default_rng(seed).permutation(n_tokens)]
    inp.x = x
    return inp


@pytest.mark.parametrize("n,shuffle", [(511, False), (511, True), (4000, False), (4000, True)])
def test_long_chain_needs_many_rounds(n, shuffle):
    """Threshold graphs that are paths: a decision chain as long as the
    bucket, which the grid rounds leave mostly undecided; the finishing
    pass takes a few rounds and then visits the rest once each in priority
    order (4000 positions: the sorted pass over a list of thousands)."""
    print_case("path", n=n, shuffle=shuffle)
    inp = _path_inputs(n, (n // 64 + 2) * 64, shuffle, seed=6)
    g = run_gpu(inp)
    o = run_oracle(inp)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    assert_output_close(g, o, "bf16")


def test_deterministic_indices():
    inp = G.make_inputs("c3", seed=0, **REDUCED["c3"])
    a = run_gpu(inp)
    b = run_gpu(inp)
    for key in ("topk_idx", "slot_pos", "perm_token", "rep_of_pos", "rep_row", "rep_token",
                "degree"):
        assert np.array_equal(a[key], b[key]), key
    assert np.array_equal(a["y"], b["y"])


@pytest.mark.parametrize("name", ["c1", "c2"])
def test_norms_computed_by_condense(name):
    # luffy_condense computing the norms itself (no inv_norm from luffy_route)
    inp = G.make_inputs(name, seed=0, **REDUCED[name])
    g = run_gpu(inp, norms_from_route=False)
    o = run_oracle(inp)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    assert_output_close(g, o, inp.cfg.dtype)


def test_gathered_rows_path_matches():
    inp = G.make_inputs("c2", seed=0, **REDUCED["c2"])
    g = run_gpu(inp, gather_x_rep=True)
    o = run_oracle(inp)
    assert_condense_equal(g, o)
    assert np.array_equal(g["x_rep"], inp.x[o.rep_token])
    assert_output_close(g, o, "bf16")


def _bf16(a):
    """Round float64 values to bfloat16 (nearest even) and back, in numpy."""
    import torch
    return torch.from_numpy(np.asarray(a, np.float64)).to(torch.bfloat16).double().numpy()


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_activation_values_bf16(act):
    """Identity weights make the expert FFN return bf16(act(x)) for every
    input element, so the device activation is compared value by value with
    the oracle's exact one: equal, or one bf16 step apart where the exact
    value lies next to a rounding boundary."""
    import torch
    import paper_2411_15419_amd as L
    d = 64
    z = _bf16(np.linspace(-9.0, 9.0, 512 * d)).reshape(512, d)
    x = torch.from_numpy(z).to(torch.bfloat16).cuda()
    eye = torch.eye(d, dtype=torch.bfloat16, device="cuda")[None]
    off = torch.tensor([0, 512], dtype=torch.int32, device="cuda")
    y = torch.empty(512, d, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(L.expert_ffn_workspace_size(512, 1, d, L.LUFFY_BF16), dtype=torch.uint8,
                     device="cuda")
    L.luffy_expert_ffn(x, None, off, eye, eye.clone(), act, 512, y, ws)
    got = y.double().cpu().numpy()
    exact = O.activation(z, act)
    ref = _bf16(exact)
    step = np.maximum(np.abs(ref), 2.0 ** -126) * 2.0 ** -7   # one bf16 ulp (upper bound)
    # GELU's erf is within 1.5e-7 absolute (Abramowitz & Stegun 7.1.26), so
    # GELU is within 0.5 |z| 1.5e-7 absolute; taken as 0.5 |z| 2e-7 to cover
    # the ulps of the hardware exp2 and reciprocal.  That is below one bf16
    # step except where GELU(z) is tiny (z < -4).
    slack = 0.5 * np.abs(z) * 2e-7 if act == "gelu" else 0.0
    bad = np.abs(got - ref) > step + slack
    assert not bad.any(), (f"{bad.sum()} values off by more than one bf16 step, e.g. "
                           f"x={z[bad][:4]} got={got[bad][:4]} want={ref[bad][:4]}")
    # away from rounding boundaries the device value rounds to the same bf16
    core = z >= -4.0
    assert np.mean(got[core] == ref[core]) > 0.99


@pytest.mark.parametrize("d,d_ff", [(256, 512), (256, 1024), (64, 64), (128, 192), (192, 576), (64, 2048),
                                   (1280, 768)])
def test_expert_ffn_tile_shapes(d, d_ff):
    """The bf16 expert FFN on expert sizes that pick every tile shape: empty,
    1 row, 255-257 rows (narrow tiles, one of them partial), 300 and 320
    (one 320-row tile instead of 256 + rest), 321 (narrow again), 600 (two
    320-row tiles instead of three) and 700 (narrow); representative rows
    gathered through a permuted row index.  On 256 CUs the second product
    (14 token tiles times d/256 column tiles) splits K in 2 at d_ff = 512,
    in 4 at 1024 and 2048, in 2 parts of 4 and 5 64-wide K stages at 576,
    and in 3 parts of 4 stages at d = 1280, d_ff = 768 (70 tiles).  d and
    d_ff of 64 to 192
    give products of 1 to 3 stages (the pipeline's prologue and tail only).
    Each output row within the bf16 tolerance of the oracle's fp64 product
    on the same bf16 inputs; run twice, bit-identical (the parts are summed
    in a fixed order)."""
    import torch
    import paper_2411_15419_amd as L
    from tests.layer_runner import TOL, rel_err_rows
    sizes = [0, 1, 255, 256, 257, 300, 320, 321, 600, 700]
    print_case("expert_ffn", d=d, d_ff=d_ff, sizes=sizes)
    E = len(sizes)
    R = sum(sizes)
    rng = np.random.default_rng(11)
    x_all = _bf16(rng.standard_normal((R + 100, d)))
    row_index = rng.permutation(R + 100)[:R].astype(np.int32)
    w1 = _bf16(0.05 * rng.standard_normal((E, d_ff, d)))
    w2 = _bf16(0.05 * rng.standard_normal((E, d, d_ff)))
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    dev = lambda a, dt=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(dt).cuda()
    y = torch.empty(R, d, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(L.expert_ffn_workspace_size(R, E, d_ff, L.LUFFY_BF16), dtype=torch.uint8, device="cuda")
    args = (dev(x_all), dev(row_index, torch.int32), dev(offsets, torch.int32), dev(w1), dev(w2))
    ref = O.expert_ffn(x_all[row_index], offsets, w1, w2, "gelu")
    first = None
    for call in range(2):
        y.fill_(float("nan"))
        L.luffy_expert_ffn(*args, "gelu", R, y, ws)
        got = y.double().cpu().numpy()
        err, _ = rel_err_rows(got, ref)
        assert err.max() <= TOL["bf16"], f"call {call}: max row rel err {err.max():.3g}"
        if first is None:
            first = got
        else:
            assert np.array_equal(first, got), "the split sum differs between calls"


def test_expert_ffn_split_tail():
    """More second-product tiles than blocks with a partial round left: 40
    experts of 1, 60, 128, 129, 256, 257, 300 and 320 rows (every tile
    shape) times 8 column tiles (d = 2048) make 320 tiles; on 256 CUs the
    first 256 run whole and the 64 left over (the last 8 experts, every
    shape again) run in 4 parts of 4 K-stages each (d_ff = 1024), finished
    by the reduction.  Each output row within the bf16 tolerance of the
    oracle; two calls bit-identical."""
    import torch
    import paper_2411_15419_amd as L
    from tests.layer_runner import TOL, rel_err_rows
    d, d_ff = 2048, 1024
    sizes = [1, 60, 128, 129, 256, 257, 300, 320] * 5
    print_case("expert_ffn_split_tail", d=d, d_ff=d_ff, E=len(sizes))
    E, R = len(sizes), sum(sizes)
    rng = np.random.default_rng(12)
    x = _bf16(rng.standard_normal((R, d)))
    w1 = _bf16(0.03 * rng.standard_normal((E, d_ff, d)))
    w2 = _bf16(0.03 * rng.standard_normal((E, d, d_ff)))
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    dev = lambda a, dt=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(dt).cuda()
    y = torch.empty(R, d, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(L.expert_ffn_workspace_size(R, E, d_ff, L.LUFFY_BF16), dtype=torch.uint8, device="cuda")
    args = (dev(x), None, dev(offsets, torch.int32), dev(w1), dev(w2))
    ref = O.expert_ffn(x, offsets, w1, w2, "gelu")
    first = None
    for call in range(2):
        y.fill_(float("nan"))
        L.luffy_expert_ffn(*args, "gelu", R, y, ws)
        got = y.double().cpu().numpy()
        err, _ = rel_err_rows(got, ref)
        assert err.max() <= TOL["bf16"], f"call {call}: max row rel err {err.max():.3g}"
        if first is None:
            first = got
        else:
            assert np.array_equal(first, got), "the split sum differs between calls"


@pytest.mark.parametrize("T,d,E,k", [(32768, 256, 24, 2), (32768, 2560, 24, 2), (70001, 2560, 24, 2),
                                     (66000, 1024, 40, 1), (5000, 3072, 48, 2), (80000, 2048, 64, 1)])
def test_route_large_batch(T, d, E, k):
    """luffy_route on a large batch: top-k, gates, dispatch with capacity,
    and 1/|x_t| against the oracle.  With a weight matrix of at most 128 KB
    and at least one 16-token chunk per wave of its grid (T >= 65536 on 256
    CUs) the streaming gate runs (T = 70001 ragged; E = 24 or 40 leave part
    of the last 16-expert MFMA block unused; d = 2560 is not a power of
    two); otherwise the blocked gate, with 64-token chunks at T >= 32768 and
    32-token ones below, and for weights of 288 KB (48 x 3072) or 256 KB
    (64 x 2048) at any T."""
    import torch
    import paper_2411_15419_amd as L
    cf = 1.25
    print_case("route", T=T, d=d, E=E, k=k)
    rng = np.random.default_rng(13)
    x = _bf16(rng.standard_normal((T, d)))
    wg = _bf16(rng.standard_normal((E, d)) / np.sqrt(d))
    bg = (0.1 * rng.standard_normal(E)).astype(np.float32)
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dt).cuda()
    i32 = dict(dtype=torch.int32, device="cuda")
    ti, sp = torch.empty(T, k, **i32), torch.empty(T, k, **i32)
    tg = torch.empty(T, k, dtype=torch.float32, device="cuda")
    pt, off = torch.empty(T * k, **i32), torch.empty(E + 1, **i32)
    nrm = torch.empty(T, dtype=torch.float32, device="cuda")
    ws = torch.empty(L.route_workspace_size(T, E, k), dtype=torch.uint8, device="cuda")
    L.luffy_route(dev(x, torch.bfloat16), dev(wg, torch.bfloat16), dev(bg, torch.float32), k, cf, ti, tg, sp, pt,
                  off, ws, inv_norm=nrm)
    o_idx, o_gate, _ = O.gate(x, wg, bg, k)
    o_off, o_perm, o_pos = O.dispatch(o_idx, E, O.capacity_of(T, k, E, cf))
    assert np.array_equal(ti.cpu().numpy(), o_idx), "topk_idx differs"
    assert np.allclose(tg.cpu().numpy(), o_gate, rtol=0, atol=2e-6)
    assert np.array_equal(off.cpu().numpy(), o_off), "offsets differ"
    assert np.array_equal(sp.cpu().numpy(), o_pos), "slot_pos differs"
    assert np.array_equal(pt.cpu().numpy()[:o_off[-1]], o_perm), "perm_token differs"
    ref = 1.0 / np.sqrt((x.astype(np.float64) ** 2).sum(axis=1))
    assert np.allclose(nrm.cpu().numpy(), ref, rtol=2e-6, atol=0)


@pytest.mark.parametrize("dtype,k,d", [("bf16", 2, 2048), ("bf16", 1, 1024), ("bf16", 1, 4096),
                                       ("bf16", 2, 8192), ("bf16", 2, 64), ("f32", 1, 256), ("f32", 2, 64),
                                       ("f32", 2, 256), ("bf16", 2, 192), ("f32", 1, 192)])
def test_combine_shapes(dtype, k, d):
    """luffy_combine alone against the oracle's combine on synthetic rows:
    top-2 on the column-sliced kernel (a row's 16-byte chunks split into
    eight slices of 1, 2, 32 and 2 x 64 chunks), top-1 and d = 192 (slices
    of 3 chunks) on the one-wave-per-token kernel.  About a
    sixth of the slots are dropped, some tokens lose every slot (their rows
    must be exactly zero), and T is not a multiple of any block's tokens."""
    import torch
    import paper_2411_15419_amd as L
    T, R = 3001, 517
    print_case("combine", dtype=dtype, k=k, d=d, T=T, R=R)
    rng = np.random.default_rng(100 + d + k)
    y_rep = rng.standard_normal((R, d))
    if dtype == "bf16":
        y_rep = _bf16(y_rep)
    S = T * k
    rep_row = rng.integers(0, R, size=S).astype(np.int32)
    slot_pos = rng.permutation(S).astype(np.int32).reshape(T, k)
    slot_pos[rng.random((T, k)) < 0.17] = -1
    slot_pos[:7] = -1                                  # tokens with no kept slot
    gate = rng.random((T, k)).astype(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dt).cuda()
    y = torch.full((T, d), float("nan"), dtype=tdt, device="cuda")
    L.luffy_combine(dev(y_rep, tdt), dev(rep_row, torch.int32), dev(slot_pos, torch.int32),
                    dev(gate, torch.float32), y)
    got = y.double().cpu().numpy()
    ref = O.combine(y_rep, rep_row, slot_pos, gate.astype(np.float64))
    assert np.all(got[:7] == 0.0), "tokens without a kept slot must be zero"
    # per element: bf16 rounding of an fp32 sum (2^-9 relative) or the fp32
    # sum of at most two products
    scale = sum(np.abs(gate[:, j:j + 1].astype(np.float64) *
                       np.where(slot_pos[:, j:j + 1] >= 0, y_rep[rep_row[np.maximum(slot_pos[:, j], 0)]], 0.0))
                for j in range(k))
    rtol = 2.0 ** -8 if dtype == "bf16" else 1e-6
    bad = np.abs(got - ref) > rtol * scale + 1e-30
    assert not bad.any(), f"{bad.sum()} elements out of tolerance, first at {np.argwhere(bad)[0]}"


def test_graph_replay_matches_eager():
    """The whole layer captured once in a HIP graph (every call is
    asynchronous, allocates nothing and clears its scratch with kernels, so
    it captures) and replayed four times, with unrelated eager work and a
    synchronisation between replays and the input changed in place before
    two of them: every replay equals the eager run on the same input,
    indices and outputs bit for bit."""
    import torch
    from tests.layer_runner import make_layer, upload
    inp = G.make_inputs("c2", seed=3, **REDUCED["c2"])
    print_case("graph_replay", **REDUCED["c2"])
    dev = upload(inp)
    x = dev["x"]
    x_other = torch.flip(x, dims=[0]).contiguous()
    x_orig = x.clone()
    layer = make_layer(inp, dev)
    names = ["topk_idx", "slot_pos", "perm_token", "offsets", "rep_of_pos", "rep_row",
             "rep_offsets", "rep_token", "y"]

    def snapshot():
        torch.cuda.synchronize()
        return {n: getattr(layer.buf, n).clone() for n in names}

    def eager(src):
        x.copy_(src)
        layer(x)
        return snapshot()

    # warm up on a side stream, as capture requires
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        layer(x)
    torch.cuda.current_stream().wait_stream(s)
    ref = {"orig": eager(x_orig), "other": eager(x_other)}
    x.copy_(x_orig)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer(x)
    junk = torch.zeros(1 << 20, device="cuda")
    for i, which in enumerate(["orig", "orig", "other", "orig"]):
        x.copy_(x_orig if which == "orig" else x_other)
        junk.add_(1.0)                     # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        got = snapshot()
        for n in names:
            assert torch.equal(got[n], ref[which][n]), f"replay {i} ({which}): {n} differs"
