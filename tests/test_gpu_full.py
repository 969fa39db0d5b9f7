"""GPU parity at the full workload sizes, in the launch configuration the
throughput benchmark times (one MoELayer call on inputs resident in HBM).

Indices (routing, buckets, degrees, representatives, compaction) are compared
bit-exactly with the oracle over the whole batch.  Layer outputs are compared
on every row: the oracle evaluates the expert FFN in fp64 on every
representative (the index maps having been found identical first) and
combines as the layer does; Y_rep and y are held to the per-row relative
tolerance.  The generator's margins (similarity 0.01 from every threshold,
routing gaps) are asserted on the same oracle buckets."""
import numpy as np
import pytest

import luffy_gen as G
from oracle import luffy_oracle as O
from tests.layer_runner import (TOL, assert_condense_equal, assert_route_equal, fetch,
                                make_layer, rel_err_rows, upload)
from tests.test_generator_margins import check_margins

pytestmark = [pytest.mark.gpu, pytest.mark.slow]



@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_15419_amd as L
    L.load_library()


def print_case(name, **kw):
    print(f"[case] {name} {kw}", flush=True)


def run_layer(inp, dev, h):
    layer = make_layer(inp, dev, h)
    layer(dev["x"])
    return fetch(layer)


def full_expected(inp, o):
    """fp64 Y_rep of every representative and y of every token, from the
    oracle's own indices (found identical to the GPU's first)."""
    cfg = inp.cfg
    y_rep = O.expert_ffn(inp.x[o.rep_token].astype(np.float64), o.rep_offsets, inp.w1, inp.w2, cfg.act)
    y = O.combine(y_rep, o.rep_row, o.slot_pos, o.topk_gate)
    return y_rep, y


def assert_all_rows_close(g, inp, o, y_rep_ref, y_ref):
    """Every row of Y_rep and of y within the dtype's per-row relative
    tolerance; fully dropped tokens exactly zero."""
    tol = TOL[inp.cfg.dtype]
    R = y_rep_ref.shape[0]
    err_rep, _ = rel_err_rows(g["y_rep"][:R], y_rep_ref)
    assert err_rep.max() <= tol, f"Y_rep max row rel err {err_rep.max():.3g} (row {int(err_rep.argmax())})"
    dropped = (o.slot_pos < 0).all(axis=1)
    assert np.all(g["y"][dropped] == 0), "fully dropped tokens must be zero"
    err, _ = rel_err_rows(g["y"], y_ref)
    assert err.max() <= tol, f"y max row rel err {err.max():.3g}"
    print(f"[all rows] {R} representatives, {int((~dropped).sum())} tokens with a kept slot, "
          f"{int(dropped.sum())} fully dropped; max row rel err Y_rep {err_rep.max():.3g}, y {err.max():.3g}",
          flush=True)


def assert_clique_union(inp, o):
    """On clustered inputs the threshold graph is a union of cliques, one per
    centre and bucket, so the representative of a slot is the first position
    of its bucket drawn from the same centre (independent of any similarity
    code; the oracle's own cosines confirm the premise in the CPU tests)."""
    cid = inp.centre_id[o.perm_token]
    for e in range(len(o.offsets) - 1):
        lo, hi = int(o.offsets[e]), int(o.offsets[e + 1])
        _, first = np.unique(cid[lo:hi], return_index=True)
        first_of = dict(zip(cid[lo:hi][first].tolist(), (first + lo).tolist()))
        want = np.array([first_of[c] for c in cid[lo:hi].tolist()], np.int64)
        assert np.array_equal(o.rep_of_pos[lo:hi], want), f"bucket {e} is not a clique union"


# The fp64 oracle's Gram and expert FFN over the largest workloads take tens
# of seconds on the host, so these tests get longer limits than the default.
@pytest.mark.parametrize("name", [
    pytest.param("c2", marks=pytest.mark.timeout(300)),
    pytest.param("c3", marks=pytest.mark.timeout(600)),
    pytest.param("c5", marks=pytest.mark.timeout(300)),
])
def test_full_size_layer(name):
    inp = G.make_inputs(name, seed=0)
    cfg = inp.cfg
    print_case(name, T=cfg.T, d=cfg.d, E=cfg.E, k=cfg.k, d_ff=cfg.d_ff, h=cfg.h)
    dev = upload(inp)
    g = run_layer(inp, dev, cfg.h)
    o = run_oracle_indices(inp, cfg.h)
    check_margins(inp, o.logits, o.perm_token, o.offsets)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    assert_clique_union(inp, o)
    y_rep_ref, y_ref = full_expected(inp, o)
    assert_all_rows_close(g, inp, o, y_rep_ref, y_ref)


def run_oracle_indices(inp, h):
    cfg = inp.cfg
    return O.moe_layer(inp.x, inp.w_g, inp.b_g, None, None, k=cfg.k, h=h, act=cfg.act,
                       capacity_factor=cfg.capacity_factor, with_ffn=False)


@pytest.mark.timeout(900)
def test_full_size_c4_threshold_sweep():
    inp = G.make_inputs("c4", seed=0)
    cfg = inp.cfg
    dev = upload(inp)
    ref = None
    for h in cfg.thresholds:
        print_case("c4", T=cfg.T, d=cfg.d, E=cfg.E, d_ff=cfg.d_ff, h=h)
        g = run_layer(inp, dev, h)
        o = run_oracle_indices(inp, h)
        assert_route_equal(g, o)
        assert_condense_equal(g, o)
        assert o.rep_offsets[-1] == o.offsets[-1], "i.i.d. tokens should not merge"
        if ref is None:
            check_margins(inp, o.logits, o.perm_token, o.offsets)
            ref = full_expected(inp, o)     # nothing merges: the same at every threshold
        assert_all_rows_close(g, inp, o, *ref)


@pytest.mark.timeout(300)
def test_full_size_backward_c2():
    """The backward at the full c2 size (T = 8192, d = 1024, E = 16,
    d_ff = 4096), as `bench.py --backward` runs it (MoELayer.backward after
    one forward whose indices match the oracle's), checked on seeded samples
    the oracle computes one by one from the GPU's own forward values:
    dgate of sampled slots, dy_rep of sampled representatives (their member
    sums), dx_rep of sampled representatives (the FFN gradient of one row),
    and sampled entries of dW1 and dW2 of two experts (sums over all their
    representatives, held to 2e-2 of the sum of the terms' magnitudes)."""
    import torch
    inp = G.make_inputs("c2", seed=0)
    print_case("backward c2 full")
    dev = upload(inp)
    layer = make_layer(inp, dev)
    layer(dev["x"])
    g = fetch(layer)
    o = O.moe_layer(inp.x.astype(np.float64), inp.w_g, inp.b_g, inp.w1, inp.w2, k=inp.cfg.k, h=inp.cfg.h,
                    act=inp.cfg.act, capacity_factor=inp.cfg.capacity_factor, with_ffn=False)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    T, d = layer.buf.y.shape
    act = inp.cfg.act
    rng = np.random.default_rng(31)
    dy = torch.randn(T, d, generator=torch.Generator().manual_seed(31)).to(torch.bfloat16)
    dy_np = dy.double().numpy()
    dgate, dx_rep, dw1, dw2 = layer.backward(dev["x"], dy.cuda())
    torch.cuda.synchronize()
    dy_rep = layer._bwd["dy_rep"].double().cpu().numpy()
    dgate, dx_rep = dgate.double().cpu().numpy(), dx_rep.double().cpu().numpy()
    y_rep = g["y_rep"].astype(np.float64)
    R = int(g["rep_offsets"][-1])
    # dgate of sampled kept slots
    kept_t, kept_j = np.nonzero(g["slot_pos"] >= 0)
    for i in rng.choice(kept_t.size, 64, replace=False):
        t, j = kept_t[i], kept_j[i]
        r = g["rep_row"][g["slot_pos"][t, j]]
        ref = dy_np[t] @ y_rep[r]
        assert abs(dgate[t, j] - ref) <= 1e-4 * np.linalg.norm(dy_np[t]) * np.linalg.norm(y_rep[r]), (t, j)
    # dy_rep of sampled representatives: the gate-weighted sum of their members' dy
    S = int(g["offsets"][-1])
    pos_t = g["perm_token"]
    pos_gate = np.zeros(S)
    for j in range(g["slot_pos"].shape[1]):
        kept = g["slot_pos"][:, j] >= 0
        pos_gate[g["slot_pos"][kept, j]] = g["topk_gate"][kept, j]
    reps = rng.choice(R, 32, replace=False)
    for r in reps:
        members = np.flatnonzero(g["rep_row"][:S] == r)
        ref = (pos_gate[members, None] * dy_np[pos_t[members]]).sum(axis=0)
        err = np.abs(dy_rep[r] - ref).max() / np.abs(ref).max()
        assert err <= TOL["bf16"], f"dy_rep row {r}: {err:.3g}"
    # dx_rep of sampled representatives, from the GPU's dy_rep rows
    ro = g["rep_offsets"]
    xr = inp.x.astype(np.float64)[g["rep_token"]]
    for r in reps:
        e = int(np.searchsorted(ro, r, side="right") - 1)
        z = xr[r] @ inp.w1[e].T
        dz = (dy_rep[r] @ inp.w2[e]) * O.activation_grad(z, act)
        ref = dz @ inp.w1[e]
        err = np.abs(dx_rep[r] - ref).max() / np.abs(ref).max()
        assert err <= TOL["bf16"], f"dx_rep row {r}: {err:.3g}"
    # sampled weight-gradient entries of two experts
    gw1, gw2 = dw1.double().cpu().numpy(), dw2.double().cpu().numpy()
    for e in (0, inp.cfg.E - 1):
        lo, hi = int(ro[e]), int(ro[e + 1])
        z = xr[lo:hi] @ inp.w1[e].T
        a = O.activation(z, act)
        da = dy_rep[lo:hi] @ inp.w2[e]
        dz = da * O.activation_grad(z, act)
        for _ in range(16):
            i, c = rng.integers(inp.cfg.d_ff), rng.integers(d)
            ref1 = dz[:, i] @ xr[lo:hi, c]
            b1 = (np.abs(da[:, i]) * (np.abs(O.activation_grad(z[:, i], act)) + np.abs(z[:, i]))) @ np.abs(xr[lo:hi, c])
            assert abs(gw1[e, i, c] - ref1) <= TOL["bf16"] * b1, ("dW1", e, i, c)
            ref2 = dy_rep[lo:hi, c] @ a[:, i]
            b2 = np.abs(dy_rep[lo:hi, c]) @ (np.abs(a[:, i]) + np.abs(z[:, i]) * np.abs(O.activation_grad(z[:, i], act)))
            assert abs(gw2[e, c, i] - ref2) <= TOL["bf16"] * b2, ("dW2", e, c, i)
    print(f"[sampled backward] R={R}, 64 gate slots, {reps.size} rows, 64 weight entries ok", flush=True)
