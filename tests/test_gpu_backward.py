"""GPU parity of the condensed layer's backward, called through the C ABI,
against the oracle's gradients on the same arrays.  The forward runs on the
GPU first (its indices are checked against the oracle's, so the backward is
compared on the same condensation) and the backward's oracle takes the
GPU's forward values as inputs."""
import numpy as np
import pytest

import luffy_gen as G
from oracle import luffy_oracle as O
from tests.layer_runner import TOL, assert_condense_equal, assert_route_equal, fetch, make_layer, \
    rel_err_rows, run_oracle, upload
from tests.test_gpu_parity import REDUCED, print_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_15419_amd as L
    L.load_library()


def _forward(name, seed=0, **kw):
    inp = G.make_inputs(name, seed=seed, **{**REDUCED[name], **kw})
    dev = upload(inp)
    layer = make_layer(inp, dev)
    layer(dev["x"])
    g = fetch(layer)
    o = run_oracle(inp)
    assert_route_equal(g, o)
    assert_condense_equal(g, o)
    return inp, dev, layer, g


def _bf16_exact(a):
    import torch
    return torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).float().numpy().astype(np.float64)


@pytest.mark.parametrize("name", ["c1", "c2", "c5"])
def test_combine_backward(name):
    """dy_rep and dgate of luffy_combine_backward against the oracle's
    transpose of combine, per representative row within the dtype's
    tolerance; dgate within 1e-4 of |dy_t| |y_rep_r| (float32 sums of exact
    products); dropped slots get dgate = 0."""
    import torch
    import paper_2411_15419_amd as L
    print_case("combine_backward", config=name, **REDUCED[name])
    inp, dev, layer, g = _forward(name)
    b = layer.buf
    T, d = b.y.shape
    k = b.slot_pos.shape[1]
    rng = np.random.default_rng(17)
    dy_np = rng.standard_normal((T, d))
    if inp.cfg.dtype == "bf16":
        dy_np = _bf16_exact(dy_np)
    dt = b.y.dtype
    dy = torch.from_numpy(dy_np.astype(np.float32)).to(dt).cuda()
    dy_rep = torch.full_like(b.y_rep, float("nan"))
    dgate = torch.full((T, k), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(L.combine_backward_workspace_size(T, k, b.y_rep.shape[0]), dtype=torch.uint8,
                     device="cuda")
    for rep in range(2):                        # a second call on the written outputs and workspace
        L.luffy_combine_backward(dy, b.y_rep, b.rep_row, b.perm_token, b.slot_pos, b.topk_gate, b.offsets,
                                 b.rep_offsets, dy_rep, dgate, ws)
        torch.cuda.synchronize()
        R = int(g["rep_offsets"][-1])
        ref_rep, ref_gate = O.combine_backward(dy_np, g["y_rep"].astype(np.float64), g["rep_row"],
                                               g["slot_pos"], g["topk_gate"].astype(np.float64))
        got_rep = dy_rep[:R].double().cpu().numpy()
        err, _ = rel_err_rows(got_rep, ref_rep[:R])
        assert err.size and err.max() <= TOL[inp.cfg.dtype], f"call {rep}: dy_rep max row rel err {err.max():.3g}"
        got_gate = dgate.double().cpu().numpy()
        kept = g["slot_pos"] >= 0
        assert np.all(got_gate[~kept] == 0.0)
        rows = g["rep_row"][g["slot_pos"][kept]]
        scale = np.linalg.norm(dy_np, axis=1)[np.nonzero(kept)[0]] * np.linalg.norm(g["y_rep"][rows], axis=1)
        gerr = np.abs(got_gate[kept] - ref_gate[kept])
        assert np.all(gerr <= 1e-4 * scale + 1e-30), f"call {rep}: dgate max err / scale {(gerr / scale).max():.3g}"


@pytest.mark.parametrize("d,d_ff,act,dw", [(256, 512, "gelu", "f32"), (256, 1024, "silu", "f32"),
                                            (128, 192, "gelu", "f32"), (256, 512, "gelu", "bf16"),
                                            (192, 320, "silu", "bf16")])
def test_expert_ffn_backward(d, d_ff, act, dw):
    """luffy_expert_ffn_backward on the expert sizes of the forward tile
    test (empty, 1 row, 255-257, 300, 320, 321, 600, 700: every tile shape,
    split second products, Kp padding of the weight gradients), rows
    gathered through a permuted index, against the oracle's fp64 gradients
    on the same bf16 inputs: dx_rep per row within the bf16 tolerance, each
    entry of dW1 and dW2 (float32, or rounded to bf16: one more relative
    2^-9, well inside the bound) within it too, and exact zeros for the
    empty expert."""
    import torch
    import paper_2411_15419_amd as L
    sizes = [0, 1, 255, 256, 257, 300, 320, 321, 600, 700]
    print_case("expert_ffn_backward", d=d, d_ff=d_ff, act=act, dw=dw, sizes=sizes)
    E = len(sizes)
    R = sum(sizes)
    rng = np.random.default_rng(23)
    x_all = _bf16_exact(rng.standard_normal((R + 50, d)))
    row_index = rng.permutation(R + 50)[:R].astype(np.int32)
    w1 = _bf16_exact(0.05 * rng.standard_normal((E, d_ff, d)))
    w2 = _bf16_exact(0.05 * rng.standard_normal((E, d, d_ff)))
    dy = _bf16_exact(rng.standard_normal((R, d)))
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).astype(np.float32)).to(torch.bfloat16).cuda()
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.int32).cuda()
    dx = torch.full((R, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    wdt = torch.float32 if dw == "f32" else torch.bfloat16
    dw1 = torch.full((E, d_ff, d), float("nan"), dtype=wdt, device="cuda")
    dw2 = torch.full((E, d, d_ff), float("nan"), dtype=wdt, device="cuda")
    ws = torch.empty(L.expert_ffn_backward_workspace_size(R, E, d, d_ff, L.LUFFY_BF16), dtype=torch.uint8,
                     device="cuda")
    L.luffy_expert_ffn_backward(bf(x_all), i32(row_index), i32(offsets), bf(w1), bf(w2), act, R, bf(dy), dx, dw1,
                                dw2, ws)
    torch.cuda.synchronize()
    if dw == "bf16":
        # same call with float32 gradients: the bf16 ones are those rounded
        # to nearest even, bit for bit (same sums in the same order)
        f1 = torch.empty((E, d_ff, d), dtype=torch.float32, device="cuda")
        f2 = torch.empty((E, d, d_ff), dtype=torch.float32, device="cuda")
        dx32 = torch.empty_like(dx)
        L.luffy_expert_ffn_backward(bf(x_all), i32(row_index), i32(offsets), bf(w1), bf(w2), act, R, bf(dy), dx32,
                                    f1, f2, ws)
        torch.cuda.synchronize()
        assert torch.equal(dw1, f1.to(torch.bfloat16)) and torch.equal(dw2, f2.to(torch.bfloat16))
        assert torch.equal(dx, dx32)
    rdx, rdw1, rdw2 = O.expert_ffn_backward(x_all[row_index], offsets, w1, w2, act, dy)
    tol = TOL["bf16"]
    err, _ = rel_err_rows(dx.double().cpu().numpy(), rdx)
    assert err.max() <= tol, f"dx_rep max row rel err {err.max():.3g}"
    # Weight gradients are sums over an expert's rows of products whose
    # factors carry bf16 rounding: Z, dA = dY W2 and dZ are bf16
    # intermediates, so a factor act'(Z) or act(Z) is off by up to about
    # |z| |act''(z)| or |z| |act'(z)| times the bf16 step, which is large
    # next to act'(z) itself near its zero (z = -0.75 for GELU).  Each entry
    # is held to tol times the sum over rows of the absolute term plus that
    # rounding term: (|dA| (|act'(Z)| + |Z|))^T |X| for dW1 (|act''| < 1)
    # and |dY|^T (|act(Z)| + |Z| |act'(Z)|) for dW2.
    xr = x_all[row_index]
    for name, got, ref in (("dW1", dw1, rdw1), ("dW2", dw2, rdw2)):
        g = got.double().cpu().numpy()
        assert not np.isnan(g).any(), f"{name} has unwritten entries"
        for e in range(E):
            lo, hi = offsets[e], offsets[e + 1]
            if hi == lo:
                assert not g[e].any(), f"{name} of an empty expert is not zero"
                continue
            z = xr[lo:hi] @ w1[e].T
            if name == "dW1":
                da = dy[lo:hi] @ w2[e]
                bound = (np.abs(da) * (np.abs(O.activation_grad(z, act)) + np.abs(z))).T @ np.abs(xr[lo:hi])
            else:
                bound = np.abs(dy[lo:hi]).T @ (np.abs(O.activation(z, act)) +
                                               np.abs(z) * np.abs(O.activation_grad(z, act)))
            viol = np.abs(g[e] - ref[e]) - tol * bound
            assert viol.max() <= 1e-12, \
                f"{name} expert {e} (rows {hi - lo}): worst entry {np.unravel_index(viol.argmax(), viol.shape)}"



@pytest.mark.parametrize("name,dw", [("c2", "f32"), ("c5", "f32"), ("c2", "bf16")])
def test_layer_backward_end_to_end(name, dw):
    """MoELayer.backward (both backward entry points in a row) on c2 and c5
    reduced (top-2; top-1 over 64 experts with dropped slots and experts
    without representatives), against the oracle's chain on the GPU
    forward's condensation: dgate within 1e-4 |dy_t| |y_rep_r|, the
    representatives' dx rows within the bf16 tolerance, the weight
    gradients of experts without representatives exactly zero, and a second
    call with a different dy."""
    import torch
    print_case("layer_backward", config=name, dw=dw, **REDUCED[name])
    inp, dev, layer, g = _forward(name)
    x = dev["x"]
    T, d = layer.buf.y.shape
    R = int(g["rep_offsets"][-1])
    xr = inp.x.astype(np.float64)[g["rep_token"]]
    rng = np.random.default_rng(29)
    for call in range(2):
        dy_np = _bf16_exact(rng.standard_normal((T, d)))
        dy = torch.from_numpy(dy_np.astype(np.float32)).to(torch.bfloat16).cuda()
        dgate, dx_rep, dw1, dw2 = layer.backward(x, dy, dw_dtype=torch.float32 if dw == "f32" else torch.bfloat16)
        torch.cuda.synchronize()
        ref_rep, ref_gate = O.combine_backward(dy_np, g["y_rep"].astype(np.float64), g["rep_row"],
                                               g["slot_pos"], g["topk_gate"].astype(np.float64))
        ref_dx, _, _ = O.expert_ffn_backward(xr, g["rep_offsets"], inp.w1, inp.w2, inp.cfg.act, ref_rep[:R])
        got_gate = dgate.double().cpu().numpy()
        kept = g["slot_pos"] >= 0
        rows = g["rep_row"][g["slot_pos"][kept]]
        scale = np.linalg.norm(dy_np, axis=1)[np.nonzero(kept)[0]] * np.linalg.norm(g["y_rep"][rows], axis=1)
        assert np.all(np.abs(got_gate[kept] - ref_gate[kept]) <= 1e-4 * scale), f"call {call}: dgate"
        err, _ = rel_err_rows(dx_rep[:R].double().cpu().numpy(), ref_dx)
        assert err.max() <= TOL["bf16"], f"call {call}: dx_rep max row rel err {err.max():.3g}"
        empty = np.flatnonzero(np.diff(g["rep_offsets"]) == 0)
        if empty.size:
            assert not dw1[torch.from_numpy(empty).cuda()].any() and not dw2[torch.from_numpy(empty).cuda()].any()
        if dw == "bf16":
            # the FFN backward again on the same dy_rep (the layer's own
            # buffer: a second combine backward may differ in its last bits)
            # with float32 gradients: the bf16 ones are those rounded to
            # nearest even, bit for bit
            import paper_2411_15419_amd as L
            b, bw = layer.buf, layer._bwd
            src, idx = (b.x_rep, None) if b.x_rep is not None else (x, b.rep_token)
            f1 = torch.empty(dw1.shape, dtype=torch.float32, device="cuda")
            f2 = torch.empty(dw2.shape, dtype=torch.float32, device="cuda")
            L.luffy_expert_ffn_backward(src, idx, b.rep_offsets, layer.w1, layer.w2, layer.act, layer.T * layer.k,
                                        bw["dy_rep"], torch.empty_like(dx_rep), f1, f2, bw["ws_f"])
            torch.cuda.synchronize()
            assert torch.equal(dw1, f1.to(torch.bfloat16)) and torch.equal(dw2, f2.to(torch.bfloat16))
