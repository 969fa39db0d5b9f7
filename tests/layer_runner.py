"""Shared helpers of the GPU parity tests: run the HIP layer through the C ABI
on seeded inputs, run the oracle on the same arrays, compare."""
from __future__ import annotations

import numpy as np

import luffy_gen as G
from oracle import luffy_oracle as O

TOL = {"bf16": 2e-2, "f32": 1e-5}


def torch_dtype(cfg):
    import torch
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def to_device(a, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype == torch.bfloat16:
        t = t.to(torch.bfloat16)          # exact: values are bf16-representable
    return t.to("cuda")


def upload(inp):
    import torch
    dt = torch_dtype(inp.cfg)
    dev = dict(
        x=to_device(inp.x, dt),
        w_g=to_device(inp.w_g, dt),
        b_g=to_device(inp.b_g.astype(np.float32), torch.float32),
        w1=to_device(inp.w1, dt) if inp.w1 is not None else None,
        w2=to_device(inp.w2, dt) if inp.w2 is not None else None,
    )
    return dev


def make_layer(inp, dev, h=None, gather_x_rep=False, norms_from_route=True):
    import paper_2411_15419_amd as L
    cfg = inp.cfg
    w1, w2 = dev["w1"], dev["w2"]
    if w1 is None:   # route/condense-only runs still need weight shapes
        import torch
        w1 = torch.zeros(cfg.E, 64, cfg.d, dtype=dev["x"].dtype, device="cuda")
        w2 = torch.zeros(cfg.E, cfg.d, 64, dtype=dev["x"].dtype, device="cuda")
    return L.MoELayer(dev["w_g"], dev["b_g"], w1, w2, k=cfg.k, act=cfg.act,
                      threshold=cfg.h if h is None else h,
                      capacity_factor=cfg.capacity_factor, T=cfg.T,
                      gather_x_rep=gather_x_rep, norms_from_route=norms_from_route)


def fetch(layer, with_ffn=True):
    """Copies the layer's outputs to numpy, truncated to the device counts."""
    import torch
    torch.cuda.synchronize()
    b = layer.buf
    off = b.offsets.cpu().numpy()
    S = int(off[-1])
    ro = b.rep_offsets.cpu().numpy()
    R = int(ro[-1])
    out = dict(
        topk_idx=b.topk_idx.cpu().numpy(), topk_gate=b.topk_gate.cpu().numpy(),
        slot_pos=b.slot_pos.cpu().numpy(), offsets=off,
        perm_token=b.perm_token[:S].cpu().numpy(),
        rep_of_pos=b.rep_of_pos[:S].cpu().numpy(), rep_row=b.rep_row[:S].cpu().numpy(),
        rep_offsets=ro, rep_token=b.rep_token[:R].cpu().numpy(),
        degree=b.degree[:S].cpu().numpy() if b.degree is not None else None,
    )
    if b.x_rep is not None:
        out["x_rep"] = b.x_rep[:R].float().cpu().numpy()
    if with_ffn:
        out["y_rep"] = b.y_rep[:R].float().cpu().numpy()
        out["y"] = b.y.float().cpu().numpy()
    return out


def run_gpu(inp, h=None, with_ffn=True, gather_x_rep=False, dev=None, norms_from_route=True):
    dev = dev or upload(inp)
    layer = make_layer(inp, dev, h, gather_x_rep, norms_from_route)
    x = dev["x"]
    layer.route(x)
    layer.condense(x, threshold=h)
    if with_ffn:
        layer.expert_ffn(x)
        layer.combine()
    return fetch(layer, with_ffn)


def run_oracle(inp, h=None, with_ffn=True):
    cfg = inp.cfg
    return O.moe_layer(inp.x.astype(np.float64), inp.w_g, inp.b_g, inp.w1, inp.w2,
                       k=cfg.k, h=cfg.h if h is None else h, act=cfg.act,
                       capacity_factor=cfg.capacity_factor, with_ffn=with_ffn)


def rel_err_rows(y, ref):
    """Per row ||y - ref||_inf / ||ref||_inf over rows with a non-zero reference."""
    den = np.abs(ref).max(axis=1)
    num = np.abs(y - ref).max(axis=1)
    nz = den > 0
    return num[nz] / den[nz], nz


def assert_route_equal(g, o):
    assert np.array_equal(g["topk_idx"], o.topk_idx), "topk_idx differs"
    assert np.allclose(g["topk_gate"], o.topk_gate, rtol=0, atol=2e-6), \
        f"gate max err {np.abs(g['topk_gate'] - o.topk_gate).max()}"
    assert np.array_equal(g["offsets"], o.offsets), "offsets differ"
    assert np.array_equal(g["perm_token"], o.perm_token), "perm_token differs"
    assert np.array_equal(g["slot_pos"], o.slot_pos), "slot_pos differs"


def assert_condense_equal(g, o):
    if g["degree"] is not None:
        bad = np.flatnonzero(g["degree"] != o.degree)
        assert bad.size == 0, f"degree differs at {bad[:10]}"
    bad = np.flatnonzero(g["rep_of_pos"] != o.rep_of_pos)
    assert bad.size == 0, f"rep_of_pos differs at {bad[:10]}"
    assert np.array_equal(g["rep_offsets"], o.rep_offsets), "rep_offsets differ"
    assert np.array_equal(g["rep_row"], o.rep_row), "rep_row differs"
    assert np.array_equal(g["rep_token"], o.rep_token), "rep_token differs"


def assert_output_close(g, o, dtype):
    tol = TOL[dtype]
    err, nz = rel_err_rows(g["y"], o.y)
    assert err.size == 0 or err.max() <= tol, f"max row rel err {err.max():.3g} > {tol}"
    dropped = (o.slot_pos < 0).all(axis=1)
    assert np.all(g["y"][dropped] == 0), "fully dropped tokens must be zero"
    return float(err.max()) if err.size else 0.0
