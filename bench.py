"""Throughput of the condensed MoE layer on one MI355X.

One step = luffy_route + luffy_condense + luffy_expert_ffn + luffy_combine
over one batch of synthetic tokens already resident in HBM.  Prints one JSON
line with tokens/s, the roofline of the dominant kernel (timed live with HIP
events on the stream it runs on) and the CPU oracle timed on the host cores.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--config c2]
    python bench.py --copy-calibration      # plain 1 GiB device copies, for
                                            # scaling the HBM byte counters

The roofline's "traffic" field is the HBM bytes per launch of the dominant
kernel read back from rocprofv3 FETCH_SIZE / WRITE_SIZE runs recorded under
profiles/ (hbm_traffic_<config>.md), each counter scaled by what it reads for
the plain copy; it is null when the kernel sources have changed since.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, 8 TB/s
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense MFMA (fp32: vector/matrix fp32 peak)

WORKLOAD_NAMES = {
    "c1": "tiny MoE layer fp32, T=512 d=256 E=4 top-1",
    "c2": "MoE layer bf16, T=8192 d=1024 E=16 top-2 cf=1.25",
    "c3": "expert-parallel share bf16, T=32768 d=2048 E=32 top-2 Zipf(1.1)",
    "c4": "condensation worst case bf16, T=16384 d=4096 E=8 top-1 i.i.d.",
    "c5": "many-expert skewed bf16, T=65536 d=1024 E=64 top-1 Zipf(1.3) cf=1.0",
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_work(name, cfg, counts):
    """Algorithmic flops and HBM bytes of one launch of a kernel."""
    b = 2 if cfg.dtype == "bf16" else 4
    T, d, E, k, dff = cfg.T, cfg.d, cfg.E, cfg.k, cfg.d_ff
    S, R = counts["S"], counts["R"]
    used = counts["used_experts"]
    if name == "gram":
        n = counts["bucket_sizes"]
        return dict(flops=2.0 * d * sum(x * (x + 1) / 2 for x in n),
                    bytes=float(S * d * b))
    if name == "ffn1":
        return dict(flops=2.0 * R * d * dff, bytes=float(used * d * dff * b + R * d * b + R * dff * b))
    if name == "ffn2":
        return dict(flops=2.0 * R * d * dff, bytes=float(used * d * dff * b + R * dff * b + R * d * b))
    if name == "gate":
        return dict(flops=2.0 * T * d * E, bytes=float(T * d * b + E * d * b + 12 * T * k))
    if name == "norm":
        return dict(flops=2.0 * T * d, bytes=float(T * d * b))
    if name == "combine":
        return dict(flops=2.0 * S * d, bytes=float(R * d * b + 12 * T * k + T * d * b))
    if name == "gather":
        return dict(flops=0.0, bytes=float(2 * R * d * b + 8 * S))
    # backward (per launch)
    if name == "bwd_wt":       # one weight tensor read and written transposed
        return dict(flops=0.0, bytes=float(2 * E * d * dff * b))
    if name in ("bwd_z", "bwd_da"):
        return dict(flops=2.0 * R * d * dff, bytes=float(used * d * dff * b + R * d * b + R * dff * b))
    if name == "bwd_dx":
        return dict(flops=2.0 * R * d * dff, bytes=float(used * d * dff * b + R * dff * b + R * d * b))
    if name in ("bwd_dw1", "bwd_dw2"):
        return dict(flops=2.0 * R * d * dff, bytes=float(E * d * dff * counts.get("dw_bytes", 4) + R * (d + dff) * b))
    if name == "cbwd_rows":
        return dict(flops=2.0 * S * d, bytes=float(S * d * b + R * d * b + 12 * S))
    if name == "cbwd_gate":
        return dict(flops=2.0 * S * d, bytes=float(T * d * b + S * d * b + 12 * T * k))
    return dict(flops=0.0, bytes=0.0)


def roofline(name, cfg, counts, sec_per_launch):
    w = kernel_work(name, cfg, counts)
    mfma_peak = MFMA_PEAK_TFLOPS[cfg.dtype]
    ridge = mfma_peak * 1e12 / (HBM_PEAK_GBS * 1e9)
    mfma_kernel = name in ("gram", "ffn1", "ffn2", "bwd_z", "bwd_da", "bwd_dx", "bwd_dw1", "bwd_dw2")
    if mfma_kernel and (w["bytes"] == 0 or w["flops"] / w["bytes"] >= ridge):
        ach = w["flops"] / sec_per_launch / 1e12
        return dict(bound="mfma", achieved=ach, peak=mfma_peak, unit="TFLOP/s",
                    frac=ach / mfma_peak, traffic=None)
    ach = w["bytes"] / sec_per_launch / 1e9
    return dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                frac=ach / HBM_PEAK_GBS, traffic=None)


def source_digest():
    """sha256 over the HIP sources of the library (file names and contents)."""
    h = hashlib.sha256()
    for path in sorted(glob.glob(os.path.join(ROOT, "paper_2411_15419_amd", "csrc", "*"))):
        h.update(os.path.basename(path).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(config, kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary of
    this workload, or None if there is none or the sources have changed."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{config}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_sha256") != source_digest() or kernel not in rec.get("kernels", {}):
        return None
    k = rec["kernels"][kernel]
    return (k["fetch_kib"] * 1024 * rec["fetch_scale"] + k["write_kib"] * 1024 * rec["write_scale"])


def copy_calibration(n_bytes=1 << 30, reps=5):
    """Plain device-to-device copies of a known size; rocprofv3 counter runs
    over this give the FETCH_SIZE / WRITE_SIZE scale factors."""
    import torch
    src = torch.ones(n_bytes // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n_bytes, "copy_bytes_written": n_bytes, "reps": reps}))


def cpu_baseline(inp, h, budget_s=15.0):
    """The oracle as it stands, on the host cores, on a bounded sample."""
    import numpy as np
    from oracle import luffy_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = len(os.sched_getaffinity(0))
    cfg = inp.cfg
    # sample: the first T' tokens of the batch (all of it when it fits the budget)
    T_s = cfg.T if cfg.T <= 8192 else max(1024, cfg.T // 8)
    x = inp.x[:T_s].astype(np.float64)
    runs, t0 = 0, time.perf_counter()
    while True:
        O.moe_layer(x, inp.w_g, inp.b_g, inp.w1, inp.w2, k=cfg.k, h=h, act=cfg.act,
                    capacity_factor=cfg.capacity_factor)
        runs += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    sample = (f"whole layer on the first {T_s} of {cfg.T} tokens" if T_s < cfg.T
              else f"whole layer on all {cfg.T} tokens") + f", {runs} run(s), {el:.1f} s"
    return dict(value=T_s * runs / el, unit="tokens/s", cores=int(threads), kind="oracle",
                sample=sample)


BACKWARD_KERNELS = ("cbwd_group", "cbwd_rows", "cbwd_gate", "bwd_z", "bwd_act", "bwd_da", "bwd_dx",
                    "bwd_dx_reduce", "bwd_gather", "bwd_dw2", "bwd_dw1")


def bench_backward(args, cfg, layer, x, L, torch, np):
    """One step = luffy_combine_backward + luffy_expert_ffn_backward for a
    synthetic dL/dy after one forward (the condensation of that forward is
    held fixed); prints one JSON line like the forward's."""
    if cfg.dtype != "bf16":
        print("bench.py --backward: the expert FFN backward is bf16 only", file=sys.stderr)
        sys.exit(2)
    b = layer.buf
    T, d = b.y.shape
    k = cfg.k
    E, dff, _ = layer.w1.shape
    S = T * k
    g = torch.Generator(device="cuda").manual_seed(args.seed)
    dy = torch.randn(T, d, device="cuda", generator=g).to(b.y.dtype)
    dy_rep = torch.empty_like(b.y_rep)
    dgate = torch.empty(T, k, dtype=torch.float32, device="cuda")
    dx_rep = torch.empty(S, d, dtype=b.y.dtype, device="cuda")
    wdt = torch.bfloat16 if args.dw_dtype == "bf16" else torch.float32
    dw1 = torch.empty(E, dff, d, dtype=wdt, device="cuda")
    dw2 = torch.empty(E, d, dff, dtype=wdt, device="cuda")
    ws_c = torch.empty(L.combine_backward_workspace_size(T, k, S), dtype=torch.uint8, device="cuda")
    ws_f = torch.empty(L.expert_ffn_backward_workspace_size(S, E, d, dff, L.LUFFY_BF16), dtype=torch.uint8,
                       device="cuda")

    def step():
        L.luffy_combine_backward(dy, b.y_rep, b.rep_row, b.perm_token, b.slot_pos, b.topk_gate, b.offsets,
                                 b.rep_offsets, dy_rep, dgate, ws_c)
        L.luffy_expert_ffn_backward(x, b.rep_token, b.rep_offsets, layer.w1, layer.w2, cfg.act, S, dy_rep,
                                    dx_rep, dw1, dw2, ws_f)

    for _ in range(max(args.warmup, 1)):
        step()
    torch.cuda.synchronize()
    per_kernel = {}
    for name in BACKWARD_KERNELS:
        L.profile_kernel(name)
        for _ in range(3):
            step()
        ms, n = L.profile_read()
        if n:
            per_kernel[name] = dict(ms_per_step=ms / 3, launches_per_step=n / 3, ms_per_launch=ms / n)
    L.profile_kernel(None)
    dominant = max(per_kernel, key=lambda kname: per_kernel[kname]["ms_per_step"])
    L.profile_kernel(dominant)
    L.profile_read()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_per_step = start.elapsed_time(stop) / args.steps
    dom_ms, dom_n = L.profile_read()
    L.profile_kernel(None)
    off = b.offsets.cpu().numpy()
    ro = b.rep_offsets.cpu().numpy()
    counts = dict(S=int(off[-1]), R=int(ro[-1]), bucket_sizes=np.diff(off).tolist(),
                  used_experts=int((np.diff(ro) > 0).sum()), dw_bytes=2 if args.dw_dtype == "bf16" else 4)
    rl = roofline(dominant, cfg, counts, dom_ms / dom_n / 1e3)
    rl.update(traffic=None, algorithmic_bytes=kernel_work(dominant, cfg, counts)["bytes"], kernel=dominant,
              us_per_launch=dom_ms / dom_n * 1e3)
    kernels = {}
    for name, v in per_kernel.items():
        r = roofline(name, cfg, counts, v["ms_per_launch"] / 1e3)
        kernels[name] = dict(us_per_launch=round(v["ms_per_launch"] * 1e3, 2),
                             launches_per_step=v["launches_per_step"], bound=r["bound"],
                             achieved=round(r["achieved"], 1), unit=r["unit"], frac=round(r["frac"], 4))
    out = {
        "metric": "condensed MoE-layer backward tokens/s on 1 MI355X",
        "value": cfg.T / (ms_per_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "wall_s": wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded clustered tokens, random-init weights, normal dL/dy)",
        "config": {"workload": WORKLOAD_NAMES[args.config] + ", backward (combine + expert FFN)",
                   "name": args.config, "T": cfg.T, "d_model": cfg.d, "E": cfg.E, "top_k": cfg.k,
                   "d_ff": cfg.d_ff, "act": cfg.act, "dw_dtype": args.dw_dtype},
        "condensation": {"slots_kept": counts["S"], "representatives": counts["R"]},
        "roofline": rl,
        "kernels": kernels,
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c2", choices=sorted(WORKLOAD_NAMES))
    ap.add_argument("--threshold", type=float, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward of the layer (combine and expert FFN) instead of the forward")
    ap.add_argument("--dw-dtype", default="f32", choices=("f32", "bf16"),
                    help="type of the backward's weight gradients: f32, or bf16 (the weights' own type, as "
                         "a bf16 parameter's gradient)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this layer is built and timed on a single "
              "MI355X (no collectives); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import luffy_gen as G
    import paper_2411_15419_amd as L

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        copy_calibration()
        return
    L.load_library()
    torch.cuda.set_device(0)
    cfg = G.config(args.config)
    h = cfg.h if args.threshold is None else args.threshold
    log(f"generating {args.config} (seed {args.seed})")
    inp = G.make_inputs(cfg, seed=args.seed)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

    def dev(a, dtype=dt):
        t = torch.from_numpy(np.ascontiguousarray(a))
        return t.to(dtype).to("cuda")

    x = dev(inp.x)
    layer = L.MoELayer(dev(inp.w_g), dev(inp.b_g, torch.float32), dev(inp.w1), dev(inp.w2),
                       k=cfg.k, act=cfg.act, threshold=h, capacity_factor=cfg.capacity_factor,
                       T=cfg.T)
    torch.cuda.synchronize()
    log("warmup")
    for _ in range(max(args.warmup, 1)):
        layer(x)
    torch.cuda.synchronize()

    if args.backward:
        bench_backward(args, cfg, layer, x, L, torch, np)
        return

    # per-kernel breakdown (untimed pass) to find the dominant kernel
    per_kernel = {}
    for name in L.KERNELS:
        L.profile_kernel(name)
        for _ in range(3):
            layer(x)
        ms, n = L.profile_read()
        if n:
            per_kernel[name] = dict(ms_per_step=ms / 3, launches_per_step=n / 3, ms_per_launch=ms / n)
    L.profile_kernel(None)
    dominant = max(per_kernel, key=lambda kname: per_kernel[kname]["ms_per_step"])
    log(f"dominant kernel: {dominant}")

    # timed region: K steps, only the dominant kernel bracketed by events
    L.profile_kernel(dominant)
    L.profile_read()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        layer(x)
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_total = start.elapsed_time(stop)
    dom_ms, dom_n = L.profile_read()
    L.profile_kernel(None)
    ms_per_step = ms_total / args.steps
    tokens_per_s = cfg.T / (ms_per_step / 1e3)

    b = layer.buf
    off = b.offsets.cpu().numpy()
    ro = b.rep_offsets.cpu().numpy()
    sizes = np.diff(off).tolist()
    counts = dict(S=int(off[-1]), R=int(ro[-1]), bucket_sizes=sizes,
                  used_experts=int((np.diff(ro) > 0).sum()))
    dropped = cfg.T * cfg.k - counts["S"]

    rl = roofline(dominant, cfg, counts, dom_ms / dom_n / 1e3)
    traffic = recorded_traffic(args.config, dominant)
    rl["traffic"] = traffic
    rl["traffic_unit"] = "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-scaled)"
    rl["algorithmic_bytes"] = kernel_work(dominant, cfg, counts)["bytes"]
    rl["kernel"] = dominant
    rl["us_per_launch"] = dom_ms / dom_n * 1e3
    kernels = {}
    for name, v in per_kernel.items():
        r = roofline(name, cfg, counts, v["ms_per_launch"] / 1e3)
        kernels[name] = dict(us_per_launch=round(v["ms_per_launch"] * 1e3, 2),
                             launches_per_step=v["launches_per_step"],
                             bound=r["bound"], achieved=round(r["achieved"], 1), unit=r["unit"],
                             frac=round(r["frac"], 4))

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        cpu = cpu_baseline(inp, h)

    out = {
        "metric": "condensed MoE-layer tokens/s on 1 MI355X",
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "wall_s": wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded clustered tokens, random-init weights)",
        "config": {"workload": WORKLOAD_NAMES[args.config], "name": args.config, "T": cfg.T,
                   "d_model": cfg.d, "E": cfg.E, "top_k": cfg.k, "d_ff": cfg.d_ff,
                   "act": cfg.act, "threshold": h, "capacity_factor": cfg.capacity_factor,
                   "seed": args.seed},
        "condensation": {"slots_kept": counts["S"], "representatives": counts["R"],
                         "ratio": counts["R"] / max(counts["S"], 1), "dropped_slots": dropped},
        "roofline": rl,
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
