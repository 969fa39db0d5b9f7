"""Throughput of the condensed MoE layer on one MI355X.

One step = luffy_route + luffy_condense + luffy_expert_ffn + luffy_combine
over one batch of synthetic tokens already resident in HBM.  Prints one JSON
line with tokens/s, the roofline of the dominant kernel (timed live with HIP
events on the stream it runs on) and the CPU oracle timed on the host cores.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--config c3] [--extras c2,c4,c5]
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
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0, "f32": 157.3}   # dense MFMA (fp32: vector/matrix fp32 peak)

WORKLOAD_NAMES = {
    "c1": "tiny MoE layer fp32, T=512 d=256 E=4 top-1",
    "c2": "MoE layer bf16, T=8192 d=1024 E=16 top-2 cf=1.25",
    "c3": "expert-parallel share bf16, T=32768 d=2048 E=32 top-2 Zipf(1.1)",
    "c4": "condensation worst case bf16, T=16384 d=4096 E=8 top-1 i.i.d.",
    "c5": "many-expert skewed bf16, T=65536 d=1024 E=64 top-1 Zipf(1.3) cf=1.0",
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_work(name, cfg, counts, norms_from_route=True):
    """Work of one launch of a kernel: flops, the algorithmic HBM bytes of the
    measurement plan ("bytes": the FFN counts only its weights, d*d_ff*b per
    used expert and product; combine 8 bytes of indices per slot), and the
    bytes with the activation rows the kernel also moves ("bytes_act")."""
    b = 2 if cfg.dtype == "bf16" else 4
    T, d, E, k, dff = cfg.T, cfg.d, cfg.E, cfg.k, cfg.d_ff
    S, R = counts["S"], counts["R"]
    used = counts["used_experts"]

    def w(flops, nbytes, nbytes_act=None):
        return dict(flops=float(flops), bytes=float(nbytes),
                    bytes_act=float(nbytes if nbytes_act is None else nbytes_act))

    if name == "gram":
        # on the fp8 screen the rows it streams are fp8 (one byte a value)
        n = counts["bucket_sizes"]
        return w(2.0 * d * sum(x * (x + 1) / 2 for x in n), S * d * (1 if counts.get("screen") else b))

    if name in ("ffn1", "ffn2"):
        wb = used * d * dff * b
        return w(2.0 * R * d * dff, wb, wb + R * d * b + R * dff * b)
    if name == "gate":
        return w(2.0 * T * d * E, T * d * b + E * d * b + 12 * T * k)
    if name == "norm":
        # with the norms from the gate pass it only clears the per-position
        # state (degree, walk state, claim key: 16 bytes a position); with the
        # fp8 similarity screen it also reads the rows and writes their fp8
        # copies and quantisation errors
        screen = bool(counts.get("screen"))
        nbytes = 16 * S + (T * d * b if screen or not norms_from_route else 0) + (T * d + 4 * T if screen else 0)
        return w(0.0 if norms_from_route else 2.0 * T * d, nbytes)
    if name == "combine":
        return w(2.0 * S * d, R * d * b + 8 * T * k + T * d * b, R * d * b + 12 * T * k + T * d * b)
    if name == "gather":
        return w(0.0, 2 * R * d * b + 8 * S)
    # backward (per launch)
    if name in ("bwd_z", "bwd_da", "bwd_dx"):
        wb = used * d * dff * b
        return w(2.0 * R * d * dff, wb, wb + R * d * b + R * dff * b)
    if name in ("bwd_dw1", "bwd_dw2"):
        ob = E * d * dff * counts.get("dw_bytes", 4)
        return w(2.0 * R * d * dff, ob, ob + R * (d + dff) * b)
    if name == "cbwd_rows":
        return w(2.0 * S * d, S * d * b + R * d * b + 12 * S)
    if name == "cbwd_gate":
        return w(2.0 * S * d, T * d * b + S * d * b + 12 * T * k)
    return w(0.0, 0.0)


MFMA_KERNELS = ("gram", "ffn1", "ffn2", "bwd_z", "bwd_da", "bwd_dx", "bwd_dw1", "bwd_dw2")


def roofline(name, cfg, counts, sec_per_launch, norms_from_route=True):
    """Roofline of one kernel: MFMA kernels whose flops per algorithmic byte
    reach the ridge (peak flops / 8 TB/s) are bound by the MFMA peak, every
    other kernel by HBM.  `attainable` = min(MFMA peak, intensity x 8 TB/s)
    in the kernel's unit; `frac_attainable` = achieved / attainable."""
    wk = kernel_work(name, cfg, counts, norms_from_route)
    # the screened similarity kernel multiplies fp8
    mfma_peak = MFMA_PEAK_TFLOPS["fp8" if name == "gram" and counts.get("screen") else cfg.dtype]
    ridge = mfma_peak * 1e12 / (HBM_PEAK_GBS * 1e9)
    tflops = wk["flops"] / sec_per_launch / 1e12
    gbs = wk["bytes"] / sec_per_launch / 1e9
    gbs_act = wk["bytes_act"] / sec_per_launch / 1e9
    extra = dict(tflops=tflops, mfma_frac=tflops / mfma_peak, hbm_gbs=gbs, hbm_frac=gbs / HBM_PEAK_GBS,
                 hbm_gbs_with_activations=gbs_act)
    if name in MFMA_KERNELS and wk["bytes"] > 0:
        intensity = wk["flops"] / wk["bytes"]
        att = min(mfma_peak, intensity * HBM_PEAK_GBS / 1e3)
        if intensity >= ridge:
            return dict(bound="mfma", achieved=tflops, peak=mfma_peak, unit="TFLOP/s", frac=tflops / mfma_peak,
                        traffic=None, attainable=att, frac_attainable=tflops / att, intensity=intensity, **extra)
        return dict(bound="hbm", achieved=gbs, peak=HBM_PEAK_GBS, unit="GB/s", frac=gbs / HBM_PEAK_GBS,
                    traffic=None, attainable=att, frac_attainable=tflops / att, intensity=intensity, **extra)
    return dict(bound="hbm", achieved=gbs, peak=HBM_PEAK_GBS, unit="GB/s", frac=gbs / HBM_PEAK_GBS,
                traffic=None, attainable=HBM_PEAK_GBS, frac_attainable=gbs / HBM_PEAK_GBS, **extra)


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


def cpu_baseline(inp, h, full_bucket_sizes, budget_s=15.0):
    """The oracle as it stands, on the host cores, on a bounded sample: the
    whole layer (its steps called in order, each timed) on the first T' tokens
    of the batch (all of them when T <= 8192), repeated for about budget_s.

    The similarity step costs the square of a bucket's size, so a sample of
    T/8 tokens does about 1/64 of the full batch's similarity work per bucket;
    `full_layer_estimate` scales the sample's similarity time by the ratio of
    sum(n_e^2) over the full batch's buckets to the sample's, and the other
    steps by T/T'."""
    import numpy as np
    from oracle import luffy_oracle as O
    affinity = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        blas = None
    cfg = inp.cfg
    T_s = cfg.T if cfg.T <= 8192 else max(1024, cfg.T // 8)
    x = inp.x[:T_s].astype(np.float64)
    E = cfg.E
    t_sim = t_other = 0.0
    runs = 0
    sizes = None
    t_start = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        idx, gates, _ = O.gate(x, inp.w_g, inp.b_g, cfg.k)
        C = O.capacity_of(T_s, cfg.k, E, cfg.capacity_factor)
        offsets, perm_token, slot_pos = O.dispatch(idx, E, C)
        t1 = time.perf_counter()
        cz = O.condense(x, perm_token, offsets, h)
        t2 = time.perf_counter()
        y_rep = O.expert_ffn(x[cz.rep_token], cz.rep_offsets, inp.w1, inp.w2, cfg.act)
        O.combine(y_rep, cz.rep_row, slot_pos, gates)
        t3 = time.perf_counter()
        t_other += (t1 - t0) + (t3 - t2)
        t_sim += t2 - t1
        sizes = np.diff(offsets)
        runs += 1
        if time.perf_counter() - t_start >= budget_s:
            break
    el = t_sim + t_other
    sq_s = float((sizes.astype(np.float64) ** 2).sum())
    sq_f = float((np.asarray(full_bucket_sizes, np.float64) ** 2).sum())
    est = (t_other / runs) * (cfg.T / T_s) + (t_sim / runs) * (sq_f / max(sq_s, 1.0))
    sample = (f"whole layer on the first {T_s} of {cfg.T} tokens" if T_s < cfg.T
              else f"whole layer on all {cfg.T} tokens") + f", {runs} run(s), {el:.1f} s"
    return dict(value=T_s * runs / el, unit="tokens/s", cores=int(blas or affinity), kind="oracle",
                sample=sample, affinity_cores=affinity, blas_threads=blas,
                similarity_share=t_sim / el,
                full_layer_estimate=dict(value=cfg.T / est, unit="tokens/s", seconds=est,
                                         note="sample similarity time x sum(n_e^2) full/sample, "
                                              "other steps x T/T'"))


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
    kernels = kernel_table(per_kernel, cfg, counts)
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


def kernel_table(per_kernel, cfg, counts, norms_from_route=True):
    out = {}
    for name, v in per_kernel.items():
        r = roofline(name, cfg, counts, v["ms_per_launch"] / 1e3, norms_from_route)
        out[name] = dict(us_per_launch=round(v["ms_per_launch"] * 1e3, 2), launches_per_step=v["launches_per_step"],
                         bound=r["bound"], achieved=round(r["achieved"], 1), unit=r["unit"], frac=round(r["frac"], 4),
                         tflops=round(r["tflops"], 1), mfma_frac=round(r["mfma_frac"], 4),
                         hbm_gbs=round(r["hbm_gbs"], 1), hbm_frac=round(r["hbm_frac"], 4))
    return out


def measure_forward(name, thresholds, args, torch, np, G, L, with_cpu):
    """Times the forward step of workload `name` at each threshold (the
    inputs are drawn and uploaded once).  Returns one record per threshold."""
    cfg = G.config(name)
    log(f"generating {name} (seed {args.seed})")
    inp = G.make_inputs(cfg, seed=args.seed)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

    def dev(a, dtype=dt):
        t = torch.from_numpy(np.ascontiguousarray(a))
        return t.to(dtype).to("cuda")

    x = dev(inp.x)
    weights = (dev(inp.w_g), dev(inp.b_g, torch.float32), dev(inp.w1), dev(inp.w2))
    records = []
    for h in thresholds:
        layer = L.MoELayer(*weights, k=cfg.k, act=cfg.act, threshold=h, capacity_factor=cfg.capacity_factor,
                           T=cfg.T)
        torch.cuda.synchronize()
        log(f"{name} h={h}: warmup")
        for _ in range(max(args.warmup, 1)):
            layer(x)
        torch.cuda.synchronize()
        if args.backward:
            bench_backward(args, cfg, layer, x, L, torch, np)
            return None
        # per-kernel breakdown (untimed passes) to find the dominant kernel
        per_kernel = {}
        for kname in L.KERNELS:
            L.profile_kernel(kname)
            for _ in range(3):
                layer(x)
            ms, n = L.profile_read()
            if n:
                per_kernel[kname] = dict(ms_per_step=ms / 3, launches_per_step=n / 3, ms_per_launch=ms / n)
        L.profile_kernel(None)
        dominant = max(per_kernel, key=lambda kk: per_kernel[kk]["ms_per_step"])
        log(f"{name} h={h}: dominant kernel {dominant}; timing {args.steps} steps")
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
        b = layer.buf
        off = b.offsets.cpu().numpy()
        ro = b.rep_offsets.cpu().numpy()
        counts = dict(S=int(off[-1]), R=int(ro[-1]), bucket_sizes=np.diff(off).tolist(),
                      used_experts=int((np.diff(ro) > 0).sum()),
                      screen=L.similarity_screen_applies(cfg.T, cfg.d, cfg.E, cfg.k,
                                                         L.LUFFY_BF16 if cfg.dtype == "bf16" else L.LUFFY_F32))
        rl = roofline(dominant, cfg, counts, dom_ms / dom_n / 1e3)
        wk = kernel_work(dominant, cfg, counts)
        rl.update(traffic=recorded_traffic(name, dominant),
                  traffic_unit="HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-scaled)",
                  algorithmic_flops=wk["flops"], algorithmic_bytes=wk["bytes"],
                  algorithmic_bytes_with_activations=wk["bytes_act"], kernel=dominant,
                  us_per_launch=dom_ms / dom_n * 1e3, launches_timed=dom_n)
        rec = dict(name=name, threshold=h, cfg=cfg, value=cfg.T / (ms_per_step / 1e3), ms_per_step=ms_per_step,
                   wall_s=wall,
                   condensation={"slots_kept": counts["S"], "representatives": counts["R"],
                                 "ratio": counts["R"] / max(counts["S"], 1),
                                 "dropped_slots": cfg.T * cfg.k - counts["S"],
                                 "largest_bucket": int(max(counts["bucket_sizes"])),
                                 "used_experts": counts["used_experts"]},
                   roofline=rl, kernels=kernel_table(per_kernel, cfg, counts), cpu_baseline=None)
        if with_cpu and h == thresholds[0]:
            log(f"{name}: cpu baseline (oracle)")
            rec["cpu_baseline"] = cpu_baseline(inp, h, counts["bucket_sizes"])
        records.append(rec)
        del layer
    del x, weights, inp
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return records


HISTORY_SETTINGS = ((0.8, 0.2), (0.7, 0.3), (0.6, 0.4), (0.5, 0.5))
HISTORY_DRIFTS = {"stable routing": dict(token_drift=0.1, gate_drift=0.0),
                  "drifting routing": dict(token_drift=1.0, gate_drift=0.05)}


def measure_history(name, args, torch, np, G, L):
    """Historical similarity (Sec. 5.1 step 2) on a two-block stack at the
    workload's shape (block 1 reads block 0's record): the condense call of
    block 1 with history against the plain condense call on the same input,
    per (S1, S2) and per drift of the tokens and router between the blocks
    (one token in twenty a mixture of two centres, whose pairs fall between
    S2 and S1)."""
    cfg = G.config(name)
    h = cfg.h
    out = {}
    for label, drift in HISTORY_DRIFTS.items():
        log(f"history {name} ({label}): generating a two-block stack")
        stack = G.make_stack(cfg, 2, seed=args.seed, mix_fraction=0.05, **drift)
        dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        xs = [torch.from_numpy(b.x).to(dt).cuda() for b in stack]
        wg = [torch.from_numpy(b.w_g).to(dt).cuda() for b in stack]
        bg = torch.from_numpy(stack[0].b_g).cuda()
        w1 = torch.zeros(cfg.E, 64, cfg.d, dtype=dt, device="cuda")
        w2 = torch.zeros(cfg.E, cfg.d, 64, dtype=dt, device="cuda")
        mk = lambda b, hist: L.MoELayer(wg[b], bg, w1, w2, k=cfg.k, act=cfg.act, threshold=h,  # noqa: E731
                                        capacity_factor=cfg.capacity_factor, T=cfg.T, history=hist)

        def timed(fn, kernel="gram"):
            for _ in range(2):
                fn()
            L.profile_kernel(kernel)
            L.profile_read()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(args.steps):
                fn()
            b.record()
            torch.cuda.synchronize()
            kms, kn = L.profile_read()
            L.profile_kernel(None)
            return a.elapsed_time(b) / args.steps * 1e3, kms / max(kn, 1) * 1e3

        plain = mk(1, None)
        plain.route(xs[1])
        plain_us, plain_gram = timed(lambda: plain.condense(xs[1]))
        runs = []
        for S1, S2 in HISTORY_SETTINGS:
            b0, b1 = mk(0, (S1, S2)), mk(1, (S1, S2))
            b0.route(xs[0])
            b0.condense(xs[0])
            b1.route(xs[1])
            us, gram_us = timed(lambda: b1.condense(xs[1], hist_in=b0.record))
            _, gather_us = timed(lambda: b1.condense(xs[1], hist_in=b0.record), "hist_gather")
            breakdown = {}
            for kname in ("hist_cols", "norm", "hist_header", "greedy_round", "greedy_more", "greedy_finish",
                          "rep_local", "rep_finalize"):
                breakdown[kname] = round(timed(lambda: b1.condense(xs[1], hist_in=b0.record), kname)[1], 1)
            st = b1.hist_stats.cpu().numpy().tolist()
            same = bool(torch.equal(b1.buf.rep_offsets, plain.buf.rep_offsets))
            runs.append(dict(S1=S1, S2=S2, condense_us=us, gram_us=gram_us, gather_us=gather_us,
                             saved_us=plain_us - us, undecided_pairs=st[0], decided_pairs=st[1],
                             undecided_frac=st[0] / max(st[0] + st[1], 1), tiles_computed=st[2],
                             tiles_skipped=st[3], same_representative_counts_as_plain=same,
                             other_kernels_us=breakdown))
            log(f"history {name} {label} S1={S1} S2={S2}: {us:.1f} us (plain {plain_us:.1f}), "
                f"undecided {st[0] / max(st[0] + st[1], 1):.3f}, tiles {st[2]} computed {st[3]} skipped")
            del b0, b1
        out[label] = dict(drift=drift, plain_condense_us=plain_us, plain_gram_us=plain_gram, settings=runs)
        del plain, xs, wg, stack
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def compact(rec):
    """Summary of a workload measured beside the headline one."""
    rl = rec["roofline"]
    return {"workload": WORKLOAD_NAMES[rec["name"]], "threshold": rec["threshold"],
            "tokens_per_s": rec["value"], "ms_per_step": rec["ms_per_step"], "condensation": rec["condensation"],
            "dominant": {k: rl[k] for k in ("kernel", "bound", "achieved", "unit", "frac", "tflops", "mfma_frac",
                                            "hbm_gbs", "hbm_frac", "us_per_launch")},
            "kernels_us": {k: v["us_per_launch"] for k, v in rec["kernels"].items()}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c3", choices=sorted(WORKLOAD_NAMES),
                    help="headline workload (default c3: one GPU's share of an expert-parallel layer)")
    ap.add_argument("--extras", default="c2,c4,c5",
                    help="workloads measured beside the headline one, reported under 'workloads' "
                         "(c4 at each of its four thresholds); 'none' for none")
    ap.add_argument("--history", default="c3",
                    help="workload whose two-block stack times the historical similarity beside the headline "
                         "(reported under 'history'); 'none' for none")
    ap.add_argument("--threshold", type=float, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-screen", action="store_true",
                    help="similarity on bf16 MFMA for every tile (the fp8 screen off)")
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
    if args.no_screen:
        L.set_similarity_screen(False)
    torch.cuda.set_device(0)
    cfg = G.config(args.config)
    h = cfg.h if args.threshold is None else args.threshold
    recs = measure_forward(args.config, [h], args, torch, np, G, L, with_cpu=not args.no_cpu_baseline)
    if recs is None:      # --backward printed its own line
        return
    head = recs[0]
    extras = {}
    if not args.backward and args.extras and args.extras != "none":
        for name in [n.strip() for n in args.extras.split(",") if n.strip()]:
            if name == args.config or name not in WORKLOAD_NAMES:
                continue
            ecfg = G.config(name)
            for r in measure_forward(name, list(ecfg.thresholds), args, torch, np, G, L, with_cpu=False):
                key = name if len(ecfg.thresholds) == 1 else f"{name}_h{r['threshold']:.2f}"
                extras[key] = compact(r)
    history = None
    if args.history and args.history != "none" and args.history in WORKLOAD_NAMES:
        history = measure_history(args.history, args, torch, np, G, L)
    out = {
        "metric": "condensed MoE-layer tokens/s on 1 MI355X",
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "wall_s": head["wall_s"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded clustered tokens, random-init weights)",
        "config": {"workload": WORKLOAD_NAMES[args.config], "name": args.config, "T": cfg.T,
                   "d_model": cfg.d, "E": cfg.E, "top_k": cfg.k, "d_ff": cfg.d_ff,
                   "act": cfg.act, "threshold": h, "capacity_factor": cfg.capacity_factor,
                   "seed": args.seed,
                   "similarity": ("fp8 (E4M3) screen, undecided tiles recomputed in bf16"
                                  if L.similarity_screen_applies(cfg.T, cfg.d, cfg.E, cfg.k,
                                                                 L.LUFFY_BF16 if cfg.dtype == "bf16" else L.LUFFY_F32)
                                  else cfg.dtype)},
        "condensation": head["condensation"],
        "roofline": head["roofline"],
        "kernels": head["kernels"],
        "cpu_baseline": head["cpu_baseline"],
        "workloads": extras,
        "history": history,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
