"""GPU parity of the historical similarity (Sec. 5.1 step 2) over stacks of
blocks: every block's routing, degrees and representatives bit-exact with
the oracle's condense(history=(previous record, S1, S2)); the pair counts
the record decided / left undecided equal the oracle's, bucket by bucket;
and the record each block leaves holds, for every pair of every bucket, the
oracle's classes of that block's weight (w > S1, w < S2)."""
import numpy as np
import pytest

import luffy_gen as G
from oracle import luffy_oracle as O
from tests.layer_runner import assert_condense_equal, assert_route_equal, fetch, upload

pytestmark = pytest.mark.gpu

MARGIN = 1e-3   # computed cosines this far from h, S1, S2 (float32 vs float64 decisions)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_15419_amd as L
    L.load_library()


def oracle_chain(stack, h, S1, S2):
    """Per block: the oracle's layer indices with history, its record, and
    the per-bucket counts of undecided / decided pairs (a < b)."""
    T = stack[0].cfg.T
    prev = np.full((T, T), np.nan)
    out = []
    for inp in stack:
        cfg = inp.cfg
        x = inp.x.astype(np.float64)
        idx, gates, logits = O.gate(x, inp.w_g, inp.b_g, cfg.k)
        C = O.capacity_of(cfg.T, cfg.k, cfg.E, cfg.capacity_factor)
        offsets, perm_token, slot_pos = O.dispatch(idx, cfg.E, C)
        cz = O.condense(x, perm_token, offsets, h, history=(prev, S1, S2))
        und = dec = 0
        worst = np.inf
        for e in range(cfg.E):
            tok = perm_token[offsets[e]:offsets[e + 1]]
            if tok.size < 2:
                continue
            w, comp = O.historical_weights(x, tok, prev, S1, S2)
            up = np.triu(np.ones_like(comp), 1)
            und += int((comp & up).sum())
            dec += int((~comp & up).sum())
            if comp.any():
                cw = w[comp]
                worst = min(worst, float(np.min(np.abs(cw[:, None] - np.array([h, S1, S2])[None, :]))))
        assert worst >= MARGIN, f"a computed cosine lies within {worst:.2e} of h, S1 or S2"
        rec, n_comp = O.historical_record(x, perm_token, offsets, prev, S1, S2)
        out.append(dict(topk_idx=idx, topk_gate=gates, offsets=offsets, perm_token=perm_token, slot_pos=slot_pos,
                        cz=cz, rec=rec, undecided=und, decided=dec))
        prev = rec
    return out


def as_oracle_ns(o):
    from types import SimpleNamespace
    return SimpleNamespace(topk_idx=o["topk_idx"], topk_gate=o["topk_gate"], offsets=o["offsets"],
                           perm_token=o["perm_token"], slot_pos=o["slot_pos"], **vars(o["cz"]))


def decode_record(raw, T, E, k, max_bucket):
    """Sections of a record as the header lays them out."""
    def take(off, n, dt):
        off = (off + 255) // 256 * 256
        a = np.frombuffer(raw[off:off + n * np.dtype(dt).itemsize].tobytes(), dtype=dt)
        return a, off + n * np.dtype(dt).itemsize
    S = T * k
    W = S * ((max_bucket + 63) // 64)
    info, o = take(0, 8, np.int32)
    slot_pos, o = take(o, S, np.int32)
    offsets, o = take(o, E + 1, np.int32)
    word_off, o = take(o, E + 1, np.int64)
    hi, o = take(o, W, np.uint64)
    lo, o = take(o, W, np.uint64)
    return info, slot_pos, offsets, word_off, hi, lo


def assert_record(raw, o, cfg, max_bucket, S1, S2):
    info, slot_pos, offsets, word_off, hi, lo = decode_record(raw, cfg.T, cfg.E, cfg.k, max_bucket)
    assert info[1:5].tolist() == [cfg.T, cfg.E, cfg.k, max_bucket] and info[0] != 0
    assert np.array_equal(slot_pos.reshape(cfg.T, cfg.k), o["slot_pos"])
    assert np.array_equal(offsets, o["offsets"])
    rec = o["rec"]
    with np.errstate(invalid="ignore"):
        for e in range(cfg.E):
            lo_, hi_ = int(offsets[e]), int(offsets[e + 1])
            n = hi_ - lo_
            if n == 0:
                continue
            Wn = (n + 63) // 64
            words = np.arange(n)[:, None] * Wn + np.arange(Wn)[None, :] + word_off[e]
            tok = o["perm_token"][lo_:hi_]
            r = rec[np.ix_(tok, tok)]
            for mask, want in ((hi, r > S1), (lo, r < S2)):
                bits = np.unpackbits(mask[words].view(np.uint8).reshape(n, Wn, 8), axis=2,
                                     bitorder="little").reshape(n, Wn * 64)[:, :n].astype(bool)
                assert np.array_equal(bits, want), f"record bucket {e}: {np.argwhere(bits != want)[:5]}"


def run_stack(stack, h, S1, S2, check_record=True, expect=None):
    import torch
    import paper_2411_15419_amd as L
    from tests.layer_runner import make_layer
    ref = oracle_chain(stack, h, S1, S2)
    prev = None
    layers = []
    all_stats = []
    for b, (inp, o) in enumerate(zip(stack, ref)):
        cfg = inp.cfg
        print(f"[case] history block {b} T={cfg.T} d={cfg.d} E={cfg.E} k={cfg.k} dtype={cfg.dtype} "
              f"h={h} S1={S1} S2={S2}", flush=True)
        dev = upload(inp)
        layer = make_layer(inp, dev, h)
        lh = L.MoELayer(layer.w_gate, layer.b_gate, layer.w1, layer.w2, k=cfg.k, act=cfg.act, threshold=h,
                        capacity_factor=cfg.capacity_factor, T=cfg.T, history=(S1, S2))
        lh.route(dev["x"])
        lh.condense(dev["x"], hist_in=prev)
        g = fetch(lh, with_ffn=False)
        stats = lh.hist_stats.cpu().numpy()
        on = as_oracle_ns(o)
        assert_route_equal(g, on)
        assert_condense_equal(g, on)
        assert int(stats[0]) == o["undecided"] and int(stats[1]) == o["decided"], \
            (b, stats.tolist(), o["undecided"], o["decided"])
        if check_record:
            torch.cuda.synchronize()
            assert_record(lh.record.cpu().numpy(), o, cfg, lh.max_bucket, S1, S2)
        print(f"[history] block {b}: undecided {stats[0]} decided {stats[1]} tiles computed {stats[2]} "
              f"skipped {stats[3]}; R={int(g['rep_offsets'][-1])} of S={int(g['offsets'][-1])}", flush=True)
        all_stats.append(stats)
        layers.append(lh)
        prev = lh.record
    return all_stats


def test_stack_bf16_top2_drifting():
    """Three blocks, top-2 with capacity drops, tokens and router drifting,
    one token in ten a mixture of two centres (pairs in the S2..S1 band are
    computed in every block)."""
    stack = G.make_stack("c2", 3, seed=0, T=2048, d=1024, E=8, n_centres=256, mix_fraction=0.1,
                         token_drift=0.3, gate_drift=0.05)
    st = run_stack(stack, h=0.9, S1=0.8, S2=0.3)
    assert st[0][1] == 0 and st[1][1] > 0 and st[1][0] > 0


def test_stack_identical_blocks_skip_every_tile():
    """Identical blocks: block 1 and 2 find every pair decided and compute no
    similarity tile (the record alone gives their graph)."""
    stack = G.make_stack("c2", 3, seed=1, T=2048, d=1024, E=4, n_centres=64, token_drift=0.0,
                         gate_drift=0.0, capacity_factor=0.0)
    st = run_stack(stack, h=0.9, S1=0.8, S2=0.3)
    assert st[0][2] > 0 and st[0][3] == 0
    for s in st[1:]:
        assert s[0] == 0 and s[2] == 0 and s[3] > 0


def test_stack_top1_capacity():
    stack = G.make_stack("c5", 2, seed=2, T=4096, d=512, E=16, n_centres=512, mix_fraction=0.05,
                         token_drift=0.2, gate_drift=0.0)
    run_stack(stack, h=0.95, S1=0.8, S2=0.35)


def test_stack_f32():
    stack = G.make_stack("c1", 3, seed=3, mix_fraction=0.1, token_drift=0.5, gate_drift=0.02)
    run_stack(stack, h=0.95, S1=0.8, S2=0.45)


@pytest.mark.parametrize("S1,S2", [(2.0, -2.0), (-2.0, 2.0), (0.6, 0.6)])
def test_stack_threshold_extremes(S1, S2):
    """S1 above every weight and S2 below: nothing decided; S1 below every
    weight: every pair that shared a bucket is decided similar (S1 first);
    S1 = S2: only the pairs at exactly that value stay undecided."""
    stack = G.make_stack("c2", 2, seed=4, T=1024, d=1024, E=4, n_centres=128, mix_fraction=0.0,
                         token_drift=0.1, gate_drift=0.0)
    st = run_stack(stack, h=0.9, S1=S1, S2=S2)
    if S1 > 1:
        assert st[1][1] == 0
