"""luffy_route_noalloc (the route entry point that allocates nothing, for
callers that cannot allocate) against luffy_route through the C ABI: the
same inputs give bit-identical routing (indices, slot positions, buckets,
offsets, gates and norms) on two calls in a row, the second on a smaller
batch, so the second call runs on the scratch the first one left behind."""
import numpy as np
import pytest

import luffy_gen as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_15419_amd as L
    L.load_library()


def route_call(inp, dev, noalloc):
    import torch
    import paper_2411_15419_amd as L
    cfg = inp.cfg
    T, k, E = cfg.T, cfg.k, cfg.E
    o = dict(topk_idx=torch.full((T, k), -7, dtype=torch.int32, device="cuda"),
             topk_gate=torch.full((T, k), -7.0, device="cuda"),
             slot_pos=torch.full((T, k), -7, dtype=torch.int32, device="cuda"),
             perm_token=torch.full((T * k,), -7, dtype=torch.int32, device="cuda"),
             offsets=torch.full((E + 1,), -7, dtype=torch.int32, device="cuda"),
             inv_norm=torch.full((T,), -7.0, device="cuda"))
    args = (dev["x"], dev["w_g"], dev["b_g"], k, cfg.capacity_factor, o["topk_idx"], o["topk_gate"],
            o["slot_pos"], o["perm_token"], o["offsets"])
    if noalloc:
        L.luffy_route_noalloc(*args, inv_norm=o["inv_norm"])
    else:
        ws = torch.empty(max(L.route_workspace_size(T, E, k), 256), dtype=torch.uint8, device="cuda")
        L.luffy_route(*args, ws, inv_norm=o["inv_norm"])
    return o


def to_host(o):
    import torch
    torch.cuda.synchronize()
    return {n: t.cpu().numpy() for n, t in o.items()}


def assert_same(a, b):
    S = int(a["offsets"][-1])
    assert S > 0
    for n in ("topk_idx", "topk_gate", "slot_pos", "offsets", "inv_norm"):
        assert np.array_equal(a[n], b[n]), n
    assert np.array_equal(a["perm_token"][:S], b["perm_token"][:S]), "perm_token"


def test_noalloc_route_matches_route_twice():
    import paper_2411_15419_amd as L
    from tests.layer_runner import upload
    big = G.make_inputs("c5", seed=0, T=65536, d=256, d_ff=64, weights=False)   # 1 MiB of slot counts, drops
    small = G.make_inputs("c2", seed=1, T=3000, d=256, d_ff=64, n_centres=128, weights=False)
    devs = [upload(big), upload(small)]
    refs = [to_host(route_call(inp, dv, noalloc=False)) for inp, dv in zip((big, small), devs)]
    # two no-alloc calls in a row, the second on the smaller batch
    outs = []
    for inp, dv in zip((big, small), devs):
        cfg = inp.cfg
        print(f"[case] noalloc route T={cfg.T} E={cfg.E} k={cfg.k} cf={cfg.capacity_factor}", flush=True)
        outs.append(route_call(inp, dv, noalloc=True))
    for ref, out in zip(refs, outs):
        assert_same(ref, to_host(out))
    assert L.load_library().luffy_route_noalloc_max_bytes() == 4 << 20


def test_noalloc_route_rejects_oversized_batch():
    import torch
    import paper_2411_15419_amd as L
    lib = L.load_library()
    T, E, k, d = 131072, 64, 2, 64
    assert lib.luffy_route_workspace_size(T, E, k) > lib.luffy_route_noalloc_max_bytes()
    x = torch.zeros(T, d, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(E, d, dtype=torch.bfloat16, device="cuda")
    i32 = torch.zeros(T * k, dtype=torch.int32, device="cuda")
    f32 = torch.zeros(T * k, device="cuda")
    st = lib.luffy_route_noalloc(x.data_ptr(), T, d, 1, w.data_ptr(), None, E, k, 0.0, i32.data_ptr(),
                                 f32.data_ptr(), i32.data_ptr(), i32.data_ptr(), i32.data_ptr(), None, None)
    assert st == -2
    assert b"scratch" in lib.luffy_last_error()
