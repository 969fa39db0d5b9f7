"""GPU parity of the loss-driven multi-block driver (Sec. 5.2 Eq. 2 over a
stack with the historical similarity of Sec. 5.1 step 2): over several
training iterations on a synthetic falling loss, the threshold the driver
feeds every block is the oracle's adaptive_threshold of the losses so far,
and every block's condensation at that threshold is bit-exact with the
oracle's condense(history=...) chain."""
import numpy as np
import pytest

import luffy_gen as G
from oracle import luffy_oracle as O
from tests.layer_runner import assert_condense_equal, assert_route_equal, fetch, upload
from tests.test_gpu_history import as_oracle_ns, oracle_chain

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_15419_amd as L
    L.load_library()


def falling_loss(t):
    return 6.0 * 0.6 ** t + 0.5


@pytest.mark.parametrize("ffn", [False, True])
def test_driver_iterations_match_oracle(ffn):
    import torch
    import paper_2411_15419_amd as L
    from tests.layer_runner import make_layer
    S1, S2, blocks, iters = 0.8, 0.2, 3, 5
    kw = dict(T=1024, d=1024, E=8, n_centres=128, d_ff=256, mix_fraction=0.0, token_drift=0.3, gate_drift=0.02)
    # the layers of the stack are built once, from the first iteration's router weights
    first = G.make_stack("c2", blocks, seed=100, weights=True, **kw)
    layers = []
    for inp in first:
        dev = upload(inp)
        base = make_layer(inp, dev)
        layers.append(L.MoELayer(base.w_gate, base.b_gate, base.w1, base.w2, k=inp.cfg.k, act=inp.cfg.act,
                                 threshold=0.9, capacity_factor=inp.cfg.capacity_factor, T=inp.cfg.T,
                                 history=(S1, S2)))
    driver = L.CondensationDriver(L.MoEStack(layers))
    losses = []
    for it in range(iters):
        # a new batch of tokens every iteration; the router weights are the layers'
        stack = G.make_stack("c2", blocks, seed=200 + it, **kw)
        for b in range(blocks):
            stack[b].w_g, stack[b].b_g = first[b].w_g, first[b].b_g
        want_h = 0.5 if not losses else O.adaptive_threshold(losses[0], losses[-1])
        xs = [upload(inp)["x"] for inp in stack]
        h, _ = driver.step(xs, falling_loss(it), ffn=ffn)
        torch.cuda.synchronize()
        assert abs(h - want_h) <= 1e-12, (it, h, want_h)
        print(f"[case] driver iteration {it}: h={h:.6f}", flush=True)
        ref = oracle_chain(stack, h, S1, S2)
        for b, (layer, o) in enumerate(zip(layers, ref)):
            g = fetch(layer, with_ffn=False)
            on = as_oracle_ns(o)
            assert_route_equal(g, on)
            assert_condense_equal(g, on)
            st = layer.hist_stats.cpu().numpy()
            assert int(st[0]) == o["undecided"] and int(st[1]) == o["decided"], (it, b)
        losses.append(falling_loss(it))
    assert driver.thresholds[0] == 0.5
    assert all(a > b for a, b in zip(driver.thresholds[1:], driver.thresholds[2:])), driver.thresholds
    assert 1.0 / (1.0 + np.e) < min(driver.thresholds)
