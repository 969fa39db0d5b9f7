"""Pins of the oracle's backward pass (CPU): each gradient is checked against
the forward functions it differentiates, by exact linearity where the
forward is linear and by central finite differences elsewhere, so a
transposed operand, a dropped term or a wrong derivative fails."""
import math

import numpy as np
import pytest

from oracle import luffy_oracle as O


def _routing_case(rng, T=40, k=2, E=5, R=23, d=24, drop=0.2):
    """A combine problem: slot positions with some dropped slots, every kept
    position mapped to one of R representative rows."""
    S = T * k
    slot_pos = np.arange(S, dtype=np.int64).reshape(T, k)
    slot_pos[rng.random((T, k)) < drop] = -1
    rep_row = rng.integers(0, R, S)
    gate = rng.random((T, k))
    y_rep = rng.standard_normal((R, d))
    dy = rng.standard_normal((T, d))
    return y_rep, rep_row, slot_pos, gate, dy


def test_combine_backward_is_the_transpose_in_y_rep():
    # combine is linear in Y_rep: <combine(Y + D), dy> - <combine(Y), dy> = <D, dy_rep>
    rng = np.random.default_rng(1)
    for _ in range(5):
        y_rep, rep_row, slot_pos, gate, dy = _routing_case(rng)
        dy_rep, _ = O.combine_backward(dy, y_rep, rep_row, slot_pos, gate)
        D = rng.standard_normal(y_rep.shape)
        lhs = np.sum(O.combine(y_rep + D, rep_row, slot_pos, gate) * dy) - \
            np.sum(O.combine(y_rep, rep_row, slot_pos, gate) * dy)
        assert lhs == pytest.approx(np.sum(D * dy_rep), rel=1e-10)


def test_combine_backward_gate_gradient():
    # combine is linear in each gate: a step eps in gate[t, j] changes
    # <y, dy> by eps * dgate[t, j]; dropped slots have dgate = 0
    rng = np.random.default_rng(2)
    y_rep, rep_row, slot_pos, gate, dy = _routing_case(rng)
    _, dgate = O.combine_backward(dy, y_rep, rep_row, slot_pos, gate)
    base = np.sum(O.combine(y_rep, rep_row, slot_pos, gate) * dy)
    for t in range(gate.shape[0]):
        for j in range(gate.shape[1]):
            g2 = gate.copy()
            g2[t, j] += 0.5
            diff = np.sum(O.combine(y_rep, rep_row, slot_pos, g2) * dy) - base
            assert diff == pytest.approx(0.5 * dgate[t, j], rel=1e-9, abs=1e-12)
            if slot_pos[t, j] < 0:
                assert dgate[t, j] == 0.0


def test_combine_backward_hand_case():
    # two tokens, top-2; slots 0 (t0,j0) and 3 (t1,j1) share representative
    # row 0, slot 1 (t1, j0) is row 1, slot 2 (t0, j1) is dropped
    slot_pos = np.array([[0, -1], [1, 3]])
    rep_row = np.array([0, 1, 7, 0])
    gate = np.array([[0.75, 0.25], [0.5, 0.5]])
    y_rep = np.array([[1.0, 2.0], [3.0, -1.0]])
    dy = np.array([[1.0, 1.0], [2.0, 0.0]])
    dy_rep, dgate = O.combine_backward(dy, y_rep, rep_row, slot_pos, gate)
    np.testing.assert_array_equal(dy_rep, [[0.75 * 1 + 0.5 * 2, 0.75 * 1 + 0.5 * 0], [0.5 * 2, 0.0]])
    np.testing.assert_array_equal(dgate, [[3.0, 0.0], [6.0, 2.0]])


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_activation_grad_matches_finite_differences(act):
    z = np.linspace(-9.0, 9.0, 721)
    eps = 1e-5
    fd = (O.activation(z + eps, act) - O.activation(z - eps, act)) / (2 * eps)
    np.testing.assert_allclose(O.activation_grad(z, act), fd, rtol=0, atol=1e-9)
    # special values: slope 1/2 at 0, 1 far right, 0 far left
    assert O.activation_grad(0.0, act) == 0.5
    assert O.activation_grad(40.0, act) == pytest.approx(1.0, abs=1e-12)
    assert O.activation_grad(-40.0, act) == pytest.approx(0.0, abs=1e-12)


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_expert_ffn_backward_directional_derivatives(act):
    # L = <Y_rep(x, W1, W2), dY>; for random directions the central
    # difference of L matches <gradient, direction> for x, W1 and W2, with an
    # empty expert and a one-row expert in the mix
    rng = np.random.default_rng(3)
    E, d, dff = 4, 12, 20
    sizes = [5, 0, 1, 7]
    rep_offsets = np.concatenate([[0], np.cumsum(sizes)])
    R = rep_offsets[-1]
    x = rng.standard_normal((R, d))
    w1 = 0.4 * rng.standard_normal((E, dff, d))
    w2 = 0.4 * rng.standard_normal((E, d, dff))
    dy = rng.standard_normal((R, d))
    dx, dw1, dw2 = O.expert_ffn_backward(x, rep_offsets, w1, w2, act, dy)

    def L(x_, w1_, w2_):
        return float(np.sum(O.expert_ffn(x_, rep_offsets, w1_, w2_, act) * dy))

    eps = 1e-6
    for _ in range(4):
        vx, v1, v2 = rng.standard_normal(x.shape), rng.standard_normal(w1.shape), rng.standard_normal(w2.shape)
        fd_x = (L(x + eps * vx, w1, w2) - L(x - eps * vx, w1, w2)) / (2 * eps)
        fd_1 = (L(x, w1 + eps * v1, w2) - L(x, w1 - eps * v1, w2)) / (2 * eps)
        fd_2 = (L(x, w1, w2 + eps * v2) - L(x, w1, w2 - eps * v2)) / (2 * eps)
        assert np.sum(dx * vx) == pytest.approx(fd_x, rel=1e-6, abs=1e-8)
        assert np.sum(dw1 * v1) == pytest.approx(fd_1, rel=1e-6, abs=1e-8)
        assert np.sum(dw2 * v2) == pytest.approx(fd_2, rel=1e-6, abs=1e-8)
    # the empty expert gets zero weight gradients
    assert not dw1[1].any() and not dw2[1].any()


def test_expert_ffn_backward_scalar_case():
    # one expert, one row, d = d_ff = 1, worked by hand with SiLU:
    # y = w2 act(w1 x); dx = dy w2 act'(w1 x) w1, dw1 = dy w2 act'(w1 x) x,
    # dw2 = dy act(w1 x)
    x = np.array([[0.7]])
    w1 = np.array([[[1.5]]])
    w2 = np.array([[[-2.0]]])
    dy = np.array([[3.0]])
    dx, dw1, dw2 = O.expert_ffn_backward(x, np.array([0, 1]), w1, w2, "silu", dy)
    z = 1.05
    s = 1.0 / (1.0 + math.exp(-z))
    ds = s * (1 + z * (1 - s))
    assert dx[0, 0] == pytest.approx(3.0 * -2.0 * ds * 1.5, rel=1e-14)
    assert dw1[0, 0, 0] == pytest.approx(3.0 * -2.0 * ds * 0.7, rel=1e-14)
    assert dw2[0, 0, 0] == pytest.approx(3.0 * z * s, rel=1e-14)
