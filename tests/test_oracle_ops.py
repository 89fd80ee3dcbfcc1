"""Pins for the oracle's operators against things other than themselves:
closed forms, brute-force loops on tiny inputs, adjoint identities, and
torch-CPU float64 library routines."""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import ops

rng = np.random.default_rng(1234)


def brute_conv3x3(x, w, b):
    """Direct six-deep loop of z[n,o,h,w] = b[o] + sum W[o,c,r,s] x[n,c,h+r-1,w+s-1]."""
    N, C, H, W = x.shape
    O = w.shape[0]
    z = np.zeros((N, O, H, W))
    for n, o, h, ww in itertools.product(range(N), range(O), range(H), range(W)):
        acc = b[o]
        for c, r, s in itertools.product(range(C), range(3), range(3)):
            hh, wq = h + r - 1, ww + s - 1
            if 0 <= hh < H and 0 <= wq < W:
                acc += w[o, c, r, s] * x[n, c, hh, wq]
        z[n, o, h, ww] = acc
    return z


def test_conv3x3_matches_brute_force():
    x = rng.standard_normal((2, 3, 5, 4))
    w = rng.standard_normal((4, 3, 3, 3))
    b = rng.standard_normal(4)
    np.testing.assert_allclose(ops.conv3x3_forward(x, w, b), brute_conv3x3(x, w, b),
                               rtol=1e-13, atol=1e-13)


def test_conv3x3_centre_delta_is_identity_plus_bias():
    C = 5
    x = rng.standard_normal((2, C, 6, 7))
    w = np.zeros((C, C, 3, 3))
    for c in range(C):
        w[c, c, 1, 1] = 1.0
    b = rng.standard_normal(C)
    np.testing.assert_array_equal(ops.conv3x3_forward(x, w, b), x + b[None, :, None, None])


@pytest.mark.parametrize("r,s", [(0, 0), (2, 2), (0, 2), (2, 1)])
def test_conv3x3_corner_delta_shifts_with_zero_padding(r, s):
    x = rng.standard_normal((1, 1, 5, 6))
    w = np.zeros((1, 1, 3, 3))
    w[0, 0, r, s] = 1.0
    z = ops.conv3x3_forward(x, w)
    H, W = 5, 6
    for h, q in itertools.product(range(H), range(W)):
        hh, qq = h + r - 1, q + s - 1
        want = x[0, 0, hh, qq] if (0 <= hh < H and 0 <= qq < W) else 0.0
        assert z[0, 0, h, q] == want


def test_conv3x3_all_ones_interior_edge_corner():
    C, H, W = 4, 5, 6
    z = ops.conv3x3_forward(np.ones((1, C, H, W)), np.ones((2, C, 3, 3)), np.array([0.5, -1.0]))
    for o, bias in enumerate([0.5, -1.0]):
        assert z[0, o, 2, 3] == 9 * C + bias       # interior
        assert z[0, o, 0, 3] == 6 * C + bias       # edge
        assert z[0, o, 2, 0] == 6 * C + bias       # edge
        assert z[0, o, 0, 0] == 4 * C + bias       # corner
        assert z[0, o, H - 1, W - 1] == 4 * C + bias


def test_conv1x1_is_channel_matmul():
    x = rng.standard_normal((3, 6, 4, 5))
    w = rng.standard_normal((7, 6, 1, 1))
    b = rng.standard_normal(7)
    want = np.matmul(w[:, :, 0, 0][None], x.reshape(3, 6, 20)).reshape(3, 7, 4, 5)
    np.testing.assert_allclose(ops.conv1x1_forward(x, w, b), want + b[None, :, None, None],
                               rtol=1e-13, atol=1e-13)


def test_dwconv_is_per_channel_conv3x3():
    x = rng.standard_normal((2, 3, 5, 5))
    w = rng.standard_normal((3, 1, 3, 3))
    z = ops.dwconv3x3_forward(x, w)
    for c in range(3):
        wc = np.zeros((1, 1, 3, 3))
        wc[0, 0] = w[c, 0]
        np.testing.assert_allclose(z[:, c:c + 1], brute_conv3x3(x[:, c:c + 1], wc, [0.0]),
                                   rtol=1e-13, atol=1e-13)


def _dot(a, b):
    return float(np.sum(a * b))


@pytest.mark.parametrize("kind", ["3x3", "1x1", "dw"])
def test_adjoint_identities(kind):
    N, C, O, H, W = 2, 5, 6, 7, 6
    if kind == "dw":
        O = C
        w = rng.standard_normal((C, 1, 3, 3))
        fwd, dg, wg = ops.dwconv3x3_forward, ops.dwconv3x3_dgrad, ops.dwconv3x3_wgrad
    elif kind == "1x1":
        w = rng.standard_normal((O, C, 1, 1))
        fwd, dg, wg = ops.conv1x1_forward, ops.conv1x1_dgrad, ops.conv1x1_wgrad
    else:
        w = rng.standard_normal((O, C, 3, 3))
        fwd, dg, wg = ops.conv3x3_forward, ops.conv3x3_dgrad, ops.conv3x3_wgrad
    x = rng.standard_normal((N, C, H, W))
    y = rng.standard_normal((N, O, H, W))
    lhs = _dot(fwd(x, w), y)
    assert abs(lhs - _dot(x, dg(y, w))) <= 1e-12 * abs(lhs) + 1e-12
    assert abs(lhs - _dot(w, wg(x, y))) <= 1e-12 * abs(lhs) + 1e-12
    # bias gradient: <b broadcast, y> = <b, bias_grad(y)>
    b = rng.standard_normal(O)
    assert abs(_dot(b[None, :, None, None] * np.ones_like(y), y) - _dot(b, ops.bias_grad(y))) < 1e-11


def test_pool_and_upsample_adjoints():
    x = rng.standard_normal((2, 3, 6, 8))
    y, arg = ops.maxpool2_forward(x)
    dy = rng.standard_normal(y.shape)
    # with the argmax fixed, pooling is a selection; its adjoint routes dy back
    assert abs(_dot(y, dy) - _dot(x, ops.maxpool2_backward(dy, arg))) < 1e-12
    u = rng.standard_normal((2, 3, 12, 16))
    assert abs(_dot(ops.upsample2_forward(x), u) - _dot(x, ops.upsample2_backward(u))) < 1e-11


def test_maxpool_values_and_ties():
    x = np.array([[[[1.0, 3.0, 2.0, 2.0],
                    [3.0, 0.0, 2.0, 2.0],
                    [-1.0, -5.0, 0.0, 0.0],
                    [-2.0, -1.0, 0.0, 7.0]]]])
    y, arg = ops.maxpool2_forward(x)
    np.testing.assert_array_equal(y[0, 0], [[3.0, 2.0], [-1.0, 7.0]])
    # ties resolve to the first element in row-major window order
    np.testing.assert_array_equal(arg[0, 0], [[1, 0], [0, 3]])
    dx = ops.maxpool2_backward(np.array([[[[10.0, 20.0], [30.0, 40.0]]]]), arg)
    want = np.zeros((4, 4))
    want[0, 1], want[0, 2], want[2, 0], want[3, 3] = 10, 20, 30, 40
    np.testing.assert_array_equal(dx[0, 0], want)


def test_ops_match_torch_float64():
    x = rng.standard_normal((2, 4, 8, 6))
    w = rng.standard_normal((5, 4, 3, 3))
    b = rng.standard_normal(5)
    tx = torch.tensor(x)
    np.testing.assert_allclose(ops.conv3x3_forward(x, w, b),
                               F.conv2d(tx, torch.tensor(w), torch.tensor(b), padding=1).numpy(),
                               rtol=1e-12, atol=1e-12)
    wd = rng.standard_normal((4, 1, 3, 3))
    np.testing.assert_allclose(ops.dwconv3x3_forward(x, wd),
                               F.conv2d(tx, torch.tensor(wd), padding=1, groups=4).numpy(),
                               rtol=1e-12, atol=1e-12)
    y, _ = ops.maxpool2_forward(x)
    np.testing.assert_array_equal(y, F.max_pool2d(tx, 2).numpy())
    np.testing.assert_array_equal(ops.upsample2_forward(x),
                                  F.interpolate(tx, scale_factor=2, mode="nearest").numpy())


def test_round_bf16_against_hand_values_and_torch():
    one = 1.0
    ulp = 2.0 ** -7          # bf16 spacing in [1, 2)
    cases = {
        one + ulp / 2: one,                    # tie -> even (1.0)
        one + 3 * ulp / 2: one + 2 * ulp,      # tie -> even (1 + 2 ulp)
        one + ulp / 2 + 2 ** -20: one + ulp,   # above the tie -> up
        -(one + ulp / 4): -one,
        3.0: 3.0,
        0.0: 0.0,
    }
    got = ops.round_bf16(np.array(list(cases.keys())))
    np.testing.assert_array_equal(got, np.array(list(cases.values())))
    v = rng.standard_normal(10000) * 10.0
    want = torch.tensor(v, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ops.round_bf16(v), want)


def test_mse_closed_form():
    y = np.array([1.0, 2.0, 4.0])
    t = np.array([0.0, 2.0, 1.0])
    loss, dy = ops.mse(y, t, 3)
    assert loss == (1.0 + 0.0 + 9.0) / 3
    np.testing.assert_array_equal(dy, np.array([2.0, 0.0, 6.0]) / 3)
