"""The EXACT input family and its certificate (tests/exactness.py), on the
CPU: the arithmetic fact the certificate rests on, its quantum computation,
the family's properties, and the certificate holding for the networks and
sizes the GPU tests run on this family."""
import numpy as np
import pytest

import exactness
from cases import exact_network_case, exact_stage_case
from oracle import network
from workloads import specs, synth
from workloads.specs import BF16, CONV3X3


def test_quantum_hand_values():
    q = exactness.quantum
    assert q([3.0]) == 1.0
    assert q([0.75, 1.5]) == 0.25
    assert q([6.0, 4.0, -12.0]) == 2.0
    assert q([5 * 2.0 ** -13, 2.0 ** -3]) == 2.0 ** -13
    assert q([0.0, 0.0]) == float("inf")
    assert q([2.0 ** 40 + 2.0 ** 10]) == 2.0 ** 10


def test_float32_sums_within_the_bound_are_order_independent():
    """Terms that are multiples of q with sum of magnitudes <= 2^24 q: every
    float32 summation order gives the float64 sum.  Just above the bound,
    some order does not."""
    rng = np.random.default_rng(5)
    q = 2.0 ** -7
    terms = rng.integers(-300, 301, size=20000) * q
    assert np.sum(np.abs(terms)) <= 2 ** 24 * q
    want = float(np.sum(terms))
    for _ in range(20):
        perm = rng.permutation(terms).astype(np.float32)
        acc = np.float32(0)
        for chunk in np.array_split(perm, 37):      # blocked, as a K loop would be
            acc = np.float32(acc + np.sum(chunk, dtype=np.float32))
        assert float(acc) == want
    big = np.array([2.0 ** 24, 1.0, -2.0 ** 24], dtype=np.float64)
    assert np.sum(np.abs(big)) > 2 ** 24
    f32 = np.float32(np.float32(big[0]) + np.float32(big[1])) + np.float32(big[2])
    assert float(f32) != float(np.sum(big))


def test_certificate_flags_an_inexact_layer():
    """One 3x3 layer whose input holds 2^23 next to 1: the forward sum bound
    exceeds 2^24 and the certificate reports it."""
    net = specs.Net("one", (specs.Layer(CONV3X3, 1, 1, relu=False, bias=False),), 1, 3, 3)
    w = np.ones((1, 1, 3, 3))
    x = np.ones((1, 1, 3, 3))
    x[0, 0, 1, 1] = 2.0 ** 23
    x[0, 0, 0, 0] = 2.0 ** 23
    r = network.run(net, [(w, None)], x, out_grads=[np.ones((1, 1, 3, 3))], storage="bf16")
    cert = exactness.certificate(net, [(w, None)], r)
    assert cert["forward"] > 1.0 and not exactness.exact(cert)


def test_exact_family_values():
    """Integers in the stated ranges, three +-1 entries per output channel,
    and the same draws for the same seeds."""
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    for idx, L in enumerate(net.layers):
        (w, _), b = synth.layer_params(net, idx, BF16, family=synth.EXACT)
        nz = (w != 0).reshape(w.shape[0], -1).sum(axis=1)
        assert np.all(nz == synth.EXACT_NNZ) and set(np.unique(w)) <= {-1.0, 0.0, 1.0}
        if b is not None:
            assert set(np.unique(b[0])) <= {-1.0, 0.0, 1.0}
    x, _ = synth.input_x(net, 4, BF16, family=synth.EXACT)
    assert set(np.unique(x)) == {-2.0, -1.0, 0.0, 1.0, 2.0}
    g, _ = synth.upstream_grad((4, 64, 8, 8), BF16, 1, synth.EXACT)
    assert set(np.unique(g)) == {-1.0, 0.0, 1.0} and 0.4 < np.mean(g != 0) < 0.6
    x2, _ = synth.input_x(net, 4, BF16, family=synth.EXACT)
    np.testing.assert_array_equal(x, x2)
    dw = synth.layer_params(specs.amoeba_cells(1, 8, 4), 0, BF16, family=synth.EXACT)[0][0]
    assert np.all((dw != 0).reshape(8, 9).sum(axis=1) == 3)


def test_exact_runs_exercise_every_decision():
    """On the exact family the networks still decide: every ReLU layer zeroes
    some outputs and keeps others, max-pool windows hold ties (so the
    first-maximum rule is exercised), and every weight gradient is
    nonzero."""
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    case = exact_network_case(net, 4)
    r, tape = case["ref"], case["ref"]["tape"]
    for idx, (L, y) in enumerate(zip(net.layers, tape.outputs)):
        if L.relu:
            frac = np.mean(y == 0)
            assert 0.2 < frac < 0.8, (idx, frac)
    ties = 0
    for idx, arg in tape.argmax.items():
        inp = tape.outputs[idx - 1]
        n, c, h, w = inp.shape
        win = inp.reshape(n, c, h // 2, 2, w // 2, 2).transpose(0, 1, 2, 4, 3, 5).reshape(
            n, c, h // 2, w // 2, 4)
        ties += int(np.sum(np.sum(win == win.max(axis=-1, keepdims=True), axis=-1) > 1))
    assert ties > 0
    for idx, (dW, db) in r["grads"].items():
        assert np.any(dW != 0), idx


# The networks and sizes the GPU tests run on the exact family, at the sizes
# they run (the two 192x192 samples of the full-size stage test and the
# 6-level network at 64x64 are certified inside those GPU tests).
NETWORK_CASES = [
    (lambda: specs.unet(3, 64, 64, 32, "unet3-c64-32"), 4),
    (lambda: specs.unet(3, 64, 64, 32, "unet3-c64-32"), 8),
    (lambda: specs.unet(2, 64, 64, 16, "unet2-c64-16"), 4),
    (lambda: specs.unet(2, 64, 64, 64, "unet2-c64-64"), 4),
]


@pytest.mark.parametrize("make,B", NETWORK_CASES)
def test_certificate_holds_for_network_cases(make, B):
    net = make()
    case = exact_network_case(net, B)
    cert = case["cert"]
    assert exactness.exact(cert) and cert["loss_sum"] <= 1.0, cert


@pytest.mark.parametrize("name,lo,hi,B,popped", [
    ("unet5-48", 0, 7, 4, False),
    ("unet5-32", 7, 12, 4, True),
    ("unet5-32", 12, 15, 4, True),
    ("unet5-32", 15, 19, 4, True),
    ("cells", 0, 8, 4, False),
    ("poolin", 0, 3, 4, False),
])
def test_certificate_holds_for_stage_cases(name, lo, hi, B, popped):
    nets = {"unet5-48": specs.unet(5, 64, 64, 48, "unet5-c64-48"),
            "unet5-32": specs.unet(5, 64, 64, 32, "unet5-c64-32"),
            "cells": specs.amoeba_cells(4, 256, 14, "cells4-c256"),
            "poolin": specs.Net("poolin", (
                specs.Layer(CONV3X3, 64, 64, stash_id=0),
                specs.Layer(CONV3X3, 64, 128, prologue=specs.PRO_MAXPOOL2),
                specs.Layer(CONV3X3, 192, 64, prologue=specs.PRO_UPCAT2, pop_id=0)), 64, 16, 24)}
    case = exact_stage_case(nets[name], lo, hi, B, popped)
    assert exactness.exact(case["cert"]), case["cert"]
