"""Pins for the oracle's full-batch network pass and its pipeline
decomposition: torch-CPU float64 autograd, central finite differences, the
micro-batch gradient-sum and recompute invariants of Sec. 2 / Sec. 2.1, and
the clock-cycle order of Algorithm 1."""
import numpy as np
import pytest

import golden_data
import torch
import torch.nn.functional as F

import oracle
from oracle import network, ops, pipeline
from workloads import specs, synth
from workloads.specs import (CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER, CONV1X1, CONV3X3,
                             DWCONV3X3, FP32, PRO_MAXPOOL2, PRO_UPCAT2)


def tiny_unet():
    return specs.unet(2, 3, 2, 8, "unet2-c3")


def tiny_unet3():
    return specs.unet(3, 2, 3, 8, "unet3-c2")


def tiny_cells():
    return specs.amoeba_cells(2, 4, 6, "cells2-c4")


def _params(net, seed=0):
    return oracle.net_params(net, FP32, index_offset=seed)


def torch_run(net, params, x, target=None, out_grads=None, lo=0, hi=None):
    """Independent float64 reference with torch autograd (library routines)."""
    hi = len(net.layers) if hi is None else hi
    tp = []
    for w, b in params:
        tw = torch.tensor(w, requires_grad=True)
        tb = None if b is None else torch.tensor(b, requires_grad=True)
        tp.append((tw, tb))
    tx = torch.tensor(x, requires_grad=True)
    cur = tx
    stash = {}
    for idx in range(lo, hi):
        L = net.layers[idx]
        w, b = tp[idx]
        if L.prologue == PRO_MAXPOOL2:
            cur = F.max_pool2d(cur, 2)
        elif L.prologue == PRO_UPCAT2:
            cur = torch.cat([F.interpolate(cur, scale_factor=2, mode="nearest"),
                             stash[L.pop_id]], dim=1)
        if L.kind == DWCONV3X3:
            cur = F.conv2d(cur, w, b if L.bias else None, padding=1, groups=L.cin)
        elif L.kind == CONV1X1:
            cur = F.conv2d(cur, w, b if L.bias else None)
        else:
            cur = F.conv2d(cur, w, b if L.bias else None, padding=1)
        if L.relu:
            cur = F.relu(cur)
        if L.stash_id >= 0:
            stash[L.stash_id] = cur
    if target is not None:
        loss = F.mse_loss(cur, torch.tensor(target), reduction="mean")
    else:
        ex = network.exported_stashes(net, lo, hi)
        loss = (cur * torch.tensor(out_grads[0])).sum()
        for k, s in enumerate(ex):
            loss = loss + (stash[s] * torch.tensor(out_grads[1 + k])).sum()
    loss.backward()
    grads = {i: (tp[i][0].grad.numpy(), None if tp[i][1] is None else tp[i][1].grad.numpy())
             for i in range(lo, hi)}
    return float(loss), grads, tx.grad.numpy()


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


@pytest.mark.parametrize("make", [tiny_unet, tiny_unet3, tiny_cells,
                                  lambda: specs.plain_stack(3, 4, 6, 6)])
def test_network_matches_torch_autograd(make):
    net = make()
    P = _params(net)
    x = synth.normal(11, (3, net.in_channels, net.height, net.width))
    h, w = net.out_hw()
    t = synth.normal(12, (3, net.out_channels(), h, w))
    r = network.run(net, P, x, target=t)
    loss, grads, dx = torch_run(net, P, x, target=t)
    assert abs(r["loss"] - loss) <= 1e-12 * abs(loss)
    for i, (dW, db) in grads.items():
        assert _rel(r["grads"][i][0], dW) < 1e-11, (net.name, i)
        if db is not None:
            assert _rel(r["grads"][i][1], db) < 1e-11, (net.name, i)
    assert _rel(r["dx"], dx) < 1e-11


def test_stage_run_matches_torch_autograd():
    """A partition run alone with injected gradients for its main output and
    for the skips it stashes for later partitions."""
    net = specs.unet(3, 2, 3, 8, "unet3-c2")
    P = _params(net)
    lo, hi = 0, 5        # enc0a enc0b enc1a enc1b enc2a: exports skips 0 and 1
    ex = network.exported_stashes(net, lo, hi)
    assert ex == [0, 1]
    x = synth.normal(21, (2, net.in_channels, 8, 8))
    out_shapes = [(2, 8, 2, 2), (2, 2, 8, 8), (2, 4, 4, 4)]
    G = [synth.normal(30 + k, s) for k, s in enumerate(out_shapes)]
    r = network.run(net, P, x, lo=lo, hi=hi, out_grads=G)
    loss, grads, dx = torch_run(net, P, x, out_grads=G, lo=lo, hi=hi)
    assert abs(r["loss"] - loss) <= 1e-12 * abs(loss)
    for i, (dW, db) in grads.items():
        assert _rel(r["grads"][i][0], dW) < 1e-11
        assert _rel(r["grads"][i][1], db) < 1e-11
    assert _rel(r["dx"], dx) < 1e-11


def _masks(tape):
    return [o > 0 for o in tape.outputs], dict(tape.argmax)


def _same_masks(a, b):
    return all(np.array_equal(u, v) for u, v in zip(a[0], b[0])) and \
        all(np.array_equal(a[1][k], b[1][k]) for k in a[1])


def test_finite_differences_whole_network():
    """Central differences (h = 1e-6) for every parameter and input coordinate
    of a tiny U-Net with pool, upsample-concat skip and a 1x1 head; a
    coordinate whose perturbation flips a ReLU mask or a pool argmax is
    skipped (the function is not differentiable there)."""
    net = tiny_unet()
    P = _params(net, seed=5)
    x = synth.normal(41, (2, net.in_channels, 8, 8))
    t = synth.normal(42, (2, 1, 8, 8))
    base = network.run(net, P, x, target=t)
    base_masks = _masks(base["tape"])
    h = 1e-6

    def loss_at(P2, x2):
        y, tape = network.forward_layers(net, P2, 0, len(net.layers), x2, {})
        return ops.mse(y, t, t.size)[0], _masks(tape)

    checked = skipped = 0
    worst = 0.0
    targets = []
    for li, (w, b) in enumerate(P):
        targets += [("w", li, ix) for ix in np.ndindex(w.shape)]
        if b is not None:
            targets += [("b", li, ix) for ix in np.ndindex(b.shape)]
    targets += [("x", -1, ix) for ix in np.ndindex(x.shape)]
    for kind, li, ix in targets:
        vals = []
        ok = True
        for sgn in (1, -1):
            P2 = [(w.copy(), None if b is None else b.copy()) for w, b in P]
            x2 = x.copy()
            if kind == "w":
                P2[li][0][ix] += sgn * h
            elif kind == "b":
                P2[li][1][ix] += sgn * h
            else:
                x2[ix] += sgn * h
            lv, mk = loss_at(P2, x2)
            ok &= _same_masks(mk, base_masks)
            vals.append(lv)
        if not ok:
            skipped += 1
            continue
        fd = (vals[0] - vals[1]) / (2 * h)
        if kind == "w":
            an = base["grads"][li][0][ix]
        elif kind == "b":
            an = base["grads"][li][1][ix]
        else:
            an = base["dx"][ix]
        err = abs(fd - an) / max(abs(an), 1e-3)
        worst = max(worst, err)
        checked += 1
    assert checked > 0.95 * len(targets), (checked, skipped)
    assert worst < 1e-6, worst


@pytest.mark.parametrize("make,balance,m", [
    (tiny_unet, (2, 3, 2), 4),
    (tiny_unet, (7,), 2),
    (tiny_unet3, (3, 4, 2, 2), 3),
    (tiny_cells, (1, 3), 6),
    (lambda: specs.plain_stack(4, 3, 6, 6), (2, 2), 4),
])
@pytest.mark.parametrize("mode", [CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER])
def test_microbatch_sum_and_recompute_invariants(make, balance, m, mode):
    """Sum over micro-batches of g_i^j equals the full-batch gradient (Sec. 2),
    and F'_{i,j} reproduces F_{i,j}'s activations bit for bit (Sec. 3,
    referential transparency)."""
    net = make()
    P = _params(net, seed=3)
    B = 2 * m
    x = synth.normal(51, (B, net.in_channels, net.height, net.width))
    h, w = net.out_hw()
    t = synth.normal(52, (B, net.out_channels(), h, w))
    full = network.run(net, P, x, target=t)
    pipe = pipeline.run_pipeline(net, P, x, t, balance, m, mode)
    assert pipe["recompute_identical"]
    assert abs(pipe["loss"] - full["loss"]) <= 1e-12 * abs(full["loss"])
    np.testing.assert_allclose(pipe["y"], full["y"], rtol=0, atol=0)
    for i, (dW, db) in full["grads"].items():
        assert _rel(pipe["grads"][i][0], dW) < 1e-12
        if db is not None:
            assert _rel(pipe["grads"][i][1], db) < 1e-12


def test_gradients_bit_identical_across_checkpoint_modes():
    net = tiny_unet3()
    P = _params(net, seed=4)
    x = synth.normal(61, (8, 3, 8, 8))
    t = synth.normal(62, (8, 1, 8, 8))
    res = [pipeline.run_pipeline(net, P, x, t, (4, 4, 3), 4, mode, storage="bf16")
           for mode in (CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER)]
    for r in res[1:]:
        assert r["loss"] == res[0]["loss"]
        for i in res[0]["grads"]:
            np.testing.assert_array_equal(r["grads"][i][0], res[0]["grads"][i][0])


def test_pipeline_trace_policies():
    net = specs.plain_stack(3, 2, 4, 4)
    P = _params(net)
    x = synth.normal(1, (4, 2, 4, 4))
    t = synth.normal(2, (4, 2, 4, 4))
    for mode, want_r in ((CKPT_ALWAYS, {1, 2, 3, 4}), (CKPT_EXCEPT_LAST, {1, 2, 3}),
                         (CKPT_NEVER, set())):
        tr = pipeline.run_pipeline(net, P, x, t, (1, 2), 4, mode)["trace"]
        assert {i for op, i, j in tr if op == "R"} == want_r
        # every recompute immediately precedes its own backward task
        for k, (op, i, j) in enumerate(tr):
            if op == "R":
                assert tr[k + 1] == ("B", i, j)
    # m = 1 under except-last means no checkpointing at all (Sec. 4.2 footnote)
    tr = pipeline.run_pipeline(net, P, x, t, (1, 2), 1, CKPT_EXCEPT_LAST)["trace"]
    assert not any(op == "R" for op, _, _ in tr)


def test_forward_clocks_match_algorithm1_m4_n3():
    """Clock k runs every F_{i,j} with i + j - 1 = k (Algorithm 1; m=4, n=3 as
    in Fig. 1): the hand-written fixture tests/golden/clock_cycle_m4_n3.txt."""
    g = golden_data.clock_cycle()
    assert pipeline.forward_clocks(4, 3) == g["FORWARD"]
    assert pipeline.backward_clocks(4, 3) == g["BACKWARD"]


@pytest.mark.parametrize("m", range(1, 9))
@pytest.mark.parametrize("n", range(1, 9))
def test_clock_order_satisfies_dependencies(m, n):
    """F_{i,j-1} before F_{i,j} (Sec. 2), F_{i,j} before F_{i+1,j} and
    B_{i,j} before B_{i-1,j} (Sec. 2.1), B_{i,j+1} before B_{i,j}; every task
    exactly once; tasks sharing a clock are independent."""
    fw = [t for c in pipeline.forward_clocks(m, n) for t in c]
    bw = [t for c in pipeline.backward_clocks(m, n) for t in c]
    allt = sorted((i, j) for i in range(1, m + 1) for j in range(1, n + 1))
    assert sorted(fw) == allt and sorted(bw) == allt
    pf = {t: k for k, t in enumerate(fw)}
    pb = {t: k for k, t in enumerate(bw)}
    for (i, j) in allt:
        if j > 1:
            assert pf[(i, j - 1)] < pf[(i, j)]
        if i < m:
            assert pf[(i, j)] < pf[(i + 1, j)]
            assert pb[(i + 1, j)] < pb[(i, j)]
        if j < n:
            assert pb[(i, j + 1)] < pb[(i, j)]
    for c in pipeline.forward_clocks(m, n):
        assert len({i for i, _ in c}) == len(c) and len({j for _, j in c}) == len(c)
    assert len(pipeline.forward_clocks(m, n)) == m + n - 1


def test_bf16_storage_is_exact_on_representable_values():
    """With small-integer inputs and weights every stored value is exactly
    representable in bf16, so bf16 storage must reproduce float64 exactly;
    with generic values it must round, and only to bf16 values."""
    net = tiny_unet()
    g = np.random.default_rng(7)
    P = [(g.integers(-1, 2, w.shape).astype(np.float64),
          None if b is None else g.integers(-2, 3, b.shape).astype(np.float64))
         for w, b in _params(net)]
    x = g.integers(-2, 3, (2, 2, 8, 8)).astype(np.float64)
    t = g.integers(-2, 3, (2, 1, 8, 8)).astype(np.float64)
    a = network.run(net, P, x, target=t * 0 + 1, storage="f64")
    # keep values small: compare only the forward activations and weight grads
    b = network.run(net, P, x, target=t * 0 + 1, storage="bf16")
    for u, v in zip(a["tape"].outputs, b["tape"].outputs):
        if np.max(np.abs(u)) < 256:
            np.testing.assert_array_equal(u, v)
    P2 = _params(net)
    x2 = synth.normal(3, (2, 2, 8, 8))
    c = network.run(net, P2, x2, target=t, storage="bf16")
    for o in c["tape"].outputs:
        np.testing.assert_array_equal(o, ops.round_bf16(o))
    d = network.run(net, P2, x2, target=t, storage="f64")
    assert any(not np.array_equal(u, v) for u, v in zip(c["tape"].outputs, d["tape"].outputs))


# ---------------------------------------------------------------- bf16 rounding points
# Hand-computed cases for the points where the bf16-storage mode rounds
# (reading R8: every stored activation, dZ, input gradient, summed upsample
# gradient and loss gradient is bf16).  bf16 keeps 8 significant bits, so
# integers are exact up to 256, even ones up to 512, multiples of 4 up to
# 1024, of 8 up to 2048 and of 32 from 4096 to 8192; ties go to the even
# significand.  Every weight is a centre tap only, so a 3x3 convolution is a
# per-pixel scale and every value below can be followed by hand.

def _centre(c_out, c_in, vals):
    w = np.zeros((c_out, c_in, 3, 3))
    w[:, :, 1, 1] = np.asarray(vals, dtype=np.float64).reshape(c_out, c_in)
    return w


def _rounding_net():
    # L0: conv 1->1 (x3), ReLU, stashed as skip 0       at 2x2
    # L1: 2x2 max-pool, conv 1->1 (x3), ReLU           at 1x1
    # L2: upsample + concat [up, skip 0], conv 2->1 (x3, x3), no ReLU  at 2x2
    layers = (specs.Layer(CONV3X3, 1, 1, bias=False, stash_id=0),
              specs.Layer(CONV3X3, 1, 1, bias=False, prologue=PRO_MAXPOOL2),
              specs.Layer(CONV3X3, 2, 1, bias=False, relu=False, prologue=PRO_UPCAT2, pop_id=0))
    P = [(_centre(1, 1, [3]), None), (_centre(1, 1, [3]), None), (_centre(1, 2, [3, 3]), None)]
    return specs.Net("rounding", layers, 1, 2, 2), P


X_ROUND = np.array([[1.0, 2.0], [3.0, 4.0]]).reshape(1, 1, 2, 2)
G_ROUND = np.array([[171.0, 1.0], [1.0, 1.0]]).reshape(1, 1, 2, 2)


def _pinned_stage(run_fn):
    """The whole net as a stage with upstream gradient G_ROUND.

    Forward (exact): y0 = 3x = [[3, 6], [9, 12]]; pool -> 12; y1 = 36;
    y2 = 3*36 + 3*y0 = [[117, 126], [135, 144]].
    Backward: dZ2 = G = [[171, 1], [1, 1]]; the input gradient of L2 is 3G =
    [[513, 3], [3, 3]] in both channels, stored as [[512, 3], [3, 3]]
    (513 -> 512).  Its skip half goes to L0; its upsample half sums to
    512 + 3 + 3 + 3 = 521, stored as 520.  dZ1 = 520, dW1 (centre) = 520 * 12
    = 6240; L1's input gradient 3 * 520 = 1560 goes to the pool's argmax
    (pixel (1, 1)).  At L0 the skip gradient is added: [[512, 3], [3, 1563]],
    stored as dZ0 = [[512, 3], [3, 1560]] (1563 -> 1560).  dW0 (centre) =
    512*1 + 3*2 + 3*3 + 1560*4 = 6767; dx = 3 dZ0 = [[1536, 9], [9, 4680]],
    stored as [[1536, 9], [9, 4672]] (4680 -> 4672).  dW2 (centre) =
    (36 * sum G, sum G * y0) = (6264, 540)."""
    net, P = _rounding_net()
    r = run_fn(net, P, X_ROUND, out_grads=[G_ROUND], storage="bf16")
    return (r["grads"][0][0][0, 0, 1, 1], r["grads"][1][0][0, 0, 1, 1],
            tuple(r["grads"][2][0][0, :, 1, 1]), tuple(r["dx"].ravel()))


PINNED_STAGE = (6767.0, 6240.0, (6264.0, 540.0), (1536.0, 9.0, 9.0, 4672.0))


def _pinned_upcat_stage(run_fn):
    """L2 alone as a stage (input y1 = 36 at 1x1, skip 0 popped from outside
    with y0): its input gradient is the stored upsample sum, 520 (521 before
    rounding)."""
    net, P = _rounding_net()
    stash = {0: np.array([[3.0, 6.0], [9.0, 12.0]]).reshape(1, 1, 2, 2)}
    r = run_fn(net, P, np.full((1, 1, 1, 1), 36.0), lo=2, hi=3, out_grads=[G_ROUND],
               storage="bf16", stash_in=stash)
    return float(r["dx"].ravel()[0])


def _pinned_loss(run_fn):
    """One 1x1 convolution 1->1 (weight 1, bias 128, no ReLU) on x = 1:
    y = 129; target 0.5; numel 1, so dL/dy = 2 (129 - 0.5) = 257, stored (as
    the layer's dZ) as 256, a tie, to the even significand; dW = db =
    256 * 1."""
    net = specs.Net("loss", (specs.Layer(CONV1X1, 1, 1, relu=False),), 1, 1, 1)
    P = [(np.ones((1, 1, 1, 1)), np.array([128.0]))]
    r = run_fn(net, P, np.ones((1, 1, 1, 1)), target=np.full((1, 1, 1, 1), 0.5), storage="bf16")
    return float(r["grads"][0][0].ravel()[0]), float(r["grads"][0][1][0])


def test_bf16_rounding_points_hand_values():
    assert _pinned_stage(network.run) == PINNED_STAGE
    assert _pinned_upcat_stage(network.run) == 520.0
    assert _pinned_loss(network.run) == (256.0, 256.0)


def _mutants():
    """Copies of the oracle's backward_layers in which one call of the bf16
    store no longer rounds, one copy per call site, with run() calling it."""
    import inspect
    import textwrap
    src = {f: textwrap.dedent(inspect.getsource(getattr(network, f)))
           for f in ("run", "backward_layers")}
    for fname in ("backward_layers",):
        text = src[fname]
        n = text.count("_store(")
        for k in range(n):
            parts = text.split("_store(")
            mutated = "_store(".join(parts[:k + 1]) + "_keep(" + "_store(".join(parts[k + 1:])
            ns = dict(network.__dict__)
            ns["_keep"] = lambda a, storage: a
            for other, t in src.items():
                exec(compile(mutated if other == fname else t, "<mutant>", "exec"), ns)
            yield f"{fname} store #{k + 1}", ns["run"]


def test_each_bf16_store_is_pinned():
    """Removing the rounding at any single store of the backward changes a
    hand-pinned value above."""
    seen = 0
    for name, run_fn in _mutants():
        seen += 1
        same = (_pinned_stage(run_fn) == PINNED_STAGE and
                _pinned_upcat_stage(run_fn) == 520.0 and
                _pinned_loss(run_fn) == (256.0, 256.0))
        assert not same, name
    assert seen == 3   # dZ, input gradient, upsample sum
