"""GPU parity for whole networks and multi-layer stages: the HIP path through
the C ABI against the oracle on the same seeded inputs, element by element.

Forward outputs and the loss are held to the parity tolerance (2e-2
max-rel bf16, 1e-4 fp32).  Gradients of bf16 runs through several ReLU and
max-pool layers are held to that tolerance or, where larger, to 4x the
spread between the reference and the same oracle with float32 contraction;
or to rms-rel 2e-2 with max-rel 5e-2 (see gpu_util.check_grad): two valid
bf16 computations of such a network take some ReLU-mask and pool-argmax
decisions differently (their bf16 activations differ in the last bit), and
no implementation with another summation order can avoid it.
Checkpointed and non-checkpointed runs must agree bit for bit."""
import numpy as np
import pytest
import torch

from gpu_util import (TOL, check_grad, gpu_network, gpu_stage, gpu_stage_with_popped, maxrel,
                      oracle_network, oracle_network_variants, oracle_stage_variants, report, say)
import oracle
from oracle import ops
from paper_2004_09910_amd.harness import nhwc_to_nchw64
from workloads import specs
from workloads.specs import BF16, CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER, FP32

pytestmark = pytest.mark.gpu

MODES = [CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER]


def check_network(got, pair, dtype, what):
    ref, alts = pair
    errs = {}
    ok = check_grad("loss", np.array([got["loss"]]), np.array([ref["loss"]]),
                    [np.array([a["loss"]]) for a in alts], dtype, errs, strict=True)
    ok &= check_grad("y", got["y"], ref["y"], [a["y"] for a in alts], dtype, errs, strict=True)
    for idx, (dW, db) in ref["grads"].items():
        ok &= check_grad(f"dW{idx}", got["grads"][idx][0], dW, [a["grads"][idx][0] for a in alts], dtype, errs)
        if db is not None:
            ok &= check_grad(f"db{idx}", got["grads"][idx][1], db, [a["grads"][idx][1] for a in alts], dtype, errs)
    report(what, errs)
    assert ok, errs


def check_stage(got, pair, dtype, what, dx=True):
    ref, alts = pair
    errs = {}
    ok = check_grad("y", nhwc_to_nchw64(got["y"]), ref["y"], [a["y"] for a in alts], dtype, errs, strict=True)
    for sid, t in got["stash"].items():
        ok &= check_grad(f"skip{sid}", nhwc_to_nchw64(t), ref["stash"][sid], [a["stash"][sid] for a in alts],
                         dtype, errs, strict=True)
    if dx:
        ok &= check_grad("dx", nhwc_to_nchw64(got["dx"]), ref["dx"], [a["dx"] for a in alts], dtype, errs)
    for idx, (dW, db) in ref["grads"].items():
        ok &= check_grad(f"dW{idx}", got["grads"][idx][0], dW, [a["grads"][idx][0] for a in alts], dtype, errs)
        if db is not None:
            ok &= check_grad(f"db{idx}", got["grads"][idx][1], db, [a["grads"][idx][1] for a in alts], dtype, errs)
    report(what, errs)
    assert ok, errs


def same_bits(a, b):
    for idx in a["grads"]:
        np.testing.assert_array_equal(a["grads"][idx][0], b["grads"][idx][0])
        if a["grads"][idx][1] is not None:
            np.testing.assert_array_equal(a["grads"][idx][1], b["grads"][idx][1])


@pytest.mark.parametrize("mode", MODES)
def test_lanes_are_bit_identical(mode):
    """Micro-batches on 2 and 3 concurrent lane streams (each lane with its
    own transient buffers, accumulations chained in the order m..1) give the
    same bits as one stream: outputs, input gradients, exported-skip values
    and every weight and bias gradient."""
    net = specs.unet(5, 64, 64, 48, "unet5-c64-48")
    bal = (7, 5, 3, 4)
    runs = []
    for k in (1, 2, 3):
        say(f"lanes={k} mode={mode}")
        runs.append(gpu_stage(net, BF16, 8, 4, mode, bal, 1, neutral=False, lanes=k))
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert torch.equal(r["y"], runs[0]["y"])
        assert torch.equal(r["dx"], runs[0]["dx"])
        for sid in runs[0]["stash"]:
            assert torch.equal(r["stash"][sid], runs[0]["stash"][sid])


@pytest.mark.parametrize("mode", MODES)
def test_micro_batch_pairs_are_bit_identical(mode):
    """Two micro-batches per launch (tgp_stage_forward2 /
    tgp_stage_backward_recompute2 on two lanes) give the same bits as one
    micro-batch per launch on one stream, on a stage that holds both
    nine-tap kernel widths, pooling, an exported skip and a ragged mix of
    layer shapes."""
    net = specs.unet(5, 64, 64, 48, "unet5-c64-48")
    bal = (7, 5, 3, 4)
    runs = []
    for k, pairs in ((1, False), (2, True)):
        say(f"pairs={pairs} mode={mode}")
        runs.append(gpu_stage(net, BF16, 8, 4, mode, bal, 1, neutral=False, lanes=k, pairs=pairs))
    same_bits(runs[0], runs[1])
    assert torch.equal(runs[1]["y"], runs[0]["y"])
    assert torch.equal(runs[1]["dx"], runs[0]["dx"])
    for sid in runs[0]["stash"]:
        assert torch.equal(runs[1]["stash"][sid], runs[0]["stash"][sid])


def test_pair_then_single_calls_in_one_step():
    """Forwards in pairs, then a paired backward (4, 3) followed by single
    backwards of 2 and 1 on one stream: the single backward on the second
    lane must see that lane's transformed weights refreshed (the pair read
    only the first lane's).  Bits equal one micro-batch per launch."""
    import paper_2004_09910_amd as tgp
    from paper_2004_09910_amd.harness import Session

    class Mixed(Session):
        def stage_step(self, j, x, y, dy, dx, stream=0, serial=False):
            def sl(t, i):
                return t.data_ptr() + (i - 1) * (t.numel() // self.m) * t.element_size()
            for i in (1, 3):
                tgp.stage_forward2(self.h, j, i, i + 1, self.checkpointed(i),
                                   self.checkpointed(i + 1), sl(x, i), sl(x, i + 1), sl(y, i),
                                   sl(y, i + 1), stream)
            tgp.stage_backward_recompute2(self.h, j, 4, 3, sl(dy, 4), sl(dy, 3), sl(dx, 4),
                                          sl(dx, 3), stream)
            tgp.grad_accumulate(self.h, j, 4, True, stream)
            tgp.grad_accumulate(self.h, j, 3, False, stream)
            for i in (2, 1):
                tgp.stage_backward_recompute(self.h, j, i, sl(dy, i), sl(dx, i), stream)
                tgp.grad_accumulate(self.h, j, i, False, stream)

    net = specs.unet(5, 64, 64, 48, "unet5-c64-48")
    bal = (7, 5, 3, 4)
    say("mixed: reference, one per launch")
    ref = gpu_stage(net, BF16, 8, 4, CKPT_ALWAYS, bal, 1, neutral=False)
    say("mixed: pair then singles")
    sess = Mixed(net, BF16, n=len(bal), balance=bal, bind_layers=range(0, 7))
    sess.plan(8, 4, CKPT_ALWAYS, 2)
    got = gpu_stage(net, BF16, 8, 4, CKPT_ALWAYS, bal, 1, neutral=False, sess=sess)
    same_bits(ref, got)
    assert torch.equal(got["y"], ref["y"])
    assert torch.equal(got["dx"], ref["dx"])


def test_micro_batch_pairs_bench_stage():
    """The pair path on the benchmark's own stage (U-Net level-0 layers at
    192 x 192, micro-batch 4), m = 2, against one micro-batch per launch."""
    net = specs.unet(5, 64, 64, 192, "unet5-c64")
    bal = (7, 5, 3, 4)
    runs = []
    for k, pairs in ((1, False), (2, True)):
        say(f"bench stage pairs={pairs}")
        runs.append(gpu_stage(net, BF16, 8, 2, CKPT_EXCEPT_LAST, bal, 1, neutral=False, lanes=k,
                              pairs=pairs))
    same_bits(runs[0], runs[1])
    assert torch.equal(runs[1]["y"], runs[0]["y"])
    assert torch.equal(runs[1]["dx"], runs[0]["dx"])


def test_tiny_fp32_pipeline_all_modes():
    """4-layer conv3x3+bias+ReLU stack, C=16, 8x16x32x32 fp32, m=4, n=2."""
    wl = specs.tiny()
    pair = oracle_network_variants(wl.net, FP32, wl.batch)
    runs = []
    for mode in MODES:
        say(f"tiny fp32 mode={mode}")
        got = gpu_network(wl.net, FP32, wl.batch, wl.m, wl.n, mode)
        check_network(got, pair, FP32, f"tiny mode {mode}")
        runs.append(got)
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert r["loss"] == runs[0]["loss"]
    again = gpu_network(wl.net, FP32, wl.batch, wl.m, wl.n, CKPT_ALWAYS)
    same_bits(runs[0], again)


@pytest.mark.parametrize("m,n", [(2, 3), (4, 2), (1, 1), (4, 4)])
def test_small_unet_bf16_pipeline(m, n):
    """3-level U-Net (64 -> 256 channels) with pools, upsample-concat skips and a
    1-channel head, 24x24 so that every level has a ragged pixel tile."""
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    B = 4
    pair = oracle_network_variants(net, BF16, B)
    runs = []
    for mode in MODES:
        say(f"unet3 bf16 m={m} n={n} mode={mode}")
        got = gpu_network(net, BF16, B, m, n, mode)
        check_network(got, pair, BF16, f"unet3 m={m} n={n} mode={mode}")
        runs.append(got)
    for r in runs[1:]:
        same_bits(runs[0], r)


@pytest.mark.parametrize("mode", MODES)
def test_pipeline_lanes_are_bit_identical(mode):
    """tgp_pipeline_step with 2 and 3 lanes, forked onto the library's own
    streams, against one lane: loss, output and every weight and bias
    gradient, bit for bit (3-level U-Net, 3 partitions, m = 4)."""
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    runs = []
    for k in (1, 2, 3):
        say(f"pipeline lanes={k} mode={mode}")
        runs.append(gpu_network(net, BF16, 8, 4, 3, mode, lanes=k))
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert r["loss"] == runs[0]["loss"]
        assert torch.equal(r["y_t"], runs[0]["y_t"])


def test_pipeline_step_graph_capture():
    """A two-lane pipeline step captured into a HIP graph from one stream
    (the fork onto the lane streams and the join are events) and replayed
    three times, with eager work and synchronisation between replays: every
    replay matches the eager step bit for bit."""
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    say("pipeline graph capture, 2 lanes")
    eager = gpu_network(net, BF16, 8, 4, 3, CKPT_ALWAYS, lanes=2)
    sess, x, t, loss, y = eager["sess"], eager["x"], eager["t"], eager["loss_t"], eager["y_t"]
    ref_y = y.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        sess.pipeline_step(x, t, loss, y, stream=torch.cuda.current_stream().cuda_stream)
    for rep in range(3):
        loss.zero_()
        y.zero_()
        for p in sess.params.values():
            p["dw"].fill_(7.0)
        graph.replay()
        torch.cuda.synchronize()
        assert float(loss.item()) == eager["loss"], rep
        assert torch.equal(y, ref_y), rep
        same_bits(eager, {"grads": sess.grads64()})
        torch.randn(4096, device="cuda").sum().item()   # eager work between replays


@pytest.mark.parametrize("bal", [(4, 3, 4), (2, 4, 5), (4, 7)])
def test_partition_ending_at_a_stashed_layer(bal):
    """Partitions whose last layer is also stashed (enc1b with skip 1, enc0b
    with skip 0): the layer's output is the partition output and must reach
    its stash slot too, where a later partition's upsample-concat pops it."""
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    B = 4
    pair = oracle_network_variants(net, BF16, B)
    runs = []
    for mode in MODES:
        say(f"unet3 balance {bal} mode={mode}")
        got = gpu_network(net, BF16, B, 2, len(bal), mode, balance=list(bal))
        check_network(got, pair, BF16, f"unet3 balance {bal} mode={mode}")
        runs.append(got)
    for r in runs[1:]:
        same_bits(runs[0], r)


def test_microbatch_count_changes_values_only_within_tolerance():
    """Per-sample activations do not depend on m (no intra-batch computation,
    Sec. 2), but a kernel's configuration may depend on the micro-batch size
    b = B / m (for example the 24 x 24 path and the weight gradient's K
    ranges), so across m outputs and gradients agree to the bf16 tolerance,
    not bit for bit (the sum over micro-batches also changes order).  At a
    fixed m the checkpoint modes stay bit-identical (other tests)."""
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    a = gpu_network(net, BF16, 8, 1, 2, CKPT_ALWAYS)
    b = gpu_network(net, BF16, 8, 8, 2, CKPT_ALWAYS)
    assert maxrel(b["y"], a["y"]) < TOL[BF16]
    for idx in a["grads"]:
        assert maxrel(b["grads"][idx][0], a["grads"][idx][0]) < TOL[BF16]
        if a["grads"][idx][1] is not None:
            assert maxrel(b["grads"][idx][1], a["grads"][idx][1]) < TOL[BF16]


def test_unet_stage_reduced_size():
    """Partition 1 of 4 of the 5-level U-Net (real channel and layer
    structure, 64 -> 512 channels), B=4, 48x48, m=2, with injected upstream
    gradients for the output and the three exported skips."""
    net = specs.unet(5, 64, 64, 48, "unet5-c64-48")
    bal = (7, 5, 3, 4)
    runs = []
    for mode in MODES:
        say(f"unet5 stage1 48x48 mode={mode}")
        runs.append(gpu_stage(net, BF16, 4, 2, mode, bal, 1))
    pair = oracle_stage_variants(net, BF16, 0, 7, runs[0]["xv"], runs[0]["G"])
    for mode, got in zip(MODES, runs):
        check_stage(got, pair, BF16, f"unet5 stage mode {mode}")
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert torch.equal(r["dx"], runs[0]["dx"])


@pytest.mark.parametrize("j", [2, 3, 4])
def test_unet_inner_stages(j):
    """Partitions 2..4 as stages: deeper levels, upsample-concat prologues that
    pop skips stashed inside or outside the partition, and the head."""
    net = specs.unet(5, 64, 64, 32, "unet5-c64-32")
    bal = (7, 5, 3, 4)
    say(f"unet5 stage {j}")
    got = gpu_stage_with_popped(net, bal, j)
    pair = oracle_stage_variants(net, BF16, got["lo"], got["hi"], got["xv"], got["G"],
                             stash_in=got["stash_in"])
    check_stage(got, pair, BF16, f"unet5 stage {j}")


def test_amoeba_cells_stage_except_last():
    """Cells of depthwise 3x3 -> pointwise 1x1 + bias -> ReLU at C=256,
    14x14 (392 pixels per micro-batch: a ragged 1x1 tile), m=2 and m=4."""
    net = specs.amoeba_cells(4, 256, 14, "cells4-c256")
    for m in (2, 4):
        runs = []
        for mode in MODES:
            say(f"cells m={m} mode={mode}")
            runs.append(gpu_stage(net, BF16, 4, m, mode, (8,), 1))
        pair = oracle_stage_variants(net, BF16, 0, 8, runs[0]["xv"], runs[0]["G"])
        for mode, got in zip(MODES, runs):
            check_stage(got, pair, BF16, f"cells m={m} mode={mode}")
        for r in runs[1:]:
            same_bits(runs[0], r)


def test_amoeba_cells_pairs_are_bit_identical():
    """Two micro-batches per launch on the depthwise / pointwise cells (the
    depthwise kernels run once per micro-batch inside the pair) against one
    per launch, except-last."""
    net = specs.amoeba_cells(4, 256, 14, "cells4-c256")
    runs = []
    for k, pairs in ((1, False), (2, True)):
        say(f"cells pairs={pairs}")
        runs.append(gpu_stage(net, BF16, 8, 4, CKPT_EXCEPT_LAST, (8,), 1, neutral=False, lanes=k,
                              pairs=pairs))
    same_bits(runs[0], runs[1])
    assert torch.equal(runs[1]["y"], runs[0]["y"])
    assert torch.equal(runs[1]["dx"], runs[0]["dx"])


def test_six_level_unet_network():
    """The 6-level, 128-channel U-Net (128 -> 4096 channels, 503 M
    parameters) in 8 partitions, B = 2, m = 2, at 32 x 32, so that its
    deepest level is a 1 x 1 image (a 3 x 3 convolution there sees only its
    centre tap).  One float32-contraction variant bounds the decision spread
    (each oracle run of this network takes tens of seconds)."""
    net = specs.unet(6, 128, 128, 32, "unet6-c128-32")
    say("unet6 oracle")
    P = oracle.net_params(net, BF16)
    ref = oracle_network(net, BF16, 2, P)
    with ops.contraction("f32"):
        alt = oracle_network(net, BF16, 2, P)
    runs = []
    for mode in (CKPT_ALWAYS, CKPT_NEVER):
        say(f"unet6 gpu mode={mode}")
        got = gpu_network(net, BF16, 2, 2, 8, mode)
        check_network(got, (ref, [alt]), BF16, f"unet6 mode {mode}")
        got.pop("sess").close()
        runs.append(got)
    same_bits(runs[0], runs[1])


def test_micro_batch_of_one_sample():
    """b = 1 (B = m): the smallest micro-batch."""
    net = specs.unet(2, 64, 64, 16, "unet2-c64")
    pair = oracle_network_variants(net, BF16, 4)
    got = gpu_network(net, BF16, 4, 4, 2, CKPT_ALWAYS)
    check_network(got, pair, BF16, "unet2 b=1")
