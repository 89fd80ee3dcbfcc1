"""GPU parity for whole networks and multi-layer stages: the HIP path through
the C ABI against the oracle on the same seeded inputs, element by element.

Every comparison is strict.  Gradients of multi-layer bf16 runs are compared
on the EXACT input family, whose float32 sums are exact (tests/exactness.py),
to 1e-6 max-rel: each layer's ReLU and max-pool decisions, and every bf16
store, must then be the oracle's bit for bit.  N(0,1) runs are held to the
spec tolerance (2e-2 max-rel bf16, 1e-4 fp32) on their forward outputs
and loss, and on everything in fp32 runs.  Checkpointed and non-checkpointed
runs must agree bit for bit."""
import numpy as np
import pytest
import torch

from gpu_util import (TOL, check_network, check_stage, gpu_network, gpu_stage,
                      gpu_stage_with_popped, maxrel, network_inputs, oracle_network,
                      oracle_stage, say)
from workloads import specs
from workloads.specs import BF16, CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER, FP32
from workloads.synth import EXACT

pytestmark = pytest.mark.gpu

MODES = [CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER]


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
        runs.append(gpu_stage(net, BF16, 8, 4, mode, bal, 1, lanes=k))
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert torch.equal(r["y"], runs[0]["y"])
        assert torch.equal(r["dx"], runs[0]["dx"])
        for sid in runs[0]["stash"]:
            assert torch.equal(r["stash"][sid], runs[0]["stash"][sid])


@pytest.mark.parametrize("mode", MODES)
def test_micro_batch_groups_are_bit_identical(mode):
    """Two and four micro-batches per launch (tgp_stage_forward_n /
    tgp_stage_backward_recompute_n on as many lanes) give the same bits as
    one micro-batch per launch on one stream, on a stage that holds both
    nine-tap kernel widths, pooling, an exported skip and a ragged mix of
    layer shapes."""
    net = specs.unet(5, 64, 64, 48, "unet5-c64-48")
    bal = (7, 5, 3, 4)
    runs = []
    for k in (1, 2, 4):
        say(f"group={k} mode={mode}")
        runs.append(gpu_stage(net, BF16, 8, 4, mode, bal, 1, lanes=k, group=k))
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert torch.equal(r["y"], runs[0]["y"])
        assert torch.equal(r["dx"], runs[0]["dx"])
        for sid in runs[0]["stash"]:
            assert torch.equal(r["stash"][sid], runs[0]["stash"][sid])


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
    ref = gpu_stage(net, BF16, 8, 4, CKPT_ALWAYS, bal, 1)
    say("mixed: pair then singles")
    sess = Mixed(net, BF16, n=len(bal), balance=bal, bind_layers=range(0, 7))
    sess.plan(8, 4, CKPT_ALWAYS, 2)
    got = gpu_stage(net, BF16, 8, 4, CKPT_ALWAYS, bal, 1, sess=sess)
    same_bits(ref, got)
    assert torch.equal(got["y"], ref["y"])
    assert torch.equal(got["dx"], ref["dx"])


def test_group_then_pair_then_single_calls_in_one_step():
    """Forwards as one group of four, then a backward group of two (4, 3)
    and single backwards of 2 and 1, on four lanes and one stream: each
    later call on a lane whose transformed weights the group did not refresh
    must refresh them first.  Bits equal one micro-batch per launch."""
    import paper_2004_09910_amd as tgp
    from paper_2004_09910_amd.harness import Session

    class Mixed(Session):
        def stage_step(self, j, x, y, dy, dx, stream=0, serial=False):
            def sl(t, i):
                return t.data_ptr() + (i - 1) * (t.numel() // self.m) * t.element_size()
            tgp.stage_forward_n(self.h, j, 1, [self.checkpointed(i) for i in range(1, 5)],
                                [sl(x, i) for i in range(1, 5)], [sl(y, i) for i in range(1, 5)],
                                stream)
            tgp.stage_backward_recompute_n(self.h, j, 4, [sl(dy, 4), sl(dy, 3)],
                                           [sl(dx, 4), sl(dx, 3)], stream)
            tgp.grad_accumulate(self.h, j, 4, True, stream)
            tgp.grad_accumulate(self.h, j, 3, False, stream)
            for i in (2, 1):
                tgp.stage_backward_recompute(self.h, j, i, sl(dy, i), sl(dx, i), stream)
                tgp.grad_accumulate(self.h, j, i, False, stream)

    net = specs.unet(5, 64, 64, 48, "unet5-c64-48")
    bal = (7, 5, 3, 4)
    say("mixed group: reference, one per launch")
    ref = gpu_stage(net, BF16, 8, 4, CKPT_ALWAYS, bal, 1)
    say("mixed group: group of four, pair, singles")
    sess = Mixed(net, BF16, n=len(bal), balance=bal, bind_layers=range(0, 7))
    sess.plan(8, 4, CKPT_ALWAYS, 4)
    got = gpu_stage(net, BF16, 8, 4, CKPT_ALWAYS, bal, 1, sess=sess)
    same_bits(ref, got)
    assert torch.equal(got["y"], ref["y"])
    assert torch.equal(got["dx"], ref["dx"])


def test_groups_of_three_in_one_step():
    """A forward group of three (1, 2, 3) and a single forward of 4, then a
    backward group of three (4, 3, 2) and a single backward of 1: every
    group kernel runs with an unused fourth pointer set, the per-tap and
    depthwise paths as a pair and a single.  Bits equal one micro-batch per
    launch, on the reduced U-Net stage and on the cells."""
    import paper_2004_09910_amd as tgp
    from paper_2004_09910_amd.harness import Session

    class Threes(Session):
        def stage_step(self, j, x, y, dy, dx, stream=0, serial=False):
            def sl(t, i):
                return t.data_ptr() + (i - 1) * (t.numel() // self.m) * t.element_size()
            tgp.stage_forward_n(self.h, j, 1, [self.checkpointed(i) for i in (1, 2, 3)],
                                [sl(x, i) for i in (1, 2, 3)], [sl(y, i) for i in (1, 2, 3)],
                                stream)
            tgp.stage_forward(self.h, j, 4, self.checkpointed(4), sl(x, 4), sl(y, 4), stream)
            tgp.stage_backward_recompute_n(self.h, j, 4, [sl(dy, i) for i in (4, 3, 2)],
                                           [None if dx is None else sl(dx, i) for i in (4, 3, 2)],
                                           stream)
            for i in (4, 3, 2):
                tgp.grad_accumulate(self.h, j, i, i == 4, stream)
            tgp.stage_backward_recompute(self.h, j, 1, sl(dy, 1), None if dx is None else sl(dx, 1),
                                         stream)
            tgp.grad_accumulate(self.h, j, 1, False, stream)

    cases = [(specs.unet(5, 64, 64, 48, "unet5-c64-48"), (7, 5, 3, 4), CKPT_EXCEPT_LAST, 7),
             (specs.amoeba_cells(4, 256, 14, "cells4-c256"), (8,), CKPT_EXCEPT_LAST, 8)]
    for net, bal, mode, nl in cases:
        say(f"threes {net.name}: reference")
        ref = gpu_stage(net, BF16, 8, 4, mode, bal, 1)
        say(f"threes {net.name}: groups of three")
        sess = Threes(net, BF16, n=len(bal), balance=bal, bind_layers=range(0, nl))
        sess.plan(8, 4, mode, 4)
        got = gpu_stage(net, BF16, 8, 4, mode, bal, 1, sess=sess)
        same_bits(ref, got)
        assert torch.equal(got["y"], ref["y"])
        assert torch.equal(got["dx"], ref["dx"])


def test_micro_batch_groups_bench_stage():
    """The group path on the benchmark's own stage (U-Net level-0 layers at
    192 x 192, micro-batch 4), m = 4, in groups of two and four against one
    micro-batch per launch."""
    net = specs.unet(5, 64, 64, 192, "unet5-c64")
    bal = (7, 5, 3, 4)
    runs = []
    for k in (1, 2, 4):
        say(f"bench stage group={k}")
        runs.append(gpu_stage(net, BF16, 16, 4, CKPT_EXCEPT_LAST, bal, 1, lanes=k, group=k))
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert torch.equal(r["y"], runs[0]["y"])
        assert torch.equal(r["dx"], runs[0]["dx"])


def test_groups_of_eight_and_sixteen_are_bit_identical():
    """Eight micro-batches per call and launch (m = 8, eight lanes) against
    one per launch: the ragged stage (both nine-tap widths, pooling, an
    exported skip), the benchmark stage's 192 x 192 layers and the
    depthwise / pointwise cells; and sixteen (m = 16, sixteen lanes, the
    largest group) on the cells and on the ragged stage, whose nine-tap and
    row-blocked weight-gradient kernels take eight per launch; except-last."""
    cases = [
        ("unet5-c64-48", specs.unet(5, 64, 64, 48, "unet5-c64-48"), 8, 8, (7, 5, 3, 4), 8),
        ("unet5-c64", specs.unet(5, 64, 64, 192, "unet5-c64"), 16, 8, (7, 5, 3, 4), 8),
        ("cells4-c256", specs.amoeba_cells(4, 256, 14, "cells4-c256"), 8, 8, (8,), 8),
        ("cells4-c256", specs.amoeba_cells(4, 256, 14, "cells4-c256"), 16, 16, (8,), 16),
        ("unet5-c64-48", specs.unet(5, 64, 64, 48, "unet5-c64-48"), 16, 16, (7, 5, 3, 4), 16),
    ]
    for name, net, B, m, bal, g in cases:
        runs = []
        for k in (1, g):
            say(f"large groups {name} m={m} group={k}")
            runs.append(gpu_stage(net, BF16, B, m, CKPT_EXCEPT_LAST, bal, 1, lanes=k, group=k))
        same_bits(runs[0], runs[1])
        assert torch.equal(runs[1]["y"], runs[0]["y"])
        assert torch.equal(runs[1]["dx"], runs[0]["dx"])


def test_tiny_fp32_pipeline_all_modes():
    """4-layer conv3x3+bias+ReLU stack, C=16, 8x16x32x32 fp32, m=4, n=2."""
    wl = specs.tiny()
    ref = oracle_network(wl.net, FP32, wl.batch)
    runs = []
    for mode in MODES:
        say(f"tiny fp32 mode={mode}")
        got = gpu_network(wl.net, FP32, wl.batch, wl.m, wl.n, mode)
        check_network(got, ref, FP32, f"tiny mode {mode}")
        runs.append(got)
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert r["loss"] == runs[0]["loss"]
    again = gpu_network(wl.net, FP32, wl.batch, wl.m, wl.n, CKPT_ALWAYS)
    same_bits(runs[0], again)


@pytest.mark.parametrize("m,n", [(2, 3), (4, 2), (1, 1), (4, 4)])
def test_small_unet_pipeline_exact(m, n):
    """3-level U-Net (64 -> 256 channels) with pools, upsample-concat skips and a
    1-channel head, 32x32, on exact inputs: loss, output and every gradient
    equal the oracle's, in every checkpoint mode."""
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    B = 4
    inputs = network_inputs(net, BF16, B, EXACT)
    ref = oracle_network(net, BF16, B, EXACT, inputs, certify=True)
    runs = []
    for mode in MODES:
        say(f"unet3 exact m={m} n={n} mode={mode}")
        got = gpu_network(net, BF16, B, m, n, mode, family=EXACT, inputs=inputs)
        check_network(got, ref, BF16, f"unet3 exact m={m} n={n} mode={mode}", EXACT)
        runs.append(got)
    for r in runs[1:]:
        same_bits(runs[0], r)


def test_small_unet_pipeline_outputs():
    """The 3-level U-Net at 24x24 (a ragged pixel tile at every level) on
    N(0,1) inputs: loss and network output within the bf16 tolerance."""
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    B = 4
    ref = oracle_network(net, BF16, B)
    for mode in MODES:
        say(f"unet3 normal outputs mode={mode}")
        got = gpu_network(net, BF16, B, 2, 3, mode)
        check_network(got, ref, BF16, f"unet3 outputs mode={mode}", grads=False)


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
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    B = 4
    inputs = network_inputs(net, BF16, B, EXACT)
    ref = oracle_network(net, BF16, B, EXACT, inputs, certify=True)
    runs = []
    for mode in MODES:
        say(f"unet3 balance {bal} mode={mode}")
        got = gpu_network(net, BF16, B, 2, len(bal), mode, balance=list(bal), family=EXACT,
                          inputs=inputs)
        check_network(got, ref, BF16, f"unet3 balance {bal} mode={mode}", EXACT)
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
    # on exact inputs every sum is exact, so the order cannot matter
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    inputs = network_inputs(net, BF16, 8, EXACT)
    a = gpu_network(net, BF16, 8, 1, 2, CKPT_ALWAYS, family=EXACT, inputs=inputs)
    b = gpu_network(net, BF16, 8, 8, 2, CKPT_ALWAYS, family=EXACT, inputs=inputs)
    assert np.array_equal(b["y"], a["y"]) and a["loss"] == b["loss"]
    same_bits(a, b)


def test_unet_stage_reduced_size():
    """Partition 1 of 4 of the 5-level U-Net (real channel and layer
    structure, 64 -> 512 channels), B=4, 48x48, m=2, with injected upstream
    gradients for the output and the three exported skips."""
    net = specs.unet(5, 64, 64, 48, "unet5-c64-48")
    bal = (7, 5, 3, 4)
    runs = []
    for mode in MODES:
        say(f"unet5 stage1 48x48 exact mode={mode}")
        runs.append(gpu_stage(net, BF16, 4, 2, mode, bal, 1, family=EXACT))
    ref = oracle_stage(net, BF16, 0, 7, runs[0]["xv"], runs[0]["G"], family=EXACT, certify=True)
    for mode, got in zip(MODES, runs):
        check_stage(got, ref, BF16, f"unet5 stage exact mode {mode}", EXACT)
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert torch.equal(r["dx"], runs[0]["dx"])
    say("unet5 stage1 48x48 normal outputs")
    got = gpu_stage(net, BF16, 4, 2, CKPT_ALWAYS, bal, 1)
    ref = oracle_stage(net, BF16, 0, 7, got["xv"], got["G"])
    check_stage(got, ref, BF16, "unet5 stage outputs", dx=False, grads=False)


@pytest.mark.parametrize("j", [2, 3, 4])
def test_unet_inner_stages(j):
    """Partitions 2..4 as stages: deeper levels, upsample-concat prologues that
    pop skips stashed inside or outside the partition, and the head."""
    net = specs.unet(5, 64, 64, 32, "unet5-c64-32")
    bal = (7, 5, 3, 4)
    say(f"unet5 stage {j} exact")
    got = gpu_stage_with_popped(net, bal, j, family=EXACT)
    ref = oracle_stage(net, BF16, got["lo"], got["hi"], got["xv"], got["G"],
                       stash_in=got["stash_in"], family=EXACT, certify=True)
    check_stage(got, ref, BF16, f"unet5 stage {j} exact", EXACT)


def test_amoeba_cells_stage_except_last():
    """Cells of depthwise 3x3 -> pointwise 1x1 + bias -> ReLU at C=256,
    14x14 (392 pixels per micro-batch: a ragged 1x1 tile), m=2 and m=4."""
    net = specs.amoeba_cells(4, 256, 14, "cells4-c256")
    for m in (2, 4):
        runs = []
        for mode in MODES:
            say(f"cells exact m={m} mode={mode}")
            runs.append(gpu_stage(net, BF16, 4, m, mode, (8,), 1, family=EXACT))
        ref = oracle_stage(net, BF16, 0, 8, runs[0]["xv"], runs[0]["G"], family=EXACT,
                           certify=True)
        for mode, got in zip(MODES, runs):
            check_stage(got, ref, BF16, f"cells exact m={m} mode={mode}", EXACT)
        for r in runs[1:]:
            same_bits(runs[0], r)
    say("cells normal outputs")
    got = gpu_stage(net, BF16, 4, 2, CKPT_EXCEPT_LAST, (8,), 1)
    ref = oracle_stage(net, BF16, 0, 8, got["xv"], got["G"])
    check_stage(got, ref, BF16, "cells outputs", dx=False, grads=False)


def test_amoeba_cells_groups_are_bit_identical():
    """Two and four micro-batches per call on the depthwise / pointwise cells
    (the depthwise and 1x1 kernels take two micro-batches per launch, so a
    group of four runs as two launches each) against one per launch,
    except-last."""
    net = specs.amoeba_cells(4, 256, 14, "cells4-c256")
    runs = []
    for k in (1, 2, 4):
        say(f"cells group={k}")
        runs.append(gpu_stage(net, BF16, 8, 4, CKPT_EXCEPT_LAST, (8,), 1, lanes=k, group=k))
    for r in runs[1:]:
        same_bits(runs[0], r)
        assert torch.equal(r["y"], runs[0]["y"])
        assert torch.equal(r["dx"], runs[0]["dx"])


@pytest.mark.timeout(600)
def test_five_level_unet_network():
    """The whole benchmark network (5-level, 64-channel U-Net) at 64 x 64 in
    the 4 partitions of its FLOP balance, trained for one step by
    tgp_pipeline_step on exact inputs, B = 8: m = 2 and 4 under every
    checkpoint mode, once on two lanes.  Loss, output and every weight and
    bias gradient equal the oracle's full-batch run, so g = sum_i g_i holds
    through all partitions and the runs agree bit for bit."""
    net = specs.unet(5, 64, 64, 64, "unet5-c64-64")
    B = 8
    say("unet5 network oracle inputs (exact family)")
    inputs = network_inputs(net, BF16, B, EXACT, log=say)
    say("unet5 network oracle run")
    ref = oracle_network(net, BF16, B, EXACT, inputs, certify=True, log=say)
    runs = []
    for m, mode, lanes in ((2, CKPT_ALWAYS, 1), (4, CKPT_ALWAYS, 2), (4, CKPT_EXCEPT_LAST, 1),
                           (4, CKPT_NEVER, 1)):
        what = f"unet5 network m={m} mode={mode} lanes={lanes}"
        say(what)
        got = gpu_network(net, BF16, B, m, 4, mode, lanes=lanes, family=EXACT, inputs=inputs)
        assert tuple(got["sess"].balance) == (7, 5, 3, 4)
        check_network(got, ref, BF16, what, EXACT)
        got.pop("sess").close()
        runs.append(got)
    for r in runs[1:]:
        same_bits(runs[0], r)


@pytest.mark.timeout(1200)
def test_six_level_unet_network():
    """The 6-level, 128-channel U-Net (128 -> 4096 channels, 503 M
    parameters) in 8 partitions at 64 x 64, B = 4, m = 2 (its deepest level
    is a 2 x 2 image), on exact inputs, under always and never: loss, output
    and every gradient equal the oracle's."""
    import exactness
    net = specs.unet(6, 128, 128, 64, "unet6-c128-64")
    B = 4
    say("unet6 oracle inputs (exact family)")
    inputs = network_inputs(net, BF16, B, EXACT, log=say)
    say("unet6 oracle run")
    ref = oracle_network(net, BF16, B, EXACT, inputs, log=say)
    runs = []
    for mode in (CKPT_ALWAYS, CKPT_NEVER):
        say(f"unet6 gpu mode={mode}")
        got = gpu_network(net, BF16, B, 2, 8, mode, family=EXACT, inputs=inputs)
        try:
            check_network(got, ref, BF16, f"unet6 exact mode {mode}", EXACT)
        except AssertionError:
            say("unet6 exactness certificate",
                exactness.certificate(net, inputs[4], ref, target=inputs[2]))
            raise
        got.pop("sess").close()
        runs.append(got)
    same_bits(runs[0], runs[1])


def test_micro_batch_of_one_sample():
    """b = 1 (B = m): the smallest micro-batch, exact inputs."""
    net = specs.unet(2, 64, 64, 16, "unet2-c64-16")
    inputs = network_inputs(net, BF16, 4, EXACT)
    ref = oracle_network(net, BF16, 4, EXACT, inputs, certify=True)
    got = gpu_network(net, BF16, 4, 4, 2, CKPT_ALWAYS, family=EXACT, inputs=inputs)
    check_network(got, ref, BF16, "unet2 b=1 exact", EXACT)
