"""Time-based balance (the per-layer cost measurement that the paper's
partitioning is driven by): measured per-layer times, the partition the
min-max rule picks for them, and a pipeline step on that partition held to
the oracle."""
import math

import pytest
import torch

import paper_2004_09910_amd as tgp
from gpu_util import check_grad, oracle_network_variants, report, say, TOL
from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc, nhwc_to_nchw64
from test_gpu_parity import check_network
from workloads import specs, synth
from workloads.specs import BF16, CKPT_ALWAYS

pytestmark = pytest.mark.gpu


def test_layer_times_restore_the_partition():
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    sess = Session(net, BF16, n=3)
    before = tgp.get_partition(sess.h)
    say("layer times, unet3 b=2")
    us = sess.layer_times(2, CKPT_ALWAYS, iters=2)
    assert len(us) == len(net.layers)
    assert all(math.isfinite(u) and u > 0 for u in us), us
    assert tgp.get_partition(sess.h) == before
    # no plan is left behind
    assert tgp.call_status("tgp_stage_forward", sess.h, 1, 1, 1, 1 << 20, 1 << 20, None) == \
        tgp.ESTATE
    sess.close()


@pytest.mark.parametrize("n", [2, 3])
def test_balance_by_time_pipeline(n):
    """Partition on measured times, then a full pipeline step (m = 2, every
    checkpoint mode) on that partition against the oracle."""
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    B, m = 4, 2
    sess = Session(net, BF16, n=1)
    say(f"balance by time, unet3 n={n}")
    bal, us = sess.balance_by_time(B // m, n, CKPT_ALWAYS, iters=2)
    say(f"  layer us {[round(u, 1) for u in us]} -> balance {bal}")
    assert len(bal) == n and sum(bal) == len(net.layers) and min(bal) >= 1
    # the same rule on the reported times, in whole nanoseconds
    ns = [int(math.floor(float(u) * 1000.0 + 0.5)) for u in us]
    assert tgp.balance_minmax(ns, n) == bal
    pair = oracle_network_variants(net, BF16, B)
    sess.plan(B, m, CKPT_ALWAYS)
    _, xraw = synth.input_x(net, B, BF16)
    h, w = net.out_hw()
    _, traw = synth.target_like((B, net.out_channels(), h, w), BF16)
    x = nchw_to_device_nhwc(xraw, BF16)
    t = nchw_to_device_nhwc(traw, BF16)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = torch.empty((B, h, w, net.out_channels()), dtype=x.dtype, device="cuda")
    sess.pipeline_step(x, t, loss, y)
    torch.cuda.synchronize()
    got = {"loss": float(loss.item()), "y": nhwc_to_nchw64(y), "grads": sess.grads64()}
    check_network(got, pair, BF16, f"unet3 balance-by-time {bal}")
    sess.close()
