"""Time-based balance (the per-layer cost measurement that the paper's
partitioning is driven by): measured per-layer times, the partition the
min-max rule picks for them, and a pipeline step on that partition held to
the oracle."""
import math

import pytest
import torch

import paper_2004_09910_amd as tgp
from gpu_util import check_network, network_inputs, oracle_network, say
from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc, nhwc_to_nchw64
from workloads import specs
from workloads.specs import BF16, CKPT_ALWAYS
from workloads.synth import EXACT

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
    """Partition on measured times, then a full pipeline step (m = 2) on that
    partition against the oracle, on exact inputs."""
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    B, m = 4, 2
    sess = Session(net, BF16, n=1, family=EXACT)
    say(f"balance by time, unet3 n={n}")
    bal, us = sess.balance_by_time(B // m, n, CKPT_ALWAYS, iters=2)
    say(f"  layer us {[round(u, 1) for u in us]} -> balance {bal}")
    assert len(bal) == n and sum(bal) == len(net.layers) and min(bal) >= 1
    # the same rule on the reported times, in whole nanoseconds
    ns = [int(math.floor(float(u) * 1000.0 + 0.5)) for u in us]
    assert tgp.balance_minmax(ns, n) == bal
    inputs = network_inputs(net, BF16, B, EXACT)
    ref = oracle_network(net, BF16, B, EXACT, inputs, certify=True)
    sess.plan(B, m, CKPT_ALWAYS)
    _, xraw, _, traw, _ = inputs
    h, w = net.out_hw()
    x = nchw_to_device_nhwc(xraw, BF16)
    t = nchw_to_device_nhwc(traw, BF16)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = torch.empty((B, h, w, net.out_channels()), dtype=x.dtype, device="cuda")
    sess.pipeline_step(x, t, loss, y)
    torch.cuda.synchronize()
    got = {"loss": float(loss.item()), "y": nhwc_to_nchw64(y), "grads": sess.grads64()}
    check_network(got, ref, BF16, f"unet3 balance-by-time {bal}", EXACT)
    sess.close()
