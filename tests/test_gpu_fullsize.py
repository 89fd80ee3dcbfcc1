"""Parity at the benchmark's full size and launch configuration: the U-Net
stage (partition 1 of 4, input 32x64x192x192 bf16, m = 8, checkpoint
always), run as the benchmark runs it (all eight micro-batches in one
launch per layer, on the buffers of eight lanes, everything on one stream),
checked on sampled
outputs the oracle computes one sample at a time, and bit-exact against the
same run without checkpointing.

Forward outputs are checked on N(0,1) inputs to the bf16 tolerance.  The
input gradient and the weight and bias gradients are checked on the EXACT
family (float32 sums exact, tests/exactness.py) to 1e-6: with upstream
gradients zero on every sample but the first of micro-batch 1 and the last
of micro-batch 8, the step's gradient is the sum over those two samples,
which the oracle computes."""
import numpy as np
import pytest
import torch

from gpu_util import check_stage, gpu_stage, oracle_stage, say
from workloads import specs
from workloads.specs import BF16, CKPT_ALWAYS, CKPT_NEVER
from workloads.synth import EXACT

pytestmark = pytest.mark.gpu

SAMPLES = [0, 31]   # first sample of micro-batch 1 and last of micro-batch 8
BENCH = dict(lanes=8, group=8, serial=True)


@pytest.fixture(scope="module")
def runs():
    wl = specs.unet_stage()
    bal = (7, 5, 3, 4)
    say("full-size U-Net stage, always, N(0,1), benchmark launch configuration")
    a = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_ALWAYS, bal, 1, **BENCH)
    return wl, bal, a


def test_fullsize_outputs(runs):
    """Stage outputs (main + three skips) of samples 0 and 31: each depends
    only on its own sample, so the oracle runs those two samples."""
    wl, bal, a = runs
    ref = oracle_stage(wl.net, BF16, 0, 7, a["xv"], a["G"], samples=SAMPLES, log=say)
    check_stage(a, ref, BF16, "full-size sampled outputs", dx=False, grads=False,
                samples=SAMPLES)


def test_fullsize_gradients_exact(runs):
    """Exact inputs in the same launch configuration, upstream gradients zero
    except on samples 0 and 31: outputs and dx_in of those samples and every
    weight and bias gradient of the step equal the oracle's."""
    wl, bal, _ = runs
    say("full-size U-Net stage, always, exact family, gradients of samples 0 and 31")
    got = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_ALWAYS, bal, 1, family=EXACT,
                    grad_samples=SAMPLES, **BENCH)
    say("oracle on samples 0 and 31")
    ref = oracle_stage(wl.net, BF16, 0, 7, got["xv"], got["G"], samples=SAMPLES, family=EXACT,
                       certify=True, log=say)
    check_stage(got, ref, BF16, "full-size exact", EXACT, samples=SAMPLES)
    got["sess"].close()


def test_fullsize_bit_exact_against_never(runs):
    """Checkpointed and stored-activation runs give bit-identical results."""
    wl, bal, a = runs
    say("full-size U-Net stage, always (again) and never")
    a2 = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_ALWAYS, bal, 1, sess=a["sess"],
                   G_override=a["G"], **BENCH)
    b = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_NEVER, bal, 1, G_override=a["G"])
    for r in (a2, b):
        assert torch.equal(r["y"], a["y"]) and torch.equal(r["dx"], a["dx"])
        for sid in a["stash"]:
            assert torch.equal(r["stash"][sid], a["stash"][sid])
        for idx in a["grads"]:
            np.testing.assert_array_equal(r["grads"][idx][0], a["grads"][idx][0])
            np.testing.assert_array_equal(r["grads"][idx][1], a["grads"][idx][1])
