"""Parity at the benchmark's full size and launch configuration: the U-Net
stage (partition 1 of 4, input 32x64x192x192 bf16, m = 8, checkpoint
always), checked on sampled outputs the oracle computes one sample at a
time, and bit-exact against the same run without checkpointing."""
import numpy as np
import pytest
import torch

from gpu_util import (TOL, check_grad, gpu_stage, maxrel, oracle_stage_variants, report,
                      say)
from paper_2004_09910_amd.harness import nhwc_to_nchw64
from workloads import specs
from workloads.specs import BF16, CKPT_ALWAYS, CKPT_NEVER

pytestmark = pytest.mark.gpu

SAMPLES = [0, 31]   # first sample of micro-batch 1 and last of micro-batch 8


@pytest.fixture(scope="module")
def runs():
    wl = specs.unet_stage()
    bal = (7, 5, 3, 4)
    say("full-size U-Net stage, always")
    a = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_ALWAYS, bal, 1, neutral_samples=SAMPLES)
    return wl, bal, a


def test_fullsize_outputs_and_input_gradient(runs):
    """Stage outputs (main + three skips) and dx_in of samples 0 and 31: each
    depends only on its own sample, so the oracle runs those two samples."""
    wl, bal, a = runs
    ref, alts = oracle_stage_variants(wl.net, BF16, 0, 7, a["xv"], a["G"], samples=SAMPLES)
    errs = {}
    ok = check_grad("y", nhwc_to_nchw64(a["y"][SAMPLES]), ref["y"], [a["y"] for a in alts], BF16, errs,
                    strict=True)
    for sid, t in a["stash"].items():
        ok &= check_grad(f"skip{sid}", nhwc_to_nchw64(t[SAMPLES]), ref["stash"][sid],
                         [a["stash"][sid] for a in alts], BF16, errs, strict=True)
    ok &= check_grad("dx", nhwc_to_nchw64(a["dx"][SAMPLES]), ref["dx"], [a["dx"] for a in alts], BF16, errs)
    report("full-size sampled outputs", errs)
    assert ok, errs


def test_fullsize_weight_gradients_on_two_samples(runs):
    """Same launch configuration with every upstream gradient zero except on
    samples 0 and 31: then g = g(sample 0) + g(sample 31), which the oracle
    computes on those two samples."""
    wl, bal, a = runs
    G = []
    for v, raw in a["G"]:
        keep = np.zeros(v.shape[0], dtype=bool)
        keep[SAMPLES] = True
        v2 = np.where(keep[:, None, None, None], v, 0.0)
        raw2 = raw.copy()
        raw2[~keep] = 0
        G.append((v2, raw2))
    say("full-size U-Net stage, two-sample gradients")
    got = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_ALWAYS, bal, 1, G_override=G,
                    sess=a["sess"])
    ref, alts = oracle_stage_variants(wl.net, BF16, 0, 7, a["xv"], G, samples=SAMPLES)
    errs = {}
    ok = True
    for idx, (dW, db) in ref["grads"].items():
        ok &= check_grad(f"dW{idx}", got["grads"][idx][0], dW, [a["grads"][idx][0] for a in alts], BF16, errs)
        ok &= check_grad(f"db{idx}", got["grads"][idx][1], db, [a["grads"][idx][1] for a in alts], BF16, errs)
    report("full-size gradients", errs)
    assert ok, errs


def test_fullsize_bit_exact_against_never(runs):
    """Checkpointed and stored-activation runs give bit-identical results."""
    wl, bal, a = runs
    # re-run the always-mode step on its session with the original gradients
    say("full-size U-Net stage, always (again) and never")
    a2 = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_ALWAYS, bal, 1, sess=a["sess"],
                   G_override=a["G"])
    b = gpu_stage(wl.net, BF16, wl.batch, wl.m, CKPT_NEVER, bal, 1, G_override=a["G"])
    for r in (a2, b):
        assert torch.equal(r["y"], a["y"]) and torch.equal(r["dx"], a["dx"])
        for sid in a["stash"]:
            assert torch.equal(r["stash"][sid], a["stash"][sid])
        for idx in a["grads"]:
            np.testing.assert_array_equal(r["grads"][idx][0], a["grads"][idx][0])
            np.testing.assert_array_equal(r["grads"][idx][1], a["grads"][idx][1])
