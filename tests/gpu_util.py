"""Helpers for the GPU parity tests: run a workload through the C ABI and
through the oracle on the same seeded inputs, and compare them element by
element.

Two input families (workloads.synth):
  NORMAL  N(0,1) inputs, He-normal weights.  Two correct bf16 computations of
          a multi-layer ReLU / max-pool network that sum in different orders
          take some ReLU-mask and argmax decisions on values within rounding
          distance of each other, and each differing decision moves a whole
          gradient element.  NORMAL runs are therefore compared on quantities
          no decision upstream of them can move: forward outputs, and every
          output of single-layer runs (their inputs are identical bits).
  EXACT   small integers and sparse +-1 weights: every accumulation of such a
          run is exact in float32 (tests/exactness.py checks it on the
          oracle's tape), so every correct implementation produces the same
          bits.  Multi-layer gradients are compared on this family, to
          EXACT_TOL.

Every comparison is max-rel = max|got - ref| / max|ref| per tensor, against
TOL (2e-2 bf16, 1e-4 fp32) for NORMAL runs and EXACT_TOL for EXACT runs.
"""
import sys

import numpy as np
import torch

import exactness
from cases import (network_inputs, oracle_network, oracle_stage, popped_stash_values,  # noqa: F401
                   stage_values, storage)
from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc, nhwc_to_nchw64
from workloads.specs import BF16, FP32
from workloads.synth import EXACT, NORMAL

TOL = {BF16: 2e-2, FP32: 1e-4}
EXACT_TOL = 1e-6


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def maxrel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.max(np.abs(b))
    return float(np.max(np.abs(a - b)) / den) if den > 0 else float(np.max(np.abs(a)))


def rmsrel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a))


def tol_for(dtype, family):
    return EXACT_TOL if family == EXACT else TOL[dtype]


def check(name, got, ref, tol, errs):
    """max-rel of `got` against `ref`, recorded in errs[name]; True if within
    tol.  An all-zero reference passes only an all-zero result."""
    e = maxrel(got, ref)
    errs[name] = (e, tol, rmsrel(got, ref))
    return e <= tol


def report(what, errs):
    worst = max(errs, key=lambda k: errs[k][0] / errs[k][1])
    say(f"{what}: " + ", ".join(f"{k}={v[0]:.2e}" for k, v in errs.items()))
    say(f"{what}: worst {worst} max-rel {errs[worst][0]:.3e} (bound {errs[worst][1]:.1e}), "
        f"rms-rel {errs[worst][2]:.3e}")


# ---------------------------------------------------------------- networks

def gpu_network(net, dtype, B, m, n, mode, balance=None, lanes=1, family=NORMAL, inputs=None):
    sess = Session(net, dtype, n=n, balance=balance, family=family)
    sess.plan(B, m, mode, lanes)
    if inputs is None:
        inputs = network_inputs(net, dtype, B, family)
    _, xraw, _, traw, _ = inputs
    h, w = net.out_hw()
    x = nchw_to_device_nhwc(xraw, dtype)
    t = nchw_to_device_nhwc(traw, dtype)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = torch.empty((B, h, w, net.out_channels()), dtype=x.dtype, device="cuda")
    sess.pipeline_step(x, t, loss, y)
    torch.cuda.synchronize()
    out = {"loss": float(loss.item()), "y": nhwc_to_nchw64(y), "grads": sess.grads64(),
           "sess": sess, "x": x, "t": t, "loss_t": loss, "y_t": y}
    return out


def check_network(got, ref, dtype, what, family=NORMAL, grads=True):
    """Loss, output and (with `grads`) every weight and bias gradient of a
    pipeline run against the oracle."""
    tol = tol_for(dtype, family)
    errs = {}
    ok = check("loss", np.array([got["loss"]]), np.array([ref["loss"]]), tol, errs)
    ok &= check("y", got["y"], ref["y"], tol, errs)
    if grads:
        for idx, (dW, db) in ref["grads"].items():
            ok &= check(f"dW{idx}", got["grads"][idx][0], dW, tol, errs)
            if db is not None:
                ok &= check(f"db{idx}", got["grads"][idx][1], db, tol, errs)
    _finish(what, ok, errs, ref, family)
    return errs


def _finish(what, ok, errs, ref, family):
    report(what, errs)
    if "cert" in ref:
        say(f"{what}: exactness certificate " +
            ", ".join(f"{k}={v:.2e}" for k, v in ref["cert"].items()))
        if family == EXACT:
            assert exactness.exact(ref["cert"]), "inputs do not keep this run exact"
    assert ok, errs


# ---------------------------------------------------------------- stages

def only_samples(G, samples):
    """Upstream gradients with every sample outside `samples` zeroed: the
    weight gradient of the step is then the sum over `samples` alone."""
    out = []
    for v, raw in G:
        keep = np.zeros(v.shape[0], dtype=bool)
        keep[list(samples)] = True
        v2 = np.where(keep[:, None, None, None], v, 0.0)
        raw2 = raw.copy()
        raw2[~keep] = 0
        out.append((v2, raw2))
    return out


def gpu_stage(net, dtype, B, m, mode, balance, j, want_dx=True, G_override=None, sess=None,
              stash_in=None, lanes=1, group=1, serial=False, family=NORMAL,
              grad_samples=None):
    """One stage step of partition j through the C ABI.  `grad_samples`
    zeroes the upstream gradients of every other sample; `serial` issues
    everything on one stream (the benchmark's configuration)."""
    n = len(balance)
    lo = sum(balance[:j - 1])
    hi = lo + balance[j - 1]
    if sess is None:
        sess = Session(net, dtype, n=n, balance=balance, bind_layers=range(lo, hi),
                       family=family)
        sess.plan(B, m, mode, lanes)
        sess.group = group
    xv, xraw, G = stage_values(net, lo, hi, B, dtype, family)
    if G_override is not None:
        G = G_override
    elif grad_samples is not None:
        G = only_samples(G, grad_samples)
    x = nchw_to_device_nhwc(xraw, dtype)
    C, H, W = sess.part_out_shape(j)
    y = torch.empty((B, H, W, C), dtype=x.dtype, device="cuda")
    dy = nchw_to_device_nhwc(G[0][1], dtype)
    dx = torch.empty_like(x) if want_dx else None
    ex = sess.exported_stashes(j)
    b = B // m
    for k, sid in enumerate(ex):
        g = nchw_to_device_nhwc(G[1 + k][1], dtype)
        for i in range(1, m + 1):
            sess.stash_view(i, sid, True).copy_(g[(i - 1) * b:i * b])
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream().cuda_stream
    sess.stage_step(j, x, y, dy, dx, stream, serial=serial)
    torch.cuda.synchronize()
    stash = {sid: torch.cat([sess.stash_view(i, sid, False) for i in range(1, m + 1)])
             for sid in ex}
    return {"sess": sess, "y": y, "dx": dx, "stash": stash, "grads": sess.grads64(range(lo, hi)),
            "G": G, "xv": xv, "lo": lo, "hi": hi}


def check_stage(got, ref, dtype, what, family=NORMAL, dx=True, grads=True, samples=None):
    """Stage outputs (main and exported skips), dx_in and every weight and
    bias gradient against the oracle.  `samples` restricts the per-sample
    tensors of the GPU run to those samples (the oracle ran only them)."""
    tol = tol_for(dtype, family)
    sel = slice(None) if samples is None else list(samples)
    errs = {}
    ok = check("y", nhwc_to_nchw64(got["y"][sel]), ref["y"], tol, errs)
    for sid, t in got["stash"].items():
        ok &= check(f"skip{sid}", nhwc_to_nchw64(t[sel]), ref["stash"][sid], tol, errs)
    if dx:
        ok &= check("dx", nhwc_to_nchw64(got["dx"][sel]), ref["dx"], tol, errs)
    if grads:
        for idx, (dW, db) in ref["grads"].items():
            ok &= check(f"dW{idx}", got["grads"][idx][0], dW, tol, errs)
            if db is not None:
                ok &= check(f"db{idx}", got["grads"][idx][1], db, tol, errs)
    _finish(what, ok, errs, ref, family)
    return errs


def gpu_stage_with_popped(net, bal, j, dtype=BF16, B=4, m=2, mode=0, family=NORMAL):
    """Runs stage j after writing seeded values into the slots of skips that
    stage j pops but an earlier partition stashes."""
    lo = sum(bal[:j - 1])
    hi = lo + bal[j - 1]
    sess = Session(net, dtype, n=len(bal), balance=bal, bind_layers=range(lo, hi), family=family)
    sess.plan(B, m, mode)
    stash_in = {}
    b = B // m
    for sid, (v, raw) in popped_stash_values(net, lo, hi, B, dtype, family).items():
        stash_in[sid] = v
        d = nchw_to_device_nhwc(raw, dtype)
        for i in range(1, m + 1):
            sess.stash_view(i, sid, False).copy_(d[(i - 1) * b:i * b])
    got = gpu_stage(net, dtype, B, m, mode, bal, j, sess=sess, stash_in=stash_in, family=family)
    got["stash_in"] = stash_in
    return got
