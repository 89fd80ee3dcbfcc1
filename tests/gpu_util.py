"""Helpers for the GPU parity tests: run a workload through the C ABI and
through the oracle on the same seeded inputs."""
import sys

import numpy as np
import torch

import oracle
from oracle import network, ops
from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc, nhwc_to_nchw64
from workloads import specs, synth
from workloads.specs import BF16, FP32

TOL = {BF16: 2e-2, FP32: 1e-4}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def maxrel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.max(np.abs(b))
    return float(np.max(np.abs(a - b)) / den) if den > 0 else float(np.max(np.abs(a)))


def storage(dtype):
    return "bf16" if dtype == BF16 else "f64"


def gpu_network(net, dtype, B, m, n, mode, balance=None, lanes=1):
    sess = Session(net, dtype, n=n, balance=balance)
    sess.plan(B, m, mode, lanes)
    _, xraw = synth.input_x(net, B, dtype)
    h, w = net.out_hw()
    _, traw = synth.target_like((B, net.out_channels(), h, w), dtype)
    x = nchw_to_device_nhwc(xraw, dtype)
    t = nchw_to_device_nhwc(traw, dtype)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = torch.empty((B, h, w, net.out_channels()), dtype=x.dtype, device="cuda")
    sess.pipeline_step(x, t, loss, y)
    torch.cuda.synchronize()
    out = {"loss": float(loss.item()), "y": nhwc_to_nchw64(y), "grads": sess.grads64(),
           "sess": sess, "x": x, "t": t, "loss_t": loss, "y_t": y}
    return out


def oracle_network(net, dtype, B, P=None):
    if P is None:
        P = oracle.net_params(net, dtype)
    xv, _ = synth.input_x(net, B, dtype)
    h, w = net.out_hw()
    tv, _ = synth.target_like((B, net.out_channels(), h, w), dtype)
    return network.run(net, P, xv, target=tv, storage=storage(dtype))


def stage_inputs(sess, j, B, dtype):
    """Seeded partition input and upstream gradients (G_0 for the main output,
    G_k for the k-th exported skip), as float64 NCHW values and device NHWC."""
    C, H, W = sess.part_in_shape(j)
    xv, xraw = synth.quantize(synth.normal(synth.SEED_X, (B, C, H, W)), dtype)
    shapes = [sess.part_out_shape(j)] + [sess.stash_shape(s) for s in sess.exported_stashes(j)]
    G = [synth.target_like((B,) + s, dtype, k) for k, s in enumerate(shapes)]
    return xv, xraw, G


def gpu_stage(net, dtype, B, m, mode, balance, j, want_dx=True, G_override=None, sess=None,
              neutral=True, neutral_samples=None, stash_in=None, lanes=1, pairs=False):
    n = len(balance)
    lo = sum(balance[:j - 1])
    hi = lo + balance[j - 1]
    if sess is None:
        sess = Session(net, dtype, n=n, balance=balance, bind_layers=range(lo, hi))
        sess.plan(B, m, mode, lanes)
        sess.pairs = pairs
    xv, xraw, G = stage_inputs(sess, j, B, dtype)
    if G_override is not None:
        G = G_override
    elif neutral:
        G = neutral_G(net, dtype, lo, hi, xv, G, samples=neutral_samples, stash_in=stash_in)
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
    sess.stage_step(j, x, y, dy, dx, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    stash = {sid: torch.cat([sess.stash_view(i, sid, False) for i in range(1, m + 1)])
             for sid in ex}
    return {"sess": sess, "y": y, "dx": dx, "stash": stash, "grads": sess.grads64(range(lo, hi)),
            "G": G, "xv": xv, "lo": lo, "hi": hi}


def oracle_stage(net, dtype, lo, hi, xv, G, samples=None, stash_in=None):
    P = oracle.net_params(net, dtype)
    Gv = [g[0] for g in G]
    st = dict(stash_in or {})
    if samples is not None:
        xv = xv[samples]
        Gv = [g[samples] for g in Gv]
        st = {k: v[samples] for k, v in st.items()}
    return network.run(net, P, xv, lo=lo, hi=hi, out_grads=Gv, storage=storage(dtype),
                       stash_in=st)


ALTS = ("f32", "f32rev", "f32split", "f32c32")


def oracle_stage_variants(net, dtype, lo, hi, xv, G, samples=None, stash_in=None):
    """The parity reference (float64 contraction) and the same computation
    with each float32 contraction variant: the distance between the variants
    and the reference is the spread that valid bf16 runs of this network show
    (ReLU / pool decisions within rounding distance of flipping)."""
    ref = oracle_stage(net, dtype, lo, hi, xv, G, samples, stash_in)
    alts = []
    for mode in (ALTS if dtype == BF16 else ()):
        with ops.contraction(mode):
            alts.append(oracle_stage(net, dtype, lo, hi, xv, G, samples, stash_in))
    return ref, alts


def oracle_network_variants(net, dtype, B):
    ref = oracle_network(net, dtype, B)
    alts = []
    for mode in (ALTS if dtype == BF16 else ()):
        with ops.contraction(mode):
            alts.append(oracle_network(net, dtype, B))
    return ref, alts


def neutral_G(net, dtype, lo, hi, xv, G, samples=None, stash_in=None):
    """Decision-neutral upstream gradients: zero G_k wherever the ReLU
    decision of the layer that produces output k is within the rounding
    distance of flipping, i.e. |z_ref| <= 4 max|z_ref - z_alt| over the float32
    contraction variants (plus a float32-epsilon floor).  Such decisions may
    legitimately go either way; with G = 0 there they cannot change any
    gradient.  Uses only the oracle."""
    P = oracle.net_params(net, dtype)
    x = xv if samples is None else xv[samples]
    st0 = dict(stash_in or {})
    if samples is not None:
        st0 = {k: v[samples] for k, v in st0.items()}
    producers = [hi - 1] + [next(k for k in range(lo, hi) if net.layers[k].stash_id == sid)
                            for sid in network.exported_stashes(net, lo, hi)]

    def preacts(mode):
        with ops.contraction(mode):
            _, tape = network.forward_layers(net, P, lo, hi, x, dict(st0), storage(dtype))
            out = {}
            for k in producers:
                L = net.layers[k]
                w, b = P[k]
                out[k] = network._FWD[L.kind](tape.inputs[k - lo], w, b if L.bias else None)
            return out
    ref = preacts("f64")
    alts = [preacts(m) for m in ALTS]
    newG = []
    for slot, k in enumerate(producers):
        v, raw = G[slot]
        L = net.layers[k]
        if not L.relu:
            newG.append((v, raw))
            continue
        zr = ref[k]
        theta = max(float(np.max(np.abs(zr - a[k]))) for a in alts)
        theta = 4.0 * theta + 1e-6 * float(np.max(np.abs(zr)))
        amb = np.abs(zr) <= theta
        v2, raw2 = v.copy(), raw.copy()
        if samples is None:
            v2[amb] = 0.0
            raw2[amb] = 0
        else:
            sub = v2[samples]
            sub[amb] = 0.0
            v2[samples] = sub
            rs = raw2[samples]
            rs[amb] = 0
            raw2[samples] = rs
        newG.append((v2, raw2))
    return newG


def rmsrel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a))


SPREAD_FACTOR = 4.0


FLIP_MAXREL = 5e-2


def check_grad(name, got, ref, alts, dtype, errs, strict=False):
    """max-rel and rms-rel error of `got` against the reference.

    strict (single layers, forward outputs, fp32 runs): both within the
    parity tolerance.  Gradients of bf16 runs through several ReLU / pool
    layers pass if either
      (a) max-rel and rms-rel are within the tolerance or SPREAD_FACTOR times
          the largest distance of a float32-contraction variant from the
          reference, whichever is larger; or
      (b) rms-rel is within the tolerance and max-rel within FLIP_MAXREL: a few
          decision flips (each moves one whole upstream gradient element) on
          an otherwise matching tensor.  The GPU's MFMA accumulation does not
          round like an IEEE float32 sum, so its flip count need not match
          the float32 variants'."""
    tol = TOL[dtype]
    e_max, e_rms = maxrel(got, ref), rmsrel(got, ref)
    bmax = brms = tol
    sp = max((maxrel(a, ref) for a in alts), default=0.0)
    if strict or dtype != BF16 or not alts:
        errs[name] = (e_max, bmax, e_rms, brms, sp)
        return e_max <= bmax and e_rms <= brms
    bmax = max(tol, SPREAD_FACTOR * sp)
    brms = max(tol, SPREAD_FACTOR * max(rmsrel(a, ref) for a in alts))
    ok = (e_max <= bmax and e_rms <= brms) or (e_rms <= tol and e_max <= FLIP_MAXREL)
    if not (e_max <= bmax and e_rms <= brms) and ok:
        bmax = FLIP_MAXREL
    errs[name] = (e_max, bmax, e_rms, brms, sp)
    return ok


def report(what, errs):
    worst = max(errs, key=lambda k: errs[k][0] / errs[k][1])
    say(f"{what}: " + ", ".join(f"{k}={v[0]:.2e}/{v[1]:.1e}(spread {v[4]:.1e})"
                                for k, v in errs.items()))
    say(f"{what}: worst {worst} max-rel {errs[worst][0]:.3e} (bound {errs[worst][1]:.2e}), "
        f"rms-rel {errs[worst][2]:.3e} (bound {errs[worst][3]:.2e})")


def gpu_stage_with_popped(net, bal, j, dtype=BF16, B=4, m=2, mode=0):
    """Runs stage j after writing seeded values into the slots of skips that
    stage j pops but an earlier partition stashes."""
    from paper_2004_09910_amd.harness import Session
    lo = sum(bal[:j - 1])
    hi = lo + bal[j - 1]
    sess = Session(net, dtype, n=len(bal), balance=bal, bind_layers=range(lo, hi))
    sess.plan(B, m, mode)
    stashed_inside = {L.stash_id for L in net.layers[lo:hi] if L.stash_id >= 0}
    popped = [L.pop_id for L in net.layers[lo:hi]
              if L.pop_id >= 0 and L.pop_id not in stashed_inside]
    stash_in = {}
    b = B // m
    for sid in popped:
        shp = (B,) + sess.stash_shape(sid)
        v, raw = synth.quantize(synth.normal(500 + sid, shp), dtype)
        stash_in[sid] = v
        d = nchw_to_device_nhwc(raw, dtype)
        for i in range(1, m + 1):
            sess.stash_view(i, sid, False).copy_(d[(i - 1) * b:i * b])
    got = gpu_stage(net, dtype, B, m, mode, bal, j, sess=sess, stash_in=stash_in)
    got["stash_in"] = stash_in
    return got
