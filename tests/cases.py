"""Seeded inputs of the parity cases and the oracle's runs on them, without
torch or the GPU: shared by the GPU parity tests and the CPU tests that
check the EXACT family's certificate on the same cases."""
import numpy as np

import exactness
import oracle
from oracle import network
from workloads import synth
from workloads.specs import BF16
from workloads.synth import EXACT, NORMAL


def storage(dtype):
    return "bf16" if dtype == BF16 else "f64"


def exact_target(net, P, xv, dtype, log=None):
    """Target of an EXACT network run: the oracle's own output plus seeded
    values in {-1, 0, 1}, quantised to the storage type, so that the loss
    gradient 2 (y - t) / numel stays a few units per element and the backward
    sums stay exact."""
    y, _ = network.forward_layers(net, P, 0, len(net.layers), xv, {}, storage(dtype), log)
    return synth.quantize(y + synth.signs(synth.SEED_TARGET, y.shape), dtype)


def network_inputs(net, dtype, B, family=NORMAL, P=None, log=None):
    """(x values, x raw, t values, t raw, params) of a network run."""
    if P is None:
        P = oracle.net_params(net, dtype, family=family)
    xv, xraw = synth.input_x(net, B, dtype, family=family)
    h, w = net.out_hw()
    if family == EXACT:
        tv, traw = exact_target(net, P, xv, dtype, log)
    else:
        tv, traw = synth.target_like((B, net.out_channels(), h, w), dtype)
    return xv, xraw, tv, traw, P


def oracle_network(net, dtype, B, family=NORMAL, inputs=None, certify=False, log=None):
    """The oracle's full-batch run on the network inputs; with `certify`, the
    exactness certificate of the run is attached under 'cert'."""
    if inputs is None:
        inputs = network_inputs(net, dtype, B, family)
    xv, _, tv, _, P = inputs
    r = network.run(net, P, xv, target=tv, storage=storage(dtype), log=log)
    if certify:
        r["cert"] = exactness.certificate(net, P, r, target=tv)
    return r


def exact_network_case(net, B, dtype=BF16):
    inputs = network_inputs(net, dtype, B, EXACT)
    ref = oracle_network(net, dtype, B, EXACT, inputs, certify=True)
    return {"inputs": inputs, "ref": ref, "cert": ref["cert"]}


def stage_shapes(net, lo, hi):
    """(C, H, W) of the input of layers [lo, hi) (before layer lo's prologue),
    of its output, and of each exported stash in increasing id order."""
    shapes = net.shapes()
    if lo == 0:
        cin = (net.in_channels, net.height, net.width)
    else:
        cin = (net.layers[lo - 1].cout,) + tuple(shapes[lo - 1])
    out = (net.layers[hi - 1].cout,) + tuple(shapes[hi - 1])
    ex = []
    for sid in network.exported_stashes(net, lo, hi):
        k = next(i for i, L in enumerate(net.layers) if L.stash_id == sid)
        ex.append((net.layers[k].cout,) + tuple(shapes[k]))
    return cin, out, ex


def stage_values(net, lo, hi, B, dtype, family=NORMAL):
    """Seeded stage input (values, raw) and upstream gradients [(values, raw)]
    for the main output and each exported stash."""
    cin, out, ex = stage_shapes(net, lo, hi)
    xv, xraw = synth.tensor(synth.SEED_X, (B,) + cin, dtype, family)
    G = [synth.upstream_grad((B,) + s, dtype, k, family) for k, s in enumerate([out] + ex)]
    return xv, xraw, G


def popped_stash_values(net, lo, hi, B, dtype, family=NORMAL):
    """Seeded values of the skips layers [lo, hi) pop but an earlier
    partition stashes: {sid: (values, raw)}."""
    shapes = net.shapes()
    stashed_inside = {L.stash_id for L in net.layers[lo:hi] if L.stash_id >= 0}
    out = {}
    for L in net.layers[lo:hi]:
        sid = L.pop_id
        if sid >= 0 and sid not in stashed_inside:
            k = next(i for i, M in enumerate(net.layers) if M.stash_id == sid)
            shp = (B, net.layers[k].cout) + tuple(shapes[k])
            out[sid] = synth.tensor(500 + sid, shp, dtype, family)
    return out


def oracle_stage(net, dtype, lo, hi, xv, G, samples=None, stash_in=None, family=NORMAL,
                 certify=False, log=None):
    P = oracle.net_params(net, dtype, family=family)
    Gv = [g[0] for g in G]
    st = dict(stash_in or {})
    if samples is not None:
        xv = xv[samples]
        Gv = [g[samples] for g in Gv]
        st = {k: v[samples] for k, v in st.items()}
    r = network.run(net, P, xv, lo=lo, hi=hi, out_grads=Gv, storage=storage(dtype),
                    stash_in=st, log=log)
    if certify:
        r["cert"] = exactness.certificate(net, P, r, lo=lo)
    return r


def exact_stage_case(net, lo, hi, B, popped=False, dtype=BF16):
    xv, _, G = stage_values(net, lo, hi, B, dtype, EXACT)
    stash_in = None
    if popped:
        stash_in = {sid: v for sid, (v, _) in
                    popped_stash_values(net, lo, hi, B, dtype, EXACT).items()}
    ref = oracle_stage(net, dtype, lo, hi, xv, G, stash_in=stash_in, family=EXACT, certify=True)
    return {"ref": ref, "cert": ref["cert"]}
