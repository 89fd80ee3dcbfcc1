"""Oracle network pass: the full-batch float64 forward and backward of a layer
sequence, with no micro-batching, no checkpointing and no schedule.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Because the layers involve no intra-batch computation, the paper's
decomposition into tasks F_{i,j} and B_{i,j} (Sec. 2, eqs. (F_ij), (B_ij))
and the sum of g_i^j over micro-batches give exactly this full-batch
gradient in real arithmetic; micro-batching and recomputation only change
when values are computed.  So the oracle is the plain definition.

Two storage modes:
  'f64'  every value is kept in float64 (the pure definition);
  'bf16' float64 arithmetic, but every tensor a bf16 run stores is rounded to
         bfloat16 where it is stored: each layer output, each dZ and dX and
         the summed 2x2 upsample gradient.  (The loss gradient a bf16 run
         stores is rounded by the last layer's dZ store: rounding it before
         would not change the result, since round(round(g) * mask) =
         round(g * mask) for a 0/1 mask.)  Weight and bias gradients stay
         unrounded (a bf16 run accumulates them in fp32).  The ReLU mask and
         the max-pool argmax are then decided on stored values, in the storage
         precision, as a bf16 run decides them.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from . import ops
from workloads.specs import (CONV1X1, CONV3X3, DWCONV3X3, PRO_MAXPOOL2, PRO_NONE,
                             PRO_UPCAT2, Net)

_FWD = {CONV3X3: ops.conv3x3_forward, CONV1X1: ops.conv1x1_forward,
        DWCONV3X3: ops.dwconv3x3_forward}
_DGRAD = {CONV3X3: ops.conv3x3_dgrad, CONV1X1: ops.conv1x1_dgrad,
          DWCONV3X3: ops.dwconv3x3_dgrad}
_WGRAD = {CONV3X3: ops.conv3x3_wgrad, CONV1X1: ops.conv1x1_wgrad,
          DWCONV3X3: ops.dwconv3x3_wgrad}


def _store(a, storage):
    return ops.round_bf16(a) if storage == "bf16" else a


@dataclass
class Tape:
    """What a forward over layers [lo, hi) leaves for its backward."""
    lo: int
    hi: int
    inputs: List[np.ndarray] = field(default_factory=list)   # layer input after prologue
    outputs: List[np.ndarray] = field(default_factory=list)  # stored layer output Y
    argmax: Dict[int, np.ndarray] = field(default_factory=dict)
    prev_c: Dict[int, int] = field(default_factory=dict)     # channels of the upsampled part
    # filled by the backward, for diagnostics: per layer, the gradient at its
    # output (after any skip gradient was added), the skip gradient added
    # there, the stored dZ and the stored gradient of its (post-prologue) input
    dy: Dict[int, np.ndarray] = field(default_factory=dict)
    dskip: Dict[int, np.ndarray] = field(default_factory=dict)
    dz: Dict[int, np.ndarray] = field(default_factory=dict)
    dinp: Dict[int, np.ndarray] = field(default_factory=dict)


def forward_layers(net: Net, params, lo: int, hi: int, x: np.ndarray,
                   stash: Dict[int, np.ndarray], storage: str = "f64", log=None):
    """Runs layers [lo, hi) on x (the output of layer lo-1, or the network
    input).  Popped skips are read from `stash`; stashed outputs are written
    to it.  Returns (output of layer hi-1, tape).  `log`, if given, is called
    with a short message after each layer (progress of long runs)."""
    tape = Tape(lo, hi)
    cur = x
    for idx in range(lo, hi):
        L = net.layers[idx]
        w, b = params[idx]
        if L.prologue == PRO_MAXPOOL2:
            inp, arg = ops.maxpool2_forward(cur)
            tape.argmax[idx] = arg
        elif L.prologue == PRO_UPCAT2:
            tape.prev_c[idx] = cur.shape[1]
            inp = np.concatenate([ops.upsample2_forward(cur), stash[L.pop_id]], axis=1)
        else:
            inp = cur
        z = _FWD[L.kind](inp, w, b if L.bias else None)
        y = np.maximum(z, 0.0) if L.relu else z
        y = _store(y, storage)
        tape.inputs.append(inp)
        tape.outputs.append(y)
        if L.stash_id >= 0:
            stash[L.stash_id] = y
        cur = y
        if log is not None:
            log(f"oracle forward layer {idx}")
    return cur, tape


def backward_layers(net: Net, params, tape: Tape, dy: np.ndarray,
                    skip_grad: Dict[int, np.ndarray], want_dx: bool = True,
                    storage: str = "f64", log=None):
    """Backward through the layers of `tape` in reverse.  `dy` is the gradient
    of the last layer's output.  `skip_grad[id]` holds the gradient flowing
    back into stashed skip `id` (written by the popping layer, read by the
    stashing layer, which adds it after the main-path gradient).  Returns
    (dx of the input of layer lo or None, {idx: (dW, db)})."""
    grads = {}
    cur = dy
    for pos in range(tape.hi - tape.lo - 1, -1, -1):
        idx = tape.lo + pos
        L = net.layers[idx]
        w, _ = params[idx]
        if L.stash_id >= 0 and L.stash_id in skip_grad:
            tape.dskip[idx] = skip_grad.pop(L.stash_id)
            cur = cur + tape.dskip[idx]
        tape.dy[idx] = cur
        y = tape.outputs[pos]
        dz = cur * (y > 0) if L.relu else cur
        dz = _store(dz, storage)
        tape.dz[idx] = dz
        dW = _WGRAD[L.kind](tape.inputs[pos], dz)
        db = ops.bias_grad(dz) if L.bias else None
        grads[idx] = (dW, db)
        if log is not None:
            log(f"oracle backward layer {idx}")
        if pos == 0 and not want_dx:
            return None, grads
        dinp = _store(_DGRAD[L.kind](dz, w), storage)
        tape.dinp[idx] = dinp
        if L.prologue == PRO_MAXPOOL2:
            cur = ops.maxpool2_backward(dinp, tape.argmax[idx])
        elif L.prologue == PRO_UPCAT2:
            pc = tape.prev_c[idx]
            skip_grad[L.pop_id] = dinp[:, pc:]
            cur = _store(ops.upsample2_backward(dinp[:, :pc]), storage)
        else:
            cur = dinp
    return cur, grads


def exported_stashes(net: Net, lo: int, hi: int):
    """Stash ids written by layers [lo, hi) and popped by a layer outside it,
    in increasing id order: the extra outputs of a partition run as a stage."""
    made = [L.stash_id for L in net.layers[lo:hi] if L.stash_id >= 0]
    popped_inside = {L.pop_id for L in net.layers[lo:hi] if L.pop_id >= 0}
    return sorted(s for s in made if s not in popped_inside)


def run(net: Net, params, x, *, lo: int = 0, hi: Optional[int] = None,
        target=None, out_grads=None, storage: str = "f64", want_dx: bool = True,
        stash_in: Optional[Dict[int, np.ndarray]] = None, log=None):
    """Full-batch forward + backward over layers [lo, hi).

    Network runs pass `target`: loss = sum (y-t)^2 / numel, no 1/2 factor.
    Stage runs pass `out_grads` = [G_0, G_1, ...] for the main output and the
    exported stashes (ids from exported_stashes); the loss is then
    sum_k <G_k, out_k>, so each upstream gradient is G_k itself.
    Returns a dict with loss, outputs, grads {idx: (dW, db)}, dx."""
    hi = len(net.layers) if hi is None else hi
    stash = dict(stash_in or {})
    y, tape = forward_layers(net, params, lo, hi, x, stash, storage, log)
    exports = exported_stashes(net, lo, hi)
    skip_grad = {}
    if target is not None:
        loss, dy = ops.mse(y, target, y.size)
    else:
        assert out_grads is not None and len(out_grads) == 1 + len(exports)
        dy = out_grads[0]
        loss = float(np.sum(out_grads[0] * y))
        for k, sid in enumerate(exports):
            skip_grad[sid] = out_grads[1 + k]
            loss += float(np.sum(out_grads[1 + k] * stash[sid]))
    dx, grads = backward_layers(net, params, tape, dy, skip_grad, want_dx, storage, log)
    return {"loss": loss, "y": y, "stash": {s: stash[s] for s in exports},
            "grads": grads, "dx": dx, "tape": tape}
