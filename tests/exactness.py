"""Exactness certificate for runs on the EXACT input family.

A float32 sum of terms that are all integer multiples of one power of two q
is exact, in any order and with any blocking, when the sum of the terms'
magnitudes is at most 2^24 q: every partial sum is then a multiple of q
below 2^24 q, which float32 holds exactly.  The product of two bf16 values
is exact in float32.  So if every accumulation of a run meets that bound,
every correct implementation that accumulates in float32 (or wider) holds the
same value before each bf16 store, rounds it the same way, and takes each
ReLU and max-pool decision on the same bits: its results must equal the
bf16-storage oracle's exactly.

`certificate` walks the oracle's tape of one run and returns, per kind of
accumulation, the largest ratio (sum of |terms|) / (2^24 q); every ratio at
most 1 means the run is exact.  It uses only the oracle's operators (applied
to magnitudes) and the values on the tape.
"""
from __future__ import annotations

import numpy as np

from oracle import network, ops
from workloads.specs import PRO_UPCAT2

LIMIT = float(2 ** 24)


def quantum(a) -> float:
    """Largest power of two of which every value of `a` is an integer
    multiple (inf for an all-zero array)."""
    a = np.asarray(a, dtype=np.float64).ravel()
    a = a[a != 0]
    if a.size == 0:
        return float("inf")
    m, e = np.frexp(a)                          # a = m 2^e, 0.5 <= |m| < 1
    M = np.abs(m * 2.0 ** 53).astype(np.int64)  # exact integer significand
    low = M & (-M)                              # lowest set bit
    tz = np.log2(low.astype(np.float64))        # exact for powers of two
    return float(2.0 ** np.min(e.astype(np.float64) - 53 + tz))


def _ratio(bound, q):
    mx = float(np.max(bound)) if np.size(bound) else 0.0
    if mx == 0.0:
        return 0.0
    return mx / (LIMIT * q)


def certificate(net, params, result, lo=0, target=None):
    """Largest sum-of-magnitudes ratio per accumulation kind of one oracle run
    (`result` from oracle.network.run over layers [lo, hi) of `net`, bf16
    storage).  Keys: 'forward', 'wgrad', 'bias', 'dgrad', 'skip_add',
    'upsample', 'loss_dy' and, for network runs (`target` given), 'loss_sum'
    (the sum of squares) and 'loss_scale_pow2' (1 if 2 / numel is a power of
    two, so that scaling y - t is exact, else inf)."""
    tape = result["tape"]
    out = {k: 0.0 for k in ("forward", "wgrad", "bias", "dgrad", "skip_add", "upsample")}
    for pos, inp in enumerate(tape.inputs):
        idx = lo + pos
        L = net.layers[idx]
        w, b = params[idx]
        bb = b if L.bias else None
        fwd = network._FWD[L.kind]
        S = fwd(np.abs(inp), np.abs(w), None if bb is None else np.abs(bb))
        q = quantum(inp) * quantum(w)
        if bb is not None:
            q = min(q, quantum(bb))
        out["forward"] = max(out["forward"], _ratio(S, q))
        if idx not in tape.dz:
            continue
        dz = tape.dz[idx]
        S = network._WGRAD[L.kind](np.abs(inp), np.abs(dz))
        out["wgrad"] = max(out["wgrad"], _ratio(S, quantum(inp) * quantum(dz)))
        if bb is not None:
            out["bias"] = max(out["bias"], _ratio(ops.bias_grad(np.abs(dz)), quantum(dz)))
        if idx in tape.dskip:
            sk = tape.dskip[idx]
            main = tape.dy[idx] - sk
            out["skip_add"] = max(out["skip_add"],
                                  _ratio(np.abs(main) + np.abs(sk),
                                         min(quantum(main), quantum(sk))))
        if idx in tape.dinp:
            S = network._DGRAD[L.kind](np.abs(dz), np.abs(w))
            out["dgrad"] = max(out["dgrad"], _ratio(S, quantum(dz) * quantum(w)))
            if L.prologue == PRO_UPCAT2:
                pc = tape.prev_c[idx]
                part = tape.dinp[idx][:, :pc]
                out["upsample"] = max(out["upsample"],
                                      _ratio(ops.upsample2_backward(np.abs(part)), quantum(part)))
    if target is not None:
        y = result["y"]
        d = y - target
        out["loss_dy"] = _ratio(np.abs(y) + np.abs(target), min(quantum(y), quantum(target)))
        out["loss_sum"] = _ratio(np.sum(d * d), quantum(d) ** 2)
        scale = 2.0 / y.size
        out["loss_scale_pow2"] = 1.0 if quantum(np.array([scale])) == scale else float("inf")
    return out


def exact(cert, keys=None) -> bool:
    """True if every listed ratio (default: all but the loss sum) is <= 1."""
    keys = [k for k in cert if k != "loss_sum"] if keys is None else keys
    return all(cert[k] <= 1.0 for k in keys)
