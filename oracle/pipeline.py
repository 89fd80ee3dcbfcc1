"""Oracle of the paper's micro-batch pipeline with checkpointing, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

It follows Sec. 2 step by step: the mini-batch is split into m micro-batches
x_1..x_m; forward tasks F_{i,j} run in the deterministic clock-cycle order of
Algorithm 1 (clock k = 1..m+n-1 runs every (i,j) with i+j-1 = k); backward
tasks B_{i,j} run in the reverse order, which keeps the GPipe constraints of
Sec. 2.1 (B_{i,j+1} before B_{i,j}, B_{i,j} before B_{i-1,j}); a checkpointed
F_{i,j} keeps only its input, and F'_{i,j} recomputes it right before
B_{i,j} (Sec. 2.1); the except-last policy skips checkpointing for i = m.
Weight gradients are g^j = sum_i g_i^j, added in the order i = m..1.

Used to pin the invariants the method relies on: the micro-batch gradient sum
equals the full-batch gradient, and recomputation reproduces the stored
activations bit for bit.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import ops
from .network import backward_layers, exported_stashes, forward_layers
from workloads.specs import CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER, Net


def forward_clocks(m: int, n: int) -> List[List[Tuple[int, int]]]:
    """Algorithm 1: clock k (1-based) holds the tasks (i, j) with i+j-1 = k.
    Within a clock the tasks are independent; they are listed with j
    ascending."""
    out = []
    for k in range(1, m + n):
        out.append([(k - j + 1, j) for j in range(1, n + 1) if 1 <= k - j + 1 <= m])
    return out


def backward_clocks(m: int, n: int) -> List[List[Tuple[int, int]]]:
    """Backward clocks, last forward clock first; j descending within a clock."""
    return [list(reversed(c)) for c in reversed(forward_clocks(m, n))]


def checkpointed(mode: int, i: int, m: int) -> bool:
    if mode == CKPT_ALWAYS:
        return True
    if mode == CKPT_EXCEPT_LAST:
        return i < m
    assert mode == CKPT_NEVER
    return False


def bounds_from_balance(balance: Sequence[int]) -> List[Tuple[int, int]]:
    out, lo = [], 0
    for cnt in balance:
        out.append((lo, lo + cnt))
        lo += cnt
    return out


def run_pipeline(net: Net, params, x: np.ndarray, target: np.ndarray,
                 balance: Sequence[int], m: int, mode: int, storage: str = "f64"):
    """Network run with MSE loss against `target` over the full mini-batch."""
    B = x.shape[0]
    assert B % m == 0
    b = B // m
    n = len(balance)
    bounds = bounds_from_balance(balance)
    numel = target.size
    trace = []
    xin: Dict[Tuple[int, int], np.ndarray] = {}      # x_i^{j-1}: input of F_{i,j}
    tapes: Dict[Tuple[int, int], object] = {}        # kept only when not checkpointed
    stash: Dict[int, Dict[int, np.ndarray]] = {i: {} for i in range(1, m + 1)}
    stash_at_fwd: Dict[Tuple[int, int], Dict[int, np.ndarray]] = {}
    y_out = np.zeros_like(target)
    loss_parts, dy_last = {}, {}

    for clock in forward_clocks(m, n):
        for (i, j) in clock:
            lo, hi = bounds[j - 1]
            inp = x[(i - 1) * b:i * b] if j == 1 else xin.pop(("out", i, j - 1))
            xin[(i, j)] = inp
            stash_at_fwd[(i, j)] = dict(stash[i])
            out, tape = forward_layers(net, params, lo, hi, inp, stash[i], storage)
            trace.append(("F", i, j))
            if not checkpointed(mode, i, m):
                tapes[(i, j)] = tape
            if j == n:
                y_out[(i - 1) * b:i * b] = out
                t = target[(i - 1) * b:i * b]
                d = out - t
                loss_parts[i] = float(np.sum(d * d))
                dy = 2.0 * d / numel
                dy_last[i] = ops.round_bf16(dy) if storage == "bf16" else dy
            else:
                xin[("out", i, j)] = out
                xin[("keep", i, j)] = out   # kept for B_{i,j}'s ReLU mask (it is a layer output)

    grads: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    dx_of: Dict[Tuple[int, int], np.ndarray] = {}
    skip_grad: Dict[int, Dict[int, np.ndarray]] = {i: {} for i in range(1, m + 1)}
    recompute_identical = True
    for clock in backward_clocks(m, n):
        for (i, j) in clock:
            lo, hi = bounds[j - 1]
            if checkpointed(mode, i, m):
                # F'_{i,j}: rerun from the saved input and the skips it popped.
                st = dict(stash_at_fwd[(i, j)])
                _, tape = forward_layers(net, params, lo, hi, xin[(i, j)], st, storage)
                trace.append(("R", i, j))
                keep = xin.get(("keep", i, j))
                if keep is not None and not np.array_equal(keep, tape.outputs[-1]):
                    recompute_identical = False
                for sid, v in st.items():
                    if sid in stash[i] and not np.array_equal(stash[i][sid], v):
                        recompute_identical = False
            else:
                tape = tapes.pop((i, j))
            dy = dy_last[i] if j == n else dx_of.pop((i, j))
            dx, g = backward_layers(net, params, tape, dy, skip_grad[i], want_dx=(j > 1),
                                    storage=storage)
            trace.append(("B", i, j))
            if j > 1:
                dx_of[(i, j - 1)] = dx
            for idx, (dW, db) in g.items():
                if idx not in grads:
                    grads[idx] = (dW.copy(), None if db is None else db.copy())
                else:
                    a, c = grads[idx]
                    grads[idx] = (a + dW, None if c is None else c + db)
            trace.append(("A", i, j))
    loss = sum(loss_parts[i] for i in range(1, m + 1)) / numel
    return {"loss": loss, "y": y_out, "grads": grads, "trace": trace,
            "recompute_identical": recompute_identical}
