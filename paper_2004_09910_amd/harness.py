"""Torch-side harness around the C ABI: device memory, seeded parameters and
layout conversion for tests, the benchmark and the smoke check.

Torch provides device memory, streams and exact layout permutations only;
every step of the method runs in libtgp.so.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

import paper_2004_09910_amd as tgp
from workloads import specs, synth
from workloads.specs import BF16, CONV1X1, DWCONV3X3, FP32

TORCH_DT = {BF16: torch.bfloat16, FP32: torch.float32}


def raw_to_torch(raw: np.ndarray, dtype: int) -> torch.Tensor:
    """Raw storage (float32 array, or uint16 bfloat16 bits) -> CPU tensor."""
    if dtype == FP32:
        return torch.from_numpy(np.ascontiguousarray(raw, dtype=np.float32))
    return torch.from_numpy(np.ascontiguousarray(raw).view(np.int16)).view(torch.bfloat16)


def nchw_to_device_nhwc(raw: np.ndarray, dtype: int, device="cuda") -> torch.Tensor:
    t = raw_to_torch(raw, dtype)
    return t.permute(0, 2, 3, 1).contiguous().to(device)


def nhwc_to_nchw64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().permute(0, 3, 1, 2).contiguous().numpy().astype(np.float64)


class _CAI:
    """Exposes a raw device address to torch.as_tensor (no copy)."""

    def __init__(self, ptr: int, shape, typestr: str):
        self.__cuda_array_interface__ = {"shape": tuple(shape), "typestr": typestr,
                                         "data": (int(ptr), False), "version": 2,
                                         "strides": None}


def wrap(ptr: int, shape, dtype: int, device="cuda") -> torch.Tensor:
    if dtype == FP32:
        return torch.as_tensor(_CAI(ptr, shape, "<f4"), device=device)
    return torch.as_tensor(_CAI(ptr, shape, "<i2"), device=device).view(torch.bfloat16)


def layer_tuple(L: specs.Layer):
    return (L.kind, L.cin, L.cout, int(L.relu), int(L.bias), L.prologue, L.stash_id, L.pop_id)


class Session:
    """One network on one device with seeded parameters bound."""

    def __init__(self, net: specs.Net, dtype: int, n: int = 1,
                 balance: Optional[Sequence[int]] = None, device: str = "cuda",
                 seed_offset: int = 0, bind_layers: Optional[Sequence[int]] = None,
                 family: str = synth.NORMAL, init: str = "seeded"):
        """init = 'seeded': the seeded parameters of `family` (what the oracle
        gets); 'device': He-normal weights and zero biases drawn on the device
        by torch, for memory and throughput runs of models too large to draw
        on the host (no oracle comparison possible)."""
        assert init in ("seeded", "device"), init
        self.net, self.dtype, self.device = net, dtype, device
        self.family = family
        self.init = init
        self.h = tgp.net_create([layer_tuple(L) for L in net.layers], net.in_channels,
                                net.height, net.width, dtype)
        tgp.set_partition(self.h, n, balance)
        self.n = n
        self.balance = tgp.get_partition(self.h)
        self.bounds = []
        lo = 0
        for c in self.balance:
            self.bounds.append((lo, lo + c))
            lo += c
        self.shapes = net.shapes()
        self.params: Dict[int, dict] = {}
        layers = range(len(net.layers)) if bind_layers is None else bind_layers
        for idx in layers:
            self._bind_layer(idx, seed_offset)
        self.ws = None
        self.B = self.m = self.b = self.mode = None
        self.lanes = 1
        self.group = 1          # micro-batches per stage call (1, 2 or 4)
        self._lane_streams = None

    def _bind_layer(self, idx: int, seed_offset: int):
        L = self.net.layers[idx]
        if self.init == "device":
            shape = (L.cout, 9) if L.kind == DWCONV3X3 else (L.cout, 3 if L.taps == 9 else 1,
                                                             3 if L.taps == 9 else 1, L.cin)
            wk = (torch.randn(shape, device=self.device) * (2.0 / L.fan_in()) ** 0.5).to(
                TORCH_DT[self.dtype])
            bt = torch.zeros(L.cout, dtype=torch.float32, device=self.device) if L.bias else None
            w64 = b = None
        else:
            (w64, wraw), b = synth.layer_params(self.net, idx, self.dtype, seed_offset,
                                                self.family)
            wt = raw_to_torch(wraw, self.dtype)
            if L.kind == DWCONV3X3:
                wk = wt.reshape(L.cout, 9)
            else:
                wk = wt.permute(0, 2, 3, 1)   # OIHW -> KRSC
            wk = wk.contiguous().to(self.device)
            bt = None if b is None else torch.from_numpy(b[1]).to(self.device)
        dw = torch.zeros(wk.shape, dtype=torch.float32, device=self.device)
        db = torch.zeros(L.cout, dtype=torch.float32, device=self.device) if L.bias else None
        tgp.bind_params(self.h, idx, wk.data_ptr(), None if bt is None else bt.data_ptr(),
                        dw.data_ptr(), None if db is None else db.data_ptr())
        self.params[idx] = {"w": wk, "b": bt, "dw": dw, "db": db, "w64": w64,
                            "b64": None if b is None else b[0]}

    def _set_bounds(self):
        self.balance = tgp.get_partition(self.h)
        self.n = len(self.balance)
        self.bounds = []
        lo = 0
        for c in self.balance:
            self.bounds.append((lo, lo + c))
            lo += c

    def layer_times(self, b: int, mode: int, iters: int = 3) -> List[float]:
        """Mean microseconds of F (+ F'), B and the accumulation of each layer
        for one micro-batch of b samples (tgp_layer_times).  Drops the plan."""
        nbytes = tgp.layer_times_plan(self.h, b, mode)
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        us = tgp.layer_times(self.h, ws.data_ptr(), ws.numel(), iters,
                             torch.cuda.current_stream().cuda_stream)
        self.ws = None
        return us

    def balance_by_time(self, b: int, n: int, mode: int, iters: int = 3):
        """Re-partitions into n parts on measured per-layer times
        (tgp_balance_by_time); returns (balance, per-layer microseconds).
        Drops the plan."""
        nbytes = tgp.layer_times_plan(self.h, b, mode)
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        bal, us = tgp.balance_by_time(self.h, ws.data_ptr(), ws.numel(), iters, n,
                                      torch.cuda.current_stream().cuda_stream)
        self.ws = None
        self._set_bounds()
        assert self.balance == bal
        return bal, us

    def plan(self, B: int, m: int, mode: int, lanes: int = 1) -> int:
        tgp.set_lanes(self.h, lanes)
        self.lanes = lanes
        self._lane_streams = None
        nbytes = tgp.plan(self.h, B, m, mode)
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        tgp.bind_workspace(self.h, self.ws.data_ptr(), self.ws.numel())
        self.B, self.m, self.b, self.mode = B, m, B // m, mode
        return nbytes

    def close(self):
        if self.h:
            tgp.net_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- shapes

    def part_in_shape(self, j: int):
        """(C, H, W) of partition j's input (pre-prologue)."""
        lo, _ = self.bounds[j - 1]
        if lo == 0:
            return (self.net.in_channels, self.net.height, self.net.width)
        h, w = self.shapes[lo - 1]
        return (self.net.layers[lo - 1].cout, h, w)

    def part_out_shape(self, j: int):
        _, hi = self.bounds[j - 1]
        h, w = self.shapes[hi - 1]
        return (self.net.layers[hi - 1].cout, h, w)

    def exported_stashes(self, j: int) -> List[int]:
        lo, hi = self.bounds[j - 1]
        made = [L.stash_id for L in self.net.layers[lo:hi] if L.stash_id >= 0]
        popped = {L.pop_id for L in self.net.layers[lo:hi] if L.pop_id >= 0}
        return sorted(s for s in made if s not in popped)

    def stash_shape(self, sid: int):
        idx = [k for k, L in enumerate(self.net.layers) if L.stash_id == sid][0]
        h, w = self.shapes[idx]
        return (self.net.layers[idx].cout, h, w)

    def stash_view(self, i: int, sid: int, grad: bool) -> torch.Tensor:
        c, h, w = self.stash_shape(sid)
        return wrap(tgp.stash_ptr(self.h, i, sid, grad), (self.b, h, w, c), self.dtype,
                    self.device)

    def esz(self) -> int:
        return 2 if self.dtype == BF16 else 4

    # ---------------------------------------------------------------- runs

    def checkpointed(self, i: int) -> bool:
        return self.mode == specs.CKPT_ALWAYS or (self.mode == specs.CKPT_EXCEPT_LAST and i < self.m)

    def stage_step(self, j: int, x: torch.Tensor, y: torch.Tensor, dy: torch.Tensor,
                   dx: Optional[torch.Tensor], stream: int = 0, serial: bool = False):
        """All m forwards of partition j, then backward + accumulate for
        i = m..1 (one stage's work per mini-batch).  Tensors are full-batch
        NHWC; micro-batch slices are pointer offsets.  With several lanes the
        micro-batches run on lane streams forked from torch's current stream
        (`stream` is then unused) unless `serial`, which issues everything on
        `stream` in order (`group` micro-batches per call when above 1)."""
        def sl(t, i):
            return t.data_ptr() + (i - 1) * (t.numel() // self.m) * t.element_size()
        if self.group > 1:
            return self._stage_step_groups(j, x, y, dy, dx, sl, stream if serial else None)
        if self.lanes > 1 and not serial:
            return self._stage_step_lanes(j, x, y, dy, dx, sl)
        for i in range(1, self.m + 1):
            tgp.stage_forward(self.h, j, i, self.checkpointed(i), sl(x, i), sl(y, i), stream)
        for i in range(self.m, 0, -1):
            tgp.stage_backward_recompute(self.h, j, i, sl(dy, i),
                                         None if dx is None else sl(dx, i), stream)
            tgp.grad_accumulate(self.h, j, i, i == self.m, stream)

    def _stage_step_lanes(self, j, x, y, dy, dx, sl):
        """stage_step with micro-batch i on lane stream (i - 1) % lanes and the
        accumulations, in the order m..1, on one more stream that waits for
        each backward; all forked from and joined back into the current
        stream.  Every cross-stream dependency points from a lane to the
        accumulation stream, never back."""
        cur = torch.cuda.current_stream()
        K = min(self.lanes, self.m)
        if self._lane_streams is None:
            self._lane_streams = [torch.cuda.Stream() for _ in range(K + 1)]
        lanes, acc = self._lane_streams[:K], self._lane_streams[K]
        for s in self._lane_streams:
            s.wait_stream(cur)
        for i in range(1, self.m + 1):
            s = lanes[(i - 1) % K]
            tgp.stage_forward(self.h, j, i, self.checkpointed(i), sl(x, i), sl(y, i), s.cuda_stream)
        # the events stay referenced until the next step
        self._events = []
        for i in range(self.m, 0, -1):
            s = lanes[(i - 1) % K]
            tgp.stage_backward_recompute(self.h, j, i, sl(dy, i), None if dx is None else sl(dx, i),
                                         s.cuda_stream)
            ev = torch.cuda.Event()
            ev.record(s)
            self._events.append(ev)
            acc.wait_event(ev)
            tgp.grad_accumulate(self.h, j, i, i == self.m, acc.cuda_stream)
        for s in self._lane_streams:
            cur.wait_stream(s)

    def _stage_step_groups(self, j, x, y, dy, dx, sl, serial_stream=None):
        """stage_step with G = `group` micro-batches per call: forwards
        (1..G), (G+1..2G), ..., backwards (m..m-G+1), ..., each group on the
        stream of its lanes, and each group's accumulations (one call, in
        the order m..1) on one more stream that waits for the group's
        backward (all on `serial_stream`, in that order, when given).  Needs
        G to divide the lanes and m."""
        G = self.group
        K = min(self.lanes, self.m)
        if K % G or self.m % G:
            raise ValueError(f"groups of {G} need lanes and m divisible by {G} "
                             f"(lanes={self.lanes}, m={self.m})")
        h = self.h

        def fwd(i, s):
            ks = range(G)
            tgp.stage_forward_n(h, j, i, [self.checkpointed(i + k) for k in ks],
                                [sl(x, i + k) for k in ks], [sl(y, i + k) for k in ks], s)

        def bwd(i, s):
            ks = range(G)
            tgp.stage_backward_recompute_n(h, j, i, [sl(dy, i - k) for k in ks],
                                           [None if dx is None else sl(dx, i - k) for k in ks], s)

        if serial_stream is not None:
            for i in range(1, self.m + 1, G):
                fwd(i, serial_stream)
            for i in range(self.m, 0, -G):
                bwd(i, serial_stream)
                tgp.grad_accumulate_n(h, j, i, G, i == self.m, serial_stream)
            return
        cur = torch.cuda.current_stream()
        if self._lane_streams is None:
            self._lane_streams = [torch.cuda.Stream() for _ in range(K // G + 1)]
        streams, acc = self._lane_streams[:K // G], self._lane_streams[K // G]
        for s in self._lane_streams:
            s.wait_stream(cur)

        def group_stream(i_lo):            # the group of micro-batches i_lo .. i_lo + G - 1
            return streams[((i_lo - 1) % K) // G]
        for i in range(1, self.m + 1, G):
            fwd(i, group_stream(i).cuda_stream)
        self._events = []
        for i in range(self.m, 0, -G):
            s = group_stream(i - G + 1)
            bwd(i, s.cuda_stream)
            ev = torch.cuda.Event()
            ev.record(s)
            self._events.append(ev)
            acc.wait_event(ev)
            tgp.grad_accumulate_n(h, j, i, G, i == self.m, acc.cuda_stream)
        for s in self._lane_streams:
            cur.wait_stream(s)

    def pipeline_step(self, x: torch.Tensor, target: torch.Tensor, loss: torch.Tensor,
                      y: Optional[torch.Tensor] = None, stream: int = 0):
        tgp.pipeline_step(self.h, x.data_ptr(), target.data_ptr(), self.B, self.m, self.n,
                          self.mode, loss.data_ptr(), None if y is None else y.data_ptr(),
                          stream)

    def grads64(self, layers: Optional[Sequence[int]] = None):
        """{idx: (dW as float64 OIHW, db as float64 or None)}"""
        out = {}
        for idx in (layers if layers is not None else sorted(self.params)):
            L = self.net.layers[idx]
            p = self.params[idx]
            dw = p["dw"].double().cpu()
            if L.kind == DWCONV3X3:
                dw = dw.reshape(L.cout, 1, 3, 3)
            else:
                dw = dw.permute(0, 3, 1, 2)
            out[idx] = (dw.contiguous().numpy(),
                        None if p["db"] is None else p["db"].double().cpu().numpy())
        return out
