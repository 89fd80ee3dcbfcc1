"""Network structures and workload shapes shared by the HIP path's harness and
the oracle.  This module holds structure only (layer lists, sizes, modes); it
does no arithmetic of the method.

A network is the paper's sequence of black-box layers (Sec. 3, "Users must
specify ... a sequence of layers"), cut into n contiguous partitions
f^1..f^n (Sec. 2).  Each layer is one convolution with an optional prologue
that reshapes its input first:

  NONE     input = previous layer output
  MAXPOOL2 input = 2x2/2 max-pool of the previous layer output
  UPCAT2   input = channel concat [nearest 2x upsample(previous output),
                                   popped skip tensor]

A layer may stash its output under a skip id (Sec. 3.3, long skip
connections) so that a later UPCAT2 layer pops it.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional, Tuple

# layer kinds (values are the C-ABI enum values)
CONV3X3 = 0
CONV1X1 = 1
DWCONV3X3 = 2

# prologues
PRO_NONE = 0
PRO_MAXPOOL2 = 1
PRO_UPCAT2 = 2

# checkpoint modes (Sec. 2.1: checkpoint every micro-batch, or all but the last)
CKPT_ALWAYS = 0
CKPT_EXCEPT_LAST = 1
CKPT_NEVER = 2
CKPT_NAMES = {"always": CKPT_ALWAYS, "except_last": CKPT_EXCEPT_LAST, "never": CKPT_NEVER}

# dtypes
BF16 = 0
FP32 = 1


@dataclass(frozen=True)
class Layer:
    kind: int
    cin: int
    cout: int
    relu: bool = True
    bias: bool = True
    prologue: int = PRO_NONE
    stash_id: int = -1
    pop_id: int = -1
    name: str = ""

    @property
    def taps(self) -> int:
        return 1 if self.kind == CONV1X1 else 9

    def weight_shape(self) -> Tuple[int, ...]:
        """Logical OIHW weight shape (depthwise: C x 1 x 3 x 3)."""
        if self.kind == DWCONV3X3:
            return (self.cout, 1, 3, 3)
        k = 1 if self.kind == CONV1X1 else 3
        return (self.cout, self.cin, k, k)

    def fan_in(self) -> int:
        if self.kind == DWCONV3X3:
            return 9
        return self.cin * self.taps


@dataclass(frozen=True)
class Net:
    name: str
    layers: Tuple[Layer, ...]
    in_channels: int
    height: int
    width: int

    def shapes(self):
        """Per layer: (H, W) of the layer's input after its prologue, which is
        also its output size (all convolutions are stride 1, 'same')."""
        out = []
        h, w = self.height, self.width
        for L in self.layers:
            if L.prologue == PRO_MAXPOOL2:
                h, w = h // 2, w // 2
            elif L.prologue == PRO_UPCAT2:
                h, w = h * 2, w * 2
            out.append((h, w))
        return out

    def check(self) -> None:
        c = self.in_channels
        stash_c = {}
        h, w = self.height, self.width
        for idx, L in enumerate(self.layers):
            if L.prologue == PRO_MAXPOOL2:
                assert h % 2 == 0 and w % 2 == 0, (self.name, idx)
                h, w = h // 2, w // 2
                want = c
            elif L.prologue == PRO_UPCAT2:
                h, w = h * 2, w * 2
                sc, sh, sw = stash_c[L.pop_id]
                assert (sh, sw) == (h, w), (self.name, idx)
                want = c + sc
            else:
                want = c
            assert L.cin == want, (self.name, idx, L.cin, want)
            if L.kind == DWCONV3X3:
                assert L.cin == L.cout
            c = L.cout
            if L.stash_id >= 0:
                stash_c[L.stash_id] = (c, h, w)

    def flops_per_sample(self) -> List[int]:
        """Forward multiply-add FLOPs (2 per MAC) per layer per sample."""
        out = []
        for L, (h, w) in zip(self.layers, self.shapes()):
            if L.kind == DWCONV3X3:
                out.append(2 * h * w * L.cout * 9)
            else:
                out.append(2 * h * w * L.cout * L.cin * L.taps)
        return out

    def out_channels(self) -> int:
        return self.layers[-1].cout

    def out_hw(self) -> Tuple[int, int]:
        return self.shapes()[-1]


def plain_stack(n_layers: int, c: int, h: int, w: int, name="stack") -> Net:
    layers = tuple(Layer(CONV3X3, c, c, name=f"conv{i}") for i in range(n_layers))
    return Net(name, layers, c, h, w)


def unet(levels: int, base: int, in_ch: int, hw: int, name="unet", head=True,
         blocks: int = 2) -> Net:
    """Symmetric U-Net: per level `blocks` conv3x3+bias+ReLU (two in every
    benchmark network); max-pool between encoder levels; decoder level l =
    nearest 2x upsample of level l+1, concat with the stashed encoder output
    of level l, then `blocks` conv3x3+ReLU; a 1x1 head to one channel without
    ReLU.  Channels double at each down-sampling (base at level 0)."""
    assert blocks >= 1
    C = [base * (2 ** l) for l in range(levels)]

    def nm(prefix, k):
        return f"{prefix}{chr(ord('a') + k)}" if k < 26 else f"{prefix}_{k}"

    layers = []
    prev = in_ch
    for l in range(levels):
        for k in range(blocks):
            pro = PRO_MAXPOOL2 if (l > 0 and k == 0) else PRO_NONE
            stash = l if (k == blocks - 1 and l < levels - 1) else -1
            layers.append(Layer(CONV3X3, prev if k == 0 else C[l], C[l], prologue=pro,
                                stash_id=stash, name=nm(f"enc{l}", k)))
        prev = C[l]
    for l in range(levels - 2, -1, -1):
        for k in range(blocks):
            if k == 0:
                layers.append(Layer(CONV3X3, prev + C[l], C[l], prologue=PRO_UPCAT2, pop_id=l,
                                    name=nm(f"dec{l}", 0)))
            else:
                layers.append(Layer(CONV3X3, C[l], C[l], name=nm(f"dec{l}", k)))
        prev = C[l]
    if head:
        layers.append(Layer(CONV1X1, prev, 1, relu=False, name="head"))
    net = Net(name, tuple(layers), in_ch, hw, hw)
    net.check()
    return net


def amoeba_cells(n_cells: int, c: int, hw: int, name="cells") -> Net:
    """Cell = depthwise 3x3 (no bias, no ReLU) -> pointwise 1x1 + bias -> ReLU."""
    layers = []
    for i in range(n_cells):
        layers.append(Layer(DWCONV3X3, c, c, relu=False, bias=False, name=f"cell{i}.dw"))
        layers.append(Layer(CONV1X1, c, c, name=f"cell{i}.pw"))
    net = Net(name, tuple(layers), c, hw, hw)
    net.check()
    return net


def subnet(net: Net, lo: int, hi: int, name: Optional[str] = None) -> Net:
    """Layers [lo, hi) of `net` as a network of their own (a partition run as a
    stage).  Input size and channels are those of layer lo's pre-prologue
    input."""
    shapes = net.shapes()
    if lo == 0:
        in_c, h, w = net.in_channels, net.height, net.width
    else:
        in_c = net.layers[lo - 1].cout
        h, w = shapes[lo - 1]
    return Net(name or f"{net.name}[{lo}:{hi}]", tuple(net.layers[lo:hi]), in_c, h, w)


@dataclass(frozen=True)
class Workload:
    name: str
    net: Net
    batch: int
    m: int
    n: int
    mode: int
    dtype: int
    # 'network': MSE loss on the final output against a seeded target.
    # 'stage'  : partition `stage_j` of the n-way split runs alone with seeded
    #            upstream gradients for its main output and exported skips.
    kind: str = "network"
    stage_j: int = 1
    balance: Optional[Tuple[int, ...]] = None

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def tiny() -> Workload:
    """4-layer conv3x3+bias+ReLU stack, C=16, 8x16x32x32 fp32, m=4, n=2, always."""
    return Workload("tiny-stack", plain_stack(4, 16, 32, 32, "stack4-c16"), 8, 4, 2,
                    CKPT_ALWAYS, FP32)


def unet_stage() -> Workload:
    """Partition 1 of 4 of the 5-level U-Net (base 64 -> 1024), input
    32x64x192x192 bf16, m=8, always."""
    return Workload("unet5-stage1of4", unet(5, 64, 64, 192, "unet5-c64"), 32, 8, 4,
                    CKPT_ALWAYS, BF16, kind="stage", stage_j=1)


def unet_network() -> Workload:
    return Workload("unet5-network", unet(5, 64, 64, 192, "unet5-c64"), 32, 8, 4,
                    CKPT_ALWAYS, BF16)


def amoeba_stage() -> Workload:
    """18 cells of [dw3x3, pw1x1+bias, ReLU] at C=256, 128x256x56x56 bf16,
    m=32, except-last, one partition."""
    return Workload("amoeba18-c256-stage", amoeba_cells(18, 256, 56, "cells18-c256"), 128,
                    32, 1, CKPT_EXCEPT_LAST, BF16, kind="stage", stage_j=1)


def large_unet() -> Workload:
    """6-level U-Net, base 128 -> 4096, input 64x128x256x256 bf16, m=32, n=8."""
    return Workload("unet6-c128-network", unet(6, 128, 128, 256, "unet6-c128"), 64, 32, 8,
                    CKPT_ALWAYS, BF16)


def sweep():
    """Checkpoint / micro-batch sweep over the 5-level U-Net network."""
    base = unet_network()
    out = []
    for m in (1, 4, 16, 32):
        for mode in ("always", "except_last", "never"):
            out.append(base.with_(name=f"unet5-network-m{m}-{mode}", m=m,
                                  mode=CKPT_NAMES[mode]))
    return out


ALL = {w.name: w for w in (tiny(), unet_stage(), unet_network(), amoeba_stage(), large_unet())}
