"""Oracle operators: plain float64 NCHW definitions of every layer operation.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
package; only tests, the smoke check and the benchmark's CPU-baseline leg do.

Each forward op is written straight from its textbook definition; each
backward op is the vector-Jacobian product of that definition (the paper's
partial_x f and partial_theta f of Sec. 2, eq. (B_ij)), written as the exact
adjoint of the forward loop.  A library matmul (numpy.tensordot) is the only
primitive used, and only for the sum over channels at one filter tap.
"""
from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------- rounding

def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (via float32, nearest-even at each
    step) and return them as float64.  Used only by the bf16-storage mode,
    which rounds exactly where a bf16 run stores a tensor."""
    a32 = np.asarray(a, dtype=np.float64).astype(np.float32)
    u = a32.view(np.uint32).astype(np.uint64)
    keep = (u >> np.uint64(16)) & np.uint64(1)
    u = (u + np.uint64(0x7FFF) + keep) >> np.uint64(16) << np.uint64(16)
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- contraction precision
# Parity references always contract in float64.  A float32 contraction mode
# exists only to measure how far two equally valid bf16-storage computations
# of a deep ReLU network drift apart when their summation precision differs
# (ReLU masks and pool argmaxes taken on values that differ in the last bf16
# bit flip, and each flip moves a whole upstream gradient element).

_CONTRACT = ["f64"]
CONTRACTIONS = ("f64", "f32", "f32rev", "f32split", "f32c32")


class contraction:
    """Context for the channel contraction used by the conv ops:
    'f64'      float64 (every parity reference);
    'f32'      float32 operands and accumulation;
    'f32rev'   float32 with the contracted channel order reversed;
    'f32split' float32 in two halves of the channels, added at the end;
    'f32c32'   float32 in blocks of 32 channels, the block sums added one by
               one in channel order (the blocking of a K loop that contracts
               32 channels per step).
    The float32 variants are equally valid ways to evaluate the same
    bf16-storage network; the spread among them and the float64 reference
    measures how many ReLU / pool decisions are within rounding distance of
    flipping."""

    def __init__(self, mode):
        assert mode in CONTRACTIONS
        self.mode = mode

    def __enter__(self):
        _CONTRACT.append(self.mode)

    def __exit__(self, *exc):
        _CONTRACT.pop()


def _td(a, b, axes):
    mode = _CONTRACT[-1]
    if mode == "f64":
        return np.tensordot(a, b, axes=axes)
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    ax_a, ax_b = axes
    k = ax_a[0]
    if mode == "f32rev":
        a = np.flip(a, axis=k)
        b = np.flip(b, axis=ax_b[0])
    if mode == "f32c32" and a.shape[k] > 32:
        out = None
        for c0 in range(0, a.shape[k], 32):
            sa = [slice(None)] * a.ndim
            sb = [slice(None)] * b.ndim
            sa[k], sb[ax_b[0]] = slice(c0, c0 + 32), slice(c0, c0 + 32)
            t = np.tensordot(a[tuple(sa)], b[tuple(sb)], axes=axes)
            out = t if out is None else out + t
        return out
    if mode == "f32split" and a.shape[k] > 1:
        h = a.shape[k] // 2
        sa = [slice(None)] * a.ndim
        sb = [slice(None)] * b.ndim
        sa[k], sb[ax_b[0]] = slice(0, h), slice(0, h)
        lo = np.tensordot(a[tuple(sa)], b[tuple(sb)], axes=axes)
        sa[k], sb[ax_b[0]] = slice(h, None), slice(h, None)
        hi = np.tensordot(a[tuple(sa)], b[tuple(sb)], axes=axes)
        return lo + hi
    return np.tensordot(a, b, axes=axes)


def _acc():
    """Accumulator type of the conv sums over taps: float64, or float32 in
    the float32 contraction variants (as a float32-accumulating kernel)."""
    return np.float64 if _CONTRACT[-1] == "f64" else np.float32


# ---------------------------------------------------------------- convolution
# Cross-correlation, stride 1, zero padding 1 for 3x3 and 0 for 1x1:
#   z[n,o,h,w] = b[o] + sum_{c,r,s} W[o,c,r,s] * x[n,c,h+r-1,w+s-1]

def _pad1(x):
    return np.pad(x, ((0, 0), (0, 0), (1, 1), (1, 1)))


def conv3x3_forward(x, w, b=None):
    n, c, h, wd = x.shape
    xp = _pad1(x)
    z = np.zeros((n, w.shape[0], h, wd), dtype=_acc())
    for r in range(3):
        for s in range(3):
            t = _td(w[:, :, r, s], xp[:, :, r:r + h, s:s + wd], axes=([1], [1]))
            z += t.transpose(1, 0, 2, 3)
    if b is not None:
        z += b[None, :, None, None].astype(z.dtype)
    return z.astype(np.float64)


def conv3x3_dgrad(dz, w):
    """dx[n,c,h',w'] = sum_{o,r,s} dz[n,o,h'-r+1,w'-s+1] W[o,c,r,s]: the adjoint
    of the forward, scattered tap by tap into a padded buffer."""
    n, o, h, wd = dz.shape
    dxp = np.zeros((n, w.shape[1], h + 2, wd + 2), dtype=_acc())
    for r in range(3):
        for s in range(3):
            t = _td(w[:, :, r, s], dz, axes=([0], [1]))  # (c, n, h, w)
            dxp[:, :, r:r + h, s:s + wd] += t.transpose(1, 0, 2, 3)
    return dxp[:, :, 1:-1, 1:-1].astype(np.float64)


def conv3x3_wgrad(x, dz):
    """dW[o,c,r,s] = sum_{n,h,w} dz[n,o,h,w] x[n,c,h+r-1,w+s-1]."""
    n, c, h, wd = x.shape
    xp = _pad1(x)
    dw = np.zeros((dz.shape[1], c, 3, 3))
    for r in range(3):
        for s in range(3):
            dw[:, :, r, s] = _td(dz, xp[:, :, r:r + h, s:s + wd], axes=([0, 2, 3], [0, 2, 3]))
    return dw.astype(np.float64)


def conv1x1_forward(x, w, b=None):
    z = _td(w[:, :, 0, 0], x, axes=([1], [1])).transpose(1, 0, 2, 3)
    if b is not None:
        z = z + b[None, :, None, None].astype(z.dtype)
    return z.astype(np.float64)


def conv1x1_dgrad(dz, w):
    return _td(w[:, :, 0, 0], dz, axes=([0], [1])).transpose(1, 0, 2, 3).astype(np.float64)


def conv1x1_wgrad(x, dz):
    return _td(dz, x, axes=([0, 2, 3], [0, 2, 3]))[:, :, None, None].astype(np.float64)


# depthwise 3x3, pad 1, no channel mixing:
#   z[n,c,h,w] = sum_{r,s} W[c,0,r,s] * x[n,c,h+r-1,w+s-1]

def dwconv3x3_forward(x, w, b=None):
    n, c, h, wd = x.shape
    xp = _pad1(x)
    z = np.zeros_like(x)
    for r in range(3):
        for s in range(3):
            z += w[None, :, 0, r, s, None, None] * xp[:, :, r:r + h, s:s + wd]
    if b is not None:
        z += b[None, :, None, None]
    return z


def dwconv3x3_dgrad(dz, w):
    n, c, h, wd = dz.shape
    dxp = np.zeros((n, c, h + 2, wd + 2))
    for r in range(3):
        for s in range(3):
            dxp[:, :, r:r + h, s:s + wd] += w[None, :, 0, r, s, None, None] * dz
    return dxp[:, :, 1:-1, 1:-1]


def dwconv3x3_wgrad(x, dz):
    n, c, h, wd = x.shape
    xp = _pad1(x)
    dw = np.zeros((c, 1, 3, 3))
    for r in range(3):
        for s in range(3):
            dw[:, 0, r, s] = np.sum(dz * xp[:, :, r:r + h, s:s + wd], axis=(0, 2, 3))
    return dw


def bias_grad(dz):
    """db[o] = sum_{n,h,w} dz[n,o,h,w]."""
    return dz.sum(axis=(0, 2, 3))


# ---------------------------------------------------------------- pooling

def maxpool2_forward(x):
    """2x2 window, stride 2.  Returns (y, argmax) where argmax in 0..3 indexes
    the window in row-major order (dh*2 + dw); ties go to the first index."""
    n, c, h, w = x.shape
    win = x.reshape(n, c, h // 2, 2, w // 2, 2).transpose(0, 1, 2, 4, 3, 5)
    win = win.reshape(n, c, h // 2, w // 2, 4)
    arg = np.argmax(win, axis=-1)  # numpy returns the first maximal index
    y = np.take_along_axis(win, arg[..., None], axis=-1)[..., 0]
    return y, arg


def maxpool2_backward(dy, arg):
    """Route each output gradient to its window's argmax element."""
    n, c, h2, w2 = dy.shape
    win = np.zeros((n, c, h2, w2, 4))
    np.put_along_axis(win, arg[..., None], dy[..., None], axis=-1)
    win = win.reshape(n, c, h2, w2, 2, 2).transpose(0, 1, 2, 4, 3, 5)
    return win.reshape(n, c, 2 * h2, 2 * w2)


# ---------------------------------------------------------------- upsample

def upsample2_forward(x):
    """Nearest neighbour: u[n,c,h,w] = x[n,c,h//2,w//2]."""
    return np.repeat(np.repeat(x, 2, axis=2), 2, axis=3)


def upsample2_backward(du):
    """Adjoint of nearest 2x upsampling: sum over each 2x2 block."""
    n, c, h, w = du.shape
    return du.reshape(n, c, h // 2, 2, w // 2, 2).sum(axis=(3, 5))


# ---------------------------------------------------------------- loss

def mse(y, t, numel):
    """L = sum (y-t)^2 / numel over the full mini-batch; dL/dy = 2 (y-t)/numel."""
    d = y - t
    return float(np.sum(d * d) / numel), 2.0 * d / numel
