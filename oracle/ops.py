"""Oracle operators: plain float64 NCHW definitions of every layer operation.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
package; only tests, the smoke check and the benchmark's CPU-baseline leg do.

Each forward op is written straight from its textbook definition; each
backward op is the vector-Jacobian product of that definition (the paper's
partial_x f and partial_theta f of Sec. 2, eq. (B_ij)), written as the exact
adjoint of the forward loop.  A library matmul (numpy.tensordot, in float64) is the only
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


# ---------------------------------------------------------------- convolution
# Cross-correlation, stride 1, zero padding 1 for 3x3 and 0 for 1x1:
#   z[n,o,h,w] = b[o] + sum_{c,r,s} W[o,c,r,s] * x[n,c,h+r-1,w+s-1]

def _pad1(x):
    return np.pad(x, ((0, 0), (0, 0), (1, 1), (1, 1)))


def conv3x3_forward(x, w, b=None):
    n, c, h, wd = x.shape
    xp = _pad1(x)
    z = np.zeros((n, w.shape[0], h, wd), dtype=np.float64)
    for r in range(3):
        for s in range(3):
            t = np.tensordot(w[:, :, r, s], xp[:, :, r:r + h, s:s + wd], axes=([1], [1]))
            z += t.transpose(1, 0, 2, 3)
    if b is not None:
        z += b[None, :, None, None]
    return z


def conv3x3_dgrad(dz, w):
    """dx[n,c,h',w'] = sum_{o,r,s} dz[n,o,h'-r+1,w'-s+1] W[o,c,r,s]: the adjoint
    of the forward, scattered tap by tap into a padded buffer."""
    n, o, h, wd = dz.shape
    dxp = np.zeros((n, w.shape[1], h + 2, wd + 2), dtype=np.float64)
    for r in range(3):
        for s in range(3):
            t = np.tensordot(w[:, :, r, s], dz, axes=([0], [1]))  # (c, n, h, w)
            dxp[:, :, r:r + h, s:s + wd] += t.transpose(1, 0, 2, 3)
    return dxp[:, :, 1:-1, 1:-1]


def conv3x3_wgrad(x, dz):
    """dW[o,c,r,s] = sum_{n,h,w} dz[n,o,h,w] x[n,c,h+r-1,w+s-1]."""
    n, c, h, wd = x.shape
    xp = _pad1(x)
    dw = np.zeros((dz.shape[1], c, 3, 3))
    for r in range(3):
        for s in range(3):
            dw[:, :, r, s] = np.tensordot(dz, xp[:, :, r:r + h, s:s + wd], axes=([0, 2, 3], [0, 2, 3]))
    return dw


def conv1x1_forward(x, w, b=None):
    z = np.tensordot(w[:, :, 0, 0], x, axes=([1], [1])).transpose(1, 0, 2, 3)
    if b is not None:
        z = z + b[None, :, None, None]
    return z


def conv1x1_dgrad(dz, w):
    return np.tensordot(w[:, :, 0, 0], dz, axes=([0], [1])).transpose(1, 0, 2, 3)


def conv1x1_wgrad(x, dz):
    return np.tensordot(dz, x, axes=([0, 2, 3], [0, 2, 3]))[:, :, None, None]


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
