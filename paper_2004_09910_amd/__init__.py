"""Python binding of libtgp.so, the MI355X micro-batch pipeline stage with
checkpointing (C ABI in include/tgp.h).

Argument marshalling only: every step of the method runs in the library's
HIP kernels.  Device buffers are passed as integer device addresses (for
example torch tensors' data_ptr()), streams as integer hipStream_t handles.
Importing fails loudly when the library has not been built; there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtgp.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2004_09910_amd/build.py`")

# torch ships its own HIP runtime.  Load it before libtgp.so so that the
# library's libamdhip64.so.7 dependency resolves to that same, already loaded
# runtime: two HIP runtimes in one process do not see each other's devices,
# streams or memory.
try:
    import torch  # noqa: F401
except ImportError:  # host-only use (schedule trace, partitioner, validation)
    pass

_lib = ctypes.CDLL(LIB_PATH)

OK, EINVAL, ESTATE, ENOSPACE, EHIP, EUNSUPPORTED = range(6)
STATUS_NAMES = {0: "OK", 1: "EINVAL", 2: "ESTATE", 3: "ENOSPACE", 4: "EHIP", 5: "EUNSUPPORTED"}
BF16, FP32 = 0, 1
CKPT_ALWAYS, CKPT_EXCEPT_LAST, CKPT_NEVER = 0, 1, 2
OP_FORWARD, OP_RECOMPUTE, OP_BACKWARD, OP_ACCUMULATE, OP_LOSS = range(5)


class TgpError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("cin", ctypes.c_int32), ("cout", ctypes.c_int32),
                ("relu", ctypes.c_int32), ("bias", ctypes.c_int32), ("prologue", ctypes.c_int32),
                ("stash_id", ctypes.c_int32), ("pop_id", ctypes.c_int32)]


_P = ctypes.c_void_p
_I = ctypes.c_int
_SIG = {
    "tgp_net_create": [ctypes.POINTER(Layer), _I, _I, _I, _I, _I, ctypes.POINTER(_P)],
    "tgp_layer_flops": [_P, _I, ctypes.POINTER(ctypes.c_int64)],
    "tgp_set_partition": [_P, _I, ctypes.POINTER(_I)],
    "tgp_get_partition": [_P, ctypes.POINTER(_I), ctypes.POINTER(_I)],
    "tgp_balance_minmax": [ctypes.POINTER(ctypes.c_int64), _I, _I, ctypes.POINTER(_I)],
    "tgp_bind_params": [_P, _I, _P, _P, _P, _P],
    "tgp_plan": [_P, _I, _I, _I, ctypes.POINTER(ctypes.c_size_t)],
    "tgp_bind_workspace": [_P, _P, ctypes.c_size_t],
    "tgp_stash_ptr": [_P, _I, _I, _I, ctypes.POINTER(_P)],
    "tgp_stage_forward": [_P, _I, _I, _I, _P, _P, _P],
    "tgp_stage_backward_recompute": [_P, _I, _I, _P, _P, _P],
    "tgp_grad_accumulate": [_P, _I, _I, _I, _P],
    "tgp_grad_accumulate_n": [_P, _I, _I, _I, _I, _P],
    "tgp_pipeline_step": [_P, _P, _P, _I, _I, _I, _I, _P, _P, _P],
    "tgp_pipeline_step_static": [_P, _P, _P, _I, _I, _I, _I, _P, _P, _P],
    "tgp_schedule_trace": [_I, _I, _I, ctypes.POINTER(ctypes.c_int32), _I, ctypes.POINTER(_I)],
    "tgp_stage_forward2": [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P],
    "tgp_stage_backward_recompute2": [_P, _I, _I, _I, _P, _P, _P, _P, _P],
    "tgp_stage_forward_n": [_P, _I, _I, _I, ctypes.POINTER(_I), ctypes.POINTER(_P),
                            ctypes.POINTER(_P), _P],
    "tgp_stage_backward_recompute_n": [_P, _I, _I, _I, ctypes.POINTER(_P), ctypes.POINTER(_P),
                                       _P],
    "tgp_layer_times_plan": [_P, _I, _I, ctypes.POINTER(ctypes.c_size_t)],
    "tgp_layer_times": [_P, _P, ctypes.c_size_t, _I, ctypes.POINTER(ctypes.c_float), _P],
    "tgp_balance_by_time": [_P, _P, ctypes.c_size_t, _I, _I, ctypes.POINTER(_I),
                            ctypes.POINTER(ctypes.c_float), _P],
}
for _name, _args in _SIG.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = ctypes.c_int


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 96), ("launches", ctypes.c_int64),
                ("ms", ctypes.c_double), ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


_lib.tgp_profile_enable.argtypes = [_I]
_lib.tgp_profile_enable.restype = ctypes.c_int
_lib.tgp_profile_read.argtypes = [ctypes.POINTER(KernelStat), _I, ctypes.POINTER(_I)]
_lib.tgp_profile_read.restype = ctypes.c_int
_lib.tgp_profile_clear.argtypes = []
_lib.tgp_profile_clear.restype = ctypes.c_int
_lib.tgp_set_lanes.argtypes = [_P, _I]
_lib.tgp_set_lanes.restype = ctypes.c_int
_lib.tgp_debug_set_fwd_variant.argtypes = [_I]
_lib.tgp_debug_set_fwd_variant.restype = _I
_lib.tgp_debug_set_rowtile_mask.argtypes = [_I]
_lib.tgp_debug_set_rowtile_mask.restype = _I
_lib.tgp_debug_fail_launch.argtypes = [_I]
_lib.tgp_debug_fail_launch.restype = _I
_lib.tgp_net_destroy.argtypes = [_P]
_lib.tgp_net_destroy.restype = None
_lib.tgp_last_error.argtypes = []
_lib.tgp_last_error.restype = ctypes.c_char_p


def last_error() -> str:
    return _lib.tgp_last_error().decode()


def _check(status: int, where: str) -> None:
    if status != OK:
        raise TgpError(status, where, last_error())


def call_status(name: str, *args) -> int:
    """Calls a tgp_* entry point and returns its raw status (for tests of the
    error paths)."""
    return getattr(_lib, name)(*args)


def _vp(x) -> Optional[int]:
    return None if x is None or x == 0 else int(x)


def net_create(layers: Sequence[Tuple[int, ...]], in_c: int, H: int, W: int, dtype: int) -> int:
    arr = (Layer * len(layers))(*[Layer(*map(int, l)) for l in layers])
    h = _P()
    _check(_lib.tgp_net_create(arr, len(layers), in_c, H, W, dtype, ctypes.byref(h)),
           "tgp_net_create")
    return h.value


def net_destroy(net: int) -> None:
    _lib.tgp_net_destroy(net)


def layer_flops(net: int, layer: int) -> int:
    v = ctypes.c_int64()
    _check(_lib.tgp_layer_flops(net, layer, ctypes.byref(v)), "tgp_layer_flops")
    return v.value


def set_partition(net: int, n: int, balance: Optional[Sequence[int]] = None) -> None:
    arr = None if balance is None else (_I * n)(*balance)
    _check(_lib.tgp_set_partition(net, n, arr), "tgp_set_partition")


def get_partition(net: int) -> List[int]:
    n = _I()
    bal = (_I * 4096)()
    _check(_lib.tgp_get_partition(net, ctypes.byref(n), bal), "tgp_get_partition")
    return list(bal[:n.value])


def balance_minmax(cost: Sequence[int], n: int) -> List[int]:
    c = (ctypes.c_int64 * len(cost))(*cost)
    out = (_I * n)()
    _check(_lib.tgp_balance_minmax(c, len(cost), n, out), "tgp_balance_minmax")
    return list(out)


def layer_times_plan(net: int, b: int, ckpt_mode: int) -> int:
    v = ctypes.c_size_t()
    _check(_lib.tgp_layer_times_plan(net, b, ckpt_mode, ctypes.byref(v)), "tgp_layer_times_plan")
    return v.value


def _n_layers(net: int) -> int:
    return sum(get_partition(net))


def layer_times(net: int, ws: int, nbytes: int, iters: int, stream: int = 0) -> List[float]:
    us = (ctypes.c_float * _n_layers(net))()
    _check(_lib.tgp_layer_times(net, _vp(ws), nbytes, iters, us, _vp(stream)), "tgp_layer_times")
    return list(us)


def balance_by_time(net: int, ws: int, nbytes: int, iters: int, n: int,
                    stream: int = 0) -> Tuple[List[int], List[float]]:
    us = (ctypes.c_float * _n_layers(net))()
    out = (_I * n)()
    _check(_lib.tgp_balance_by_time(net, _vp(ws), nbytes, iters, n, out, us, _vp(stream)),
           "tgp_balance_by_time")
    return list(out), list(us)


def bind_params(net: int, layer: int, w: int, b: Optional[int], dw_acc: int,
                db_acc: Optional[int]) -> None:
    _check(_lib.tgp_bind_params(net, layer, _vp(w), _vp(b), _vp(dw_acc), _vp(db_acc)),
           "tgp_bind_params")


def set_lanes(net: int, lanes: int) -> None:
    _check(_lib.tgp_set_lanes(net, int(lanes)), "tgp_set_lanes")


def plan(net: int, B: int, m: int, ckpt_mode: int) -> int:
    v = ctypes.c_size_t()
    _check(_lib.tgp_plan(net, B, m, ckpt_mode, ctypes.byref(v)), "tgp_plan")
    return v.value


def bind_workspace(net: int, ptr: int, nbytes: int) -> None:
    _check(_lib.tgp_bind_workspace(net, _vp(ptr), nbytes), "tgp_bind_workspace")


def stash_ptr(net: int, i: int, stash_id: int, grad: bool) -> int:
    p = _P()
    _check(_lib.tgp_stash_ptr(net, i, stash_id, int(grad), ctypes.byref(p)), "tgp_stash_ptr")
    return p.value


def stage_forward(net: int, j: int, i: int, checkpoint: bool, x_in: int, y_out: int,
                  stream: int = 0) -> None:
    _check(_lib.tgp_stage_forward(net, j, i, int(checkpoint), _vp(x_in), _vp(y_out),
                                  _vp(stream)), "tgp_stage_forward")


def stage_backward_recompute(net: int, j: int, i: int, dy_out: int, dx_in: Optional[int],
                             stream: int = 0) -> None:
    _check(_lib.tgp_stage_backward_recompute(net, j, i, _vp(dy_out), _vp(dx_in), _vp(stream)),
           "tgp_stage_backward_recompute")


def stage_forward2(net: int, j: int, i0: int, i1: int, checkpoint0: bool, checkpoint1: bool,
                   x0: int, x1: int, y0: int, y1: int, stream: int = 0) -> None:
    _check(_lib.tgp_stage_forward2(net, j, i0, i1, int(checkpoint0), int(checkpoint1),
                                   _vp(x0), _vp(x1), _vp(y0), _vp(y1), _vp(stream)),
           "tgp_stage_forward2")


def stage_backward_recompute2(net: int, j: int, i0: int, i1: int, dy0: int, dy1: int,
                              dx0: Optional[int], dx1: Optional[int], stream: int = 0) -> None:
    _check(_lib.tgp_stage_backward_recompute2(net, j, i0, i1, _vp(dy0), _vp(dy1), _vp(dx0),
                                              _vp(dx1), _vp(stream)),
           "tgp_stage_backward_recompute2")


def stage_forward_n(net: int, j: int, i0: int, checkpoints: Sequence[bool], xs: Sequence[int],
                    ys: Sequence[int], stream: int = 0) -> None:
    """F_{i,j} for i = i0 .. i0 + len(xs) - 1 (element k: micro-batch i0 + k)."""
    n = len(xs)
    _check(_lib.tgp_stage_forward_n(net, j, i0, n, (_I * n)(*[int(c) for c in checkpoints]),
                                    (_P * n)(*[_vp(x) for x in xs]),
                                    (_P * n)(*[_vp(y) for y in ys]), _vp(stream)),
           "tgp_stage_forward_n")


def stage_backward_recompute_n(net: int, j: int, i0: int, dys: Sequence[int],
                               dxs: Sequence[Optional[int]], stream: int = 0) -> None:
    """F'_{i,j} + B_{i,j} for i = i0, i0 - 1, .. (element k: micro-batch i0 - k)."""
    n = len(dys)
    _check(_lib.tgp_stage_backward_recompute_n(net, j, i0, n, (_P * n)(*[_vp(d) for d in dys]),
                                               (_P * n)(*[_vp(d) for d in dxs]), _vp(stream)),
           "tgp_stage_backward_recompute_n")


def grad_accumulate(net: int, j: int, i: int, overwrite: bool, stream: int = 0) -> None:
    _check(_lib.tgp_grad_accumulate(net, j, i, int(overwrite), _vp(stream)),
           "tgp_grad_accumulate")


def grad_accumulate_n(net: int, j: int, i0: int, count: int, overwrite: bool,
                      stream: int = 0) -> None:
    """The accumulations of micro-batches i0, i0 - 1, .., i0 - count + 1."""
    _check(_lib.tgp_grad_accumulate_n(net, j, i0, count, int(overwrite), _vp(stream)),
           "tgp_grad_accumulate_n")


def pipeline_step(net: int, x: int, target: int, B: int, m: int, n: int, ckpt_mode: int,
                  loss_dev: int, y_out: Optional[int] = None, stream: int = 0) -> None:
    _check(_lib.tgp_pipeline_step(net, _vp(x), _vp(target), B, m, n, ckpt_mode, _vp(loss_dev),
                                  _vp(y_out), _vp(stream)), "tgp_pipeline_step")


STATIC_SCRATCH_BYTES = 64 << 20   # TGP_STATIC_SCRATCH_BYTES


def pipeline_step_static(net: int, x: int, target: int, B: int, m: int, n: int, ckpt_mode: int,
                         loss_dev: int, y_out: Optional[int] = None, stream: int = 0) -> None:
    """tgp_pipeline_step on the library's static device scratch (no bound
    workspace, no allocation; one lane)."""
    _check(_lib.tgp_pipeline_step_static(net, _vp(x), _vp(target), B, m, n, ckpt_mode,
                                         _vp(loss_dev), _vp(y_out), _vp(stream)),
           "tgp_pipeline_step_static")


def schedule_trace(m: int, n: int, ckpt_mode: int) -> List[Tuple[int, int, int]]:
    cnt = _I()
    _lib.tgp_schedule_trace(m, n, ckpt_mode, None, 0, ctypes.byref(cnt))
    buf = (ctypes.c_int32 * (3 * max(cnt.value, 1)))()
    _check(_lib.tgp_schedule_trace(m, n, ckpt_mode, buf, cnt.value, ctypes.byref(cnt)),
           "tgp_schedule_trace")
    return [tuple(buf[3 * k:3 * k + 3]) for k in range(cnt.value)]


def profile_enable(enable: bool) -> None:
    _check(_lib.tgp_profile_enable(int(enable)), "tgp_profile_enable")


def profile_read() -> List[dict]:
    """Per-kernel launch count, summed event-timed duration (ms) and the
    algorithmic FLOPs / bytes of those launches since the last read."""
    cnt = _I()
    buf = (KernelStat * 256)()
    _check(_lib.tgp_profile_read(buf, 256, ctypes.byref(cnt)), "tgp_profile_read")
    return [{"name": buf[k].name.decode(), "launches": buf[k].launches, "ms": buf[k].ms,
             "flops": buf[k].flops, "bytes": buf[k].bytes} for k in range(cnt.value)]


def profile_clear() -> None:
    _check(_lib.tgp_profile_clear(), "tgp_profile_clear")


def debug_set_fwd_variant(v: int) -> int:
    """Forces the convolution kernel configuration (0 = automatic plan);
    returns the previous value.  Testing and tuning only."""
    return _lib.tgp_debug_set_fwd_variant(int(v))


def debug_fail_launch(n: int) -> int:
    """Makes the n-th kernel launch from now on (on this thread) fail, with
    every later launch of that call skipped; 0 disarms.  Error-path tests
    only.  Returns the previous countdown."""
    return _lib.tgp_debug_fail_launch(int(n))


def debug_set_rowtile_mask(m: int) -> int:
    """Enables kernel families in the automatic plan (bit mask); returns the
    previous mask.  Testing and tuning only."""
    return _lib.tgp_debug_set_rowtile_mask(int(m))
