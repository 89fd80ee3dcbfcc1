"""Error paths on the GPU, forced from the host: a kernel launch made to fail
with tgp_debug_fail_launch (the failing launch and the rest of the call are
skipped, so nothing faulty reaches the device).  The call must return
TGP_EHIP naming the operation, leave no lane fork open (also under graph
capture), and leave the net ready: the next step gives the reference bits."""
import numpy as np
import pytest
import torch

import paper_2004_09910_amd as tgp
from gpu_util import gpu_network, say
from workloads import specs
from workloads.specs import BF16, CKPT_ALWAYS

pytestmark = pytest.mark.gpu

B, M, N = 8, 4, 3


def _step_status(sess, x, t, loss, y):
    return tgp.call_status("tgp_pipeline_step", sess.h, x.data_ptr(), t.data_ptr(), B, M, N,
                           CKPT_ALWAYS, loss.data_ptr(), y.data_ptr(),
                           torch.cuda.current_stream().cuda_stream)


def _same_as(ref, sess, loss, y):
    assert float(loss.item()) == ref["loss"]
    assert torch.equal(y, ref["y_ref"])
    got = sess.grads64()
    for idx, (dW, db) in ref["grads"].items():
        np.testing.assert_array_equal(got[idx][0], dW)
        if db is not None:
            np.testing.assert_array_equal(got[idx][1], db)


@pytest.fixture(scope="module")
def ref():
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    say("reference step, two lanes")
    r = gpu_network(net, BF16, B, M, N, CKPT_ALWAYS, lanes=2)
    r["y_ref"] = r["y_t"].clone()
    # launches per step: arm far ahead, run one step, read what is left
    big = 1 << 30
    tgp.debug_fail_launch(big)
    assert _step_status(r["sess"], r["x"], r["t"], r["loss_t"], r["y_t"]) == tgp.OK
    r["launches"] = big - tgp.debug_fail_launch(0)
    torch.cuda.synchronize()
    say(f"  {r['launches']} launches per step")
    return r


def test_failed_step_then_good_step(ref):
    sess, x, t, loss, y = ref["sess"], ref["x"], ref["t"], ref["loss_t"], ref["y_t"]
    L = ref["launches"]
    assert L > 20
    for k in (1, L // 3, L - 1):
        say(f"failing launch {k} of {L}")
        tgp.debug_fail_launch(k)
        assert _step_status(sess, x, t, loss, y) == tgp.EHIP
        msg = tgp.last_error()
        assert ":" in msg and msg.split(":")[0], msg
        assert tgp.debug_fail_launch(0) == 0          # the countdown fired
        torch.cuda.synchronize()
        loss.zero_()
        y.zero_()
        assert _step_status(sess, x, t, loss, y) == tgp.OK, tgp.last_error()
        torch.cuda.synchronize()
        _same_as(ref, sess, loss, y)


def test_failed_step_under_capture_leaves_no_open_fork(ref):
    """A step that fails while being captured still joins its lanes into the
    capturing stream, so the capture ends cleanly (the partial graph is
    discarded, never replayed)."""
    sess, x, t, loss, y = ref["sess"], ref["x"], ref["t"], ref["loss_t"], ref["y_t"]
    g = torch.cuda.CUDAGraph()
    tgp.debug_fail_launch(ref["launches"] // 2)
    with torch.cuda.graph(g):
        status = _step_status(sess, x, t, loss, y)
    assert status == tgp.EHIP
    assert tgp.debug_fail_launch(0) == 0
    del g
    torch.cuda.synchronize()
    assert _step_status(sess, x, t, loss, y) == tgp.OK
    torch.cuda.synchronize()
    _same_as(ref, sess, loss, y)


def test_failed_stage_forward_can_be_retried():
    """A stage forward whose launch fails is not marked as run: the same
    call succeeds afterwards."""
    from paper_2004_09910_amd.harness import Session
    net = specs.unet(3, 64, 64, 24, "unet3-c64")
    sess = Session(net, BF16, n=1)
    sess.plan(2, 2, CKPT_ALWAYS)
    x = torch.zeros((2, 24, 24, 64), dtype=torch.bfloat16, device="cuda")
    y = torch.empty((2, 24, 24, 1), dtype=torch.bfloat16, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    tgp.debug_fail_launch(2)
    assert tgp.call_status("tgp_stage_forward", sess.h, 1, 1, 1, x.data_ptr(), y.data_ptr(),
                           st) == tgp.EHIP
    assert tgp.debug_fail_launch(0) == 0
    assert tgp.call_status("tgp_stage_forward", sess.h, 1, 1, 1, x.data_ptr(), y.data_ptr(),
                           st) == tgp.OK
    torch.cuda.synchronize()
    sess.close()
