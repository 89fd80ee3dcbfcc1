"""tgp_pipeline_step_static, the step that allocates nothing: it runs on the
library's static device scratch and must give the bits of tgp_pipeline_step
on a caller-bound workspace.  Two calls in a row on one device (the second
with a smaller input, so it runs on what the first left in the scratch), each
against the bound-workspace step; and the host-side refusals."""
import numpy as np
import pytest
import torch

import paper_2004_09910_amd as tgp
from gpu_util import gpu_network, network_inputs, say
from paper_2004_09910_amd.harness import Session, nchw_to_device_nhwc, nhwc_to_nchw64
from workloads import specs
from workloads.specs import BF16, CKPT_ALWAYS

pytestmark = pytest.mark.gpu


def _static_step(net, B, m, n, mode, inputs):
    """A session whose net is planned but never given a workspace; the step
    runs through tgp_pipeline_step_static."""
    sess = Session(net, BF16, n=n)
    tgp.set_lanes(sess.h, 1)
    nbytes = tgp.plan(sess.h, B, m, mode)
    assert nbytes <= tgp.STATIC_SCRATCH_BYTES, nbytes
    _, xraw, _, traw, _ = inputs
    h, w = net.out_hw()
    x = nchw_to_device_nhwc(xraw, BF16)
    t = nchw_to_device_nhwc(traw, BF16)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = torch.empty((B, h, w, net.out_channels()), dtype=x.dtype, device="cuda")
    tgp.pipeline_step_static(sess.h, x.data_ptr(), t.data_ptr(), B, m, n, mode, loss.data_ptr(),
                             y.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    out = {"loss": float(loss.item()), "y": nhwc_to_nchw64(y), "grads": sess.grads64()}
    sess.close()
    return out


def test_static_step_matches_bound_workspace_twice():
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    for B, m in ((4, 2), (2, 2)):
        say(f"static scratch step B={B} m={m}")
        inputs = network_inputs(net, BF16, B)
        ref = gpu_network(net, BF16, B, m, 3, CKPT_ALWAYS, inputs=inputs)
        ref.pop("sess").close()
        got = _static_step(net, B, m, 3, CKPT_ALWAYS, inputs)
        assert got["loss"] == ref["loss"]
        assert np.array_equal(got["y"], ref["y"])
        for idx, (dW, db) in ref["grads"].items():
            np.testing.assert_array_equal(got["grads"][idx][0], dW)
            if db is not None:
                np.testing.assert_array_equal(got["grads"][idx][1], db)


def test_static_step_refusals():
    """Too large a plan and more than one lane are refused on the host,
    before anything is enqueued."""
    net = specs.unet(3, 64, 64, 32, "unet3-c64-32")
    sess = Session(net, BF16, n=3)
    tgp.set_lanes(sess.h, 1)
    assert tgp.plan(sess.h, 16, 2, CKPT_ALWAYS) > tgp.STATIC_SCRATCH_BYTES
    assert tgp.call_status("tgp_pipeline_step_static", sess.h, 1 << 20, 1 << 20, 16, 2, 3, 0,
                           1 << 20, None, None) == tgp.ENOSPACE
    tgp.set_lanes(sess.h, 2)
    tgp.plan(sess.h, 2, 2, CKPT_ALWAYS)
    assert tgp.call_status("tgp_pipeline_step_static", sess.h, 1 << 20, 1 << 20, 2, 2, 3, 0,
                           1 << 20, None, None) == tgp.EINVAL
    sess.close()
