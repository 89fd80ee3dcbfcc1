"""Single-layer parity: each kernel family through the C ABI, as a one-layer
stage with an injected upstream gradient.  Both sides start from identical
bf16 inputs, so only the layer's own output ReLU decides anything, and
every output (y, dx, dW, db) is held to the parity tolerance: 2e-2 max-rel
for bf16, 1e-4 for fp32, on N(0,1) inputs.  Stages of several layers in one
partition take the EXACT input family in bf16 (1e-6).  Shapes include
ragged pixel tiles and the benchmark's own level-0 and deepest layer shapes
at its micro-batch size."""
import pytest
import torch

from gpu_util import check_stage, gpu_stage, gpu_stage_with_popped, oracle_stage, say
from workloads import specs
from workloads.specs import (BF16, CONV1X1, CONV3X3, DWCONV3X3, FP32, PRO_MAXPOOL2,
                             PRO_UPCAT2, Layer, Net)
from workloads.synth import EXACT, NORMAL

pytestmark = pytest.mark.gpu


def one_layer(L, h, w, name="one"):
    return Net(name, (L,), L.cin, h, w)


def run_and_check(net, bal, j, dtype, B, m, what, popped=False, family=NORMAL):
    say(what)
    if popped:
        got = gpu_stage_with_popped(net, bal, j, dtype=dtype, B=B, m=m, family=family)
    else:
        got = gpu_stage(net, dtype, B, m, 0, bal, j, family=family)
    ref = oracle_stage(net, dtype, got["lo"], got["hi"], got["xv"], got["G"],
                       stash_in=got.get("stash_in"), family=family,
                       certify=(family == EXACT))
    check_stage(got, ref, dtype, what, family)
    got["sess"].close()


@pytest.mark.parametrize("cin,cout,h,w,B,m", [
    (64, 64, 32, 32, 4, 2),      # 64-channel tile (BN = 64, BM = 256)
    (64, 128, 20, 12, 6, 3),     # ragged pixel tile, 128-channel tile
    (128, 256, 10, 10, 4, 4),    # b = 1
    (512, 512, 6, 6, 2, 1),      # deep K, one partial tile
    (64, 128, 7, 48, 4, 2),      # row-blocked weight gradient: 4 rows a stage, ragged row block
    (128, 64, 5, 96, 2, 1),      # 2 rows a stage, two input-channel tiles
    (64, 64, 3, 192, 2, 2),      # 1 row a stage, K ranges of one row
    (128, 128, 5, 24, 4, 2),     # 4 rows a stage, 16-pixel k steps across rows
    (512, 512, 24, 24, 8, 2),    # weight-gradient partials too large to keep: reduced at once
])
def test_conv3x3(cin, cout, h, w, B, m):
    net = one_layer(Layer(CONV3X3, cin, cout), h, w)
    run_and_check(net, (1,), 1, BF16, B, m, f"conv3x3 {cin}->{cout} @{h}x{w} B={B} m={m}")


@pytest.mark.parametrize("cin,cout,h,w", [(64, 64, 3, 256), (64, 128, 5, 128), (64, 64, 7, 64),
                                          (128, 64, 9, 32), (64, 64, 11, 16), (128, 128, 9, 8),
                                          (512, 512, 5, 8), (512, 512, 7, 32)])
def test_wgrad_rows_other_widths(cin, cout, h, w):
    """The row-blocked weight gradient at the 6-level U-Net's widths 256 ...
    8 (stages of one to eight image rows), with a ragged last row block; the
    two 512-channel cases take one K range over both samples of the
    micro-batch (no partial slices)."""
    net = one_layer(Layer(CONV3X3, cin, cout), h, w)
    run_and_check(net, (1,), 1, BF16, 2, 1, f"wgrad rows {cin}->{cout} @{h}x{w}")


# Configurations of the nine-tap whole-row kernel: (index, W, rows per tile).
ROWS32 = [(0, 192, 3), (1, 192, 1), (2, 96, 6), (3, 96, 3), (4, 96, 2), (5, 48, 12),
          (6, 48, 6), (7, 48, 4), (8, 24, 24), (9, 24, 12), (10, 24, 8),
          # eight-wave layouts
          (11, 192, 3), (12, 96, 3), (13, 96, 2), (14, 48, 4), (15, 24, 8),
          # widths 64 and 32
          (18, 64, 4), (19, 64, 6), (20, 32, 8), (21, 32, 12),
          # eight waves, twelve fragments
          (22, 48, 8), (23, 96, 4)]


@pytest.mark.parametrize("cfg,w,r", ROWS32)
def test_rows32_configurations(cfg, w, r):
    """Each configuration of the nine-tap whole-row kernel, forced, on a layer
    whose last row block is ragged (H = R + 1), with four 16-channel stages
    and two output-channel tiles; the data gradient (64 output channels from
    128) runs the same configuration on the transposed weights."""
    import paper_2004_09910_amd as tgp
    old = tgp.debug_set_fwd_variant(401 + cfg)
    try:
        net = one_layer(Layer(CONV3X3, 64, 128), r + 1, w)
        run_and_check(net, (1,), 1, BF16, 2, 1, f"rows32 cfg {cfg} 64->128 @{r + 1}x{w}")
    finally:
        tgp.debug_set_fwd_variant(old)


@pytest.mark.parametrize("w,h", [(24, 25), (96, 13)])
def test_rows32_configurations_agree_bitwise(w, h):
    """Every configuration of the nine-tap kernel at one width sums each
    output in the same order (16-channel chunk, tap, channel), whatever its
    tile, fragment layout or wave count: forced one after another on the
    same layer and inputs (H leaves a ragged last row block in each), they
    give the same bits for y and dx_in."""
    import paper_2004_09910_amd as tgp
    cfgs = [(c, r) for c, cw, r in ROWS32 if cw == w]
    net = one_layer(Layer(CONV3X3, 64, 128), h, w)
    ref = None
    for cfg, r in cfgs:
        assert r < h and h % r
        old = tgp.debug_set_fwd_variant(401 + cfg)
        try:
            say(f"rows32 cfg {cfg} @{h}x{w}")
            tgp.profile_enable(True)
            tgp.profile_read()
            got = gpu_stage(net, BF16, 2, 1, 0, (1,), 1)
            ran = {k["name"] for k in tgp.profile_read()}
        finally:
            tgp.profile_enable(False)
            tgp.debug_set_fwd_variant(old)
        got["sess"].close()
        assert any(n.startswith(f"conv3x3_rows32<{w},{r},") for n in ran), ran
        if ref is None:
            ref = got
            continue
        for key in ("y", "dx"):
            assert torch.equal(got[key], ref[key]), f"cfg {cfg} {key} differs from cfg {cfgs[0][0]}"


@pytest.mark.parametrize("cfg,r", [(16, 2), (17, 3)])
def test_rows32_resident_weights(cfg, r):
    """The nine-tap kernel's configurations that keep the weights of all 64
    input channels in LDS (64 -> 64 channels only), forced, with a ragged
    last row block; the data gradient takes the same configuration."""
    import paper_2004_09910_amd as tgp
    old = tgp.debug_set_fwd_variant(401 + cfg)
    try:
        net = one_layer(Layer(CONV3X3, 64, 64), r + 1, 192)
        run_and_check(net, (1,), 1, BF16, 2, 1, f"rows32 resident cfg {cfg} @{r + 1}x192")
    finally:
        tgp.debug_set_fwd_variant(old)


# Configurations of the row-tiled 16x16x32 kernel (widths the nine-tap kernel
# is not built for): (index, W, rows per tile).  Rows per tile follow from the
# configuration's sub-tiles per wave and its LDS slot: 4, 2, 1 at width 128
# and 2, 1 at width 256 (the third does not fit a 256-pixel row).
ROWTILE = [(0, 128, 4), (1, 128, 2), (2, 128, 1), (0, 256, 2), (1, 256, 1)]


@pytest.mark.parametrize("cfg,w,r", ROWTILE)
def test_rowtile_configurations(cfg, w, r):
    """Each configuration of the row-tiled kernel, forced, on a layer whose
    last row block is ragged (H = R + 1), with two 32-channel chunks and two
    output-channel tiles; the data gradient (64 output channels from 128)
    runs the same configuration."""
    import paper_2004_09910_amd as tgp
    old = tgp.debug_set_fwd_variant(301 + cfg)
    try:
        net = one_layer(Layer(CONV3X3, 64, 128), r + 1, w)
        run_and_check(net, (1,), 1, BF16, 2, 1, f"rowtile cfg {cfg} 64->128 @{r + 1}x{w}")
    finally:
        tgp.debug_set_fwd_variant(old)


@pytest.mark.parametrize("cfg", [None, 0, 1, 2])
def test_rowtile_128x128(cfg):
    """A whole 128 x 128 image (the 6-level U-Net's level 1 at 128 channels):
    the automatic plan (the row-tiled kernel) and each configuration forced."""
    import paper_2004_09910_amd as tgp
    old = tgp.debug_set_fwd_variant(0 if cfg is None else 301 + cfg)
    try:
        net = one_layer(Layer(CONV3X3, 128, 128), 128, 128)
        run_and_check(net, (1,), 1, BF16, 2, 1, f"rowtile 128->128 @128x128 cfg {cfg}")
    finally:
        tgp.debug_set_fwd_variant(old)


@pytest.mark.parametrize("cin,cout,h,w", [(64, 128, 7, 48), (128, 64, 5, 96), (64, 64, 3, 192),
                                          (128, 128, 5, 24)])
def test_wgrad_rows_four_wave_layout(cin, cout, h, w):
    """The row-blocked weight gradient's four-wave layout forced at every
    width (the automatic choice takes the eight-wave one at widths 192 and
    48), on the same shapes as the conv3x3 cases above."""
    import paper_2004_09910_amd as tgp
    old = tgp.debug_set_rowtile_mask(15 | 32)
    try:
        net = one_layer(Layer(CONV3X3, cin, cout), h, w)
        run_and_check(net, (1,), 1, BF16, 2, 1, f"wgrad four-wave {cin}->{cout} @{h}x{w}")
    finally:
        tgp.debug_set_rowtile_mask(old)


@pytest.mark.parametrize("cin,cout,h,w", [(64, 128, 5, 96), (128, 128, 3, 96), (128, 256, 7, 48),
                                          (256, 256, 4, 48), (512, 256, 2, 48), (128, 128, 5, 24),
                                          (256, 512, 3, 24)])
def test_wgrad_three_filter_rows(cin, cout, h, w):
    """The weight gradient with all three filter rows per work item (micro-
    batches of four samples at widths 96, 48 and 24, in launches of eight
    micro-batches; 512 -> 256 at 48 and 256 -> 512 at 24 take one K range
    over the whole micro-batch): against the oracle, and bit for bit the
    same weight gradient as the one-filter-row kernel in its four-wave layout
    (forced), which sums each K range in the same order, and as one
    micro-batch per launch, which runs that layout by itself."""
    import numpy as np
    import paper_2004_09910_amd as tgp
    net = one_layer(Layer(CONV3X3, cin, cout), h, w)
    what = f"wgrad three rows {cin}->{cout} @{h}x{w}"
    say(what)
    tgp.profile_enable(True)
    tgp.profile_read()
    try:
        got = gpu_stage(net, BF16, 32, 8, 0, (1,), 1, lanes=8, group=8)
        ran = {k["name"] for k in tgp.profile_read()}
    finally:
        tgp.profile_enable(False)
    assert any(n.startswith("conv_wgrad_rows3<") for n in ran), ran
    ref = oracle_stage(net, BF16, got["lo"], got["hi"], got["xv"], got["G"])
    check_stage(got, ref, BF16, what)
    got["sess"].close()
    old = tgp.debug_set_rowtile_mask(15 | 32 | 64)
    try:
        forced = gpu_stage(net, BF16, 32, 8, 0, (1,), 1, lanes=8, group=8)
    finally:
        tgp.debug_set_rowtile_mask(old)
    forced["sess"].close()
    single = gpu_stage(net, BF16, 32, 8, 0, (1,), 1)
    single["sess"].close()
    for other in (forced, single):
        for idx in got["grads"]:
            np.testing.assert_array_equal(got["grads"][idx][0], other["grads"][idx][0])
            np.testing.assert_array_equal(got["grads"][idx][1], other["grads"][idx][1])
        assert torch.equal(got["dx"], other["dx"])


def test_conv1x1_and_depthwise():
    net = one_layer(Layer(CONV1X1, 256, 256), 14, 14)
    run_and_check(net, (1,), 1, BF16, 4, 2, "conv1x1 256->256 @14x14")
    net = one_layer(Layer(DWCONV3X3, 256, 256, relu=False, bias=False), 14, 14)
    run_and_check(net, (1,), 1, BF16, 4, 2, "dwconv3x3 256 @14x14")


@pytest.mark.parametrize("cin,h,w,B,m", [(256, 20, 20, 2, 1), (128, 9, 7, 4, 2), (64, 56, 56, 4, 2)])
def test_conv1x1_resident_weights(cin, h, w, B, m):
    """The 1x1 kernel with all weights resident in LDS (256 output
    channels): against the oracle on y, dx, dW and db, with a ragged last
    64-pixel tile; and bit for bit the same y and dx as the per-tap kernel
    (forced), whose K order it shares."""
    import paper_2004_09910_amd as tgp
    net = one_layer(Layer(CONV1X1, cin, 256), h, w)
    tgp.profile_enable(True)
    tgp.profile_read()
    try:
        run_and_check(net, (1,), 1, BF16, B, m, f"conv1x1_res {cin}->256 @{h}x{w} B={B} m={m}")
        ran = {k["name"] for k in tgp.profile_read()}
    finally:
        tgp.profile_enable(False)
    assert "conv1x1_res" in ran, ran
    got = gpu_stage(net, BF16, B, m, 0, (1,), 1)
    got["sess"].close()
    old = tgp.debug_set_fwd_variant(101)
    try:
        ref = gpu_stage(net, BF16, B, m, 0, (1,), 1)
    finally:
        tgp.debug_set_fwd_variant(old)
    ref["sess"].close()
    assert torch.equal(got["y"], ref["y"]) and torch.equal(got["dx"], ref["dx"])


@pytest.mark.parametrize("c,h,w,relu", [(64, 15, 9, True), (16, 7, 33, False), (2048, 5, 5, True),
                                         (24, 6, 6, True)])
def test_depthwise_shapes(c, h, w, relu):
    """Depthwise 3x3 with one to 256 channel packs per pixel, ragged row
    strips and column chunks; 24 channels (three packs, not a divisor of the
    block) takes the per-element kernels."""
    net = one_layer(Layer(DWCONV3X3, c, c, relu=relu, bias=relu), h, w)
    run_and_check(net, (1,), 1, BF16, 4, 2, f"dwconv3x3 {c} @{h}x{w} relu={relu}")


def test_head_without_relu():
    net = one_layer(Layer(CONV1X1, 64, 1, relu=False), 16, 16)
    run_and_check(net, (1,), 1, BF16, 4, 2, "head 1x1 64->1")


@pytest.mark.parametrize("dtype,cin,cout,relu", [(BF16, 64, 3, True), (BF16, 128, 4, False),
                                                 (FP32, 16, 2, True)])
def test_small_output_1x1(dtype, cin, cout, relu):
    """1x1 convolutions with at most four output channels (the head's path:
    one thread per pixel forward, block-reduced weight gradient)."""
    net = one_layer(Layer(CONV1X1, cin, cout, relu=relu), 20, 12)
    run_and_check(net, (1,), 1, dtype, 4, 2, f"1x1 {cin}->{cout} relu={relu}")


def test_maxpool_prologue():
    net = Net("pool", (Layer(CONV3X3, 64, 64), Layer(CONV3X3, 64, 128, prologue=PRO_MAXPOOL2)),
              64, 24, 20)
    run_and_check(net, (1, 1), 2, BF16, 4, 2, "maxpool prologue + conv 64->128")


def test_upcat_prologue():
    net = Net("upcat", (Layer(CONV3X3, 64, 64, stash_id=0),
                        Layer(CONV3X3, 64, 128, prologue=PRO_MAXPOOL2),
                        Layer(CONV3X3, 192, 64, prologue=PRO_UPCAT2, pop_id=0)), 64, 16, 24)
    run_and_check(net, (1, 1, 1), 3, BF16, 4, 2, "upsample-concat prologue + conv 192->64",
                  popped=True)


@pytest.mark.parametrize("dtype,c,bias", [(BF16, 64, True), (BF16, 64, False), (FP32, 16, True)])
def test_pool_backward_inside_a_partition(dtype, c, bias):
    """A max-pool prologue that is not its partition's first layer: its
    backward is formed inside the previous layer's fused ReLU-backward / bias
    kernel (without a bias there, by the plain pool backward).  The pooled
    layer's output is also stashed and popped by an upsample-concat in the
    same partition, so a skip gradient joins the routed one."""
    net = Net("poolin", (Layer(CONV3X3, c, c, bias=bias, stash_id=0),
                         Layer(CONV3X3, c, 2 * c, prologue=PRO_MAXPOOL2),
                         Layer(CONV3X3, 3 * c, c, prologue=PRO_UPCAT2, pop_id=0)), c, 16, 24)
    run_and_check(net, (3,), 1, dtype, 4, 2,
                  f"pool inside a partition, {'bf16' if dtype == BF16 else 'fp32'} c={c} bias={bias}",
                  family=EXACT if dtype == BF16 else NORMAL)


def test_fp32_direct_conv():
    net = one_layer(Layer(CONV3X3, 16, 16), 32, 32)
    run_and_check(net, (1,), 1, FP32, 8, 4, "fp32 conv3x3 16->16")
    net = Net("pool32", (Layer(CONV3X3, 16, 16, stash_id=0),
                         Layer(CONV3X3, 16, 32, prologue=PRO_MAXPOOL2),
                         Layer(CONV3X3, 48, 16, prologue=PRO_UPCAT2, pop_id=0)), 16, 8, 8)
    run_and_check(net, (1, 1, 1), 3, FP32, 4, 2, "fp32 upcat", popped=True)
    run_and_check(net, (1, 2), 2, FP32, 4, 2, "fp32 pool + upcat", popped=True)


@pytest.mark.parametrize("cin,cout,h", [(64, 64, 192), (256, 512, 24)])
def test_benchmark_layer_shapes(cin, cout, h):
    """The stage's level-0 layer (147456 x 64 x 576 per micro-batch) and its
    deepest layer (2304 x 512 x 2304) at the benchmark's micro-batch size 4."""
    net = one_layer(Layer(CONV3X3, cin, cout), h, h)
    run_and_check(net, (1,), 1, BF16, 4, 1, f"bench layer {cin}->{cout} @{h}x{h} b=4")


@pytest.mark.parametrize("cin,cout,h,B", [
    (4096, 4096, 8, 2),     # 6-level U-Net enc5b: 128 x 4096 x 36864 at micro-batch 2
    (6144, 2048, 16, 2),    # 6-level U-Net dec4a (upsample-concat input): K = 55296
    (1536, 512, 24, 4),     # 5-level U-Net dec3a: 9216 x 512 x 13824 at micro-batch 4
    (128, 128, 256, 2),     # 6-level U-Net level 0: 131072 x 128 x 1152 at micro-batch 2
])
def test_largest_layers_at_full_shape(cin, cout, h, B):
    """The layers with the longest K (and the 6-level network's widest image)
    at their real per-micro-batch shape: forward, data gradient, weight and
    bias gradient against the float64 oracle."""
    net = one_layer(Layer(CONV3X3, cin, cout), h, h)
    run_and_check(net, (1,), 1, BF16, B, 1, f"full-shape layer {cin}->{cout} @{h}x{h} b={B}")
