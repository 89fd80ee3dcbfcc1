"""Host-side tests of the C ABI (no GPU needed): exported symbols, the
clock-cycle schedule against the oracle's Algorithm 1 enumeration, the FLOP
partitioner against brute force, and argument / state validation, none of
which enqueues device work."""
import itertools
import os
import random
import re

import pytest

import golden_data

import paper_2004_09910_amd as tgp
from oracle import pipeline as opipe
from paper_2004_09910_amd.harness import layer_tuple
from workloads import specs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "tgp.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    names = set(re.findall(r"\b(tgp_[a-z_]+)\s*\(", hdr))
    assert len(names) >= 16
    for nm in sorted(names):
        assert hasattr(tgp._lib, nm), nm


@pytest.mark.parametrize("mode", [0, 1, 2])
@pytest.mark.parametrize("m", range(1, 7))
@pytest.mark.parametrize("n", range(1, 6))
def test_schedule_trace_follows_clock_cycle(m, n, mode):
    ops = tgp.schedule_trace(m, n, mode)
    fwd = [(i, j) for op, i, j in ops if op == tgp.OP_FORWARD]
    bwd = [(i, j) for op, i, j in ops if op == tgp.OP_BACKWARD]
    assert fwd == [t for c in opipe.forward_clocks(m, n) for t in c]
    assert bwd == [t for c in opipe.backward_clocks(m, n) for t in c]
    # every forward precedes every backward; the loss of micro-batch i comes
    # right after F_{i,n}
    last_f = max(k for k, o in enumerate(ops) if o[0] == tgp.OP_FORWARD)
    first_b = min(k for k, o in enumerate(ops) if o[0] in (tgp.OP_BACKWARD, tgp.OP_RECOMPUTE))
    assert last_f < first_b
    for k, (op, i, j) in enumerate(ops):
        if op == tgp.OP_FORWARD and j == n:
            assert ops[k + 1] == (tgp.OP_LOSS, i, 0)
        if op == tgp.OP_RECOMPUTE:
            assert ops[k + 1] == (tgp.OP_BACKWARD, i, j)
            assert opipe.checkpointed(mode, i, m)
        if op == tgp.OP_BACKWARD:
            assert ops[k + 1] == (tgp.OP_ACCUMULATE, i, j)
            assert (ops[k - 1] == (tgp.OP_RECOMPUTE, i, j)) == opipe.checkpointed(mode, i, m)
    assert sum(op == tgp.OP_RECOMPUTE for op, _, _ in ops) == \
        n * sum(opipe.checkpointed(mode, i, m) for i in range(1, m + 1))


def test_schedule_trace_m4_n3_written_out():
    """The library's clock order for m=4, n=3 (except-last) against the
    hand-written fixture tests/golden/clock_cycle_m4_n3.txt (Algorithm 1)."""
    g = golden_data.clock_cycle()
    ops = tgp.schedule_trace(4, 3, 1)   # except-last
    assert [(i, j) for op, i, j in ops if op == tgp.OP_FORWARD] == \
        [t for c in g["FORWARD"] for t in c]
    assert [(i, j) for op, i, j in ops if op == tgp.OP_RECOMPUTE] == \
        [t for c in g["RECOMPUTE_EXCEPT_LAST"] for t in c]


def _brute_balance(cost, n):
    L = len(cost)
    best = None
    for cuts in itertools.combinations(range(1, L), n - 1):
        edges = (0,) + cuts + (L,)
        parts = [sum(cost[edges[k]:edges[k + 1]]) for k in range(n)]
        key = (max(parts), sum(p * p for p in parts), cuts)
        if best is None or key < best[0]:
            best = (key, [edges[k + 1] - edges[k] for k in range(n)])
    return best[1]


def test_partitioner_matches_brute_force():
    rnd = random.Random(5)
    for _ in range(300):
        L = rnd.randint(1, 10)
        n = rnd.randint(1, min(L, 4))
        cost = [rnd.choice([0, 1, 2, 3, 5, 8, 13, 10 ** 12]) for _ in range(L)]
        assert tgp.balance_minmax(cost, n) == _brute_balance(cost, n), (cost, n)


def _net(net, dtype=0):
    return tgp.net_create([layer_tuple(L) for L in net.layers], net.in_channels, net.height,
                          net.width, dtype)


def test_unet_partition_and_flops():
    net = specs.unet(5, 64, 64, 192)
    h = _net(net)
    try:
        assert [tgp.layer_flops(h, k) for k in range(len(net.layers))] == net.flops_per_sample()
        tgp.set_partition(h, 4)
        assert tgp.get_partition(h) == [7, 5, 3, 4]
        tgp.set_partition(h, 2, [10, 9])
        assert tgp.get_partition(h) == [10, 9]
        with pytest.raises(tgp.TgpError):
            tgp.set_partition(h, 2, [10, 10])
        with pytest.raises(tgp.TgpError):
            tgp.set_partition(h, 20)
    finally:
        tgp.net_destroy(h)
    h = _net(specs.unet(6, 128, 128, 256))
    tgp.set_partition(h, 8)
    assert tgp.get_partition(h) == [4, 4, 4, 2, 2, 2, 2, 3]
    tgp.net_destroy(h)


def _status(layers, in_c=8, H=8, W=8, dtype=0):
    return tgp.call_status("tgp_net_create", (tgp.Layer * len(layers))(*[tgp.Layer(*l) for l in layers]),
                           len(layers), in_c, H, W, dtype, tgp.ctypes.byref(tgp.ctypes.c_void_p()))


def test_net_create_validation():
    C3, C1, DW = 0, 1, 2
    ok = [(C3, 8, 8, 1, 1, 0, 0, -1), (C3, 8, 16, 1, 1, 1, -1, -1), (C3, 24, 8, 1, 1, 2, -1, 0)]
    assert _status(ok) == tgp.OK
    assert _status([(C3, 4, 8, 1, 1, 0, -1, -1)]) == tgp.EINVAL          # cin mismatch
    assert _status([(C3, 8, 8, 1, 1, 2, -1, 3)]) == tgp.EINVAL           # pop of missing skip
    assert _status([(C3, 8, 8, 1, 1, 1, -1, -1)], H=7) == tgp.EINVAL     # odd pool
    assert _status([(DW, 8, 16, 0, 0, 0, -1, -1)]) == tgp.EINVAL         # depthwise cin != cout
    assert _status([(C3, 8, 8, 1, 1, 0, 0, -1), (C3, 8, 8, 1, 1, 0, 0, -1)]) == tgp.EINVAL
    assert _status([(9, 8, 8, 1, 1, 0, -1, -1)]) == tgp.EINVAL           # bad kind
    assert _status([(C3, 4, 4, 1, 1, 1, -1, -1)], in_c=4) == tgp.EUNSUPPORTED  # bf16 pool, 4 ch
    assert _status([(C3, 4, 4, 1, 1, 1, -1, -1)], in_c=4, dtype=1) == tgp.OK
    assert _status([]) == tgp.EINVAL


FAKE = 1 << 20   # a non-null address; never dereferenced by these tests


def _bound_net(mode=0, B=4, m=2, n=2):
    net = specs.plain_stack(4, 8, 8, 8)
    h = _net(net, dtype=1)
    tgp.set_partition(h, n)
    for k in range(4):
        tgp.bind_params(h, k, FAKE, FAKE, FAKE, FAKE)
    nbytes = tgp.plan(h, B, m, mode)
    return h, nbytes


def test_plan_and_workspace_validation():
    h, nbytes = _bound_net()
    assert nbytes > 0
    sz = tgp.ctypes.c_size_t()
    assert tgp.call_status("tgp_plan", h, 5, 2, 0, tgp.ctypes.byref(sz)) == tgp.EINVAL
    assert tgp.call_status("tgp_plan", h, 4, 2, 7, tgp.ctypes.byref(sz)) == tgp.EINVAL
    assert tgp.call_status("tgp_plan", h, 4, 2, 0, tgp.ctypes.byref(sz)) == tgp.OK
    assert tgp.call_status("tgp_bind_workspace", h, FAKE, sz.value - 1) == tgp.ENOSPACE
    assert tgp.call_status("tgp_bind_workspace", h, FAKE + 16, sz.value) == tgp.EINVAL
    assert tgp.call_status("tgp_bind_workspace", h, None, sz.value) == tgp.EINVAL
    # no workspace bound yet
    assert tgp.call_status("tgp_stage_forward", h, 1, 1, 1, FAKE, FAKE, None) == tgp.ESTATE
    # checkpoint memory: never > except_last > always for m > 1
    sizes = [_bound_net(mode)[1] for mode in (0, 1, 2)]
    assert sizes[0] < sizes[1] < sizes[2]
    tgp.net_destroy(h)


def test_layer_times_plan_and_error_paths():
    """tgp_layer_times_plan: one-layer partitions for one micro-batch, a
    workspace at least the plan's plus four activation buffers; the caller's
    partition comes back only through tgp_layer_times, and the checks that
    run before any GPU work."""
    h, plan_bytes = _bound_net(mode=0, B=4, m=2, n=2)
    try:
        assert tgp.get_partition(h) == [2, 2]
        us = (tgp.ctypes.c_float * 4)()
        bal = (tgp.ctypes.c_int * 2)()
        # no timing plan yet
        assert tgp.call_status("tgp_layer_times", h, FAKE, 1 << 30, 1, us, None) == tgp.ESTATE
        nbytes = tgp.layer_times_plan(h, 2, 0)
        assert tgp.get_partition(h) == [1, 1, 1, 1]
        act = 2 * 8 * 8 * 8 * 4          # the largest activation of one 2-sample micro-batch
        assert nbytes >= 4 * act
        # a second timing plan keeps the original partition aside, not the singletons
        assert tgp.layer_times_plan(h, 2, 0) == nbytes
        assert tgp.call_status("tgp_layer_times", h, FAKE, nbytes, 0, us, None) == tgp.EINVAL
        assert tgp.call_status("tgp_layer_times", h, FAKE, nbytes - 1, 1, us, None) == tgp.ENOSPACE
        assert tgp.call_status("tgp_balance_by_time", h, FAKE, nbytes, 1, 0, bal, us, None) == \
            tgp.EINVAL
        assert tgp.call_status("tgp_balance_by_time", h, FAKE, nbytes, 1, 5, bal, us, None) == \
            tgp.EINVAL
        # the failed binding kept the timing plan; a new partition drops it
        tgp.set_partition(h, 2)
        assert tgp.call_status("tgp_layer_times", h, FAKE, nbytes, 1, us, None) == tgp.ESTATE
        assert tgp.call_status("tgp_layer_times_plan", h, 0, 0, tgp.ctypes.byref(
            tgp.ctypes.c_size_t())) == tgp.EINVAL
    finally:
        tgp.net_destroy(h)


def test_lanes_replicate_only_the_transient_buffers():
    """tgp_set_lanes: 1..TGP_MAX_LANES, invalidates the plan, and each extra
    lane adds the same per-lane block (stash slots, stored activations and
    pipeline boundaries are not replicated); several lanes add one gradient
    slot per micro-batch."""
    h, one = _bound_net(mode=0, B=8, m=4, n=2)
    assert tgp.call_status("tgp_set_lanes", h, 0) == tgp.EINVAL
    assert tgp.call_status("tgp_set_lanes", h, 17) == tgp.EINVAL
    sizes = []
    for k in (1, 2, 3, 4):
        tgp.set_lanes(h, k)
        # the plan is gone until tgp_plan runs again
        assert tgp.call_status("tgp_bind_workspace", h, FAKE, 1 << 40) == tgp.ESTATE
        sizes.append(tgp.plan(h, 8, 4, 0))
    assert sizes[0] == one
    # from two lanes on, each lane adds the same block (the per-micro-batch
    # gradient slots appear once, at two lanes)
    step = sizes[2] - sizes[1]
    assert step > 0 and sizes[3] - sizes[2] == step
    assert sizes[1] - sizes[0] > step
    assert step < sizes[0]
    tgp.net_destroy(h)


def test_stage_state_machine_rejects_out_of_order_calls():
    h, nbytes = _bound_net(mode=1, B=4, m=2, n=2)
    tgp.bind_workspace(h, FAKE, nbytes)
    st = lambda name, *a: tgp.call_status(name, h, *a)
    # checkpoint flag must match the planned policy (except-last: i=1 yes, i=2 no)
    assert st("tgp_stage_forward", 1, 1, 0, FAKE, FAKE, None) == tgp.EINVAL
    assert st("tgp_stage_forward", 1, 2, 1, FAKE, FAKE, None) == tgp.EINVAL
    assert st("tgp_stage_forward", 3, 1, 1, FAKE, FAKE, None) == tgp.EINVAL   # bad j
    assert st("tgp_stage_forward", 1, 3, 1, FAKE, FAKE, None) == tgp.EINVAL   # bad i
    assert st("tgp_stage_forward", 1, 1, 1, None, FAKE, None) == tgp.EINVAL   # NULL x
    # backward before forward, accumulate before backward
    assert st("tgp_stage_backward_recompute", 1, 2, FAKE, None, None) == tgp.ESTATE
    assert st("tgp_grad_accumulate", 1, 2, 1, None) == tgp.ESTATE
    assert st("tgp_grad_accumulate", 1, 1, 1, None) == tgp.EINVAL             # overwrite only at i=m
    # pipeline step arguments must match the plan
    assert st("tgp_pipeline_step", FAKE, FAKE, 8, 2, 2, 1, FAKE, None, None) == tgp.EINVAL
    assert st("tgp_pipeline_step", FAKE, FAKE, 4, 2, 1, 1, FAKE, None, None) == tgp.EINVAL
    assert st("tgp_pipeline_step", FAKE, FAKE, 4, 2, 2, 0, FAKE, None, None) == tgp.EINVAL
    assert st("tgp_pipeline_step", None, FAKE, 4, 2, 2, 1, FAKE, None, None) == tgp.EINVAL
    assert "match" in tgp.last_error() or "NULL" in tgp.last_error()
    tgp.net_destroy(h)


def test_paired_stage_calls_check_lanes_and_order():
    """tgp_stage_forward2 / tgp_stage_backward_recompute2: the two
    micro-batches must sit on different lanes, the backward pair must be
    (i0, i0 - 1) with per-micro-batch gradient slots, and each micro-batch
    passes the single call's checks (checkpoint policy, NULLs, state)."""
    h, _ = _bound_net(mode=1, B=8, m=4, n=2)
    tgp.set_lanes(h, 2)
    tgp.bind_workspace(h, FAKE, tgp.plan(h, 8, 4, 1))
    st = lambda name, *a: tgp.call_status(name, h, *a)
    F = FAKE
    assert st("tgp_stage_forward2", 1, 1, 1, 1, 1, F, F, F, F, None) == tgp.EINVAL   # same i
    assert st("tgp_stage_forward2", 1, 1, 3, 1, 1, F, F, F, F, None) == tgp.EINVAL   # same lane
    assert st("tgp_stage_forward2", 1, 3, 4, 1, 1, F, F, F, F, None) == tgp.EINVAL   # i=4 is not checkpointed
    assert st("tgp_stage_forward2", 1, 1, 5, 1, 1, F, F, F, F, None) == tgp.EINVAL   # bad i
    assert st("tgp_stage_forward2", 1, 1, 2, 1, 1, F, None, F, F, None) == tgp.EINVAL
    assert st("tgp_stage_backward_recompute2", 1, 4, 3, F, F, None, None, None) == tgp.ESTATE
    assert st("tgp_stage_backward_recompute2", 1, 4, 2, F, F, None, None, None) == tgp.EINVAL
    assert st("tgp_stage_backward_recompute2", 1, 1, 0, F, F, None, None, None) == tgp.EINVAL
    assert st("tgp_stage_backward_recompute2", 1, 4, 3, F, None, None, None, None) == tgp.EINVAL
    assert st("tgp_stage_backward_recompute2", 1, 4, 3, F, F, F, None, None) == tgp.EINVAL
    assert "all or none" in tgp.last_error()
    # one lane: a single gradient slot, so no backward pair
    tgp.set_lanes(h, 1)
    tgp.bind_workspace(h, FAKE, tgp.plan(h, 8, 4, 1))
    assert st("tgp_stage_forward2", 1, 1, 2, 1, 1, F, F, F, F, None) == tgp.EINVAL
    assert st("tgp_stage_backward_recompute2", 1, 4, 3, F, F, None, None, None) == tgp.EINVAL
    assert "lanes" in tgp.last_error()
    tgp.net_destroy(h)


def test_group_stage_calls_check_count_lanes_and_order():
    """tgp_stage_forward_n / tgp_stage_backward_recompute_n: 1..16 tasks on
    distinct lanes, consecutive micro-batches (i0 upwards for the forward,
    downwards for the backward), each passing the single call's checks.
    Every call here fails a host check, so nothing is enqueued."""
    import ctypes
    h, _ = _bound_net(mode=1, B=8, m=4, n=2)
    tgp.set_lanes(h, 4)
    tgp.bind_workspace(h, FAKE, tgp.plan(h, 8, 4, 1))
    st = lambda name, *a: tgp.call_status(name, h, *a)
    F = FAKE
    I4 = lambda *v: (ctypes.c_int * 4)(*v)
    P4 = lambda *v: (ctypes.c_void_p * 4)(*v)
    ck = I4(1, 1, 1, 0)                       # except-last: only i = 4 keeps its activations
    xs, none = P4(F, F, F, F), P4(None, None, None, None)
    assert st("tgp_stage_forward_n", 1, 1, 0, ck, xs, xs, None) == tgp.EINVAL      # count 0
    assert st("tgp_stage_forward_n", 1, 1, 17, ck, xs, xs, None) == tgp.EINVAL     # count 17
    assert "count 17" in tgp.last_error()
    assert st("tgp_stage_forward_n", 1, 1, 5, ck, xs, xs, None) == tgp.EINVAL      # i = 5
    assert st("tgp_stage_forward_n", 1, 2, 4, ck, xs, xs, None) == tgp.EINVAL      # i = 5
    assert st("tgp_stage_forward_n", 1, 1, 4, I4(1, 1, 1, 1), xs, xs, None) == tgp.EINVAL
    assert "checkpoint" in tgp.last_error()
    assert st("tgp_stage_forward_n", 1, 1, 4, ck, P4(F, None, F, F), xs, None) == tgp.EINVAL
    assert st("tgp_stage_forward_n", 3, 1, 2, ck, xs, xs, None) == tgp.EINVAL      # j = 3
    assert st("tgp_stage_backward_recompute_n", 1, 4, 4, xs, none, None) == tgp.ESTATE
    assert st("tgp_stage_backward_recompute_n", 1, 3, 4, xs, none, None) == tgp.EINVAL   # 3..0
    assert st("tgp_stage_backward_recompute_n", 1, 4, 4, xs, P4(F, None, None, None),
              None) == tgp.EINVAL
    assert "all or none" in tgp.last_error()
    assert st("tgp_stage_backward_recompute_n", 1, 4, 4, P4(F, F, None, F), none,
              None) == tgp.EINVAL
    # grouped accumulation: count and range, overwrite exactly for i0 = m,
    # and every micro-batch's backward first
    assert st("tgp_grad_accumulate_n", 1, 4, 0, 1, None) == tgp.EINVAL        # count 0
    assert st("tgp_grad_accumulate_n", 1, 4, 17, 1, None) == tgp.EINVAL       # count 17
    assert st("tgp_grad_accumulate_n", 1, 4, 5, 1, None) == tgp.EINVAL        # 4..0
    assert st("tgp_grad_accumulate_n", 1, 4, 4, 0, None) == tgp.EINVAL        # overwrite
    assert "overwrite" in tgp.last_error()
    assert st("tgp_grad_accumulate_n", 1, 3, 2, 1, None) == tgp.EINVAL        # overwrite
    assert st("tgp_grad_accumulate_n", 3, 4, 4, 1, None) == tgp.EINVAL        # j = 3
    assert st("tgp_grad_accumulate_n", 1, 4, 4, 1, None) == tgp.ESTATE        # no B yet
    assert "needs B" in tgp.last_error()
    # two lanes: micro-batches 1 and 3 share one, and a backward of four
    # needs four
    tgp.set_lanes(h, 2)
    tgp.bind_workspace(h, FAKE, tgp.plan(h, 8, 4, 1))
    assert st("tgp_stage_forward_n", 1, 1, 4, ck, xs, xs, None) == tgp.EINVAL
    assert "share a lane" in tgp.last_error()
    assert st("tgp_stage_backward_recompute_n", 1, 4, 4, xs, none, None) == tgp.EINVAL
    assert "lanes" in tgp.last_error()
    tgp.net_destroy(h)


def test_unbound_layers_are_rejected():
    net = specs.plain_stack(2, 8, 8, 8)
    h = _net(net, dtype=1)
    nbytes = tgp.plan(h, 2, 1, 0)
    tgp.bind_workspace(h, FAKE, nbytes)
    assert tgp.call_status("tgp_stage_forward", h, 1, 1, 1, FAKE, FAKE, None) == tgp.ESTATE
    assert "bound" in tgp.last_error()
    tgp.net_destroy(h)


def test_misaligned_pointers_are_rejected():
    """Whole tensors must be 16-byte aligned (loss 4-byte); micro-batch
    slices to the largest power of two up to 16 dividing their channel row.
    The fp32 8-channel stack has 32-byte rows, so its slices need 16."""
    h, nbytes = _bound_net(mode=0, B=4, m=2, n=2)
    tgp.bind_workspace(h, FAKE, nbytes)
    st = lambda name, *a: tgp.call_status(name, h, *a)
    for args in ((FAKE + 8, FAKE, FAKE, FAKE), (FAKE, FAKE + 4, FAKE, FAKE),
                 (FAKE, FAKE, FAKE + 8, FAKE), (FAKE, FAKE, FAKE, FAKE + 2)):
        assert st("tgp_bind_params", 0, *args) == tgp.EINVAL
        assert "aligned" in tgp.last_error()
    assert st("tgp_bind_params", 0, FAKE, FAKE, FAKE, FAKE) == tgp.OK
    assert st("tgp_stage_forward", 1, 1, 1, FAKE + 8, FAKE, None) == tgp.EINVAL
    assert st("tgp_stage_forward", 1, 1, 1, FAKE, FAKE + 4, None) == tgp.EINVAL
    assert "aligned" in tgp.last_error()
    assert st("tgp_stage_backward_recompute", 1, 2, FAKE + 8, None, None) == tgp.EINVAL
    assert st("tgp_stage_backward_recompute", 1, 2, FAKE, FAKE + 8, None) == tgp.EINVAL
    assert st("tgp_pipeline_step", FAKE + 8, FAKE, 4, 2, 2, 0, FAKE, None, None) == tgp.EINVAL
    assert st("tgp_pipeline_step", FAKE, FAKE + 8, 4, 2, 2, 0, FAKE, None, None) == tgp.EINVAL
    assert st("tgp_pipeline_step", FAKE, FAKE, 4, 2, 2, 0, FAKE + 2, None, None) == tgp.EINVAL
    assert st("tgp_pipeline_step", FAKE, FAKE, 4, 2, 2, 0, FAKE, FAKE + 8, None) == tgp.EINVAL
    tgp.net_destroy(h)
    # a 1-channel output (the U-Net head) has 2-byte bf16 rows: any even
    # address is a valid slice of it
    net = specs.Net("head", (specs.Layer(specs.CONV1X1, 64, 1, relu=False),), 64, 4, 4)
    h = _net(net, dtype=0)
    tgp.bind_params(h, 0, FAKE, FAKE, FAKE, FAKE)
    tgp.bind_workspace(h, FAKE, tgp.plan(h, 2, 2, 0))
    assert tgp.call_status("tgp_stage_forward", h, 1, 1, 1, FAKE + 8, FAKE, None) == tgp.EINVAL
    assert tgp.call_status("tgp_stage_forward", h, 1, 1, 1, FAKE, FAKE + 1, None) == tgp.EINVAL
    tgp.net_destroy(h)


def test_launch_failure_hook_arms_and_disarms():
    """tgp_debug_fail_launch returns the previous countdown; 0 disarms."""
    assert tgp.debug_fail_launch(5) == 0
    assert tgp.debug_fail_launch(0) == 5
    assert tgp.debug_fail_launch(0) == 0
