"""The C ABI: both libraries load and export every function of
include/rtcc.h; the release controller, driven through the host test
library (controller + C ABI linked against a recording executor), follows
the state machine, validation and release rules of Sec. IV-C."""

import ctypes
import math
import os
import re
import threading
import time

import numpy as np
import pytest

import synth
from oracle import network as N
from paper_2608_08330_amd import rtcc as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    text = open(os.path.join(ROOT, "include", "rtcc.h")).read()
    return sorted(set(re.findall(r"RTCC_API\s+[\w\s\*]+?\b(rtcc_\w+)\s*\(", text)))


def test_header_and_binding_agree():
    assert sorted(R.EXPORTS) == _header_functions()


@pytest.mark.parametrize("kind", ["gpu", "host"])
def test_library_loads_and_exports_every_symbol(kind):
    lib = R.load(kind)
    for name in _header_functions():
        assert hasattr(lib, name), name
    assert R.load(kind).rtcc_status_str(6) == b"RTCC_E_INFEASIBLE"


# --------------------------------------------------------------- controller

def _host_log(clear=True):
    lib = R.load("host")
    buf = ctypes.create_string_buffer(1 << 20)
    lib.rtcc_hosttest_log(buf, len(buf), 1 if clear else 0)
    return [l for l in buf.value.decode().splitlines() if l]


@pytest.fixture
def host_ctx():
    cfg = synth.config("t_attn")
    fr = synth.make_frame(cfg)
    ctx = R.rtcc_create(R.model_desc(cfg), R.weights_blob(cfg, fr["weights"]), kind="host")
    _host_log()
    yield cfg, fr, ctx
    ctx.close()


def _status(fn, *a):
    try:
        fn(*a)
        return R.RTCC_OK
    except R.RtccError as e:
        return e.status


def test_release_mode_dispatches_each_branch_at_its_event(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 10)
    order = [2, 0, 3, 1]
    for i, k in enumerate(order):
        assert R.rtcc_get_branch_state(ctx, k) == R.RTCC_WAITING
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.1 * i)
        # released = input received and encoder enqueued (eq. branch_state)
        assert R.rtcc_get_branch_state(ctx, k) == R.RTCC_RELEASED
        assert _host_log()[-1].startswith("dispatch %d " % k)
    det = R.rtcc_join_and_detect(ctx)
    assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_FINISHED for k in range(4))
    np.testing.assert_allclose(det["arrival_s"], [0.1, 0.3, 0.0, 0.2])
    assert _host_log()[-1].startswith("join")


def test_barrier_mode_dispatches_all_at_last_event_in_index_order(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_set_mode(ctx, R.RTCC_MODE_BARRIER)
    R.rtcc_begin_frame(ctx, time.monotonic() - 10)
    for i, k in enumerate([3, 1, 2]):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.1 * i)
        # recorded, not released: the barrier releases every encoder at A
        assert R.rtcc_get_branch_state(ctx, k) == R.RTCC_WAITING
        assert _status(R.rtcc_release_branch, ctx, k, fr["points"][k], fr["poses"][k], 0.0) == R.RTCC_E_DUPLICATE
    assert not any(l.startswith("dispatch") for l in _host_log(clear=False))
    R.rtcc_release_branch(ctx, 0, fr["points"][0], fr["poses"][0], 0.5)
    disp = [l.split()[1] for l in _host_log() if l.startswith("dispatch")]
    assert disp == ["0", "1", "2", "3"]
    assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_RELEASED for k in range(4))
    R.rtcc_join_and_detect(ctx)
    assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_FINISHED for k in range(4))


def test_branch_state_follows_the_device(host_ctx):
    """RELEASED -> RUNNING -> FINISHED as the executor reports the encoder
    started and finished (eq. branch_state; Alg. 1): FINISHED at encoder
    completion, before the join."""
    cfg, fr, ctx = host_ctx
    lib = R.load("host")
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    for k in range(cfg["K"]):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
    assert R.rtcc_get_branch_state(ctx, 1) == R.RTCC_RELEASED
    lib.rtcc_hosttest_set_progress(1, 1)
    assert R.rtcc_get_branch_state(ctx, 1) == R.RTCC_RUNNING
    lib.rtcc_hosttest_set_progress(1, 2)
    assert R.rtcc_get_branch_state(ctx, 1) == R.RTCC_FINISHED
    # states never go back, and the others are untouched
    lib.rtcc_hosttest_set_progress(1, 0)
    assert R.rtcc_get_branch_state(ctx, 1) == R.RTCC_FINISHED
    assert R.rtcc_get_branch_state(ctx, 0) == R.RTCC_RELEASED
    lib.rtcc_hosttest_set_progress(2, 2)
    assert R.rtcc_get_branch_state(ctx, 2) == R.RTCC_FINISHED
    R.rtcc_join_and_detect(ctx)
    assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_FINISHED for k in range(cfg["K"]))


@pytest.mark.parametrize("mode", ["release", "barrier"])
def test_failed_dispatch_withholds_the_join(host_ctx, mode):
    """An encoder whose enqueue fails never reaches its slot: the join
    returns an error without running the post-join subgraph, a barrier
    release (one group of all K) leaves every branch undispatched, and the
    next frame runs normally."""
    cfg, fr, ctx = host_ctx
    lib = R.load("host")
    R.rtcc_set_mode(ctx, R.RTCC_MODE_BARRIER if mode == "barrier" else R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    lib.rtcc_hosttest_fail_dispatch(1)
    st = [_status(R.rtcc_release_branch, ctx, k, fr["points"][k], fr["poses"][k], 0.0) for k in range(cfg["K"])]
    if mode == "release":
        assert st == [R.RTCC_OK, R.RTCC_E_HIP, R.RTCC_OK, R.RTCC_OK]
    else:
        assert st == [R.RTCC_OK, R.RTCC_OK, R.RTCC_OK, R.RTCC_E_HIP]
    assert R.rtcc_get_branch_state(ctx, 1) == R.RTCC_WAITING
    disp = [l.split()[1] for l in _host_log() if l.startswith("dispatch")]
    assert disp == (["0", "2", "3"] if mode == "release" else [])
    if mode == "barrier":
        assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_WAITING for k in range(cfg["K"]))
    # a repeated event for the failed branch is still a duplicate
    assert _status(R.rtcc_release_branch, ctx, 1, fr["points"][1], fr["poses"][1], 0.0) == R.RTCC_E_DUPLICATE
    assert _status(R.rtcc_join_and_detect, ctx) == R.RTCC_E_STATE
    assert not any(l.startswith("join") for l in _host_log())
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    for k in range(cfg["K"]):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
    R.rtcc_join_and_detect(ctx)
    assert any(l.startswith("join") for l in _host_log())


def test_validation_errors_leave_branch_waiting(host_ctx):
    cfg, fr, ctx = host_ctx
    pts, pose = fr["points"][0], fr["poses"][0]
    # no frame open
    assert _status(R.rtcc_release_branch, ctx, 0, pts, pose, 0.0) == R.RTCC_E_STATE
    t0 = time.monotonic()
    R.rtcc_begin_frame(ctx, t0)
    assert _status(R.rtcc_release_branch, ctx, 7, pts, pose, 0.0) == R.RTCC_E_ARG
    assert _status(R.rtcc_release_branch, ctx, -1, pts, pose, 0.0) == R.RTCC_E_ARG
    too_many = np.zeros((cfg["n_points"] + 1, 4), np.float32)
    assert _status(R.rtcc_release_branch, ctx, 0, too_many, pose, 0.0) == R.RTCC_E_MALFORMED
    assert _status(R.rtcc_release_branch, ctx, 0, None, pose, 0.0, 5) == R.RTCC_E_MALFORMED
    assert _status(R.rtcc_release_branch, ctx, 0, pts, (math.nan, 0, 0), 0.0) == R.RTCC_E_MALFORMED
    assert _status(R.rtcc_release_branch, ctx, 0, pts, pose, math.inf) == R.RTCC_E_MALFORMED
    assert _status(R.rtcc_release_branch, ctx, 0, pts, pose, -1.0) == R.RTCC_E_MALFORMED
    # an event claiming an arrival 100 s from now is premature
    assert _status(R.rtcc_release_branch, ctx, 0, pts, pose, 100.0) == R.RTCC_E_PREMATURE
    assert R.rtcc_get_branch_state(ctx, 0) == R.RTCC_WAITING
    assert not any(l.startswith("dispatch") for l in _host_log())
    # a valid event, then a duplicate
    R.rtcc_release_branch(ctx, 0, pts, pose, 0.0)
    assert _status(R.rtcc_release_branch, ctx, 0, pts, pose, 0.0) == R.RTCC_E_DUPLICATE
    # mode change inside a frame
    assert _status(R.rtcc_set_mode, ctx, R.RTCC_MODE_BARRIER) == R.RTCC_E_STATE
    assert _status(R.rtcc_begin_frame, ctx, t0) == R.RTCC_E_STATE


def test_infeasible_frame_withholds_fusion(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    for k in (0, 1, 3):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
    assert _status(R.rtcc_join_and_detect, ctx) == R.RTCC_E_INFEASIBLE
    assert not any(l.startswith("join") for l in _host_log())
    # the frame is closed; a new one can start and complete
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    for k in range(4):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
    R.rtcc_join_and_detect(ctx)


def test_barrier_infeasible_dispatches_nothing(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_set_mode(ctx, R.RTCC_MODE_BARRIER)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    for k in (0, 1, 2):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
    assert _status(R.rtcc_join_and_detect, ctx) == R.RTCC_E_INFEASIBLE
    assert not any(l.startswith(("dispatch", "join")) for l in _host_log())


def test_staging_buffer_is_zero_copy(host_ctx):
    cfg, fr, ctx = host_ctx
    stg = R.rtcc_staging_buffer(ctx, 2)
    assert stg.shape == (cfg["n_points"], 4)
    n = 100
    stg[:n] = fr["points"][2][:n]
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    R.rtcc_release_branch(ctx, 2, stg[:n], fr["poses"][2], 0.0)
    assert _host_log()[-1].startswith("dispatch 2 n=100 src=staging staged=1 affine=[")


def test_concurrent_releases_from_threads(host_ctx):
    cfg, fr, ctx = host_ctx
    for _ in range(20):
        R.rtcc_begin_frame(ctx, time.monotonic() - 1)
        errs = []

        def rel(k):
            try:
                R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
            except Exception as e:  # pragma: no cover
                errs.append(e)

        th = [threading.Thread(target=rel, args=(k,)) for k in range(4)]
        for t in th:
            t.start()
        for t in th:
            t.join()
        assert not errs
        R.rtcc_join_and_detect(ctx)
        log = _host_log()
        assert sorted(l.split()[1] for l in log if l.startswith("dispatch")) == ["0", "1", "2", "3"]


def test_pose_affines_match_oracle(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    for k in range(4):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
    R.rtcc_join_and_detect(ctx)
    line = [l for l in _host_log() if l.startswith("join")][-1]
    mats = [list(map(float, m.split(","))) for m in re.findall(r"\[([^\]]+)\]", line)]
    for k in range(4):
        M, t = N.index_affine(fr["poses"][k], cfg)
        want = [M[0, 0], M[0, 1], t[0], M[1, 0], M[1, 1], t[1]]
        np.testing.assert_allclose(mats[k], want, rtol=1e-4, atol=1e-4)
    assert mats[0] == [1.0, 0.0, 0.0, 0.0, 1.0, 0.0] or mats[0][:3] == [1.0, 0.0, 0.0]


def test_dispatch_carries_the_agents_pose_warp(host_ctx):
    """The branch receives its own warp at dispatch (for a warp placed in
    the branch), the same affine the join receives."""
    cfg, fr, ctx = host_ctx
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    _host_log()
    R.rtcc_begin_frame(ctx, time.monotonic())
    for k in range(cfg["K"]):
        R.rtcc_release_branch(ctx, k, fr["points"][k], fr["poses"][k], 0.0)
    R.rtcc_join_and_detect(ctx)
    log = _host_log()
    disp = {int(l.split()[1]): l.split("affine=")[1] for l in log if l.startswith("dispatch")}
    join = [l for l in log if l.startswith("join")][-1]
    mats = join.split(" ", 1)[1].split(" ")
    assert [disp[k] for k in range(cfg["K"])] == mats


@pytest.mark.parametrize("field,value", [
    ("n_agents", 0), ("n_agents", 17), ("c_pfn", 48), ("pillar_size", 0.0), ("n_anchors", 3),
    ("precision", 5), ("fusion", 9), ("max_points", 0), ("abi_version", 99),
    ("nms_max_candidates", -1), ("nms_max_candidates", 16385), ("nms_iou_threshold", 1.5),
    ("nms_iou_threshold", -0.5), ("nms_iou_threshold", float("nan")), ("warp_in_branch", 2),
    ("warp_in_branch", -1), ("multiscale", 2),
])
def test_bad_descriptor_rejected(field, value):
    cfg = synth.config("t_max")
    w = R.weights_blob(cfg, synth.make_weights(cfg))
    d = R.model_desc(cfg)
    setattr(d, field, value)
    with pytest.raises(R.RtccError) as ei:
        R.rtcc_create(d, w, kind="host")
    assert ei.value.status == R.RTCC_E_ARG


def test_weight_blob_size_and_values_checked():
    cfg = synth.config("t_max")
    w = R.weights_blob(cfg, synth.make_weights(cfg))
    with pytest.raises(R.RtccError) as ei:
        R.rtcc_create(R.model_desc(cfg), w[:-1], kind="host")
    assert ei.value.status == R.RTCC_E_ARG
    bad = w.copy()
    bad[3] = np.nan
    with pytest.raises(R.RtccError):
        R.rtcc_create(R.model_desc(cfg), bad, kind="host")


def test_nms_off_and_threshold_edges_accepted():
    cfg = synth.config("t_max")
    w = R.weights_blob(cfg, synth.make_weights(cfg))
    for cap, thr in ((0, 7.0), (1, 0.0), (16384, 1.0)):
        d = R.model_desc(cfg)
        d.nms_max_candidates, d.nms_iou_threshold = cap, thr
        R.rtcc_create(d, w, kind="host").close()


def test_host_library_nms_entry_reports_no_gpu():
    lib = R.load("host")
    kept = ctypes.c_int64(5)
    assert lib.rtcc_rotated_nms(None, 0, 16, 0.15, None, ctypes.byref(kept)) == R.RTCC_E_STATE
    assert kept.value == 0 and b"GPU" in lib.rtcc_last_error(None)


def test_multiscale_needs_upsampling_and_a_post_join_warp():
    for name, extra in (("c1", {}), ("t_attn", {"warp_in_branch": True})):
        cfg = dict(synth.config(name), multiscale=True, **extra)
        fr = synth.make_frame(name)
        with pytest.raises(R.RtccError) as e:
            R.rtcc_create(R.model_desc(cfg), R.weights_blob(cfg, fr["weights"]), kind="host")
        assert e.value.status == R.RTCC_E_ARG
    cfg = dict(synth.config("t_attn"), multiscale=True)
    fr = synth.make_frame("t_attn")
    R.rtcc_create(R.model_desc(cfg), R.weights_blob(cfg, fr["weights"]), kind="host").close()


@pytest.mark.parametrize("field,value", [("use_graphs", 2), ("use_graphs", -1), ("node_timing", 3)])
def test_bad_runtime_opts_rejected(field, value):
    cfg = synth.config("t_max")
    w = R.weights_blob(cfg, synth.make_weights(cfg))
    o = R.rtcc_runtime_opts()
    o.exec = R.RTCC_EXEC_PER_BRANCH_STREAMS
    o.premature_tol_s = 1e-6
    setattr(o, field, value)
    with pytest.raises(R.RtccError) as ei:
        R.rtcc_create(R.model_desc(cfg), w, o, kind="host")
    assert ei.value.status == R.RTCC_E_ARG
    o.use_graphs, o.node_timing = 1, 0
    ctx = R.rtcc_create(R.model_desc(cfg), w, o, kind="host")
    assert R.rtcc_graph_stats(ctx) == (0, 0, 0)   # the recording executor runs no graphs
    ctx.close()


# --------------------------------------------------------- batched events

def _events(cfg, fr, agents, arrival=0.0):
    return [dict(agent=k, points=fr["points"][k], pose=fr["poses"][k], arrival_t=arrival) for k in agents]


def test_batch_release_is_one_group_in_index_order(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    _host_log()
    st = []
    R.rtcc_release_branches(ctx, _events(cfg, fr, [2, 0, 3, 1]), st)
    assert st == [R.RTCC_OK] * 4
    log = _host_log()
    assert log[0] == "group 0 1 2 3"
    assert [l.split()[1] for l in log[1:] if l.startswith("dispatch")] == ["0", "1", "2", "3"]
    assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_RELEASED for k in range(cfg["K"]))
    det = R.rtcc_join_and_detect(ctx)
    # released together: one dispatch time for the whole group
    assert len(set(det["dispatch_s"])) == 1


def test_batch_release_events_are_checked_one_by_one(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    R.rtcc_release_branch(ctx, 3, fr["points"][3], fr["poses"][3], 0.0)
    _host_log()
    ev = _events(cfg, fr, [0, 1, 0, 3, 2])
    ev[1]["pose"] = (math.nan, 0.0, 0.0)       # malformed
    ev[4]["arrival_t"] = 100.0                 # premature
    st = []
    with pytest.raises(R.RtccError) as e:
        R.rtcc_release_branches(ctx, ev, st)
    # the first rejected event names the call's status
    assert e.value.status == R.RTCC_E_MALFORMED and "event 1" in str(e.value)
    assert st == [R.RTCC_OK, R.RTCC_E_MALFORMED, R.RTCC_E_DUPLICATE, R.RTCC_E_DUPLICATE, R.RTCC_E_PREMATURE]
    # the one accepted event was released (a group of one: no group line)
    log = _host_log()
    assert [l.split()[1] for l in log if l.startswith("dispatch")] == ["0"]
    assert not any(l.startswith("group") for l in log)
    assert [R.rtcc_get_branch_state(ctx, k) for k in range(4)] == [
        R.RTCC_RELEASED, R.RTCC_WAITING, R.RTCC_WAITING, R.RTCC_RELEASED]
    # the rejected branches can still be released
    R.rtcc_release_branches(ctx, _events(cfg, fr, [1, 2]))
    R.rtcc_join_and_detect(ctx)


def test_batch_release_under_barrier(host_ctx):
    cfg, fr, ctx = host_ctx
    R.rtcc_set_mode(ctx, R.RTCC_MODE_BARRIER)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    _host_log()
    R.rtcc_release_branches(ctx, _events(cfg, fr, [3, 1]))
    assert not any(l.startswith("dispatch") for l in _host_log())
    assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_WAITING for k in range(4))
    R.rtcc_release_branch(ctx, 0, fr["points"][0], fr["poses"][0], 0.0)
    assert not _host_log()
    R.rtcc_release_branches(ctx, _events(cfg, fr, [2]))
    log = _host_log()
    assert log[0] == "group 0 1 2 3"
    assert [l.split()[1] for l in log if l.startswith("dispatch")] == ["0", "1", "2", "3"]
    R.rtcc_join_and_detect(ctx)


def test_batch_release_argument_errors(host_ctx):
    cfg, fr, ctx = host_ctx
    lib = R.load("host")
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    _host_log()
    st = (ctypes.c_int * 1)()
    assert lib.rtcc_release_branches(ctx.handle, 1, None, st) == R.RTCC_E_ARG
    assert lib.rtcc_release_branches(ctx.handle, -1, None, None) == R.RTCC_E_ARG
    assert lib.rtcc_release_branches(ctx.handle, R.RTCC_MAX_AGENTS + 1, None, None) == R.RTCC_E_ARG
    assert lib.rtcc_release_branches(None, 0, None, None) == R.RTCC_E_ARG
    assert lib.rtcc_release_branches(ctx.handle, 0, None, None) == R.RTCC_OK
    ev = _events(cfg, fr, [0])
    ev[0]["device"] = 2
    st = []
    assert _status(R.rtcc_release_branches, ctx, ev, st) == R.RTCC_E_MALFORMED
    assert st == [R.RTCC_E_MALFORMED]
    assert not any(l.startswith("dispatch") for l in _host_log())
    assert R.rtcc_get_branch_state(ctx, 0) == R.RTCC_WAITING


def test_batch_release_dispatch_failure_leaves_the_group_waiting(host_ctx):
    cfg, fr, ctx = host_ctx
    lib = R.load("host")
    R.rtcc_set_mode(ctx, R.RTCC_MODE_RELEASE)
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    lib.rtcc_hosttest_fail_dispatch(2)
    st = []
    assert _status(R.rtcc_release_branches, ctx, _events(cfg, fr, [0, 1, 2, 3]), st) == R.RTCC_E_HIP
    assert st == [R.RTCC_OK] * 4  # every event valid; the enqueue failed
    assert all(R.rtcc_get_branch_state(ctx, k) == R.RTCC_WAITING for k in range(4))
    assert _status(R.rtcc_join_and_detect, ctx) == R.RTCC_E_STATE
    R.rtcc_begin_frame(ctx, time.monotonic() - 1)
    R.rtcc_release_branches(ctx, _events(cfg, fr, [0, 1, 2, 3]))
    R.rtcc_join_and_detect(ctx)
