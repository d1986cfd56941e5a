"""ctypes binding of include/rtcc.h (argument marshalling only).

Every computation runs in ``lib/librtcc.so``.  The functions keep the C
names; a non-OK status raises :class:`RtccError` carrying the status and the
library's message.  Loading the library fails loudly when it is missing; there
is no fallback.

HIP runtime: PyTorch ships its own ``libamdhip64``; its libraries load it by
file name, so if this library loaded the system copy first a later
``import torch`` would bring a second runtime into the process.  The loader
therefore imports torch (when installed) before the library, so that the
library binds to the runtime already in the process.
"""

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_DIR = os.path.join(HERE, "lib")

RTCC_ABI_VERSION = 6
RTCC_MAX_AGENTS = 16
RTCC_MAX_STAGES = 4

STATUS = {
    0: "RTCC_OK", 1: "RTCC_E_ARG", 2: "RTCC_E_STATE", 3: "RTCC_E_DUPLICATE",
    4: "RTCC_E_MALFORMED", 5: "RTCC_E_PREMATURE", 6: "RTCC_E_INFEASIBLE",
    7: "RTCC_E_NOMEM", 8: "RTCC_E_HIP", 9: "RTCC_E_INTERNAL",
}
RTCC_OK, RTCC_E_ARG, RTCC_E_STATE, RTCC_E_DUPLICATE, RTCC_E_MALFORMED = 0, 1, 2, 3, 4
RTCC_E_PREMATURE, RTCC_E_INFEASIBLE, RTCC_E_NOMEM, RTCC_E_HIP, RTCC_E_INTERNAL = 5, 6, 7, 8, 9
RTCC_PREC_FP32, RTCC_PREC_BF16 = 0, 1
RTCC_FUSE_MAX, RTCC_FUSE_ATTN = 0, 1
RTCC_MODE_RELEASE, RTCC_MODE_BARRIER = 0, 1
RTCC_EXEC_PER_BRANCH_STREAMS, RTCC_EXEC_SERIAL = 0, 1
RTCC_WAITING, RTCC_RELEASED, RTCC_RUNNING, RTCC_FINISHED = 0, 1, 2, 3
(RTCC_T_PILLAR_CELLS, RTCC_T_PILLAR_COUNTS, RTCC_T_CANVAS, RTCC_T_SLOT, RTCC_T_FUSED,
 RTCC_T_HEAD, RTCC_T_STAGE_OUT, RTCC_T_DECODED, RTCC_T_WARPED, RTCC_T_FUSED_STAGE,
 RTCC_T_PILLAR_MEMBERS, RTCC_T_CONV_OUT) = range(12)
(RTCC_SCHED_MAXRATE, RTCC_SCHED_MAXWEIGHT, RTCC_SCHED_EARLIEST_RELEASE, RTCC_SCHED_WEIGHTED_RATE,
 RTCC_SCHED_ROUND_ROBIN, RTCC_SCHED_PROPORTIONAL_FAIR) = range(6)


class rtcc_stage(ctypes.Structure):
    _fields_ = [("stride", ctypes.c_int32), ("c_out", ctypes.c_int32), ("n_convs", ctypes.c_int32)]


class rtcc_model_desc(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_int32),
        ("n_agents", ctypes.c_int32),
        ("max_points", ctypes.c_int64),
        ("x_min", ctypes.c_float), ("x_max", ctypes.c_float),
        ("y_min", ctypes.c_float), ("y_max", ctypes.c_float),
        ("z_min", ctypes.c_float), ("z_max", ctypes.c_float),
        ("pillar_size", ctypes.c_float),
        ("max_points_per_pillar", ctypes.c_int32),
        ("c_pfn", ctypes.c_int32),
        ("precision", ctypes.c_int32),
        ("n_stages", ctypes.c_int32),
        ("stages", rtcc_stage * RTCC_MAX_STAGES),
        ("up_channels", ctypes.c_int32),
        ("fusion", ctypes.c_int32),
        ("n_anchors", ctypes.c_int32),
        ("anchor_w", ctypes.c_float), ("anchor_l", ctypes.c_float),
        ("anchor_h", ctypes.c_float), ("anchor_z", ctypes.c_float),
        ("anchor_yaw", ctypes.c_float * 2),
        ("score_logit_threshold", ctypes.c_float),
        ("nms_max_candidates", ctypes.c_int32),
        ("nms_iou_threshold", ctypes.c_float),
        ("warp_in_branch", ctypes.c_int32),
        ("multiscale", ctypes.c_int32),
    ]


DEV_ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p)
DEV_FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)


class rtcc_runtime_opts(ctypes.Structure):
    _fields_ = [
        ("exec", ctypes.c_int32),
        ("use_graphs", ctypes.c_int32),
        ("node_timing", ctypes.c_int32),
        ("device", ctypes.c_int32),
        ("premature_tol_s", ctypes.c_double),
        ("conv_variant", ctypes.c_int32),
        ("conv_splits", ctypes.c_int32),
        ("dev_alloc", DEV_ALLOC_FN),
        ("dev_free", DEV_FREE_FN),
        ("alloc_user", ctypes.c_void_p),
        ("join_stream", ctypes.c_void_p),
    ]


def use_torch_memory(opts, device=0, stream=None):
    """Route the context's device buffers through PyTorch's caching
    allocator (and, with ``stream``, run the post-join subgraph on that
    torch stream).  The callbacks are kept on ``opts``, which rtcc_create
    keeps alive with the context."""
    import torch

    def _alloc(nbytes, _user):
        try:
            return torch.cuda.caching_allocator_alloc(int(nbytes), device)
        except RuntimeError:
            return None

    def _free(ptr, _user):
        torch.cuda.caching_allocator_delete(ptr)

    opts._callbacks = (DEV_ALLOC_FN(_alloc), DEV_FREE_FN(_free))
    opts.dev_alloc, opts.dev_free = opts._callbacks
    if stream is not None:
        opts.join_stream = stream.cuda_stream
        opts._stream = stream
    return opts


class rtcc_uplink_desc(ctypes.Structure):
    _fields_ = [
        ("slots", ctypes.c_int32),
        ("agents", ctypes.c_int32),
        ("rbs", ctypes.c_int32),
        ("policy", ctypes.c_int32),
        ("slot_s", ctypes.c_double),
        ("agent_weight", ctypes.POINTER(ctypes.c_double)),
        ("pf_window", ctypes.c_double),
        ("pf_init_rate", ctypes.c_double),
    ]


class rtcc_event(ctypes.Structure):
    _fields_ = [
        ("agent", ctypes.c_int32),
        ("device", ctypes.c_int32),
        ("points", ctypes.c_void_p),
        ("n", ctypes.c_int64),
        ("pose", ctypes.c_float * 3),
        ("arrival_t", ctypes.c_double),
    ]


class rtcc_checkpoint_info(ctypes.Structure):
    _fields_ = [
        ("config_id", ctypes.c_char * 32),
        ("seed", ctypes.c_uint64),
        ("version", ctypes.c_int32),
        ("n_tensors", ctypes.c_int32),
        ("data_bytes", ctypes.c_uint64),
        ("sha256", ctypes.c_uint8 * 32),
    ]


class rtcc_detections(ctypes.Structure):
    _fields_ = [
        ("count", ctypes.c_int64),
        ("count_decoded", ctypes.c_int64),
        ("boxes", ctypes.POINTER(ctypes.c_float)),
        ("scores", ctypes.POINTER(ctypes.c_float)),
        ("anchor_idx", ctypes.POINTER(ctypes.c_int32)),
        ("t_head_s", ctypes.c_double),
        ("t_det_s", ctypes.c_double),
        ("n_agents", ctypes.c_int32),
        ("arrival_s", ctypes.c_double * RTCC_MAX_AGENTS),
        ("dispatch_s", ctypes.c_double * RTCC_MAX_AGENTS),
    ]


EXPORTS = (
    "rtcc_create", "rtcc_read_checkpoint", "rtcc_create_from_checkpoint", "rtcc_destroy", "rtcc_set_mode", "rtcc_staging_buffer", "rtcc_begin_frame",
    "rtcc_release_branch", "rtcc_release_branch_device", "rtcc_release_branches", "rtcc_join_and_detect",
    "rtcc_get_branch_state", "rtcc_tensor_bytes", "rtcc_get_tensor", "rtcc_profile_nodes",
    "rtcc_node_times", "rtcc_node_count", "rtcc_graph_stats", "rtcc_conv_plan", "rtcc_conv_tiling", "rtcc_rotated_nms", "rtcc_rotated_nms_noalloc", "rtcc_uplink_emulate", "rtcc_schedule_model",
    "rtcc_upward_rank", "rtcc_status_str", "rtcc_last_error",
)


class RtccError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        super().__init__("%s: %s" % (STATUS.get(status, status), message))


_P = ctypes.c_void_p
_F = ctypes.POINTER(ctypes.c_float)
_I64P = ctypes.POINTER(ctypes.c_int64)


def _declare(lib):
    S = ctypes.c_int
    sig = {
        "rtcc_create": (S, [ctypes.POINTER(rtcc_model_desc), _P, ctypes.c_size_t,
                            ctypes.POINTER(rtcc_runtime_opts), ctypes.POINTER(_P)]),
        "rtcc_read_checkpoint": (S, [_P, ctypes.c_size_t, ctypes.POINTER(rtcc_checkpoint_info)]),
        "rtcc_create_from_checkpoint": (S, [ctypes.POINTER(rtcc_model_desc), _P, ctypes.c_size_t,
                                            ctypes.POINTER(rtcc_runtime_opts), ctypes.POINTER(_P)]),
        "rtcc_destroy": (None, [_P]),
        "rtcc_set_mode": (S, [_P, ctypes.c_int]),
        "rtcc_staging_buffer": (S, [_P, ctypes.c_int32, ctypes.POINTER(_F), ctypes.POINTER(ctypes.c_int64)]),
        "rtcc_begin_frame": (S, [_P, ctypes.c_double]),
        "rtcc_release_branch": (S, [_P, ctypes.c_int32, _P, ctypes.c_int64, _F, ctypes.c_double]),
        "rtcc_release_branch_device": (S, [_P, ctypes.c_int32, _P, ctypes.c_int64, _F, ctypes.c_double]),
        "rtcc_release_branches": (S, [_P, ctypes.c_int32, ctypes.POINTER(rtcc_event), ctypes.POINTER(ctypes.c_int)]),
        "rtcc_join_and_detect": (S, [_P, ctypes.POINTER(rtcc_detections)]),
        "rtcc_get_branch_state": (S, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]),
        "rtcc_tensor_bytes": (S, [_P, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]),
        "rtcc_get_tensor": (S, [_P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_size_t]),
        "rtcc_profile_nodes": (S, [_P, ctypes.c_int32, ctypes.c_int32, _F, ctypes.POINTER(ctypes.c_int32)]),
        "rtcc_node_times": (S, [_P, _F, ctypes.POINTER(ctypes.c_int32)]),
        "rtcc_node_count": (S, [_P, ctypes.POINTER(ctypes.c_int32)]),
        "rtcc_graph_stats": (S, [_P, ctypes.POINTER(ctypes.c_int64)]),
        "rtcc_conv_plan": (S, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]),
        "rtcc_conv_tiling": (S, [ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                 ctypes.POINTER(ctypes.c_int32)]),
        "rtcc_rotated_nms": (S, [_P, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, _P,
                                 ctypes.POINTER(ctypes.c_int64)]),
        "rtcc_rotated_nms_noalloc": (S, [_P, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, _P,
                                         ctypes.POINTER(ctypes.c_int64), _P]),
        "rtcc_uplink_emulate": (S, [ctypes.POINTER(rtcc_uplink_desc), _P, _P, _P, _P, _P]),
        "rtcc_schedule_model": (S, [ctypes.c_int32, _P, _P, ctypes.c_int64, ctypes.c_int32, _I64P, _I64P, _P]),
        "rtcc_upward_rank": (S, [ctypes.c_int32, _P, ctypes.c_int32, _P, _P]),
        "rtcc_status_str": (ctypes.c_char_p, [ctypes.c_int]),
        "rtcc_last_error": (ctypes.c_char_p, [_P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_LIBS = {}


def lib_path(kind="gpu"):
    if kind == "host" and os.environ.get("RTCC_HOSTTEST_LIB"):
        # a sanitizer build of the host test library (build_sanitize.py)
        return os.environ["RTCC_HOSTTEST_LIB"]
    return os.path.join(LIB_DIR, "librtcc.so" if kind == "gpu" else "librtcc_hosttest.so")


def load(kind="gpu"):
    """Load the GPU library (``kind='gpu'``) or the host test library."""
    if kind in _LIBS:
        return _LIBS[kind]
    path = lib_path(kind)
    if not os.path.exists(path):
        raise RuntimeError("%s is not built; run python -m paper_2608_08330_amd.build" % path)
    if kind == "gpu":
        try:
            import torch  # noqa: F401  (binds the library to torch's HIP runtime)
        except ImportError:
            pass
    lib = _declare(ctypes.CDLL(path))
    if kind == "host":
        lib.rtcc_hosttest_log.restype = ctypes.c_size_t
        lib.rtcc_hosttest_log.argtypes = [ctypes.c_char_p, ctypes.c_size_t, ctypes.c_int]
        lib.rtcc_hosttest_set_progress.restype = None
        lib.rtcc_hosttest_set_progress.argtypes = [ctypes.c_int, ctypes.c_int]
        lib.rtcc_hosttest_fail_dispatch.restype = None
        lib.rtcc_hosttest_fail_dispatch.argtypes = [ctypes.c_int]
    _LIBS[kind] = lib
    return lib


# ----------------------------------------------------------------------------
# descriptor and weight blob marshalling
# ----------------------------------------------------------------------------

def model_desc(cfg, max_points=None):
    """rtcc_model_desc of a workload description."""
    d = rtcc_model_desc()
    d.abi_version = RTCC_ABI_VERSION
    d.n_agents = cfg["K"]
    d.max_points = int(max_points if max_points is not None else cfg["n_points"])
    d.x_min, d.x_max = cfg["x_range"]
    d.y_min, d.y_max = cfg["y_range"]
    d.z_min, d.z_max = cfg["z_range"]
    d.pillar_size = cfg["pillar"]
    d.max_points_per_pillar = cfg["max_pts"]
    d.c_pfn = cfg["c_pfn"]
    d.precision = RTCC_PREC_BF16 if cfg["precision"] == "bf16" else RTCC_PREC_FP32
    d.n_stages = len(cfg["stages"])
    for i, (s, c, n) in enumerate(cfg["stages"]):
        d.stages[i] = rtcc_stage(s, c, n)
    d.up_channels = cfg["up_channels"]
    d.fusion = RTCC_FUSE_ATTN if cfg["fusion"] == "attn" else RTCC_FUSE_MAX
    d.n_anchors = cfg["n_anchors"]
    d.anchor_w, d.anchor_l, d.anchor_h, d.anchor_z = (
        cfg["anchor_w"], cfg["anchor_l"], cfg["anchor_h"], cfg["anchor_z"])
    d.anchor_yaw[0], d.anchor_yaw[1] = cfg["anchor_yaws"]
    d.score_logit_threshold = cfg["logit_threshold"]
    d.nms_max_candidates = cfg.get("nms_max_candidates", 0)
    d.nms_iou_threshold = cfg.get("nms_iou_threshold", 0.0)
    d.warp_in_branch = int(bool(cfg.get("warp_in_branch", False)))
    d.multiscale = int(bool(cfg.get("multiscale", False)))
    return d


def weight_order(cfg):
    """Tensor names in the order of the library's weight blob."""
    names = ["pfn_w", "pfn_b"]
    for s, (_stride, _c, n) in enumerate(cfg["stages"]):
        for l in range(n):
            names += ["s%dc%d_w" % (s, l), "s%dc%d_b" % (s, l)]
    if cfg["up_channels"]:
        for s in range(len(cfg["stages"])):
            names += ["up%d_w" % s, "up%d_b" % s]
    return names + ["head_w", "head_b"]


def weights_blob(cfg, weights):
    """Concatenate float32 tensors in blob order (little endian)."""
    parts = [np.ascontiguousarray(weights[n], dtype="<f4").ravel() for n in weight_order(cfg)]
    return np.concatenate(parts)


# ----------------------------------------------------------------------------
# C functions
# ----------------------------------------------------------------------------

class Context:
    """Owns an ``rtcc_ctx *``; the methods call the C functions of the same
    name with the context as first argument."""

    def __init__(self, lib, handle):
        self.lib = lib
        self.handle = handle

    def check(self, status):
        if status != RTCC_OK:
            msg = self.lib.rtcc_last_error(self.handle)
            raise RtccError(status, msg.decode() if msg else "")
        return status

    def close(self):
        if self.handle:
            self.lib.rtcc_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def rtcc_create(desc, blob, opts=None, kind="gpu"):
    lib = load(kind)
    blob = np.ascontiguousarray(blob, dtype="<f4")
    h = _P()
    st = lib.rtcc_create(ctypes.byref(desc), blob.ctypes.data_as(_P), blob.nbytes,
                         ctypes.byref(opts) if opts is not None else None, ctypes.byref(h))
    if st != RTCC_OK:
        msg = lib.rtcc_last_error(None)
        raise RtccError(st, msg.decode() if msg else "")
    ctx = Context(lib, h)
    ctx._opts = opts  # keeps allocator callbacks alive with the context
    return ctx


def rtcc_read_checkpoint(data, kind="gpu"):
    """Verify a checkpoint (bytes); returns a dict of its manifest."""
    lib = load(kind)
    buf = ctypes.create_string_buffer(bytes(data), len(data))
    info = rtcc_checkpoint_info()
    st = lib.rtcc_read_checkpoint(buf, len(data), ctypes.byref(info))
    if st != RTCC_OK:
        msg = lib.rtcc_last_error(None)
        raise RtccError(st, msg.decode() if msg else "")
    return dict(config_id=info.config_id.decode(), seed=int(info.seed), version=int(info.version),
                n_tensors=int(info.n_tensors), data_bytes=int(info.data_bytes), sha256=bytes(info.sha256).hex())


def rtcc_create_from_checkpoint(desc, data, opts=None, kind="gpu"):
    lib = load(kind)
    buf = ctypes.create_string_buffer(bytes(data), len(data))
    h = _P()
    st = lib.rtcc_create_from_checkpoint(ctypes.byref(desc), buf, len(data),
                                         ctypes.byref(opts) if opts is not None else None, ctypes.byref(h))
    if st != RTCC_OK:
        msg = lib.rtcc_last_error(None)
        raise RtccError(st, msg.decode() if msg else "")
    ctx = Context(lib, h)
    ctx._opts = opts
    return ctx


def rtcc_destroy(ctx):
    ctx.close()


def rtcc_set_mode(ctx, mode):
    return ctx.check(ctx.lib.rtcc_set_mode(ctx.handle, int(mode)))


def rtcc_staging_buffer(ctx, agent):
    """numpy view [capacity, 4] float32 of the agent's pinned staging buffer."""
    p = _F()
    cap = ctypes.c_int64()
    ctx.check(ctx.lib.rtcc_staging_buffer(ctx.handle, agent, ctypes.byref(p), ctypes.byref(cap)))
    return np.ctypeslib.as_array(p, shape=(cap.value, 4))


def rtcc_begin_frame(ctx, t0):
    return ctx.check(ctx.lib.rtcc_begin_frame(ctx.handle, float(t0)))


def _pose(pose):
    a = (ctypes.c_float * 3)(*[float(v) for v in pose])
    return ctypes.cast(a, _F), a


def rtcc_release_branch(ctx, agent, host_points, pose, arrival_t, n=None):
    """host_points: float32 [n, 4] numpy array (or the staging view)."""
    if host_points is None:
        ptr, n = None, int(n or 0)
    else:
        arr = np.ascontiguousarray(host_points, dtype=np.float32)
        if arr.ndim != 2 or arr.shape[1] != 4:
            raise ValueError("host_points must be [n, 4] float32")
        n = arr.shape[0] if n is None else int(n)
        ptr = arr.ctypes.data_as(_P)
    pp, keep = _pose(pose)
    return ctx.check(ctx.lib.rtcc_release_branch(ctx.handle, agent, ptr, n, pp, float(arrival_t)))


def rtcc_release_branch_device(ctx, agent, device_ptr, n, pose, arrival_t):
    pp, keep = _pose(pose)
    return ctx.check(ctx.lib.rtcc_release_branch_device(ctx.handle, agent, _P(device_ptr), int(n), pp,
                                                        float(arrival_t)))


def rtcc_release_branches(ctx, events, statuses=None):
    """Events that arrived together.  ``events``: list of dicts with agent,
    points (a float32 [n, 4] host array, or with device=1 a device pointer
    int), n (device events), pose, arrival_t.  Raises on a non-OK status; with
    ``statuses`` (a list) each event's status is appended to it."""
    m = len(events)
    arr = (rtcc_event * max(m, 1))()
    keep = []
    for i, e in enumerate(events):
        ev = arr[i]
        ev.agent = int(e["agent"])
        ev.device = int(e.get("device", 0))
        if ev.device == 1:
            ev.points = int(e["points"])
            ev.n = int(e["n"])
        else:
            p = np.ascontiguousarray(e["points"], dtype=np.float32).reshape(-1, 4)
            keep.append(p)
            ev.points = p.ctypes.data if len(p) else None
            ev.n = int(e.get("n", len(p)))
        ev.pose[:] = [float(v) for v in e["pose"]]
        ev.arrival_t = float(e["arrival_t"])
    st = (ctypes.c_int * max(m, 1))()
    r = ctx.lib.rtcc_release_branches(ctx.handle, m, arr, st)
    if statuses is not None:
        statuses.extend(int(st[i]) for i in range(m))
    return ctx.check(r)


def rtcc_join_and_detect(ctx):
    """Returns a dict with numpy copies of the detections and the timings."""
    d = rtcc_detections()
    ctx.check(ctx.lib.rtcc_join_and_detect(ctx.handle, ctypes.byref(d)))
    n = d.count
    boxes = np.ctypeslib.as_array(d.boxes, shape=(n, 7)).copy() if n else np.zeros((0, 7), np.float32)
    scores = np.ctypeslib.as_array(d.scores, shape=(n,)).copy() if n else np.zeros(0, np.float32)
    aidx = np.ctypeslib.as_array(d.anchor_idx, shape=(n,)).copy() if n else np.zeros(0, np.int32)
    K = d.n_agents
    return dict(count=n, count_decoded=d.count_decoded, boxes=boxes, scores=scores, anchor_idx=aidx,
                t_head_s=d.t_head_s,
                t_det_s=d.t_det_s, arrival_s=list(d.arrival_s[:K]), dispatch_s=list(d.dispatch_s[:K]))


def decoded_records(ctx):
    """Decoded anchors of the last frame before NMS (RTCC_T_DECODED) as a
    dict of boxes [n][7] float32, scores [n] float32, anchor_idx [n] int32."""
    raw = rtcc_get_tensor(ctx, RTCC_T_DECODED, 0, np.float32).reshape(-1, 9)
    return dict(boxes=raw[:, :7].copy(), scores=raw[:, 7].copy(),
                anchor_idx=raw[:, 8].copy().view(np.int32))


def rtcc_rotated_nms(device_records, n, max_candidates, iou_threshold, device_out, kind="gpu"):
    """Rotated NMS of [n][9] device records into device_out; returns the
    number kept.  Pointers are integers (e.g. torch ``data_ptr()``)."""
    lib = load(kind)
    kept = ctypes.c_int64()
    st = lib.rtcc_rotated_nms(_P(device_records), n, max_candidates, iou_threshold, _P(device_out),
                              ctypes.byref(kept))
    if st != 0:
        raise RtccError(st, (lib.rtcc_last_error(None) or b"").decode())
    return kept.value


def rtcc_rotated_nms_noalloc(device_records, n, max_candidates, iou_threshold, device_out, stream=0,
                             kind="gpu"):
    """rtcc_rotated_nms without device allocation, on a HIP stream handle
    (integer, 0 = the null stream); returns the number kept."""
    lib = load(kind)
    kept = ctypes.c_int64()
    st = lib.rtcc_rotated_nms_noalloc(_P(device_records), n, max_candidates, iou_threshold, _P(device_out),
                                      ctypes.byref(kept), _P(stream))
    if st != 0:
        raise RtccError(st, (lib.rtcc_last_error(None) or b"").decode())
    return kept.value


def _free_call(lib, st):
    if st != 0:
        raise RtccError(st, (lib.rtcc_last_error(None) or b"").decode())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_P)


def rtcc_uplink_emulate(rates, payload_bits, policy, slot_s, agent_weight=None, avail_slot=None,
                        pf_window=100.0, pf_init_rate=1.0, want_alloc=False, kind="gpu"):
    """Slot-level uplink emulation.  rates [T, K, F] bit/s, payload_bits [K].
    Returns the completion slot per agent (int32, 0 = undelivered) and, with
    want_alloc, the [T, F] agent given each RB (-1 idle)."""
    lib = load(kind)
    R = np.ascontiguousarray(rates, dtype=np.float64)
    if R.ndim != 3:
        raise ValueError("rates must be [T, K, F]")
    T, K, F = R.shape
    B = np.ascontiguousarray(payload_bits, dtype=np.float64)
    if B.shape != (K,):
        raise ValueError("payload_bits must be [K]")
    d = rtcc_uplink_desc(T, K, F, int(policy), float(slot_s), None, float(pf_window), float(pf_init_rate))
    w = None
    if agent_weight is not None:
        w = np.ascontiguousarray(agent_weight, dtype=np.float64)
        if w.shape != (K,):
            raise ValueError("agent_weight must be [K]")
        d.agent_weight = w.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    ell = None if avail_slot is None else np.ascontiguousarray(avail_slot, dtype=np.int32)
    if ell is not None and ell.shape != (K,):
        raise ValueError("avail_slot must be [K]")
    done = np.zeros(K, dtype=np.int32)
    alloc = np.empty((T, F), dtype=np.int32) if want_alloc else None
    _free_call(lib, lib.rtcc_uplink_emulate(ctypes.byref(d), _ptr(R), _ptr(B), _ptr(ell), _ptr(done), _ptr(alloc)))
    return (done, alloc) if want_alloc else done


def rtcc_schedule_model(arrival_ns, encoder_ns, post_ns, mode, kind="gpu"):
    """Single-stream latency of one arrival vector (integer ns).  Returns
    (latency_ns, pre_arrival_ns, start_ns[K])."""
    lib = load(kind)
    a = np.ascontiguousarray(arrival_ns, dtype=np.int64)
    c = np.ascontiguousarray(encoder_ns, dtype=np.int64)
    if a.ndim != 1 or c.shape != a.shape:
        raise ValueError("arrival_ns and encoder_ns must be [K]")
    lat, pre = ctypes.c_int64(), ctypes.c_int64()
    start = np.zeros(len(a), dtype=np.int64)
    _free_call(lib, lib.rtcc_schedule_model(len(a), _ptr(a), _ptr(c), int(post_ns), int(mode), ctypes.byref(lat),
                                            ctypes.byref(pre), _ptr(start)))
    return lat.value, pre.value, start


def rtcc_upward_rank(cost_ns, edges, kind="gpu"):
    """Upward rank (ns) of every node; edges is a sequence of (u, v) pairs,
    v depending on u."""
    lib = load(kind)
    c = np.ascontiguousarray(cost_ns, dtype=np.int64)
    e = np.ascontiguousarray(np.asarray(edges, dtype=np.int32).reshape(-1, 2))
    out = np.zeros(len(c), dtype=np.int64)
    _free_call(lib, lib.rtcc_upward_rank(len(c), _ptr(c), len(e), _ptr(e) if len(e) else None, _ptr(out)))
    return out


def rtcc_get_branch_state(ctx, agent):
    s = ctypes.c_int32()
    ctx.check(ctx.lib.rtcc_get_branch_state(ctx.handle, agent, ctypes.byref(s)))
    return s.value


def rtcc_tensor_bytes(ctx, tid, agent=0):
    b = ctypes.c_size_t()
    ctx.check(ctx.lib.rtcc_tensor_bytes(ctx.handle, tid, agent, ctypes.byref(b)))
    return b.value


def rtcc_get_tensor(ctx, tid, agent=0, dtype=np.uint8):
    nbytes = rtcc_tensor_bytes(ctx, tid, agent)
    buf = np.empty(nbytes, dtype=np.uint8)
    ctx.check(ctx.lib.rtcc_get_tensor(ctx.handle, tid, agent, buf.ctypes.data_as(_P), nbytes))
    return buf.view(dtype)


def rtcc_profile_nodes(ctx, warmup=5, reps=30):
    out = (ctypes.c_float * (RTCC_MAX_AGENTS + 1))()
    n = ctypes.c_int32()
    ctx.check(ctx.lib.rtcc_profile_nodes(ctx.handle, warmup, reps, out, ctypes.byref(n)))
    return np.array(out[:n.value], dtype=np.float64)


def rtcc_node_count(ctx):
    n = ctypes.c_int32()
    ctx.check(ctx.lib.rtcc_node_count(ctx.handle, ctypes.byref(n)))
    return n.value


def rtcc_conv_plan(ctx, layer):
    """(tiling, K slices) of 3x3 conv layer ``layer``."""
    out = (ctypes.c_int32 * 2)()
    ctx.check(ctx.lib.rtcc_conv_plan(ctx.handle, int(layer), out))
    return int(out[0]), int(out[1])


def rtcc_conv_tiling(Hi, Wi, Ci, Ho, Wo, Co, stride, n_cu, maps=1, bf16=True, lib=None):
    """(tiling, K slices) the library plans for a 3x3 conv layer of this shape
    on a GPU with n_cu compute units, in a launch over `maps` maps (host
    computation; `lib`: a loaded library, default the GPU library)."""
    lib = lib if lib is not None else load()
    shape = (ctypes.c_int32 * 8)(Hi, Wi, Ci, Ho, Wo, Co, stride, n_cu)
    out = (ctypes.c_int32 * 2)()
    st = lib.rtcc_conv_tiling(1 if bf16 else 0, shape, int(maps), out)
    if st != RTCC_OK:
        raise RtccError(st, "rtcc_conv_tiling")
    return int(out[0]), int(out[1])


def rtcc_graph_stats(ctx):
    """(instantiated, update attempts, launches) of the context's HIP graphs."""
    out = (ctypes.c_int64 * 3)()
    ctx.check(ctx.lib.rtcc_graph_stats(ctx.handle, out))
    return tuple(out)


def rtcc_node_times(ctx):
    cap = max(rtcc_node_count(ctx), 1)
    out = (ctypes.c_float * cap)()
    n = ctypes.c_int32()
    ctx.check(ctx.lib.rtcc_node_times(ctx.handle, out, ctypes.byref(n)))
    return np.array(out[:n.value], dtype=np.float64)


def rtcc_status_str(status):
    return load().rtcc_status_str(int(status)).decode()


def bf16_bits_to_f32(u16):
    """Widen raw bfloat16 bit patterns (uint16) to float32 (exact)."""
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
