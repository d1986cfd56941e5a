"""Real-time replay of arrival traces through the library (harness layer).

A trace is an arrival vector a (seconds since the frame's uplink start).
Each branch input is written to its pinned staging buffer before the frame
(inputs stay in pinned host memory until their arrival, Sec. IV-F); the
replay loop spins on CLOCK_MONOTONIC until t0 + a_k and then signals the
completion event e_k = Complete(k, a_k) through rtcc_release_branch, in
(a_k, k) order.  Both release rules leave the GPU idle before the first
arrival, so the replay starts at a_min and adds it back to the measured
latencies.
"""

import time

import numpy as np

from . import rtcc as R


def stage_inputs(ctx, points):
    views = []
    for k, p in enumerate(points):
        stg = R.rtcc_staging_buffer(ctx, k)
        stg[: len(p)] = p
        views.append(stg[: len(p)])
    return views


def replay_frame(ctx, staged, poses, a, mode, resident=False):
    """Run one frame; returns dict with T^head, T^det (s since the uplink
    start), dispatch lateness per agent and the detections count.
    ``staged`` holds the pinned staging views, or with ``resident`` the
    (device pointer, point count) of every agent's device-resident input
    (the resident-input runs of Sec. V-C)."""
    a = np.asarray(a, dtype=np.float64)
    shift = float(a.min())
    rel = a - shift
    R.rtcc_set_mode(ctx, mode)
    order = sorted(range(len(a)), key=lambda k: (a[k], k))
    t0 = time.monotonic()
    R.rtcc_begin_frame(ctx, t0)
    for k in order:
        target = t0 + rel[k]
        while time.monotonic() < target:
            pass
        if resident:
            R.rtcc_release_branch_device(ctx, k, staged[k][0], staged[k][1], poses[k], float(rel[k]))
        else:
            R.rtcc_release_branch(ctx, k, staged[k], poses[k], float(rel[k]))
    det = R.rtcc_join_and_detect(ctx)
    lateness = [det["dispatch_s"][k] - rel[k] for k in range(len(a))]
    return dict(t_head=det["t_head_s"] + shift, t_det=det["t_det_s"] + shift,
                lateness=lateness, count=det["count"], anchor_idx=det["anchor_idx"])


def bootstrap_ci(x, n=10000, seed=0, alpha=0.05):
    """Percentile bootstrap CI of the mean (independent trace-level
    observations are the statistical unit)."""
    x = np.asarray(x, dtype=np.float64)
    if len(x) < 2:
        return (float(x.mean()), float(x.mean())) if len(x) else (float("nan"), float("nan"))
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, len(x), (n, len(x)))
    means = x[idx].mean(axis=1)
    return float(np.quantile(means, alpha / 2)), float(np.quantile(means, 1 - alpha / 2))


def replay_traces(ctx, staged, poses, arrivals_s, reps, start=0, resident=False):
    """Paired RTCC / barrier replay of every trace, alternating which mode
    runs first per repetition; repetitions are averaged per trace.
    ``staged`` are the pinned staging views from :func:`stage_inputs`;
    ``start`` is the global index of the first trace (order alternation)."""
    rows = []
    identical = True
    for t, a in enumerate(arrivals_s, start):
        tr = {"R": [], "B": []}
        ids = {}
        for r in range(reps):
            modes = (("R", R.RTCC_MODE_RELEASE), ("B", R.RTCC_MODE_BARRIER))
            if (t + r) % 2:
                modes = modes[::-1]
            for key, mode in modes:
                res = replay_frame(ctx, staged, poses, a, mode, resident)
                tr[key].append(res)
                ids.setdefault(key, res["anchor_idx"])
                identical &= np.array_equal(ids[key], res["anchor_idx"])
        identical &= np.array_equal(ids["R"], ids["B"])
        rows.append(dict(
            a=[float(v) for v in a],
            A=float(np.max(a)), spread=float(np.max(a) - np.min(a)),
            R_det=float(np.mean([x["t_det"] for x in tr["R"]])),
            B_det=float(np.mean([x["t_det"] for x in tr["B"]])),
            R_det_med=float(np.median([x["t_det"] for x in tr["R"]])),
            B_det_med=float(np.median([x["t_det"] for x in tr["B"]])),
            R_head=float(np.mean([x["t_head"] for x in tr["R"]])),
            B_head=float(np.mean([x["t_head"] for x in tr["B"]])),
            lateness=[l for x in tr["R"] for l in x["lateness"]],
        ))
    return rows, identical


def summarize(rows):
    Rd = np.array([r["R_det"] for r in rows]) * 1e3
    Bd = np.array([r["B_det"] for r in rows]) * 1e3
    Rh = np.array([r["R_head"] for r in rows]) * 1e3
    Bh = np.array([r["B_head"] for r in rows]) * 1e3
    gain = Bd - Rd
    lo, hi = bootstrap_ci(gain)
    late = np.array([l for r in rows for l in r["lateness"]]) * 1e3
    return dict(
        traces=len(rows),
        A_p50_ms=float(np.median([r["A"] for r in rows]) * 1e3),
        rtcc_det_p50_ms=float(np.percentile(Rd, 50)), rtcc_det_p95_ms=float(np.percentile(Rd, 95)),
        barrier_det_p50_ms=float(np.percentile(Bd, 50)), barrier_det_p95_ms=float(np.percentile(Bd, 95)),
        rtcc_head_p50_ms=float(np.percentile(Rh, 50)), barrier_head_p50_ms=float(np.percentile(Bh, 50)),
        mean_gain_ms=float(gain.mean()), gain_ci95_ms=[lo, hi],
        wins=int(np.sum(gain > 0)),
        wins_median=int(sum(r["R_det_med"] < r["B_det_med"] for r in rows)),
        dispatch_lateness_p50_ms=float(np.percentile(late, 50)) if late.size else None,
        dispatch_lateness_p95_ms=float(np.percentile(late, 95)) if late.size else None,
    )
