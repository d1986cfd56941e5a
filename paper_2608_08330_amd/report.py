"""Latency report: RTCC vs barrier over replayed arrival traces of a config.

  python -m paper_2608_08330_amd.report --config c4 [--setting I] \
      [--traces N] [--reps R] [--exec serial|streams] --out FILE.json

For every trace the same branch-arrival vector is replayed under both
release rules (order alternating per repetition, Sec. V-A3); repetitions
are averaged per trace and traces are the statistical unit (mean paired gain
with a 10,000-resample bootstrap CI).  Uplink-driven configs derive each
agent's payload from its pillar count (pillars x 64 channels x 2 bytes) and
its completion time from the slot-level uplink emulation.  The profiled
node times (warm-up 5, median of 30, Sec. IV-A) give the DAG-predicted gain
of every trace, reported beside the measured one (Pearson r, MAE).
"""

import argparse
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

import synth  # noqa: E402
from . import dag, replay, uplink  # noqa: E402
from . import rtcc as R  # noqa: E402


def settings(cfg):
    arr = cfg["arrivals"]
    if arr["kind"] != "uplink":
        return [dict(kind=arr["kind"])]
    return [dict(kind="uplink", snr_db=s, scheduler=p) for s in arr["snr_db"] for p in arr["schedulers"]]


def arrivals_for(cfg, setting, n_traces, pillars):
    if setting["kind"] != "uplink":
        return synth.arrival_draws(cfg, n_traces) * 1e-3, 0
    arr = cfg["arrivals"]
    bits = np.asarray(pillars, dtype=np.float64) * arr["bytes_per_pillar"] * 8.0
    out, infeasible = [], 0
    for t in range(n_traces):
        g = synth.fading_draws(cfg, t)
        a = uplink.completion_times(g, bits, setting["snr_db"], arr["bandwidth_hz"], arr["slot_s"],
                                    setting["scheduler"], arr["pf_window"])
        if np.all(np.isfinite(a)):
            out.append(a)
        else:
            infeasible += 1
    return np.array(out), infeasible


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", required=True)
    ap.add_argument("--setting", type=int, default=None)
    ap.add_argument("--traces", type=int, default=None)
    ap.add_argument("--reps", type=int, default=None)
    ap.add_argument("--exec", choices=["serial", "streams"], default="serial")
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)

    cfg = synth.config(a.config)
    fr = synth.make_frame(cfg)
    o = R.rtcc_runtime_opts()
    o.exec = R.RTCC_EXEC_SERIAL if a.exec == "serial" else R.RTCC_EXEC_PER_BRANCH_STREAMS
    o.premature_tol_s = 1e-6
    ctx = R.rtcc_create(R.model_desc(cfg), R.weights_blob(cfg, fr["weights"]), o)
    staged = replay.stage_inputs(ctx, fr["points"])
    # one frame from host memory: pillar counts (payload sizes) and node profile
    R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
    for k in range(cfg["K"]):
        R.rtcc_release_branch(ctx, k, staged[k], fr["poses"][k], 0.0)
    R.rtcc_join_and_detect(ctx)
    pillars = [R.rtcc_tensor_bytes(ctx, R.RTCC_T_PILLAR_CELLS, k) // 4 for k in range(cfg["K"])]
    prof = R.rtcc_profile_nodes(ctx, 5, 30) * 1e-3
    c_enc, c_post = prof[:cfg["K"]], float(prof[cfg["K"]])
    n_traces = a.traces or cfg["traces"]
    reps = a.reps or cfg["reps"]
    sets = settings(cfg)
    idx = range(len(sets)) if a.setting is None else [a.setting]
    results = []
    for i in idx:
        st = sets[i]
        arr, infeasible = arrivals_for(cfg, st, n_traces, pillars)
        t0 = time.time()
        rows, identical = [], True
        for t in range(len(arr)):
            r, same = replay.replay_traces(ctx, staged, fr["poses"], arr[t:t + 1], reps, start=t)
            rows += r
            identical &= same
            print("# %s setting %d trace %d/%d A=%.3f s gain=%.3f ms (%.0f s)" % (
                a.config, i, t, len(arr), r[0]["A"], (r[0]["B_det"] - r[0]["R_det"]) * 1e3,
                time.time() - t0), flush=True)
        summ = replay.summarize(rows)
        pred = np.array([dag.predicted_gain(x, c_enc, c_post) for x in arr]) * 1e3
        meas = np.array([(r["B_head"] - r["R_head"]) * 1e3 for r in rows])
        summ.update(
            setting=st, reps=reps, infeasible_traces=infeasible,
            outputs_identical_rtcc_vs_barrier=bool(identical),
            rtcc_below_barrier_every_trace=bool(summ["wins_median"] == len(rows)),
            dag_pred_gain_mean_ms=float(pred.mean()), head_gain_mean_ms=float(meas.mean()),
            dag_vs_measured_r=float(np.corrcoef(pred, meas)[0, 1]) if len(rows) > 2 and pred.std() > 0 else None,
            dag_vs_measured_mae_ms=float(np.mean(np.abs(pred - meas))),
        )
        print(json.dumps(summ), flush=True)
        summ["per_trace"] = [dict(a_ms=[v * 1e3 for v in r["a"]], rtcc_det_ms=r["R_det"] * 1e3,
                                  barrier_det_ms=r["B_det"] * 1e3, rtcc_det_med_ms=r["R_det_med"] * 1e3,
                                  barrier_det_med_ms=r["B_det_med"] * 1e3, pred_gain_ms=float(p))
                             for r, p in zip(rows, pred)]
        results.append(summ)
    out = dict(config=a.config, exec=a.exec, pillars=pillars, node_ms=(prof * 1e3).tolist(), results=results)
    with open(a.out, "w") as f:
        json.dump(out, f, indent=1)
    ctx.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
