"""Measured-DAG load sweep over the OFDMA uplink (Sec. V-C and V-D).

  python -m paper_2608_08330_amd.sweep [--config s6] [--traces 30]
      [--node-ms E0,...,E5,POST | --profile] [--replay N] [--reps 3]
      [--lib gpu|host] --out FILE.json

Every trial pairs RTCC and Barrier on one arrival vector: a channel trace
(seeded OFDMA draws), a payload scale gamma, a bandwidth scale beta and one
of the five causal schedulers (MaxRate, MaxWeight, EarliestRelease, DAGRank,
Task-Weighted MaxRate) give the completion slots (rtcc_uplink_emulate); the
profiled service times of the DAG's nodes (rtcc_profile_nodes on the GPU:
warm-up 5, median of 30, Sec. IV-A) give T_R, T_B and the pre-arrival
encoder work W_pre (rtcc_schedule_model, integer nanoseconds), and the gain
identity T_B - T_R = W_pre is checked exactly on every trial.  The default
grid is 4 gammas x 5 betas x 5 schedulers x 30 traces = 3,000 trials.

Reported, as in the paper's load-robustness and scheduler-compatibility
figures: per (gamma, beta) cell the mean gain over the five schedulers, the
mean relative reduction (gain / T_B), the worst scheduler's mean gain, the
best RTCC scheduler (lowest mean T_R), and for every scheduler-load cell the
mean gain with a 10,000-resample bootstrap 95% CI; at the nominal load per
scheduler the mean Barrier and RTCC latency, the overlap window A - min a,
wins and the share of trials within the service deadline.

--replay N replays N nominal-load trials through the library on the GPU with
device-resident inputs (RTCC and Barrier, --reps repetitions each, order
alternating) and compares the measured T^head gain with the DAG prediction
(Pearson r, mean absolute error).
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
from . import channel, dag, replay, uplink  # noqa: E402
from . import rtcc as R  # noqa: E402


def grid(cfg):
    arr = cfg["arrivals"]
    return [(g, b) for g in arr["gammas"] for b in arr["betas"]]


def run_trials(cfg, c_enc_ns, c_post_ns, traces, kind="gpu", cells=None, schedulers=None):
    """Every (trace, gamma, beta, scheduler) trial; list of dicts."""
    arr = cfg["arrivals"]
    n_pts = synth.points_per_agent(cfg)
    slot_ns = int(round(arr["slot_s"] * 1e9))
    omega = dag.dagrank_weights(c_enc_ns, c_post_ns, kind=kind)
    weights = dict(dagrank=omega, tw_maxrate=list(arr["task_weights"]))
    cells = grid(cfg) if cells is None else cells
    schedulers = arr["schedulers"] if schedulers is None else schedulers
    betas = sorted({b for _, b in cells})
    out = []
    for t in traces:
        draw = synth.ofdma_draws(cfg, t)
        rates = {b: channel.rates(draw, cfg, b) for b in betas}
        for gamma, beta in cells:
            B = channel.payload_bits(cfg, n_pts, gamma)
            for s in schedulers:
                tau = uplink.completion_slots(rates[beta], B, arr["slot_s"], s, agent_weight=weights.get(s), kind=kind)
                row = dict(trace=int(t), gamma=gamma, beta=beta, scheduler=s, tau=tau.tolist(),
                           feasible=bool(np.all(tau > 0)))
                if row["feasible"]:
                    a = [int(v) * slot_ns for v in tau]
                    t_r, t_b, w = dag.paired_latency_ns(a, c_enc_ns, c_post_ns, kind=kind)
                    row.update(a_ns=a, T_R=t_r, T_B=t_b, W_pre=w)
                out.append(row)
    return out


def _ci(x):
    lo, hi = replay.bootstrap_ci(np.asarray(x, dtype=np.float64))
    return [lo, hi]


def summarize(cfg, trials):
    arr = cfg["arrivals"]
    dl_ns = arr["deadline_s"] * 1e9
    ok = [r for r in trials if r["feasible"]]
    gain = lambda r: (r["T_B"] - r["T_R"]) * 1e-6  # noqa: E731
    ident = dict(
        trials=len(trials), feasible=len(ok),
        identity_exact=sum(r["T_B"] - r["T_R"] == r["W_pre"] for r in ok),
        positive_gain=sum(r["T_B"] > r["T_R"] for r in ok),
        zero_gain=sum(r["T_B"] == r["T_R"] for r in ok),
        negative_gain=sum(r["T_B"] < r["T_R"] for r in ok),
    )
    cells = []
    for gamma, beta in grid(cfg):
        rows = [r for r in ok if r["gamma"] == gamma and r["beta"] == beta]
        per = {}
        for s in arr["schedulers"]:
            rs = [r for r in rows if r["scheduler"] == s]
            if not rs:
                continue
            g = [gain(r) for r in rs]
            per[s] = dict(n=len(rs), mean_gain_ms=float(np.mean(g)), gain_ci95_ms=_ci(g),
                          rtcc_ms=float(np.mean([r["T_R"] for r in rs]) * 1e-6),
                          barrier_ms=float(np.mean([r["T_B"] for r in rs]) * 1e-6))
        if not per:
            continue
        cells.append(dict(
            gamma=gamma, beta=beta, n=len(rows),
            mean_gain_ms=float(np.mean([gain(r) for r in rows])),
            mean_rel_reduction=float(np.mean([(r["T_B"] - r["T_R"]) / r["T_B"] for r in rows])),
            worst_scheduler_gain_ms=float(min(p["mean_gain_ms"] for p in per.values())),
            best_rtcc_scheduler=min(per, key=lambda s: per[s]["rtcc_ms"]),
            A_median_ms=float(np.median([max(r["a_ns"]) for r in rows]) * 1e-6),
            per_scheduler=per,
        ))
    g0, b0 = arr["nominal"]
    nominal = {}
    for s in arr["schedulers"]:
        rs = [r for r in ok if r["gamma"] == g0 and r["beta"] == b0 and r["scheduler"] == s]
        if not rs:
            continue
        g = [gain(r) for r in rs]
        nominal[s] = dict(
            n=len(rs), barrier_ms=float(np.mean([r["T_B"] for r in rs]) * 1e-6),
            rtcc_ms=float(np.mean([r["T_R"] for r in rs]) * 1e-6), mean_gain_ms=float(np.mean(g)),
            gain_ci95_ms=_ci(g), overlap_window_ms=float(np.mean([max(r["a_ns"]) - min(r["a_ns"]) for r in rs]) * 1e-6),
            wins=int(sum(v > 0 for v in g)),
            deadline_rtcc=float(np.mean([r["T_R"] <= dl_ns for r in rs])),
            deadline_barrier=float(np.mean([r["T_B"] <= dl_ns for r in rs])),
        )
    best = {}
    for c in cells:
        best[c["best_rtcc_scheduler"]] = best.get(c["best_rtcc_scheduler"], 0) + 1
    sc_cells = [(c, s, p) for c in cells for s, p in c["per_scheduler"].items()]
    return dict(
        identity=ident, cells=cells, nominal=nominal, best_rtcc_scheduler_cells=best,
        scheduler_load_cells=len(sc_cells),
        scheduler_load_cells_positive_mean=sum(p["mean_gain_ms"] > 0 for _, _, p in sc_cells),
        scheduler_load_cells_positive_ci_low=sum(p["gain_ci95_ms"][0] > 0 for _, _, p in sc_cells),
        mean_gain_range_ms=[min(c["mean_gain_ms"] for c in cells), max(c["mean_gain_ms"] for c in cells)],
        rel_reduction_range=[min(c["mean_rel_reduction"] for c in cells), max(c["mean_rel_reduction"] for c in cells)],
        worst_scheduler_gain_range_ms=[min(c["worst_scheduler_gain_ms"] for c in cells),
                                       max(c["worst_scheduler_gain_ms"] for c in cells)],
    )


def profile_dag(cfg, warmup=5, reps=30):
    """Context for the workload (single compute stream, the execution model
    of the profiled DAG), one frame from host staging, then the node
    profile.  Returns (ctx, frame, c_enc_ms, c_post_ms)."""
    fr = synth.make_frame(cfg)
    o = R.rtcc_runtime_opts()
    o.exec = R.RTCC_EXEC_SERIAL
    o.premature_tol_s = 1e-6
    ctx = R.rtcc_create(R.model_desc(cfg), R.weights_blob(cfg, fr["weights"]), o)
    staged = replay.stage_inputs(ctx, fr["points"])
    R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
    for k in range(cfg["K"]):
        R.rtcc_release_branch(ctx, k, staged[k], fr["poses"][k], 0.0)
    R.rtcc_join_and_detect(ctx)
    prof = R.rtcc_profile_nodes(ctx, warmup, reps)
    return ctx, fr, prof[:cfg["K"]].tolist(), [float(prof[cfg["K"]])]


def replay_resident(ctx, cfg, fr, trials, reps):
    """GPU replay of trials with device-resident inputs; returns rows with
    the measured T^head gain and the DAG-predicted gain (ms)."""
    import torch
    dev = [torch.from_numpy(p).to("cuda") for p in fr["points"]]
    torch.cuda.synchronize()
    inputs = [(int(d.data_ptr()), int(d.shape[0])) for d in dev]
    out = []
    for i, r in enumerate(trials):
        a = np.asarray(r["a_ns"], dtype=np.float64) * 1e-9
        rows, same = replay.replay_traces(ctx, inputs, fr["poses"], [a], reps, start=i, resident=True)
        meas = (rows[0]["B_head"] - rows[0]["R_head"]) * 1e3
        out.append(dict(trace=r["trace"], scheduler=r["scheduler"], pred_gain_ms=(r["T_B"] - r["T_R"]) * 1e-6,
                        head_gain_ms=meas, det_gain_ms=(rows[0]["B_det"] - rows[0]["R_det"]) * 1e3,
                        identical_outputs=bool(same)))
        print("# replay %d/%d %s trace %d: pred %.3f ms, measured %.3f ms" % (
            i + 1, len(trials), r["scheduler"], r["trace"], out[-1]["pred_gain_ms"], meas), flush=True)
    del dev
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default="s6")
    ap.add_argument("--traces", type=int, default=None)
    ap.add_argument("--node-ms", default=None, help="comma-separated encoder times then the post-join time, ms")
    ap.add_argument("--profile", action="store_true", help="profile the DAG's nodes on the GPU")
    ap.add_argument("--replay", type=int, default=0)
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--lib", choices=["gpu", "host"], default="gpu")
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)

    cfg = synth.config(a.config)
    if cfg["arrivals"]["kind"] != "ofdma":
        raise SystemExit("config %s has no OFDMA uplink" % a.config)
    K = cfg["K"]
    ctx = fr = None
    if a.profile:
        ctx, fr, c_enc_ms, c_post_ms = profile_dag(cfg)
    elif a.node_ms:
        v = [float(x) for x in a.node_ms.split(",")]
        if len(v) != K + 1:
            raise SystemExit("--node-ms needs %d values" % (K + 1))
        c_enc_ms, c_post_ms = v[:K], v[K:]
    else:
        raise SystemExit("give --profile (GPU) or --node-ms")
    if a.replay and ctx is None:
        raise SystemExit("--replay needs --profile")
    c_enc_ns = [int(round(x * 1e6)) for x in c_enc_ms]
    c_post_ns = [int(round(x * 1e6)) for x in c_post_ms]
    print("# node service times (ms): encoders %s, post-join %s" % (
        ", ".join("%.4f" % x for x in c_enc_ms), ", ".join("%.4f" % x for x in c_post_ms)), flush=True)

    t0 = time.time()
    n_tr = a.traces or cfg["traces"]
    trials = run_trials(cfg, c_enc_ns, c_post_ns, range(n_tr), kind=a.lib)
    summ = summarize(cfg, trials)
    print("# %d trials in %.1f s: %s" % (len(trials), time.time() - t0, json.dumps(summ["identity"])), flush=True)
    res = dict(config=a.config, traces=n_tr, node_ms=dict(encoders=c_enc_ms, post=c_post_ms),
               dagrank_omega=dag.dagrank_weights(c_enc_ns, c_post_ns, kind=a.lib), summary=summ)
    if a.replay:
        g0, b0 = cfg["arrivals"]["nominal"]
        nom = [r for r in trials if r["feasible"] and r["gamma"] == g0 and r["beta"] == b0][:a.replay]
        rows = replay_resident(ctx, cfg, fr, nom, a.reps)
        p = np.array([r["pred_gain_ms"] for r in rows])
        m = np.array([r["head_gain_ms"] for r in rows])
        res["replay"] = dict(
            pairs=len(rows), reps=a.reps,
            pearson_r=float(np.corrcoef(p, m)[0, 1]) if len(rows) > 2 and p.std() > 0 and m.std() > 0 else None,
            mae_ms=float(np.mean(np.abs(p - m))), positive=int(np.sum(m > 0)),
            identical_outputs=all(r["identical_outputs"] for r in rows), rows=rows)
        print("# replay: %s" % json.dumps({k: v for k, v in res["replay"].items() if k != "rows"}), flush=True)
    res["trials"] = [{k: v for k, v in r.items() if k != "a_ns"} for r in trials]
    with open(a.out, "w") as f:
        json.dump(res, f, indent=1)
    _print_tables(cfg, summ)
    if ctx is not None:
        ctx.close()
    return 0


def _print_tables(cfg, summ):
    print("\n| gamma | beta | A p50 ms | mean gain ms | rel. reduction | worst scheduler gain ms | best RTCC scheduler |")
    print("|---:|---:|---:|---:|---:|---:|---|")
    for c in summ["cells"]:
        print("| %.1f | %.1f | %.0f | %.3f | %.2f%% | %.3f | %s |" % (
            c["gamma"], c["beta"], c["A_median_ms"], c["mean_gain_ms"], 100 * c["mean_rel_reduction"],
            c["worst_scheduler_gain_ms"], c["best_rtcc_scheduler"]))
    print("\n| scheduler (nominal) | barrier ms | RTCC ms | gain ms [95% CI] | overlap window ms | wins | deadline R / B |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for s, p in summ["nominal"].items():
        print("| %s | %.2f | %.2f | %.3f [%.3f, %.3f] | %.1f | %d/%d | %.0f%% / %.0f%% |" % (
            s, p["barrier_ms"], p["rtcc_ms"], p["mean_gain_ms"], p["gain_ci95_ms"][0], p["gain_ci95_ms"][1],
            p["overlap_window_ms"], p["wins"], p["n"], 100 * p["deadline_rtcc"], 100 * p["deadline_barrier"]))


if __name__ == "__main__":
    sys.exit(main())
