#!/usr/bin/env python
"""Benchmark of the RTCC fork-join detector path on one MI355X.

One step = one complete frame through the C ABI: K branch encoders
(pillarize, point-feature net, 3x3 conv backbone, upsample) released on
device-resident inputs that all arrive at once (one batch of K completion
events: one pillar-stage launch chain over the K agents, then every backbone
on its own stream), then the join (warp, fusion, head, decode, NMS, D2H).
--warp-in-branch moves the pose warp into the branches.

Output: one JSON line with
  value       encoder throughput, TFLOP/s = algorithmic encoder FLOPs of the
              timed frames / wall time of the timed frames, with the library's
              default executor (per-branch streams)
  roofline    the dominant kernel (3x3 convolution): algorithmic FLOPs /
              summed kernel durations of its launches (HIP events that
              bracket the kernels, one compute stream), against the bf16
              dense MFMA peak
  latency     p50 / p95 complete-detection latency T^det, RTCC vs barrier,
              over replayed synthetic arrival traces (pinned host inputs,
              H2D included, as on the release path; contexts without node
              events)
  cpu_baseline  the fp64 CPU oracle's encoder throughput on a bounded sample
"""

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "p50/p95 complete-detection latency ms (RTCC vs barrier); encoder TFLOP/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 (vector / MFMA fp32)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

# HBM bytes per launch from two rocprofv3 counter runs (FETCH_SIZE x 2.0 and
# WRITE_SIZE x 1.0, the factors a plain 512 MiB copy gives; summary and
# commands in profiles/traffic_c5_bench.md).  Each figure holds only for the
# kernel source it was taken on; after a change it reads null until re-taken.
MEASURED_TRAFFIC = {
    # per 8-agent launch of a conv layer (averaged over the 13 layers)
    "conv": dict(src="paper_2608_08330_amd/csrc/kernels/igemm.hip", bytes=154.8e6,
                 sha256="1ea11a11e3bed1bdddb119fe33f47298bae88df767b509db8774190339f217c4"),
    "warp_fuse": dict(src="paper_2608_08330_amd/csrc/kernels/post.hip", bytes=472.1e6,
                      sha256="c30da5594b4491cccb79cd6bf3584f6866b3e6fc4850e9952cce71f7bad853c2"),
    # per 8-agent launch chain of the pillar stage (five kernels)
    "pillar": dict(src="paper_2608_08330_amd/csrc/kernels/pillar.hip", bytes=195e6,
                   sha256="624b87e26ad92d9196d0e1e206e92b8349c8c32de965453523b85f3ee2223d4b"),
}


def measured_traffic(kernel):
    import hashlib
    t = MEASURED_TRAFFIC.get(kernel)
    if t is None:
        return None
    try:
        with open(os.path.join(ROOT, t["src"]), "rb") as f:
            same = hashlib.sha256(f.read()).hexdigest() == t["sha256"]
    except OSError:
        same = False
    return t["bytes"] if same else None


def grid(cfg):
    W = int(round((cfg["x_range"][1] - cfg["x_range"][0]) / cfg["pillar"]))
    H = int(round((cfg["y_range"][1] - cfg["y_range"][0]) / cfg["pillar"]))
    return H, W


def layer_work(cfg):
    """Algorithmic FLOPs / bytes of every node of one agent's encoder and of
    the post-join subgraph, in node-time order."""
    H, W = grid(cfg)
    elt = 2 if cfg["precision"] == "bf16" else 4
    convs, ups = [], []
    h, w, c = H, W, cfg["c_pfn"]
    stage = []
    for stride, co, n in cfg["stages"]:
        for l in range(n):
            s = stride if l == 0 else 1
            ho, wo = -(-h // s), -(-w // s)
            convs.append(dict(flops=2.0 * ho * wo * co * 9 * c, M=ho * wo, N=co, K=9 * c,
                              bytes=(h * w * c + ho * wo * co + 9 * c * co) * elt,
                              Hi=h, Wi=w, Ci=c, stride=s, stage=len(stage), layer=l))
            h, w, c = ho, wo, co
        stage.append((h, w, c))
    H2, W2 = stage[0][0], stage[0][1]
    if cfg["up_channels"]:
        for (hs, ws, cs) in stage:
            ups.append(dict(flops=2.0 * H2 * W2 * cs * cfg["up_channels"],
                            bytes=(hs * ws * cs + H2 * W2 * cfg["up_channels"]) * elt))
        C = cfg["up_channels"] * len(cfg["stages"])
    else:
        C = stage[-1][2]
    return dict(H=H, W=W, H2=H2, W2=W2, C=C, elt=elt, convs=convs, ups=ups)


def encoder_flops(cfg, lw, n_used):
    """PFN (linear 4 -> C on every used point) + convs + upsampling."""
    pfn = 2.0 * 4 * cfg["c_pfn"] * n_used
    # multi-scale fusion upsamples the fused maps once, after the join
    ups = 0.0 if cfg.get("multiscale") else sum(u["flops"] for u in lw["ups"])
    return pfn + sum(c["flops"] for c in lw["convs"]) + ups


def timed_steps(ctx, cfg, frames, dev_pts, steps, warmup, R, torch, record_nodes=True, release_us=None, batch=True):
    """Warm-up, then exactly `steps` timed frames bracketed by device syncs.
    Step s runs stream frame s mod len(frames) (its own points and poses), as
    a live stream does.  Every agent's input arrives at once, so with
    `batch` the K completion events are released in one call (one group);
    otherwise one call per event.  Returns wall seconds and (with
    record_nodes) the per-node HIP-event times of every step; with
    release_us (a list), the host time of each frame's release calls is
    appended to it."""
    K = cfg["K"]
    F = len(frames)

    def one(f, times=None):
        fr, dev = frames[f], dev_pts[f]
        R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
        t0 = time.perf_counter()
        if batch:
            R.rtcc_release_branches(ctx, [dict(agent=k, device=1, points=dev[k].data_ptr(), n=len(fr["points"][k]),
                                               pose=fr["poses"][k], arrival_t=0.0) for k in range(K)])
        else:
            for k in range(K):
                R.rtcc_release_branch_device(ctx, k, dev[k].data_ptr(), len(fr["points"][k]), fr["poses"][k], 0.0)
        if times is not None:
            times.append((time.perf_counter() - t0) * 1e6)
        return R.rtcc_join_and_detect(ctx)

    for w in range(warmup):
        one(w % F)
    torch.cuda.synchronize()
    node = []
    t = time.perf_counter()
    for i in range(steps):
        one((warmup + i) % F, release_us)
        if record_nodes:
            node.append(R.rtcc_node_times(ctx))
    torch.cuda.synchronize()
    return time.perf_counter() - t, node


def used_points(ctx, cfg, frames, dev_pts, R):
    """Points fed to the point-feature net per frame of the stream (sum over
    agents of min(count, cap) of every pillar), from the library's pillar
    counts after running each frame once."""
    import numpy as np
    out = []
    for f, fr in enumerate(frames):
        R.rtcc_begin_frame(ctx, time.monotonic() - 1.0)
        for k in range(cfg["K"]):
            R.rtcc_release_branch_device(ctx, k, dev_pts[f][k].data_ptr(), len(fr["points"][k]), fr["poses"][k], 0.0)
        R.rtcc_join_and_detect(ctx)
        out.append([int(np.minimum(R.rtcc_get_tensor(ctx, R.RTCC_T_PILLAR_COUNTS, k, np.int32), cfg["max_pts"]).sum())
                    for k in range(cfg["K"])])
    return out


def gemm_reference(layers, torch, iters=50):
    """The vendor library's dense GEMM (torch.matmul -> hipBLASLt, bf16, fp32
    accumulation) on each conv layer's GEMM shape: the cost of the same
    FLOPs as a plain GEMM whose im2col operand is already in memory."""
    rows = []
    for l in layers:
        M, N, K = l["M"], l["N"], l["K"]
        x = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
        w = torch.randn(K, N, device="cuda", dtype=torch.bfloat16)
        for _ in range(5):
            torch.matmul(x, w)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            torch.matmul(x, w)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / iters * 1e3
        rows.append({"M": M, "N": N, "K": K, "hipblaslt_us": round(us, 2),
                     "hipblaslt_tflops": round(2.0 * M * N * K / (us * 1e-6) / 1e12, 1), "conv_us_per_agent": l["us_per_agent"]})
        del x, w
    return rows


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return os.cpu_count() or 1


def oracle_stage_times(cfg, frame, agents=(0,), post=True):
    """Wall seconds of every stage of the fp64 oracle (untuned): O1 cell ids,
    O2 pillars, O3 point-feature canvas, O4 each conv stage, O5 upsampling,
    for the listed agents' encoders; then O7 warp and O8 fusion of all K
    agents, O9 head, O10 decode (the post-join stages reuse the listed
    agents' slots for the others).  Returns (seconds by stage, FLOPs of the
    encoders run)."""
    import numpy as np
    from oracle import network as N
    pw = N.prepared_weights(cfg, frame["weights"])
    lw = layer_work(cfg)
    st = {}

    def tick(name, t0):
        st[name] = st.get(name, 0.0) + time.perf_counter() - t0

    flops = 0.0
    slots = []
    for k in agents:
        pts = frame["points"][k]
        t0 = time.perf_counter(); cell = N.cell_ids(pts, cfg); tick("O1_cell_ids", t0)
        t0 = time.perf_counter(); pil = N.pillars(cell, cfg["max_pts"]); tick("O2_pillars", t0)
        t0 = time.perf_counter(); x = N.pfn_canvas(pts, pil, pw["pfn_w"], pw["pfn_b"], cfg); tick("O3_pfn_canvas", t0)
        x = N._store(cfg, x)
        stage_out = []
        for s, (stride, _c, n) in enumerate(cfg["stages"]):
            t0 = time.perf_counter()
            for l in range(n):
                x = N._store(cfg, N.conv3x3(x, pw["s%dc%d_w" % (s, l)], pw["s%dc%d_b" % (s, l)], stride if l == 0 else 1))
            tick("O4_conv_stage%d" % s, t0)
            stage_out.append(x)
        if cfg["up_channels"]:
            t0 = time.perf_counter()
            H2, W2 = stage_out[0].shape[:2]
            parts, rel = [], 1
            for s, (stride, _c, _n) in enumerate(cfg["stages"]):
                if s > 0:
                    rel *= stride
                parts.append(N._store(cfg, N.deconv(stage_out[s], pw["up%d_w" % s], pw["up%d_b" % s], rel, H2, W2)))
            slot = np.concatenate(parts, axis=2)
            tick("O5_upsample", t0)
        else:
            slot = stage_out[-1]
        slots.append(slot)
        flops += encoder_flops(cfg, lw, int(np.minimum(pil["counts"], cfg["max_pts"]).sum()))
    if post:
        full = [slots[k % len(slots)] for k in range(cfg["K"])]
        t0 = time.perf_counter(); warped = [N.warp(full[k], frame["poses"][k], cfg) for k in range(cfg["K"])]
        tick("O7_warp", t0)
        t0 = time.perf_counter()
        fused = N._store(cfg, N.fuse_attn(warped) if cfg["fusion"] == "attn" else N.fuse_max(warped))
        tick("O8_fusion", t0)
        t0 = time.perf_counter(); Z = N.head(fused, pw["head_w"], pw["head_b"]); tick("O9_head", t0)
        t0 = time.perf_counter(); N.decode(Z, cfg); tick("O10_decode", t0)
    return st, flops


def schedule_decision_us(cfg, reps=2000):
    """Host cost of one release decision of the schedule oracle (the
    single-stream RTCC execution of K arrivals: validation-free ordering by
    (a_k, k) and the start / finish recursion), microseconds per frame."""
    import numpy as np
    from oracle import schedule as S
    rng = np.random.default_rng(0)
    a = rng.uniform(0.0, 0.1, (reps, cfg["K"]))
    c = np.full(cfg["K"], 2e-4)
    t = time.perf_counter()
    for r in range(reps):
        S.rtcc(a[r], c, [5e-5])
    return (time.perf_counter() - t) / reps * 1e6


def cpu_baseline(cfg, frame, budget_s):
    """The fp64 oracle (untuned) on the host cores: agent encoders repeated
    while the budget lasts with the BLAS library's threads (the value), the
    same single-threaded on a bounded sample, the stage split of one agent
    encoder, and the schedule oracle's cost per decision."""
    import numpy as np
    from oracle import network as N
    threads = _blas_threads()
    pw = N.prepared_weights(cfg, frame["weights"])
    lw = layer_work(cfg)
    done, flops = 0, 0.0
    t = time.perf_counter()
    stages = None
    while True:
        k = done % cfg["K"]
        if done == 0:
            stages, f = oracle_stage_times(cfg, frame, agents=(k,), post=False)
            flops += f
        else:
            enc = N.encoder(frame["points"][k], cfg, pw)
            flops += encoder_flops(cfg, lw, int(np.minimum(enc["counts"], cfg["max_pts"]).sum()))
        done += 1
        if time.perf_counter() - t >= budget_s:
            break
    dt = time.perf_counter() - t
    out = dict(value=flops / dt / 1e12, unit="TFLOP/s", cores=int(threads), kind="oracle",
               sample="%d agent encoder(s) of the %s frame (fp64 numpy oracle), %.1f s, %d BLAS threads"
                      % (done, cfg["name"], dt, threads),
               stages_ms_one_agent={k: round(v * 1e3, 1) for k, v in stages.items()})
    # single-threaded: the last conv stage of one agent (the smallest grid),
    # repeated for a few seconds
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            cl = lw["convs"][-1]
            x = np.random.default_rng(0).random((cl["Hi"], cl["Wi"], cl["Ci"]))
            w = pw["s%dc%d_w" % (cl["stage"], cl["layer"])]
            b = pw["s%dc%d_b" % (cl["stage"], cl["layer"])]
            n1, t1 = 0, time.perf_counter()
            while time.perf_counter() - t1 < min(budget_s, 5.0) or n1 == 0:
                N.conv3x3(x, w, b, cl["stride"])
                n1 += 1
            dt1 = time.perf_counter() - t1
        out["single_thread"] = dict(value=n1 * lw["convs"][-1]["flops"] / dt1 / 1e12, unit="TFLOP/s", cores=1,
                                    sample="%d x the last 3x3 conv layer (%d x %d x %d -> %d), %.1f s" % (
                                        n1, x.shape[0], x.shape[1], x.shape[2], w.shape[3], dt1))
    except Exception as e:  # pragma: no cover
        out["single_thread"] = dict(error=str(e))
    out["schedule_decision_us"] = round(schedule_decision_us(cfg), 2)
    return out


def cpu_stage_table(names=("c1", "c2", "c3", "c5")):
    """Stage-by-stage wall time of the fp64 oracle for one agent encoder and
    the post-join subgraph of each config, with all BLAS threads and with one
    (JSON on stdout)."""
    import synth
    from threadpoolctl import threadpool_limits
    rows = []
    for name in names:
        cfg = synth.config(name)
        frame = synth.make_frame(cfg)
        for threads in (None, 1):
            with threadpool_limits(limits=threads):
                n_thr = _blas_threads()
                t = time.perf_counter()
                st, flops = oracle_stage_times(cfg, frame, agents=(0,), post=True)
                total = time.perf_counter() - t
            enc = sum(v for k, v in st.items() if k[:2] in ("O1", "O2", "O3", "O4", "O5"))
            rows.append(dict(config=name, threads=n_thr, stages_ms={k: round(v * 1e3, 2) for k, v in st.items()},
                             encoder_ms=round(enc * 1e3, 2), encoder_gflops=round(flops / enc / 1e9, 2),
                             total_ms=round(total * 1e3, 2)))
            print("# %s threads=%d encoder %.1f ms" % (name, n_thr, enc * 1e3), file=sys.stderr, flush=True)
    print(json.dumps(dict(cpu=os.cpu_count(), rows=rows, schedule_decision_us=round(
        schedule_decision_us(synth.config("c5")), 2))))
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c5")
    ap.add_argument("--exec", choices=["serial", "streams"], default="streams",
                    help="executor of the throughput pass (the library's default: per-branch streams)")
    ap.add_argument("--roofline-steps", type=int, default=10,
                    help="frames of the serial, node-timed pass behind roofline and per-layer tables")
    ap.add_argument("--latency-traces", type=int, default=30)
    ap.add_argument("--latency-reps", type=int, default=3)
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--warp-in-branch", action="store_true",
                    help="place the pose warp as the last node of every branch (the join only fuses)")
    ap.add_argument("--multiscale", action="store_true",
                    help="fuse the agents at every backbone scale before upsampling")
    ap.add_argument("--no-graphs", action="store_true",
                    help="launch kernels one by one on the per-branch-stream executor too (by default it "
                         "replays each branch and the join as HIP graphs; the serial executor is eager, "
                         "graph launches on one stream being slower there)")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="also time the vendor GEMM (torch.matmul, hipBLASLt) on every conv layer's GEMM shape "
                         "(M x K times K x N, bf16) next to the conv kernel")
    ap.add_argument("--stream-frames", type=int, default=3,
                    help="distinct seeded frames (points and poses) the throughput pass cycles through, so that "
                         "HIP graphs are updated every step as on a live stream")
    ap.add_argument("--cpu-stages", action="store_true",
                    help="only time the CPU oracle stage by stage for c1, c2, c3 and c5, with all BLAS threads and "
                         "single-threaded, and print the table as JSON")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB, 5 times "
                         "(reference for the FETCH_SIZE / WRITE_SIZE counters)")
    a = ap.parse_args(argv)

    if a.cpu_stages:
        return cpu_stage_table()

    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the detector path runs on a single MI355X and has no "
              "multi-GPU mode (--gpus must be 1)", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    import synth
    from paper_2608_08330_amd import rtcc as R
    from paper_2608_08330_amd import replay

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2

    if a.copy_calibration:
        n = a.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": 5}))
        return 0

    cfg = synth.config(a.config)
    cfg["warp_in_branch"] = bool(a.warp_in_branch)
    cfg["multiscale"] = bool(a.multiscale)
    frame = synth.make_frame(cfg)
    lw = layer_work(cfg)
    K = cfg["K"]

    def make_ctx(exec_kind, timing):
        o = R.rtcc_runtime_opts()
        o.exec = R.RTCC_EXEC_SERIAL if exec_kind == "serial" else R.RTCC_EXEC_PER_BRANCH_STREAMS
        o.node_timing = 1 if timing else 0
        o.use_graphs = 1 if exec_kind == "streams" and not a.no_graphs and not timing else 0
        o.premature_tol_s = 1e-6
        return R.rtcc_create(R.model_desc(cfg), R.weights_blob(cfg, frame["weights"]), o)

    # a stream of frames: frame 0 is the config's, the others new seeded
    # points and poses (the network is the same)
    F = max(1, a.stream_frames)
    frames = [frame] + [synth.make_frame(cfg, f) for f in range(1, F)]
    dev_frames = [[torch.from_numpy(p).to("cuda") for p in fr["points"]] for fr in frames]
    dev_pts = dev_frames[0]
    torch.cuda.synchronize()

    # throughput: the library's executor, no node events, cycling the stream
    ctx_t = make_ctx(a.exec, False)
    used_f = used_points(ctx_t, cfg, frames, dev_frames, R)
    release_us = []
    wall, _ = timed_steps(ctx_t, cfg, frames, dev_frames, a.steps, a.warmup, R, torch, record_nodes=False,
                          release_us=release_us)
    ms_per_step = wall / a.steps * 1e3
    step_flops = [sum(encoder_flops(cfg, lw, u) for u in used_f[(a.warmup + i) % F]) for i in range(a.steps)]
    value = sum(step_flops) / wall / 1e12
    eager = None
    if a.exec == "streams" and not a.no_graphs:
        # the same stream launched kernel by kernel
        o = R.rtcc_runtime_opts()
        o.exec = R.RTCC_EXEC_PER_BRANCH_STREAMS
        o.premature_tol_s = 1e-6
        ctx_e = R.rtcc_create(R.model_desc(cfg), R.weights_blob(cfg, frame["weights"]), o)
        wall_e, _ = timed_steps(ctx_e, cfg, frames, dev_frames, a.steps, a.warmup, R, torch, record_nodes=False)
        ctx_e.close()
        eager = dict(ms_per_step=round(wall_e / a.steps * 1e3, 4), value=round(sum(step_flops) / wall_e / 1e12, 3),
                     unit="TFLOP/s")
    # roofline and per-node tables: one compute stream (the paper's execution
    # model), so that node durations do not overlap; conv nodes are timed by
    # events that bracket their kernels
    ctx = make_ctx("serial", True)
    wall_s, node = timed_steps(ctx, cfg, [frame], [dev_pts], a.roofline_steps, a.warmup, R, torch)
    rsteps = a.roofline_steps
    # the same frames released one event at a time: every agent's pillar
    # stage alone (a group of one)
    ctx_1 = make_ctx("serial", True)
    _, node_1 = timed_steps(ctx_1, cfg, [frame], [dev_pts], a.roofline_steps, a.warmup, R, torch, batch=False)
    ctx_1.close()

    # node layout per agent: h2d, pillar, pfn, conv[L], up[S or 1], warp (0 unless in the branch);
    # post: warp_fuse (or fuse), head, decode, nms
    L, S = len(lw["convs"]), max(len(lw["ups"]), 1)
    per_agent = 3 + L + S + 1
    node = np.array(node)  # [steps, nodes] ms
    conv_ms = 0.0
    for k in range(K):
        base = k * per_agent + 3
        conv_ms += node[:, base:base + L].sum()
    conv_flops = sum(c["flops"] for c in lw["convs"]) * K * rsteps
    # the K agents released together: one launch per conv layer serves all
    conv_launches = L * rsteps
    achieved = conv_flops / (conv_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if cfg["precision"] == "bf16" else PEAK_FP32_TFLOPS
    # pillar stage: the K agents released together run it as one launch
    # chain, so every member's pillar + PFN nodes are the group's span
    node_1 = np.array(node_1)
    # (each member's node is its share of the shared launches)
    group_ms = sum(float(node[:, k * per_agent + 1].sum() + node[:, k * per_agent + 2].sum()) for k in range(K))
    single_ms = sum(float(node_1[:, k * per_agent + 1].sum() + node_1[:, k * per_agent + 2].sum()) for k in range(K))
    P = [int(R.rtcc_tensor_bytes(ctx, R.RTCC_T_PILLAR_CELLS, k)) // 4 for k in range(K)]
    pil_bytes = sum(16 * len(frame["points"][k]) + 8 * P[k] + lw["H"] * lw["W"] * cfg["c_pfn"] * lw["elt"]
                    for k in range(K)) * rsteps
    post0 = K * per_agent
    warp_ms = node[:, post0].sum()
    slot_bytes = lw["H2"] * lw["W2"] * lw["C"] * lw["elt"]
    # warp + fusion, or fusion of the stored maps: K maps read, one written
    warp_bytes = (K + 1) * slot_bytes * rsteps
    # branch warps (agents with a non-identity pose): one slot read, one map written
    bw_ms = sum(node[:, k * per_agent + per_agent - 1].sum() for k in range(K))
    bw_launches = sum(1 for k in range(K) if node[:, k * per_agent + per_agent - 1].sum() > 0) * rsteps

    layers = []
    for l, c in enumerate(lw["convs"]):
        us = float(np.mean([node[:, k * per_agent + 3 + l] for k in range(K)])) * 1e3
        layers.append({"M": c["M"], "N": c["N"], "K": c["K"], "us_per_agent": round(us, 2),
                       "tflops": round(c["flops"] / (us * 1e-6) / 1e12, 1)})
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg["precision"] == "bf16" else "f32",
        "data": "synthetic (seeded points, poses, He-normal weights, arrival traces)",
        "config": {
            "workload": "%s: %d agents x %d points, %dx%d BEV, %s, %s fusion%s" % (
                cfg["name"], K, cfg["n_points"], lw["H"], lw["W"], cfg["precision"], cfg["fusion"],
                (", warp in the branches" if cfg["warp_in_branch"] else "")
                + (", multi-scale fusion" if cfg["multiscale"] else "")),
            "agents": K, "inputs": "device-resident",
            "executor": "per-branch streams" if a.exec == "streams" else "serial",
            "hip_graphs": bool(a.exec == "streams" and not a.no_graphs),
            "stream_frames": F,
        },
        "serial_ms_per_step": round(wall_s / rsteps * 1e3, 4),
        "eager_streams": eager,
        "release_us_per_frame_p50": round(float(np.median(release_us)), 2) if release_us else None,
        "roofline": {
            "bound": "mfma", "kernel": "3x3 conv: halo-tiled k_conv3s1 + implicit-GEMM k_igemm",
            "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": measured_traffic("conv"),
            "launches": conv_launches, "avg_launch_us": round(conv_ms * 1e3 / conv_launches, 3),
        },
        "secondary_rooflines": {
            "pillar_pfn_canvas": {"bound": "hbm", "achieved": round(pil_bytes / (group_ms * 1e-3) / 1e9, 1),
                                  "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                  "frac": round(pil_bytes / (group_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                                  "agents": K, "span_us": round(group_ms / rsteps * 1e3, 2),
                                  "traffic": measured_traffic("pillar"),
                                  "per_agent_alone": {
                                      "achieved": round(pil_bytes / (single_ms * 1e-3) / 1e9, 1),
                                      "us_per_agent": round(single_ms / (K * rsteps) * 1e3, 2)},
                                  "work": "16 n + 8 P + H*W*C_pfn*elt bytes per agent (the dense canvas as "
                                          "output; the kernels write the P pillar cells, the previous frame's "
                                          "were cleared after its join), all K agents over the span of their one "
                                          "launch chain"},
        },
        "conv_layers": layers,
        "node_ms_mean": {
            "pillar_group_of_%d" % K: round(float(sum(node[:, k * per_agent + 1].mean() for k in range(K))), 4),
            "pfn_canvas_group_of_%d" % K: round(float(sum(node[:, k * per_agent + 2].mean() for k in range(K))), 4),
            "pillar_alone": round(float(np.mean([node_1[:, k * per_agent + 1] for k in range(K)])), 4),
            "pfn_canvas_alone": round(float(np.mean([node_1[:, k * per_agent + 2] for k in range(K)])), 4),
            "conv_total_per_agent": round(conv_ms / (K * rsteps), 4),
            "up_total_per_agent": round(float(np.sum([node[:, k * per_agent + 3 + L:k * per_agent + per_agent]
                                                      for k in range(K)]) / (K * rsteps)), 4),
            "branch_warp_per_agent": round(bw_ms / (K * rsteps), 4),
            ("multiscale_fusion_upsample" if cfg["multiscale"] else "fuse" if cfg["warp_in_branch"]
             else "warp_fuse"): round(float(node[:, post0].mean()), 4),
            "head": round(float(node[:, post0 + 1].mean()), 4),
            "decode": round(float(node[:, post0 + 2].mean()), 4),
            "nms": round(float(node[:, post0 + 3].mean()), 4),
        },
    }
    if not cfg["multiscale"]:
        out["secondary_rooflines"]["fuse" if cfg["warp_in_branch"] else "warp_fuse"] = {
            "bound": "hbm", "achieved": round(warp_bytes / (warp_ms * 1e-3) / 1e9, 1),
            "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "traffic": measured_traffic("fuse" if cfg["warp_in_branch"] else "warp_fuse")}
    if cfg["warp_in_branch"] and bw_launches:
        out["secondary_rooflines"]["branch_warp"] = {
            "bound": "hbm", "achieved": round(2 * slot_bytes * bw_launches / (bw_ms * 1e-3) / 1e9, 1),
            "peak": PEAK_HBM_GBS, "unit": "GB/s", "traffic": measured_traffic("warp_slot")}
    if a.gemm_reference:
        out["gemm_reference"] = gemm_reference(layers, torch)
    if a.exec == "streams" and not a.no_graphs:
        out["graph_stats"] = dict(zip(("instantiated", "updates", "launches"), R.rtcc_graph_stats(ctx_t)))
    print("# throughput done: %.3f ms/step, %.1f TFLOP/s" % (ms_per_step, value), file=sys.stderr, flush=True)

    if a.latency_traces > 0:
        if cfg["arrivals"]["kind"] == "uplink":
            raise SystemExit("latency replay of uplink-driven configs runs in the load-sweep report")
        arr = synth.arrival_draws(cfg, a.latency_traces) * 1e-3
        # primary: one compute stream, as the paper's latency model; then the
        # per-branch-stream executor on the same traces.  Both without node
        # events, which would add their own overhead to every launch (and far
        # more of it to the barrier, which runs every branch after A).
        ctx_l = make_ctx("serial", False)
        for key, c in (("latency", ctx_l), ("latency_streams", ctx_t)):
            staged = replay.stage_inputs(c, frame["points"])
            rows, identical = replay.replay_traces(c, staged, frame["poses"], arr, a.latency_reps)
            lat = replay.summarize(rows)
            lat["reps"] = a.latency_reps
            lat["executor"] = "serial" if c is ctx_l else "per-branch streams"
            lat["outputs_identical_rtcc_vs_barrier"] = bool(identical)
            lat["rtcc_below_barrier_every_trace"] = bool(lat["wins_median"] == len(rows))
            out[key] = lat
            print("# %s done" % key, file=sys.stderr, flush=True)
        ctx_l.close()

    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, frame, a.cpu_budget)
    ctx.close()
    ctx_t.close()
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
