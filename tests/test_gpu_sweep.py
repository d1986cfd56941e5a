"""Measured-DAG sweep on the GPU: the six-agent workload's node profile
(rtcc_profile_nodes), and the resident-input replay of nominal-load OFDMA
trials under RTCC and Barrier, which must give identical detections."""

import sys

import numpy as np
import pytest

import synth
from paper_2608_08330_amd import sweep

pytestmark = pytest.mark.gpu


def test_profile_and_resident_replay():
    cfg = synth.config("s6")
    print("sweep: profile s6 (K=6)", flush=True)
    sys.stdout.flush()
    ctx, fr, c_enc, c_post = sweep.profile_dag(cfg, warmup=2, reps=5)
    try:
        assert len(c_enc) == cfg["K"] and len(c_post) == 1
        assert all(v > 0 for v in c_enc) and c_post[0] > 0
        c_enc_ns = [int(round(x * 1e6)) for x in c_enc]
        c_post_ns = [int(round(x * 1e6)) for x in c_post]
        g0, b0 = cfg["arrivals"]["nominal"]
        rows = sweep.run_trials(cfg, c_enc_ns, c_post_ns, [0], cells=[(g0, b0)],
                                schedulers=("maxrate", "maxweight"))
        rows = [r for r in rows if r["feasible"]]
        assert rows and all(r["T_B"] - r["T_R"] == r["W_pre"] for r in rows)
        print("sweep: replay %d trials" % len(rows), flush=True)
        out = sweep.replay_resident(ctx, cfg, fr, rows, reps=1)
        assert all(r["identical_outputs"] for r in out)
        assert all(np.isfinite(r["head_gain_ms"]) for r in out)
    finally:
        ctx.close()
