"""The measured-DAG sweep's product path against the oracle, on the CPU:
the library's uplink emulation (rtcc_uplink_emulate), single-stream model
(rtcc_schedule_model) and upward rank (rtcc_upward_rank), called through the
host-test build of the same source, and the harness's channel composition.
Completion slots, allocations and integer-nanosecond latencies are compared
exactly."""

import json
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import synth
from oracle import ofdma as O
from oracle import schedule as S
from oracle import uplink as U
from paper_2608_08330_amd import channel, dag, sweep, uplink
from paper_2608_08330_amd import rtcc as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST = "host"
SCHEDS = ("maxrate", "maxweight", "earliest_release", "dagrank", "tw_maxrate")
C_ENC = [205_000, 211_000, 198_000, 207_000, 203_000, 209_000]
C_POST = [812_000]


@pytest.fixture(scope="module")
def cfg():
    return synth.config("s6")


def _oracle_policy(name, K, slot_s, w):
    return U.make_policy(name, K, slot_s=slot_s, weights=w)


@pytest.mark.parametrize("trace", [0, 3])
def test_channel_rates_equal_oracle(cfg, trace):
    draw = synth.ofdma_draws(cfg, trace)
    for beta in (0.6, 1.0, 1.4):
        assert np.array_equal(channel.rates(draw, cfg, beta), O.rates(draw, cfg, beta))
    n = synth.points_per_agent(cfg)
    for gamma in (0.5, 2.0):
        assert np.array_equal(channel.payload_bits(cfg, n, gamma), O.payload_bits(cfg, n, gamma))


@pytest.mark.parametrize("sched", SCHEDS)
def test_native_emulation_equals_oracle_exactly(cfg, sched):
    arr = cfg["arrivals"]
    n = synth.points_per_agent(cfg)
    w = dict(dagrank=O.dagrank_weights(C_ENC, C_POST), tw_maxrate=list(arr["task_weights"])).get(sched)
    for trace in (1, 2):
        draw = synth.ofdma_draws(cfg, trace)
        for gamma, beta in ((0.5, 1.4), (1.0, 0.8), (2.0, 0.6)):
            Rt = O.rates(draw, cfg, beta)
            B = O.payload_bits(cfg, n, gamma)
            ref = U.emulate(Rt, B, arr["slot_s"], _oracle_policy(sched, cfg["K"], arr["slot_s"], w))
            tau, alloc = R.rtcc_uplink_emulate(Rt, B, uplink.SCHEDULERS[sched], arr["slot_s"], agent_weight=w,
                                               want_alloc=True, kind=HOST)
            assert tau.tolist() == ref["tau"].tolist()
            T = ref["x"].shape[0]
            want = np.where(ref["x"].any(axis=1), ref["x"].argmax(axis=1), -1)
            assert np.array_equal(alloc[:T], want)
            assert np.all(alloc[T:] == -1)


@pytest.mark.parametrize("sched", ["rr", "pf"])
def test_native_single_rb_policies_equal_oracle(sched):
    rng = np.random.default_rng(4)
    K, F = 4, 3
    Rt = rng.exponential(1e6, (3000, K, F))
    B = rng.uniform(1e5, 4e5, K)
    pol = U.RoundRobin(K) if sched == "rr" else U.ProportionalFair(K, 100, 1e6)
    ref = U.emulate(Rt, B, 1e-3, pol, ell=np.array([1, 5, 1, 40]))
    tau, alloc = R.rtcc_uplink_emulate(Rt, B, uplink.SCHEDULERS[sched], 1e-3, avail_slot=[1, 5, 1, 40],
                                       pf_window=100.0, pf_init_rate=1e6, want_alloc=True, kind=HOST)
    assert tau.tolist() == ref["tau"].tolist()
    T = ref["x"].shape[0]
    assert np.array_equal(alloc[:T], np.where(ref["x"].any(axis=1), ref["x"].argmax(axis=1), -1))


def test_native_emulation_reports_undelivered_branches():
    Rt = np.full((10, 3, 1), 1000.0)
    tau = R.rtcc_uplink_emulate(Rt, [5.0, 5.0, 5.0], R.RTCC_SCHED_MAXRATE, 1e-3, kind=HOST)
    ref = U.emulate(Rt, np.array([5.0, 5.0, 5.0]), 1e-3, U.make_policy("maxrate", 3))
    assert tau.tolist() == ref["tau"].tolist() and 0 in tau.tolist()


def test_scale_invariance_of_the_grid(cfg):
    """Payload x2 and rate x2 scale every backlog, payload and score by a
    power of two (exact in floating point), so (gamma, beta) and
    (2 gamma, 2 beta) give identical completion slots for every rule; the
    grid holds two such pairs."""
    arr = cfg["arrivals"]
    n = synth.points_per_agent(cfg)
    draw = synth.ofdma_draws(cfg, 5)
    for (g1, b1), (g2, b2) in (((0.5, 0.6), (1.0, 1.2)), ((1.0, 0.6), (2.0, 1.2))):
        R1, R2 = O.rates(draw, cfg, b1), O.rates(draw, cfg, b2)
        for s in SCHEDS:
            w = dict(dagrank=O.dagrank_weights(C_ENC, C_POST), tw_maxrate=arr["task_weights"]).get(s)
            a = U.emulate(R1, O.payload_bits(cfg, n, g1), arr["slot_s"], _oracle_policy(s, 6, arr["slot_s"], w))
            b = U.emulate(R2, O.payload_bits(cfg, n, g2), arr["slot_s"], _oracle_policy(s, 6, arr["slot_s"], w))
            assert a["tau"].tolist() == b["tau"].tolist()


def test_native_schedule_model_equals_oracle():
    rng = np.random.default_rng(9)
    for _ in range(2000):
        K = int(rng.integers(1, 17))
        a = (rng.integers(0, 40, K) * 1_000_000).tolist()       # slot-quantised, with ties
        c = rng.integers(0, 3_000_000, K).tolist()
        post = rng.integers(0, 5_000_000, int(rng.integers(1, 4))).tolist()
        TR, TB, W = S.paired_int(a, c, post)
        assert dag.paired_latency_ns(a, c, post, kind=HOST) == (TR, TB, W)
        r = S.execute_int(a, c, post)
        _, _, start = R.rtcc_schedule_model(a, c, sum(post), R.RTCC_MODE_RELEASE, kind=HOST)
        assert start.tolist() == r["start"]


def test_native_upward_rank_equals_oracle():
    rng = np.random.default_rng(2)
    for _ in range(300):
        n = int(rng.integers(1, 30))
        perm = rng.permutation(n)  # random topological order
        edges = [(int(perm[i]), int(perm[j])) for i in range(n) for j in range(i + 1, n) if rng.random() < 0.2]
        cost = rng.integers(0, 10**7, n).tolist()
        succ = {}
        for u, v in edges:
            succ.setdefault(u, []).append(v)
        want = O.upward_rank(dict(enumerate(cost)), succ)
        got = R.rtcc_upward_rank(cost, edges, kind=HOST)
        assert got.tolist() == [want[v] for v in range(n)]
    assert dag.dagrank_weights(C_ENC, C_POST, kind=HOST) == O.dagrank_weights(C_ENC, C_POST)
    assert dag.dagrank_weights([100, 300, 200], [50, 50], kind=HOST) == [0.5, 1.0, 0.75]


def test_native_argument_errors():
    ok = np.ones((4, 2, 2))
    bad_calls = [
        lambda: R.rtcc_uplink_emulate(ok, [1.0, 1.0], 17, 1e-3, kind=HOST),
        lambda: R.rtcc_uplink_emulate(ok, [1.0, 1.0], R.RTCC_SCHED_WEIGHTED_RATE, 1e-3, kind=HOST),
        lambda: R.rtcc_uplink_emulate(-ok, [1.0, 1.0], R.RTCC_SCHED_MAXRATE, 1e-3, kind=HOST),
        lambda: R.rtcc_uplink_emulate(ok * np.nan, [1.0, 1.0], R.RTCC_SCHED_MAXRATE, 1e-3, kind=HOST),
        lambda: R.rtcc_uplink_emulate(ok, [0.0, 1.0], R.RTCC_SCHED_MAXRATE, 1e-3, kind=HOST),
        lambda: R.rtcc_uplink_emulate(ok, [1.0, 1.0], R.RTCC_SCHED_MAXRATE, 0.0, kind=HOST),
        lambda: R.rtcc_uplink_emulate(ok, [1.0, 1.0], R.RTCC_SCHED_MAXRATE, 1e-3, avail_slot=[0, 1], kind=HOST),
        lambda: R.rtcc_uplink_emulate(ok, [1.0, 1.0], R.RTCC_SCHED_PROPORTIONAL_FAIR, 1e-3, pf_window=0.5,
                                      kind=HOST),
        lambda: R.rtcc_schedule_model([-1, 0], [1, 1], 0, R.RTCC_MODE_RELEASE, kind=HOST),
        lambda: R.rtcc_schedule_model([0, 0], [1, 1], 0, 7, kind=HOST),
        lambda: R.rtcc_schedule_model([0, 2**61], [1, 1], 0, R.RTCC_MODE_RELEASE, kind=HOST),
        lambda: R.rtcc_upward_rank([1, 1], [(0, 1), (1, 0)], kind=HOST),
        lambda: R.rtcc_upward_rank([1, 1], [(0, 0)], kind=HOST),
        lambda: R.rtcc_upward_rank([1, 1], [(0, 2)], kind=HOST),
        lambda: R.rtcc_upward_rank([-1], [], kind=HOST),
    ]
    for call in bad_calls:
        with pytest.raises(R.RtccError) as e:
            call()
        assert e.value.status == R.RTCC_E_ARG


def test_sweep_trials_equal_oracle_trials(cfg):
    cells = [(0.5, 1.4), (1.0, 0.8), (2.0, 0.6)]
    rows = sweep.run_trials(cfg, C_ENC, C_POST, [0, 4], kind=HOST, cells=cells)
    assert len(rows) == 2 * 3 * 5
    n = synth.points_per_agent(cfg)
    for r in rows:
        draw = synth.ofdma_draws(cfg, r["trace"])
        ref = O.trial(O.rates(draw, cfg, r["beta"]), O.payload_bits(cfg, n, r["gamma"]), cfg, r["scheduler"],
                      C_ENC, C_POST)
        assert r["tau"] == ref["tau"] and r["feasible"] == ref["feasible"]
        if ref["feasible"]:
            assert (r["T_R"], r["T_B"], r["W_pre"]) == (ref["T_R"], ref["T_B"], ref["W_pre"])
            assert r["T_B"] - r["T_R"] == r["W_pre"]


def test_sweep_cli_small_grid(tmp_path):
    out = tmp_path / "sweep.json"
    node = ",".join("%.3f" % (c * 1e-6) for c in C_ENC + C_POST)
    r = subprocess.run([sys.executable, "-m", "paper_2608_08330_amd.sweep", "--lib", "host", "--traces", "2",
                        "--node-ms", node, "--out", str(out)], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr
    res = json.loads(out.read_text())
    s = res["summary"]
    assert s["identity"]["trials"] == 2 * 20 * 5
    assert s["identity"]["identity_exact"] == s["identity"]["feasible"]
    assert s["identity"]["negative_gain"] == 0
    assert len(s["cells"]) == 20 and set(s["nominal"]) == set(SCHEDS)
    for c in s["cells"]:
        assert math.isfinite(c["mean_gain_ms"]) and c["mean_gain_ms"] >= 0
