"""Host-side harness logic against the oracle: the product's uplink
emulation (the library's rtcc_uplink_emulate, through the host-test build of
the same source) and DAG gain model reproduce the oracle's, and the
ergodic-rate closed form agrees with scipy."""

import math

import numpy as np
import pytest

import synth
from oracle import schedule as S
from oracle import uplink as U
from paper_2608_08330_amd import dag, uplink


@pytest.mark.parametrize("snr", [0.0, 10.0, 20.0])
def test_mean_rate_matches_oracle(snr):
    assert math.isclose(uplink.mean_rate(snr, 20e6), U.ergodic_rate(snr, 20e6), rel_tol=1e-12)


@pytest.mark.parametrize("sched", ["rr", "pf"])
def test_uplink_completion_times_match_oracle(sched):
    cfg = synth.config("c4")
    rng = np.random.default_rng(11)
    for t in range(3):
        g = synth.fading_draws(cfg, t, n_slots=8000)
        B = rng.uniform(1e6, 2.5e7, 5)
        for snr in (0.0, 10.0, 20.0):
            a = uplink.completion_times(g, B, snr, 20e6, 1e-3, sched, 100, kind="host")
            ref = U.trace_arrivals(cfg, g, B / 8.0, snr, sched)["a"]
            assert np.array_equal(np.isfinite(a), np.isfinite(ref))
            fin = np.isfinite(a)
            np.testing.assert_allclose(a[fin], ref[fin], rtol=0, atol=1e-12)


def test_dag_gain_matches_schedule_oracle():
    rng = np.random.default_rng(5)
    for _ in range(500):
        K = int(rng.integers(1, 9))
        a = rng.exponential(10.0, K)
        c = rng.uniform(0.1, 5.0, K)
        post = float(rng.uniform(0.1, 3.0))
        want = S.barrier(a, c, [post])["T"] - S.rtcc(a, c, [post])["T"]
        assert math.isclose(dag.predicted_gain(a, c, post), want, rel_tol=1e-9, abs_tol=1e-9)
