"""Pins of the five causal evaluation schedulers (oracle/uplink.py), the
OFDMA channel and the measured-DAG trial (oracle/ofdma.py): hand-computed
allocations and traces, closed forms of the schedulers on constant rates,
reductions between schedulers, and statistics of the channel draws."""

import math

import numpy as np
import pytest

import synth
from oracle import ofdma as O
from oracle import schedule as S
from oracle import uplink as U


def _run(R_tkf, B, sched, weights=None, ell=None, slot_s=1.0):
    R = np.asarray(R_tkf, dtype=np.float64)
    pol = U.make_policy(sched, R.shape[1], slot_s=slot_s, weights=weights)
    return U.emulate(R, np.asarray(B, dtype=np.float64), slot_s, pol, ell=ell)


def _one_slot(R_kf, Q, sched, weights=None):
    """Agent given each RB in one slot with slot-start backlog Q (slot 1 s,
    so a rate is units per slot)."""
    res = _run([R_kf], Q, sched, weights)
    x = res["x"][0]
    return [int(np.argmax(x[:, f])) if x[:, f].any() else -1 for f in range(x.shape[1])]


# ------------------------------------------------------------ score rules

def test_one_slot_decisions_by_hand():
    # R[k][f]: agent 0 is strong on RB 0, agent 1 on RB 1; backlog Q = (1, 5)
    R = [[3.0, 1.0], [1.0, 2.0]]
    Q = [1.0, 5.0]
    assert _one_slot(R, Q, "maxrate") == [0, 1]            # 3 > 1;  1 < 2
    assert _one_slot(R, Q, "maxweight") == [1, 1]          # 3 < 5;  1 < 10
    assert _one_slot(R, Q, "earliest_release") == [0, 0]   # -1/3 > -5;  -1 > -5/2
    assert _one_slot(R, Q, "dagrank", [0.25, 1.0]) == [1, 1]  # 0.75 < 1;  0.25 < 2
    # task weights (1.00, 0.80): 1 * 1 > 0.8 * 1.2 although 1 < 1.2
    assert _one_slot([[3.0, 1.0], [1.0, 1.2]], Q, "tw_maxrate", [1.0, 0.8]) == [0, 0]
    assert _one_slot([[3.0, 1.0], [1.0, 1.2]], Q, "maxrate") == [0, 1]


def test_ties_go_to_the_smallest_index():
    R = [[2.0, 2.0], [2.0, 2.0], [2.0, 2.0]]
    for s, w in (("maxrate", None), ("dagrank", [1.0, 1.0, 1.0]), ("tw_maxrate", [0.5, 0.5, 0.5])):
        assert _one_slot(R, [4.0, 4.0, 4.0], s, w) == [0, 0]
    assert _one_slot(R, [4.0, 4.0, 4.0], "maxweight") == [0, 0]
    assert _one_slot(R, [4.0, 4.0, 4.0], "earliest_release") == [0, 0]
    # an RB that carries nothing for anyone: every EarliestRelease score is
    # -inf, and the smallest eligible index still takes the RB
    assert _one_slot([[0.0], [0.0]], [1.0, 1.0], "earliest_release") == [0]
    # finished agents are not eligible: agent 0 has no backlog
    assert _one_slot(R, [0.0, 4.0, 4.0], "maxrate") == [1, 1]


def test_earliest_release_is_shortest_remaining_first():
    # one RB, unit rate for everyone: each slot serves the smallest backlog,
    # so agents finish in ascending payload order, back to back:
    # B = (5, 2, 3) -> agent 1 at slot 2, agent 2 at 2 + 3, agent 0 at 5 + 5
    res = _run(np.ones((20, 3, 1)), [5.0, 2.0, 3.0], "earliest_release")
    assert res["tau"].tolist() == [10, 2, 5]


def test_maxweight_is_longest_queue_first():
    # one RB, unit rate, equal payloads n = 2: the largest backlog is served
    # (ties to the smallest index), so the queues drain together and the
    # agents finish in the last K slots: a_k = K (n - 1) + k + 1
    res = _run(np.ones((20, 3, 1)), [2.0, 2.0, 2.0], "maxweight")
    assert res["tau"].tolist() == [4, 5, 6]
    # two RBs: agent 0 (rate 2) takes both RBs while Q0 R0 > Q1 R1, and the
    # second slot's surplus is wasted (payload 6 = 4 + 2): a = (2, 4)
    R = np.tile(np.array([[2.0, 2.0], [1.0, 1.0]]), (10, 1, 1))
    res = _run(R, [6.0, 3.0], "maxweight")
    assert res["tau"].tolist() == [2, 4]
    assert res["d"][:4].tolist() == [[4.0, 0.0], [4.0, 0.0], [0.0, 2.0], [0.0, 2.0]]


def test_maxrate_serves_the_fastest_first_and_waits_for_local_availability():
    # constant rates (1, 3, 2) per slot on one RB, payloads (3, 3, 4):
    # agent 1 done in slot 1, agent 2 in slots 2-3, agent 0 in slots 4-6
    R = np.tile(np.array([[1.0], [3.0], [2.0]]), (10, 1, 1))
    assert _run(R, [3.0, 3.0, 4.0], "maxrate")["tau"].tolist() == [6, 1, 3]
    # agent 1 (faster) only becomes available in slot 3 (eq. eligible_set)
    R = np.tile(np.array([[1.0], [5.0]]), (10, 1, 1))
    res = _run(R, [2.0, 5.0], "maxrate", ell=np.array([1, 3]))
    assert res["tau"].tolist() == [2, 3]
    assert res["x"][:2, 1, 0].sum() == 0


def _random_ofdma(seed, T=400, K=6, F=8):
    rng = np.random.default_rng(seed)
    R = rng.uniform(250e3, 4500e3, (1, K, F)) * rng.exponential(1.0, (T, K, F))
    B = rng.uniform(0.4e6, 0.6e6, K)
    return R, B


def test_reductions_between_schedulers():
    for seed in range(3):
        R, B = _random_ofdma(seed)
        mr = _run(R, B, "maxrate", slot_s=1e-3)
        # equal DAG ranks or equal task weights reduce to MaxRate
        for s, w in (("dagrank", [1.0] * 6), ("tw_maxrate", [0.7] * 6)):
            other = _run(R, B, s, w, slot_s=1e-3)
            assert np.array_equal(other["x"], mr["x"]) and np.array_equal(other["tau"], mr["tau"])
        # one agent alone: every rule gives it every RB until done
        one = [_run(R[:, :1], B[:1], s, [1.0], slot_s=1e-3)["tau"][0]
               for s in ("maxrate", "maxweight", "earliest_release", "dagrank", "tw_maxrate")]
        assert len(set(one)) == 1


@pytest.mark.parametrize("sched", ["maxrate", "maxweight", "earliest_release", "dagrank", "tw_maxrate"])
def test_arrival_definition_and_orthogonality(sched):
    """a_k = Delta min{t : sum_{tau<=t} d_k[tau] >= B_k} (eq. branch_arrival)
    by brute force, at most one agent per RB (eq. rb_orthogonality), and
    nothing sent after completion."""
    R, B = _random_ofdma(7)
    w = [1.0, 0.8, 1.2, 0.7, 1.05, 0.6]
    res = _run(R, B, sched, w, slot_s=1e-3)
    assert res["feasible"]
    assert np.all(res["x"].sum(axis=1) <= 1)
    for k in range(6):
        cum = np.cumsum(res["d"][:, k])
        t_star = int(np.nonzero(cum >= B[k] * (1 - 1e-12))[0][0]) + 1
        assert res["tau"][k] == t_star
        assert res["x"][t_star:, k].sum() == 0
    # every slot with an eligible agent uses every RB (work-conserving RBs)
    busy = res["x"].sum(axis=(1, 2))
    assert np.all(busy[:max(res["tau"])] == R.shape[2])


# ------------------------------------------------------------ DAG rank

def test_upward_rank_by_hand():
    #   A(2) -> B(3) -> D(1);  A -> C(4) -> D
    cost = {"A": 2, "B": 3, "C": 4, "D": 1}
    succ = {"A": ["B", "C"], "B": ["D"], "C": ["D"]}
    assert O.upward_rank(cost, succ) == {"A": 7, "B": 4, "C": 5, "D": 1}
    # encoders (100, 300, 200) before a post-join chain (50, 50): ranks
    # (200, 400, 300) normalised by 400
    assert O.dagrank_weights([100, 300, 200], [50, 50]) == [0.5, 1.0, 0.75]


# ------------------------------------------------------------ channel

def test_reflection_closed_form():
    assert O.reflect(85.0, 80.0) == 75.0
    assert O.reflect(-5.0, 80.0) == 5.0
    assert O.reflect(165.0, 80.0) == 5.0
    assert O.reflect(80.0, 80.0) == 80.0
    assert O.reflect(31.5, 80.0) == 31.5
    arr = synth.config("s6")["arrivals"]
    draw = dict(speed_mps=np.array([10.0]), heading=np.array([0.0]), pos0_m=np.array([[75.0, 25.0]]))
    assert O.position(draw, arr, 0, 1) == (75.0, 25.0)
    x, y = O.position(draw, arr, 0, 1001)  # 1 s later: 85 m folds back to 75 m
    assert x == pytest.approx(75.0, abs=1e-12) and y == 25.0


def test_path_gain_closed_form():
    arr = synth.config("s6")["arrivals"]
    d0 = arr["ref_distance_m"]
    assert O.path_gain(0.0, arr) == 1.0 and O.path_gain(d0, arr) == 1.0 and O.path_gain(0.5 * d0, arr) == 1.0
    assert O.path_gain(2 * d0, arr) == pytest.approx(2.0 ** -2.15, rel=1e-15)
    ds = np.linspace(d0, 60.0, 50)
    g = [O.path_gain(d, arr) for d in ds]
    assert all(a > b for a, b in zip(g, g[1:]))
    slope = np.polyfit(np.log(ds[1:]), np.log(g[1:]), 1)[0]
    assert slope == pytest.approx(-2.15, abs=1e-9)


def test_blockage_chain_statistics():
    arr = dict(synth.config("s6")["arrivals"])
    T, K = 400_000, 2
    rng = np.random.default_rng(3)
    draw = dict(block_u0=rng.uniform(0, 1, K), block_u=rng.uniform(0, 1, (T, K)))
    st = np.array(O.blockage(draw, arr, T, K))
    rho, D = arr["blockage_fraction"], arr["blockage_dwell_slots"]
    assert abs(st.mean() - rho) < 0.03
    runs = []
    for k in range(K):
        s = st[:, k].astype(int)
        edges = np.flatnonzero(np.diff(np.concatenate([[0], s, [0]])))
        runs += list(edges[1::2] - edges[::2])
    assert abs(np.mean(runs) - D) < 0.1 * D


def test_rates_closed_form_and_scaling():
    cfg = synth.config("s6")
    arr = cfg["arrivals"]
    draw = synth.ofdma_draws(cfg, 0)
    lo, hi = arr["ref_rate_bps"]
    assert draw["ref_rate_bps"].min() >= lo and draw["ref_rate_bps"].max() < hi
    R1 = O.rates(draw, cfg, 1.0)
    R8 = O.rates(draw, cfg, 0.8)
    np.testing.assert_allclose(R8, 0.8 * R1, rtol=1e-15, atol=0)
    # without fading and blockage the rate is Rref * G(distance)
    plain = dict(draw, fading=np.ones_like(draw["fading"]), block_u0=np.ones(cfg["K"]),
                 block_u=np.ones_like(draw["block_u"]))
    Rp = O.rates(plain, cfg, 1.0)
    sx, sy = arr["server_m"]
    for t in (1, 450, 900):
        for k in range(cfg["K"]):
            x, y = O.position(draw, arr, k, t)
            g = min(1.0, (arr["ref_distance_m"] / math.hypot(x - sx, y - sy)) ** arr["path_loss_exp"])
            np.testing.assert_allclose(Rp[t - 1, k], draw["ref_rate_bps"][k] * g, rtol=1e-14)
    # fading has unit mean: the time-average rate is close to the plain one
    # times the blockage factor
    blocked = np.array(O.blockage(draw, arr, arr["t_max_slots"], cfg["K"]))
    zb = 10 ** (-arr["blockage_loss_db"] / 10)
    expect = (Rp * np.where(blocked, zb, 1.0)[:, :, None]).mean()
    assert R1.mean() == pytest.approx(expect, rel=0.05)


def test_payload_bits():
    cfg = synth.config("s6")
    n = synth.points_per_agent(cfg)
    B = O.payload_bits(cfg, n, 1.0)
    assert np.all(B / 8 / 1024 >= 60.6 - 0.01) and np.all(B / 8 / 1024 <= 65.2 + 0.01)
    np.testing.assert_array_equal(O.payload_bits(cfg, n, 2.0), 2.0 * B)


# ------------------------------------------------------------ trials

def test_measured_dag_trials_identity_exact():
    """T_B - T_R = W_pre exactly, on integer-nanosecond trials over the
    (gamma, beta) corners and the five schedulers."""
    cfg = synth.config("s6")
    arr = cfg["arrivals"]
    n = synth.points_per_agent(cfg)
    c_enc = [6_110_000, 6_520_000, 6_300_000, 6_250_000, 6_400_000, 6_200_000]
    c_post = [16_760_000]
    draw = synth.ofdma_draws(cfg, 1)
    positive = 0
    for gamma, beta in ((0.5, 1.4), (1.0, 0.8), (2.0, 0.6)):
        R = O.rates(draw, cfg, beta)
        B = O.payload_bits(cfg, n, gamma)
        for s in arr["schedulers"]:
            r = O.trial(R, B, cfg, s, c_enc, c_post)
            assert r["feasible"]
            assert r["T_B"] - r["T_R"] == r["W_pre"] >= 0
            assert r["T_B"] == max(r["a_ns"]) + sum(c_enc) + sum(c_post)
            assert all(a % 1_000_000 == 0 for a in r["a_ns"])
            positive += r["W_pre"] > 0
    assert positive > 0


def test_zero_overlap_boundary():
    # all branches complete in the same slot: no encoder can start before
    # A, RTCC and barrier coincide
    TR, TB, W = S.paired_int([5_000_000] * 4, [1000, 2000, 3000, 4000], [500])
    assert TR == TB and W == 0
    # out-of-order arrivals with a tie, hand-computed (ns):
    # a = (4, 0, 4), c = (1, 2, 3), post 1 -> order 1, 0, 2; T_R = 9, T_B = 11
    TR, TB, W = S.paired_int([4, 0, 4], [1, 2, 3], [1])
    assert (TR, TB, W) == (9, 11, 2)
