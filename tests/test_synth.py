"""The seeded generators are deterministic and produce the stated shapes."""

import numpy as np

import synth


def test_generators_are_deterministic_and_shaped():
    for name in synth.CONFIG_NAMES:
        cfg = synth.config(name)
        a = synth.make_frame(name)
        b = synth.make_frame(name)
        assert len(a["points"]) == cfg["K"]
        for pa, pb, n in zip(a["points"], b["points"], synth.points_per_agent(cfg)):
            assert pa.dtype == np.float32 and pa.shape == (n, 4) and n <= cfg["n_points"]
            assert np.array_equal(pa, pb)
        assert np.array_equal(a["poses"][0], [0.0, 0.0, 0.0])
        for n, arr in a["weights"].items():
            assert np.array_equal(arr, b["weights"][n])


def test_load_sweep_reuses_config3_frames():
    a = synth.make_frame("c3")
    b = synth.make_frame("c4")
    for pa, pb in zip(a["points"], b["points"]):
        assert np.array_equal(pa, pb)
    assert np.array_equal(a["poses"], b["poses"])


def test_arrival_draws():
    c1 = synth.arrival_draws(synth.config("c1"))
    assert c1.tolist() == [[0.0, 5.0]]
    c2 = synth.arrival_draws(synth.config("c2"))
    assert c2.shape == (30, 3) and np.all(c2 > 0)
    c5 = synth.arrival_draws(synth.config("c5"))
    assert c5.shape == (30, 8)
    assert 10 < np.median(c5) < 40
    g = synth.fading_draws(synth.config("c4"), 0, n_slots=100)
    assert g.shape == (100, 5, 1)


def test_ofdma_draws_are_deterministic_and_independent_per_trace():
    cfg = synth.config("s6")
    arr = cfg["arrivals"]
    a, b, c = synth.ofdma_draws(cfg, 0), synth.ofdma_draws(cfg, 0), synth.ofdma_draws(cfg, 1)
    T, K, F = arr["t_max_slots"], cfg["K"], arr["n_rb"]
    assert a["fading"].shape == (T, K, F) and a["ref_rate_bps"].shape == (K, F)
    assert a["block_u"].shape == (T, K) and a["pos0_m"].shape == (K, 2)
    for key in a:
        assert np.array_equal(a[key], b[key])
        assert not np.array_equal(a[key], c[key])
    assert np.all((a["pos0_m"] >= 0) & (a["pos0_m"] <= np.array(arr["area_m"])))
    lo, hi = arr["speed_mps"]
    assert np.all((a["speed_mps"] >= lo) & (a["speed_mps"] < hi))
    # branch inputs of 60.6 to 65.2 KiB of 16-byte points
    kib = np.array(synth.points_per_agent(cfg)) * arr["bytes_per_point"] / 1024
    assert abs(kib.min() - 60.6) < 0.01 and abs(kib.max() - 65.2) < 0.01


def test_stream_frames_differ_and_frame_zero_is_the_config_frame():
    a = synth.make_frame("t_attn")
    b = synth.make_frame("t_attn", 0)
    c = synth.make_frame("t_attn", 1)
    d = synth.make_frame("t_attn", 1)
    for k in range(len(a["points"])):
        assert np.array_equal(a["points"][k], b["points"][k])
        assert not np.array_equal(a["points"][k], c["points"][k])
        assert np.array_equal(c["points"][k], d["points"][k])
    assert np.array_equal(a["poses"], b["poses"]) and not np.array_equal(a["poses"][1:], c["poses"][1:])
    assert np.all(c["poses"][0] == 0.0)
    for name in a["weights"]:
        assert np.array_equal(a["weights"][name], c["weights"][name])
