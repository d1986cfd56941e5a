"""The seeded generators are deterministic and produce the stated shapes."""

import numpy as np

import synth


def test_generators_are_deterministic_and_shaped():
    for name in synth.CONFIG_NAMES:
        cfg = synth.config(name)
        a = synth.make_frame(name)
        b = synth.make_frame(name)
        assert len(a["points"]) == cfg["K"]
        for pa, pb in zip(a["points"], b["points"]):
            assert pa.dtype == np.float32 and pa.shape == (cfg["n_points"], 4)
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
