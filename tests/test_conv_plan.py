"""The conv planner through the C ABI (host computation, no GPU): the c5
plan at 256 CUs for launches over 1, 2, 4 and 8 agents' maps, and on every
layer shape of the configs, for several CU counts and every batch size, the
invariant that lets a group release equal separate releases bit for bit:
all tilings a layer takes accumulate each output element in the same order
(the same channel chunks and taps, so the same chunk width and one wave
group), with the same K split."""

import pytest

import synth
from paper_2608_08330_amd import rtcc as R

IMPLICIT = (0,)         # implicit GEMM, 128 x 128 tiles
IMPLICIT256 = (12,)     # 256 x 128 tiles, every other tile's K steps backwards
HALO_RULE = (1, 2, 9)   # halo tilings whose chunk width follows the channel rule
HALO_C64 = (8, 10)      # halo tilings with 64-byte chunks
HALO_S2 = (3, 4, 11)    # stride-2 halo tilings (64-byte chunks)
TWO_GROUPS = (5, 6)     # split chunk sums (another order): never planned


def _lib():
    return R.load("host")


def _layers(name):
    cfg = synth.config(name)
    h = round((cfg["y_range"][1] - cfg["y_range"][0]) / cfg["pillar"])
    w = round((cfg["x_range"][1] - cfg["x_range"][0]) / cfg["pillar"])
    c = cfg["c_pfn"]
    out = []
    for stride, co, n in cfg["stages"]:
        for l in range(n):
            s = stride if l == 0 else 1
            ho, wo = -(-h // s), -(-w // s)
            out.append((h, w, c, ho, wo, co, s))
            h, w, c = ho, wo, co
    return cfg, out


def _family(variant, ci, elt):
    if variant in IMPLICIT:
        return "implicit"
    if variant in IMPLICIT256:
        return "implicit256"
    if variant in HALO_RULE:
        return ("halo", 128 if (ci * elt) % 128 == 0 and ci * elt >= 512 else 64)
    if variant in HALO_C64 or variant in HALO_S2:
        return ("halo", 64)
    raise AssertionError("tiling %d is not planned" % variant)


def test_c5_plans_at_256_cus():
    _cfg, layers = _layers("c5")
    lib = _lib()
    want = {1: (12, 1, 1, 3, 8, 8, 8, 8, 4, 2, 2, 2, 2),
            2: (12, 1, 1, 11, 10, 10, 10, 10, 4, 2, 2, 2, 2),
            4: (12, 1, 1, 11, 10, 10, 10, 10, 3, 1, 1, 1, 1),
            8: (12, 1, 1, 11, 10, 10, 10, 10, 11, 9, 9, 9, 9)}
    for maps, v in want.items():
        got = [R.rtcc_conv_tiling(*s, 256, maps, lib=lib) for s in layers]
        assert got == [(x, 1) for x in v], maps


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c5", "t_var", "t_max"])
@pytest.mark.parametrize("n_cu", [80, 104, 228, 256, 304])
def test_every_batch_size_accumulates_alike(name, n_cu):
    cfg, layers = _layers(name)
    bf16 = cfg["precision"] == "bf16"
    elt = 2 if bf16 else 4
    lib = _lib()
    for shape in layers:
        plans = [R.rtcc_conv_tiling(*shape, n_cu, m, bf16=bf16, lib=lib) for m in range(1, 17)]
        fams = {_family(v, shape[2], elt) for v, _sp in plans}
        assert len(fams) == 1, (shape, plans)
        assert len({sp for _v, sp in plans}) == 1, (shape, plans)
        for v, _sp in plans:
            assert v not in TWO_GROUPS
            if shape[6] == 1:
                assert v not in HALO_S2
            elif v not in IMPLICIT + IMPLICIT256:
                assert v in HALO_S2


def test_arguments_are_checked():
    lib = _lib()
    for bad in [dict(maps=0), dict(maps=17), dict(stride=3), dict(n_cu=0), dict(Ci=0)]:
        kw = dict(Hi=64, Wi=64, Ci=64, Ho=64, Wo=64, Co=128, stride=1, n_cu=256, maps=1)
        kw.update(bad)
        with pytest.raises(R.RtccError) as e:
            R.rtcc_conv_tiling(kw["Hi"], kw["Wi"], kw["Ci"], kw["Ho"], kw["Wo"], kw["Co"], kw["stride"],
                               kw["n_cu"], kw["maps"], lib=lib)
        assert e.value.status == R.RTCC_E_ARG
