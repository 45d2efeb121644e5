"""The training recipe around the layer (Sec. 3.3, App. A) on the CPU:
Philox4x32-10 against the published known-answer vectors, the CPU draws'
distributions, the C ABI's recipe defaults and learning-rate multipliers
against the equations, and the validation of noble_init_params (no HIP call)."""

import ctypes

import numpy as np
import pytest
from scipy import stats

from oracle import recipe as rec
from paper_2603_06492_amd import noble

OK, NULL, SHAPE, MISAL = 0, 1, 2, 4


# Known-answer vectors of Philox4x32-10 published with the Random123 library
# (counter words, key words -> output words).
KAT = [
    ((0x00000000, 0x00000000, 0x00000000, 0x00000000), (0x00000000, 0x00000000),
     (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF), (0xFFFFFFFF, 0xFFFFFFFF),
     (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,want", KAT)
def test_philox_known_answers(ctr, key, want):
    got = rec.philox4x32_10(ctr, key)
    assert tuple(int(x) for x in got) == want


def test_philox_vectorised_matches_scalar_calls():
    c = np.arange(5, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15 & 0xFFFFFFFF)
    outs = rec.philox4x32_10((c, c + np.uint64(1), c + np.uint64(2), c + np.uint64(3)), (7, 11))
    for i in range(5):
        one = rec.philox4x32_10(tuple(int(v) for v in (c[i], c[i] + 1, c[i] + 2, c[i] + 3)), (7, 11))
        assert tuple(int(o[i]) for o in outs) == tuple(int(x) for x in one)


def test_draw_distributions():
    """Uniform draws fill [lo, hi] evenly; the Box-Muller draws are N(0, std^2)
    (Kolmogorov-Smirnov against the exact distributions)."""
    n = 200_000
    u = rec.draw_uniform(5, 2, n, 0.8, 1.2)
    assert u.min() >= 0.8 and u.max() <= 1.2
    assert stats.kstest((u - 0.8) / 0.4, "uniform").pvalue > 1e-3
    z = rec.draw_normal(5, 3, n, 0.1)
    assert stats.kstest(z / 0.1, "norm").pvalue > 1e-3
    assert abs(np.std(z) - 0.1) < 0.002
    # different tensor ids and seeds give unrelated streams
    assert abs(np.corrcoef(rec.draw_normal(5, 3, n, 1.0), rec.draw_normal(5, 4, n, 1.0))[0, 1]) < 0.01
    assert abs(np.corrcoef(rec.draw_normal(5, 3, n, 1.0), rec.draw_normal(6, 3, n, 1.0))[0, 1]) < 0.01


def test_init_values_scales():
    v = rec.init_values(1024, 512, 64, seed=3, dtype="f32")
    assert abs(np.std(v["W"]) - 0.5 / np.sqrt(1024)) < 0.01 * 0.5 / np.sqrt(1024)
    assert abs(np.std(v["W_up"]) - 0.01 / np.sqrt(64)) < 0.02 * 0.01 / np.sqrt(64)
    assert np.all(np.abs(v["W_down"]) <= 1 / np.sqrt(1024))
    assert np.all(np.abs(v["M"]) <= np.sqrt(3 / 64))
    # Xavier-uniform variance 2 / (fan_in + fan_out) = 1 / r
    assert abs(np.var(v["M"]) * 64 - 1.0) < 0.05
    for k in ("omega1", "omega2"):
        assert np.all((v[k] >= 0.8) & (v[k] <= 1.2))
    assert np.all(v["b"] == 0)
    vb = rec.init_values(1024, 512, 64, seed=3, dtype="bf16")
    np.testing.assert_array_equal(vb["W"], rec.to_bf16(v["W"]))


def test_to_bf16_ties_and_rounding():
    # 1 + 2^-8 is halfway between bf16 1 and 1 + 2^-7: ties go to even (1);
    # 1 + 3 * 2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: ties go to even
    a = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -2.5], np.float32)
    np.testing.assert_array_equal(rec.to_bf16(a), np.array([1.0, 1 + 2 ** -6, 1 + 2 ** -7, -2.5], np.float32))


def test_recipe_defaults_are_the_papers():
    rc = noble.noble_recipe_defaults()
    for k, v in rec.DEFAULTS.items():
        assert getattr(rc, k) == v, k
    assert noble.noble_recipe_defaults(alpha=0.02).alpha == 0.02
    with pytest.raises(TypeError):
        noble.noble_recipe_defaults(beta=1.0)


def test_lr_multipliers_closed_form():
    """d = 2048, r = 128: the ratio is 16, so W_up takes 16^0.6 = 2^2.4 and M
    16^0.45 = 2^1.8 (Eqs. 3-4 with gamma = 0.3, gamma_M = 0.45)."""
    m = noble.noble_lr_multipliers(2048, 6144, 128)
    assert m["W_up"] == pytest.approx(2 ** 2.4, rel=1e-12)
    assert m["M"] == pytest.approx(2 ** 1.8, rel=1e-12)
    assert (m["W"], m["b"], m["W_down"], m["omega"], m["phi"]) == (1.0, 1.0, 1.0, 3.0, 5.0)


@pytest.mark.parametrize("shape", [(1024, 4096, 64), (8192, 2048, 128), (768, 3072, 32), (64, 64, 8), (64, 64, 0)])
def test_lr_multipliers_match_oracle(shape):
    got = noble.noble_lr_multipliers(*shape)
    want = rec.lr_multipliers(*shape)
    for k, v in want.items():
        assert got[k] == pytest.approx(v, rel=1e-12), k
    rc = noble.noble_recipe_defaults(gamma=0.5, gamma_M=1.0)
    got = noble.noble_lr_multipliers(*shape, recipe=rc)
    want = rec.lr_multipliers(*shape, recipe=dict(gamma=0.5, gamma_M=1.0))
    for k, v in want.items():
        assert got[k] == pytest.approx(v, rel=1e-12), k


def test_lr_multipliers_validation():
    L = noble.lib()
    d = noble.make_desc(0, 64, 64, 12, noble.NOBLE_BF16)
    rc, out = noble.noble_recipe_defaults(), noble.noble_lr_mults()
    assert L.noble_lr_multipliers(ctypes.byref(d), ctypes.byref(rc), ctypes.byref(out)) == SHAPE
    d = noble.make_desc(0, 64, 64, 16, noble.NOBLE_BF16)
    assert L.noble_lr_multipliers(ctypes.byref(d), None, ctypes.byref(out)) == NULL
    assert L.noble_lr_multipliers(ctypes.byref(d), ctypes.byref(rc), None) == NULL
    assert L.noble_lr_multipliers(None, ctypes.byref(rc), ctypes.byref(out)) == NULL


def test_param_groups():
    groups = noble.param_groups({"W": "w", "b": None, "W_down": "d", "omega1": "o1", "omega2": "o2",
                                 "phi1": "p1", "phi2": "p2", "M": "m", "W_up": "u"}, 1e-3, 2048, 2048, 128)
    lr = {g["name"]: (g["lr"], g["params"]) for g in groups}
    assert lr["W"] == (1e-3, ["w"]) and lr["W_down"] == (1e-3, ["d"])
    assert lr["omega"] == (pytest.approx(3e-3), ["o1", "o2"]) and lr["phi"] == (pytest.approx(5e-3), ["p1", "p2"])
    assert lr["W_up"][0] == pytest.approx(1e-3 * 2 ** 2.4) and lr["M"][0] == pytest.approx(1e-3 * 2 ** 1.8)
    assert "b" not in lr
    with pytest.raises(KeyError):
        noble.param_groups({"V": "v"}, 1e-3, 64, 64, 8)


def test_init_params_validation_makes_no_hip_call():
    L = noble.lib()
    rc = noble.noble_recipe_defaults()
    d = noble.make_desc(0, 64, 64, 16, noble.NOBLE_BF16)
    none = [None] * 9
    assert L.noble_init_params(ctypes.byref(d), ctypes.byref(rc), 1, *none, None) == OK
    assert L.noble_init_params(ctypes.byref(d), None, 1, *none, None) == NULL
    bad = list(none)
    bad[0] = 0x100001          # W, bf16: odd address
    assert L.noble_init_params(ctypes.byref(d), ctypes.byref(rc), 1, *bad, None) == MISAL
    bad = list(none)
    bad[3] = 0x100002          # omega1, float32: not 4-byte aligned
    assert L.noble_init_params(ctypes.byref(d), ctypes.byref(rc), 1, *bad, None) == MISAL
    d = noble.make_desc(0, 64, 64, 20, noble.NOBLE_BF16)
    assert L.noble_init_params(ctypes.byref(d), ctypes.byref(rc), 1, *none, None) == SHAPE


def test_init_values_three_layer_form_continues_the_streams():
    """The 3-layer form's M [2, r, r] and omega2 / phi2 [2, r]: the first
    halves are the two-layer draws, the second halves continue the same
    streams (and the same distributions)."""
    two = rec.init_values(256, 128, 32, seed=9, dtype="bf16")
    three = rec.init_values(256, 128, 32, seed=9, dtype="bf16", layers=3)
    assert three["M"].shape == (2, 32, 32) and three["omega2"].shape == (2, 32)
    np.testing.assert_array_equal(three["M"][0], two["M"])
    for k in ("omega2", "phi2"):
        np.testing.assert_array_equal(three[k][0], two[k])
    for k in ("W", "W_down", "W_up", "omega1", "phi1", "b"):
        np.testing.assert_array_equal(three[k], two[k])
    assert not np.array_equal(three["M"][1], three["M"][0])
    assert np.all(np.abs(three["M"][1]) <= np.sqrt(3 / 32) * (1 + 2.0 ** -8))   # bf16 rounding
    assert np.all((three["omega2"][1] >= 0.8) & (three["omega2"][1] <= 1.2))
    g = rec.init_values(64, 96, 8, seed=9, dtype="f32", groups=3, layers=3)
    assert g["M"].shape == (2, 3, 8, 8) and g["phi2"].shape == (2, 24)
