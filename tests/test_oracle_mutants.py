"""Strength of the oracle pins: plausible mistakes planted in a copy of the
oracle (on the CPU, never on a device) must each be caught by the pin battery
(hand-worked closed-form examples of the CosNet layer and of every bottleneck
activation, plus finite differences of every activation variant)."""

import importlib.util
import json
import math
import os
import types

import numpy as np
import pytest

import oracle.noble_oracle as good
from paper_2603_06492_amd import inputs as inp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

MUTATIONS = {
    "forward_mixing_transposed": ("H2 = C1 @ _f64(M)", "H2 = C1 @ _f64(M).T"),
    "phase2_dropped": ("A2 = H2 * _f64(omega2) + _f64(phi2)", "A2 = H2 * _f64(omega2)"),
    "bias_dropped": ("Y = Y + _f64(b)", "Y = Y"),
    "cos_slope_sign": ("return -np.sin(a)", "return np.sin(a)"),
    "outer_slope_sign": ("dA2 = activation_slope(f, fw[\"A2\"]) * dC2", "dA2 = -activation_slope(f, fw[\"A2\"]) * dC2"),
    "inner_slope_sign": ("dA1 = activation_slope(f, fw[\"A1\"]) * dC1", "dA1 = -activation_slope(f, fw[\"A1\"]) * dC1"),
    "dC1_not_transposed": ("dC1 = dH2 @ _f64(M).T", "dC1 = dH2 @ _f64(M)"),
    "dM_transposed": ("out[\"dM\"] = fw[\"C1\"].T @ dH2", "out[\"dM\"] = dH2.T @ fw[\"C1\"]"),
    "domega1_dropped_H": ("out[\"domega1\"] = np.sum(dA1 * H, axis=0)", "out[\"domega1\"] = np.sum(dA1, axis=0)"),
    "domega2_wrong_factor": ("out[\"domega2\"] = np.sum(dA2 * fw[\"H2\"], axis=0)",
                             "out[\"domega2\"] = np.sum(dA2 * fw[\"C1\"], axis=0)"),
    "dH_missing_omega1": ("out[\"dH\"] = dA1 * w1", "out[\"dH\"] = dA1"),
    "dH2_missing_omega2": ("dH2 = dA2 * _f64(omega2)", "dH2 = dA2"),
    "dx_missing_branch": ("out[\"dx\"] = dy @ W.T + dH @ D.T", "out[\"dx\"] = dy @ W.T"),
    "dW_up_uses_cos_argument": ("\"dW_up\": cb[\"out\"].T @ dy", "\"dW_up\": np.cos(cb[\"out\"]).T @ dy"),
    # activation variants
    "tanh_slope_not_squared": ("return 1.0 - np.tanh(a) ** 2", "return 1.0 - np.tanh(a)"),
    "tanh_value_is_sin": ("return np.tanh(a)\n", "return np.sin(a)\n"),
    "leaky_value_is_relu": ("return np.where(a > 0, a, LEAKY_SLOPE * a)", "return np.where(a > 0, a, 0.0 * a)"),
    "leaky_slope_swapped": ("return np.where(a > 0, 1.0, LEAKY_SLOPE)", "return np.where(a > 0, LEAKY_SLOPE, 1.0)"),
    "leaky_slope_value": ("LEAKY_SLOPE = 0.01", "LEAKY_SLOPE = 0.02"),
    "gelu_slope_missing_density": ("return _phi_cdf(a) + a * np.exp(-0.5 * a * a) / np.sqrt(2.0 * np.pi)",
                                   "return _phi_cdf(a)"),
    "gelu_value_is_cdf": ("return a * _phi_cdf(a)", "return _phi_cdf(a)"),
    "gelu_cdf_unscaled": ("return 0.5 * erfc(-a / np.sqrt(2.0))", "return 0.5 * erfc(-a)"),
    "gelu_cdf_through_erf": ("return 0.5 * erfc(-a / np.sqrt(2.0))",
                             "from scipy.special import erf\n    return 0.5 * (1.0 + erf(a / np.sqrt(2.0)))"),
    "one_layer_chain_mixes": ("        dC1 = dC2                                    # C2 = C1",
                              "        dC1 = 2.0 * dC2"),
    # the 3-layer CosNet
    "third_layer_phase_dropped": ("A3 = H3 * w3 + p3", "A3 = H3 * w3"),
    "third_layer_reuses_first_matrix": ("H3 = C2 @ M3", "H3 = C2 @ _f64(M)"),
    "third_layer_output_ignored": ("fw.update(H3=H3, A3=A3, C3=C3, out=C3)", "fw.update(H3=H3, A3=A3, C3=C3)"),
    "third_layer_gradient_skips_mixing": ("dC2 = dH3 @ M3.T", "dC2 = dH3"),
    "third_layer_dM_from_C1": ("dM3 = fw[\"C2\"].T @ dH3", "dM3 = fw[\"C1\"].T @ dH3"),
    "third_layer_frequency_gradient_without_H3": ("domega3 = np.sum(dA3 * fw[\"H3\"], axis=0)",
                                                  "domega3 = np.sum(dA3, axis=0)"),
    # grouped layers
    "grouped_dx_last_block_only": ('out = {"dx": sum(q["dx"] for q in parts),', 'out = {"dx": parts[-1]["dx"],'),
    "grouped_rank_slice_fixed": ("rs = slice(g * r, (g + 1) * r)", "rs = slice(0, r)"),
    "grouped_first_M_only": ("Mg = _f64(M)[:, g] if layers == 3 else _f64(M)[g]",
                             "Mg = _f64(M)[:, 0] if layers == 3 else _f64(M)[0]"),
    "grouped_column_block_shifted": ("return (slice(g * dg, (g + 1) * dg),", "return (slice((G - 1 - g) * dg, (G - g) * dg),"),
}


def _mutant(name):
    old, new = MUTATIONS[name]
    src = open(good.__file__).read()
    assert src.count(old) == 1, name
    mod = types.ModuleType(f"oracle_mutant_{name}")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def _eval(v):
    if isinstance(v, list):
        return np.array([_eval(e) for e in v], dtype=np.float64)
    if isinstance(v, str):
        return float(eval(v, {"__builtins__": {}}, {"pi": math.pi, "sqrt": math.sqrt, "atanh": math.atanh}))
    return float(v)


def _battery_passes(mod):
    """True when every pin in the battery holds for oracle module ``mod``."""
    def fwd(p):
        return mod.forward(p["x"], p["W"], p["b"], p["W_down"], p["omega1"], p["phi1"],
                           p["M"], p["omega2"], p["phi2"], p["W_up"])

    def bwd(p):
        return mod.backward(p["dy"], p["x"], p["W"], p["W_down"], p["omega1"], p["phi1"],
                            p["M"], p["omega2"], p["phi2"], p["W_up"])

    with open(os.path.join(GOLDEN, "hand_examples.json")) as f:
        for ex in json.load(f)["examples"]:
            p = {k: _eval(v) for k, v in ex["inputs"].items()}
            e = {k: _eval(v) for k, v in ex["expected"].items()}
            Y, _ = fwd(p)
            if not np.allclose(Y, e["y"], rtol=0, atol=1e-12):
                return False
            g = bwd(p)
            for k in e:
                if k in g and not np.allclose(g[k], e[k], rtol=0, atol=1e-11):
                    return False
    with open(os.path.join(GOLDEN, "activation_examples.json")) as f:
        for ex in json.load(f)["examples"]:
            act = ex["activation"]
            p = {k: _eval(v) for k, v in ex["inputs"].items()}
            Y, _ = mod.forward(p["x"], p["W"], p["b"], p["W_down"], p["omega1"], p["phi1"], p["M"],
                               p["omega2"], p["phi2"], p["W_up"], activation=act)
            g = mod.backward(p["dy"], p["x"], p["W"], p["W_down"], p["omega1"], p["phi1"], p["M"],
                             p["omega2"], p["phi2"], p["W_up"], activation=act)
            for k, v in ex["expected"].items():
                got = Y if k == "y" else g[k]
                if not np.allclose(got, _eval(v), rtol=0, atol=1e-12):
                    return False
    for act, (_, layers) in sorted(good.ACTIVATIONS.items()):
        p = {k: v.astype(np.float64) for k, v in
             inp.draw_projection("t", 4, 5, 6, 3, "f32", 21, bias_std=0.5, layers=layers).arrays.items()}
        g = mod.backward(p["dy"], p["x"], p["W"], p["W_down"], p["omega1"], p["phi1"], p["M"],
                         p["omega2"], p["phi2"], p["W_up"], activation=act)

        def loss(q):
            Y, _ = mod.forward(q["x"], q["W"], q["b"], q["W_down"], q["omega1"], q["phi1"], q["M"],
                               q["omega2"], q["phi2"], q["W_up"], activation=act)
            return float(np.sum(q["dy"] * Y))

        pairs = {"x": "dx", "W": "dW", "b": "db", "W_down": "dW_down", "W_up": "dW_up",
                 "omega1": "domega1", "phi1": "dphi1"}
        if layers >= 2:
            pairs.update({"M": "dM", "omega2": "domega2", "phi2": "dphi2"})
        for pn, gn in pairs.items():
            for idx in np.ndindex(p[pn].shape):
                qp, qm = dict(p), dict(p)
                qp[pn] = p[pn].copy()
                qm[pn] = p[pn].copy()
                qp[pn][idx] += 1e-6
                qm[pn][idx] -= 1e-6
                fd = (loss(qp) - loss(qm)) / 2e-6
                if abs(fd - g[gn][idx]) > 1e-6 * max(1.0, abs(g[gn][idx])):
                    return False
    return _grouped_pin(mod) and _tail_pin(mod)


def _grouped_pin(mod):
    """A 3-group layer against the single layer with block-diagonal M and
    W_up (the one-branch oracle, checked by the rest of the battery)."""
    G, r, dg = 3, 2, 4
    q = inp.draw_projection("grp", 5, 6, G * dg, r, "f32", 59, bias_std=0.5, groups=G)
    p = {k: v.astype(np.float64) for k, v in q.arrays.items()}
    R = G * r
    Mb, Ub = np.zeros((R, R)), np.zeros((R, G * dg))
    for g in range(G):
        Mb[g * r:(g + 1) * r, g * r:(g + 1) * r] = p["M"][g]
        Ub[g * r:(g + 1) * r, g * dg:(g + 1) * dg] = p["W_up"][g * r:(g + 1) * r]
    a = (p["W_down"], p["omega1"], p["phi1"])
    Yg, _ = mod.forward_grouped(p["x"], p["W"], p["b"], *a, p["M"], p["omega2"], p["phi2"], p["W_up"], G)
    Ys, _ = good.forward(p["x"], p["W"], p["b"], *a, Mb, p["omega2"], p["phi2"], Ub)
    if not np.allclose(Yg, Ys, rtol=0, atol=1e-12):
        return False
    gg = mod.backward_grouped(p["dy"], p["x"], p["W"], *a, p["M"], p["omega2"], p["phi2"], p["W_up"], G)
    gs = good.backward(p["dy"], p["x"], p["W"], *a, Mb, p["omega2"], p["phi2"], Ub)
    for k in ("dx", "dW", "db", "dW_down", "domega1", "dphi2"):
        if not np.allclose(gg[k], gs[k], rtol=0, atol=1e-12):
            return False
    for g in range(G):
        if not np.allclose(gg["dM"][g], gs["dM"][g * r:(g + 1) * r, g * r:(g + 1) * r], rtol=0, atol=1e-12):
            return False
    return True


def _tail_pin(mod):
    """GELU's value and slope in the lower tail lie inside the Mills-ratio
    bounds of the normal distribution function, and tanh's slope equals
    1 / cosh^2 where tanh saturates."""
    a = np.array([-6.0, -8.0, -10.0, -20.0])
    dens = np.exp(-0.5 * a * a) / math.sqrt(2.0 * math.pi)
    lo, hi = dens / np.abs(a) * (1.0 - 1.0 / (a * a)), dens / np.abs(a)
    cdf = mod.activation_value("gelu", a) / a
    d = mod.activation_slope("gelu", a)
    t = np.array([5.0, 9.5, -12.0])
    return bool(np.all(lo < cdf) and np.all(cdf < hi) and np.all(lo + a * dens < d) and np.all(d < hi + a * dens)
                and np.allclose(mod.activation_slope("tanh", t), np.cosh(t) ** -2.0, rtol=1e-5, atol=0))


def test_battery_accepts_the_oracle():
    assert _battery_passes(good)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_battery_rejects_mutant(name):
    assert not _battery_passes(_mutant(name))
