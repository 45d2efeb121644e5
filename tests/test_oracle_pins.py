"""Pins of the fp64 oracle against things fixed outside it (CPU only).

* hand-worked closed-form examples of Eq. (1)-(2) (tests/golden/hand_examples.json)
* Table 1 "Params+" from the branch's parameter shapes
* central finite differences of L = sum(dy * y) for every gradient
* an independently written torch forward differentiated by autograd (fp64)
* special cases with closed forms (W_up = 0, omega2 = 0, omega1 = 0, M = 0)
* invariants: evenness of cos, 2 pi periodicity, rescaling of W_down, row
  permutation, and the |C2| <= 1 bound on the branch
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2603_06492_amd import inputs as inp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
GRADS = ("dx", "dW", "db", "dW_down", "dM", "dW_up", "domega1", "dphi1", "domega2", "dphi2")


def _eval(v):
    if isinstance(v, str):
        return float(eval(v, {"__builtins__": {}}, {"pi": math.pi, "sqrt": math.sqrt}))
    return float(v)


def _arr(v):
    if isinstance(v, list):
        return np.array([_arr(e) for e in v], dtype=np.float64)
    return _eval(v)


def _fwd(p):
    return oracle.forward(p["x"], p["W"], p["b"], p["W_down"], p["omega1"], p["phi1"],
                          p["M"], p["omega2"], p["phi2"], p["W_up"])


def _bwd(p, **kw):
    return oracle.backward(p["dy"], p["x"], p["W"], p["W_down"], p["omega1"], p["phi1"],
                           p["M"], p["omega2"], p["phi2"], p["W_up"], **kw)


def _tiny(seed=3, T=5, d_in=7, d_out=6, r=3, layers=2):
    p = inp.draw_projection("tiny", T, d_in, d_out, r, "f32", seed, bias_std=0.5, layers=layers)
    return {k: v.astype(np.float64) for k, v in p.arrays.items()}


# ---------------------------------------------------------------- golden -----

def _hand_examples():
    with open(os.path.join(GOLDEN, "hand_examples.json")) as f:
        return json.load(f)["examples"]


@pytest.mark.parametrize("ex", _hand_examples(), ids=lambda e: e["name"])
def test_hand_worked_examples(ex):
    p = {k: _arr(v) for k, v in ex["inputs"].items()}
    exp = {k: _arr(v) for k, v in ex["expected"].items()}
    Y, H = _fwd(p)
    np.testing.assert_allclose(Y, exp["y"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(H, exp["H"], rtol=0, atol=1e-12)
    g = _bwd(p)
    for k in GRADS:
        np.testing.assert_allclose(g[k], exp[k], rtol=0, atol=1e-11, err_msg=k)


def test_mixing_orientation_is_distinguished():
    """The r = 2 example gives a different y under the transposed mixing."""
    ex = [e for e in _hand_examples() if e["name"] == "mixing_orientation_r2"][0]
    p = {k: _arr(v) for k, v in ex["inputs"].items()}
    p_t = dict(p, M=p["M"].T.copy())
    Y, _ = _fwd(p)
    Yt, _ = _fwd(p_t)
    assert abs(Y[0, 0] - Yt[0, 0]) > 1.0


def test_table1_params_plus():
    with open(os.path.join(GOLDEN, "table1_params_plus.json")) as f:
        t1 = json.load(f)
    V = t1["vocab"]
    for row in t1["rows"]:
        L, d, r = row["layers"], row["width"], row["rank"]
        h = math.ceil(8 * d / 3 / 64) * 64
        # untied input embedding and LM head, Q K V O, fused GeGLU up (d -> 2h),
        # down (h -> d), two RMSNorm gains per block and a final one
        base = 2 * V * d + L * (4 * d * d + 2 * h * d + h * d + 2 * d) + d

        def branch(di, do):
            return sum(int(np.prod(s)) for s in oracle.branch_param_shapes(di, do, r).values())

        extra = L * (4 * branch(d, d) + branch(d, 2 * h) + branch(h, d))
        pct = 100.0 * extra / base
        assert abs(pct - row["params_plus_pct"]) < 0.1, (row, pct)


# ------------------------------------------------------- finite differences --

def test_gradients_match_central_differences():
    p = _tiny()
    g = _bwd(p)

    def loss(q):
        Y, _ = _fwd(q)
        return float(np.sum(q["dy"] * Y))

    names = {"x": "dx", "W": "dW", "b": "db", "W_down": "dW_down", "M": "dM", "W_up": "dW_up",
             "omega1": "domega1", "phi1": "dphi1", "omega2": "domega2", "phi2": "dphi2"}
    for pname, gname in names.items():
        base = p[pname]
        fd = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            h = 1e-6 * max(1.0, abs(base[idx]))
            qp = dict(p)
            qp[pname] = base.copy()
            qp[pname][idx] += h
            qm = dict(p)
            qm[pname] = base.copy()
            qm[pname][idx] -= h
            fd[idx] = (loss(qp) - loss(qm)) / (2 * h)
        scale = max(1.0, float(np.max(np.abs(g[gname]))))
        assert np.max(np.abs(fd - g[gname])) <= 1e-6 * scale, gname


def test_gradients_match_torch_autograd():
    torch = pytest.importorskip("torch")
    p = _tiny(seed=11, T=9, d_in=16, d_out=24, r=8)
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
    # independent formulation: column-vector CosNet with the mixing written as
    # an explicit sum over the input rank, per token
    h = t["x"] @ t["W_down"]
    c1 = torch.cos(t["omega1"] * h + t["phi1"])
    h2 = (c1[:, :, None] * t["M"][None, :, :]).sum(dim=1)
    branch = torch.cos(t["omega2"] * h2 + t["phi2"]) @ t["W_up"]
    y = t["x"] @ t["W"] + t["b"] + branch
    (y * t["dy"]).sum().backward()
    g = _bwd(p)
    Y, _ = _fwd(p)
    np.testing.assert_allclose(Y, y.detach().numpy(), rtol=0, atol=1e-12)
    names = {"x": "dx", "W": "dW", "b": "db", "W_down": "dW_down", "M": "dM", "W_up": "dW_up",
             "omega1": "domega1", "phi1": "dphi1", "omega2": "domega2", "phi2": "dphi2"}
    for pname, gname in names.items():
        np.testing.assert_allclose(g[gname], t[pname].grad.numpy(), rtol=1e-10, atol=1e-10,
                                   err_msg=gname)


# ------------------------------------------------------------- closed forms --

def test_zero_up_projection_collapses_to_linear():
    p = _tiny(seed=5)
    p["W_up"] = np.zeros_like(p["W_up"])
    Y, _ = _fwd(p)
    np.testing.assert_array_equal(Y, p["x"] @ p["W"] + p["b"])
    g = _bwd(p)
    for k in ("dW_down", "dM", "domega1", "dphi1", "domega2", "dphi2"):
        np.testing.assert_array_equal(g[k], 0.0, err_msg=k)
    np.testing.assert_array_equal(g["dx"], p["dy"] @ p["W"].T)
    np.testing.assert_array_equal(g["dW"], p["x"].T @ p["dy"])
    np.testing.assert_allclose(g["db"], p["dy"].sum(axis=0), rtol=0, atol=1e-14)


def test_zero_second_frequency_gives_constant_branch():
    p = _tiny(seed=6)
    p["omega2"] = np.zeros_like(p["omega2"])
    Y, _ = _fwd(p)
    c = np.cos(p["phi2"])
    np.testing.assert_allclose(Y, p["x"] @ p["W"] + p["b"] + c @ p["W_up"], rtol=0, atol=1e-13)
    g = _bwd(p)
    sg = p["dy"].sum(axis=0)
    np.testing.assert_allclose(g["dW_up"], np.outer(c, sg), rtol=0, atol=1e-13)
    np.testing.assert_allclose(g["dphi2"], -np.sin(p["phi2"]) * (p["W_up"] @ sg), rtol=0, atol=1e-13)
    for k in ("dM", "domega1", "dphi1", "dW_down"):
        np.testing.assert_array_equal(g[k], 0.0, err_msg=k)
    np.testing.assert_allclose(g["dx"], p["dy"] @ p["W"].T, rtol=0, atol=1e-14)


def test_zero_first_frequency_gives_constant_branch():
    p = _tiny(seed=7)
    p["omega1"] = np.zeros_like(p["omega1"])
    Y, _ = _fwd(p)
    row = np.cos((np.cos(p["phi1"]) @ p["M"]) * p["omega2"] + p["phi2"]) @ p["W_up"]
    np.testing.assert_allclose(Y, p["x"] @ p["W"] + p["b"] + row, rtol=0, atol=1e-13)
    g = _bwd(p)
    np.testing.assert_array_equal(g["dW_down"], 0.0)
    np.testing.assert_allclose(g["dx"], p["dy"] @ p["W"].T, rtol=0, atol=1e-14)
    assert np.max(np.abs(g["domega1"])) > 1e-3


def test_zero_mixing_matrix():
    p = _tiny(seed=8)
    p["M"] = np.zeros_like(p["M"])
    Y, _ = _fwd(p)
    np.testing.assert_allclose(Y, p["x"] @ p["W"] + p["b"] + np.cos(p["phi2"]) @ p["W_up"],
                               rtol=0, atol=1e-13)
    g = _bwd(p)
    for k in ("domega1", "dphi1", "dW_down"):
        np.testing.assert_array_equal(g[k], 0.0, err_msg=k)
    assert np.max(np.abs(g["dM"])) > 1e-3
    # dM = C1^T dH2 with C1 = cos(H w1 + p1), dH2 = -sin(p2) * dC2 * w2
    C1 = np.cos((p["x"] @ p["W_down"]) * p["omega1"] + p["phi1"])
    dH2 = -np.sin(p["phi2"]) * (p["dy"] @ p["W_up"].T) * p["omega2"]
    np.testing.assert_allclose(g["dM"], C1.T @ dH2, rtol=0, atol=1e-12)


# --------------------------------------------------------------- invariants --

@pytest.mark.parametrize("k", [1, 2])
def test_evenness_of_cosine(k):
    p = _tiny(seed=9)
    q = dict(p)
    q[f"omega{k}"] = -p[f"omega{k}"]
    q[f"phi{k}"] = -p[f"phi{k}"]
    Yp, _ = _fwd(p)
    Yq, _ = _fwd(q)
    np.testing.assert_allclose(Yq, Yp, rtol=0, atol=1e-12)
    gp, gq = _bwd(p), _bwd(q)
    for n in ("dx", "dW", "dW_down", "dM", "dW_up", "db"):
        np.testing.assert_allclose(gq[n], gp[n], rtol=0, atol=1e-11, err_msg=n)
    for n in (f"domega{k}", f"dphi{k}"):
        np.testing.assert_allclose(gq[n], -gp[n], rtol=0, atol=1e-11, err_msg=n)


def test_phase_periodicity():
    p = _tiny(seed=10)
    q = dict(p, phi1=p["phi1"] + 2 * np.pi, phi2=p["phi2"] - 2 * np.pi)
    np.testing.assert_allclose(_fwd(q)[0], _fwd(p)[0], rtol=0, atol=1e-12)
    gp, gq = _bwd(p), _bwd(q)
    for n in GRADS:
        np.testing.assert_allclose(gq[n], gp[n], rtol=0, atol=1e-11, err_msg=n)


def test_down_projection_rescaling():
    p = _tiny(seed=12)
    s = np.array([0.5, 2.0, -1.5])
    q = dict(p, W_down=p["W_down"] * s, omega1=p["omega1"] / s)
    np.testing.assert_allclose(_fwd(q)[0], _fwd(p)[0], rtol=0, atol=1e-12)
    gp, gq = _bwd(p), _bwd(q)
    np.testing.assert_allclose(gq["domega1"], s * gp["domega1"], rtol=0, atol=1e-11)
    np.testing.assert_allclose(gq["dW_down"], gp["dW_down"] / s, rtol=0, atol=1e-11)
    np.testing.assert_allclose(gq["dx"], gp["dx"], rtol=0, atol=1e-11)


def test_row_permutation():
    p = _tiny(seed=13, T=11)
    perm = np.random.default_rng(0).permutation(11)
    q = dict(p, x=p["x"][perm], dy=p["dy"][perm])
    np.testing.assert_allclose(_fwd(q)[0], _fwd(p)[0][perm], rtol=0, atol=1e-13)
    gp, gq = _bwd(p), _bwd(q)
    np.testing.assert_allclose(gq["dx"], gp["dx"][perm], rtol=0, atol=1e-12)
    for n in GRADS[1:]:
        np.testing.assert_allclose(gq[n], gp[n], rtol=0, atol=1e-11, err_msg=n)


def test_branch_bound():
    p = _tiny(seed=14, T=64, d_in=32, d_out=48, r=8)
    Y, _ = _fwd(p)
    dev = np.abs(Y - p["x"] @ p["W"] - p["b"])
    assert np.all(dev <= np.abs(p["W_up"]).sum(axis=0)[None, :] + 1e-12)


def test_row_selection_matches_full():
    p = _tiny(seed=15, T=17, d_in=9, d_out=10, r=4)
    rows = np.array([0, 5, 16])
    Y, _ = _fwd(p)
    Ys, _ = _fwd(dict(p, x=p["x"][rows]))
    np.testing.assert_allclose(Ys, Y[rows], rtol=0, atol=1e-13)
    g = _bwd(p)
    gs = _bwd(p, dx_rows=rows, dW_rows=np.array([1, 8]))
    np.testing.assert_allclose(gs["dx"], g["dx"][rows], rtol=0, atol=1e-13)
    np.testing.assert_allclose(gs["dW"], g["dW"][[1, 8]], rtol=0, atol=1e-13)


# ----------------------------------------------------------- input recipe ----

def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    a = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    # exact ties: low 16 bits 0x8000 with even and odd bf16 mantissas
    ties = np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x40490000 | 0x8000], dtype=np.uint32).view(np.float32)
    a = np.concatenate([a, ties])
    mine = inp.bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(mine, ref)


def test_input_recipe_is_seeded_and_shaped():
    p = inp.draw_workload_projection("llm250m_r64", 0, T=64)
    q = inp.draw_workload_projection("llm250m_r64", 0, T=64)
    for k in p.arrays:
        np.testing.assert_array_equal(p[k], q[k])
    assert p["x"].shape == (64, 1024) and p["W"].shape == (1024, 3072)
    assert p["W_down"].shape == (1024, 64) and p["M"].shape == (64, 64)
    assert p["W_up"].shape == (64, 3072) and p["dy"].shape == (64, 3072)
    # bf16 storage tensors hold bf16-exact values
    for k in inp.STORAGE:
        np.testing.assert_array_equal(inp.round_bf16(p[k]), p[k])
    assert np.all(p["b"] == 0)
    assert 0 <= p["phi1"].min() and p["phi1"].max() < 2 * np.pi


# ------------------------------------------------- activation variants -----
# The ablation of §4.4 (Table 5): cos, tanh, LeakyReLU and GELU, as a single
# activation and as the 2-layer sandwich with M.

ACTS = sorted(oracle.ACTIVATIONS)
ONE_LAYER = [a for a in ACTS if oracle.ACTIVATIONS[a][1] == 1]


def _eval_act(v):
    if isinstance(v, list):
        return np.array([_eval_act(e) for e in v], dtype=np.float64)
    if isinstance(v, str):
        return float(eval(v, {"__builtins__": {}}, {"pi": math.pi, "sqrt": math.sqrt, "atanh": math.atanh}))
    return float(v)


def _activation_examples():
    with open(os.path.join(GOLDEN, "activation_examples.json")) as f:
        return json.load(f)["examples"]


def _fwd_a(p, act):
    return oracle.forward(p["x"], p["W"], p["b"], p["W_down"], p["omega1"], p["phi1"],
                          p["M"], p["omega2"], p["phi2"], p["W_up"], activation=act)


def _bwd_a(p, act):
    return oracle.backward(p["dy"], p["x"], p["W"], p["W_down"], p["omega1"], p["phi1"],
                           p["M"], p["omega2"], p["phi2"], p["W_up"], activation=act)


@pytest.mark.parametrize("ex", _activation_examples(), ids=lambda e: e["name"])
def test_activation_hand_examples(ex):
    """r = 1 cases whose pre-activations are chosen so that each activation's
    value and slope are known exactly (tanh(atanh t) = t, cos(pi/3) = 1/2,
    LeakyReLU(-2) = -0.02, GELU(1) = Phi(1) from a normal table)."""
    p = {k: _eval_act(v) for k, v in ex["inputs"].items()}
    Y, _ = _fwd_a(p, ex["activation"])
    g = _bwd_a(p, ex["activation"])
    for k, v in ex["expected"].items():
        got = Y if k == "y" else g[k]
        np.testing.assert_allclose(got, _eval_act(v), rtol=0, atol=1e-12, err_msg=f"{ex['name']} {k}")


@pytest.mark.parametrize("act", ACTS)
def test_activation_gradients_match_central_differences(act):
    layers = oracle.ACTIVATIONS[act][1]
    p = _tiny(seed=17, layers=layers)
    g = _bwd_a(p, act)
    two = layers >= 2

    def loss(q):
        return float(np.sum(q["dy"] * _fwd_a(q, act)[0]))

    names = {"x": "dx", "W": "dW", "b": "db", "W_down": "dW_down", "W_up": "dW_up",
             "omega1": "domega1", "phi1": "dphi1"}
    if two:
        names.update({"M": "dM", "omega2": "domega2", "phi2": "dphi2"})
    else:
        assert g["dM"] is None and g["domega2"] is None and g["dphi2"] is None
    for pname, gname in names.items():
        base = p[pname]
        fd = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            h = 1e-6 * max(1.0, abs(base[idx]))
            qp, qm = dict(p), dict(p)
            qp[pname] = base.copy()
            qm[pname] = base.copy()
            qp[pname][idx] += h
            qm[pname][idx] -= h
            fd[idx] = (loss(qp) - loss(qm)) / (2 * h)
        scale = max(1.0, float(np.max(np.abs(g[gname]))))
        assert np.max(np.abs(fd - g[gname])) <= 1e-6 * scale, (act, gname)


@pytest.mark.parametrize("act", ACTS)
def test_activation_gradients_match_torch_autograd(act):
    """An independent torch formulation (torch's own tanh, leaky_relu with
    slope 0.01, exact gelu, cos), differentiated by autograd in float64.  The
    3-layer form applies the stacked second matrix and vectors once more."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    fn = {"cos": torch.cos, "tanh": torch.tanh, "leaky_relu": lambda a: F.leaky_relu(a, 0.01),
          "gelu": lambda a: F.gelu(a)}[oracle.ACTIVATIONS[act][0]]
    layers = oracle.ACTIVATIONS[act][1]
    two = layers >= 2
    p = _tiny(seed=23, T=9, d_in=16, d_out=24, r=8, layers=layers)
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
    h = t["x"] @ t["W_down"]
    c = fn(t["omega1"] * h + t["phi1"])
    if layers == 2:
        h2 = (c[:, :, None] * t["M"][None, :, :]).sum(dim=1)
        c = fn(t["omega2"] * h2 + t["phi2"])
    elif layers == 3:
        for l in range(2):
            h2 = (c[:, :, None] * t["M"][l][None, :, :]).sum(dim=1)
            c = fn(t["omega2"][l] * h2 + t["phi2"][l])
    y = t["x"] @ t["W"] + t["b"] + c @ t["W_up"]
    (y * t["dy"]).sum().backward()
    Y, _ = _fwd_a(p, act)
    np.testing.assert_allclose(Y, y.detach().numpy(), rtol=0, atol=1e-12)
    g = _bwd_a(p, act)
    names = {"x": "dx", "W": "dW", "b": "db", "W_down": "dW_down", "W_up": "dW_up",
             "omega1": "domega1", "phi1": "dphi1"}
    if two:
        names.update({"M": "dM", "omega2": "domega2", "phi2": "dphi2"})
    for pname, gname in names.items():
        np.testing.assert_allclose(g[gname], t[pname].grad.numpy(), rtol=1e-10, atol=1e-10,
                                   err_msg=f"{act} {gname}")


def test_one_layer_ignores_the_second_layer_parameters():
    p = _tiny(seed=29)
    for act in ONE_LAYER:
        Y1, _ = _fwd_a(p, act)
        q = dict(p, M=None, omega2=None, phi2=None)
        Y2, _ = _fwd_a(q, act)
        np.testing.assert_array_equal(Y1, Y2)


def test_odd_and_even_single_activations():
    """With p1 = 0: tanh is odd, cos even; flipping the sign of W_down flips
    or keeps the branch accordingly."""
    p = _tiny(seed=31)
    p["phi1"] = np.zeros_like(p["phi1"])
    q = dict(p, W_down=-p["W_down"])
    W0 = dict(p, W_up=np.zeros_like(p["W_up"]))
    base = _fwd_a(W0, "tanh")[0]
    bt_p = _fwd_a(p, "tanh")[0] - base
    bt_q = _fwd_a(q, "tanh")[0] - base
    np.testing.assert_allclose(bt_q, -bt_p, rtol=0, atol=1e-13)
    bc_p = _fwd_a(p, "cos")[0] - base
    bc_q = _fwd_a(q, "cos")[0] - base
    np.testing.assert_allclose(bc_q, bc_p, rtol=0, atol=1e-13)


def test_leaky_relu_positive_homogeneity_and_linear_regime():
    """LeakyReLU is positively homogeneous (with p1 = 0, scaling W_down by
    c > 0 scales the 1-layer branch by c), and on positive pre-activations the
    1-layer branch is the linear map (w1 (.) H + p1) W_up."""
    p = _tiny(seed=37)
    p["phi1"] = np.zeros_like(p["phi1"])
    W0 = dict(p, W_up=np.zeros_like(p["W_up"]))
    base = _fwd_a(W0, "leaky_relu")[0]
    b1 = _fwd_a(p, "leaky_relu")[0] - base
    b3 = _fwd_a(dict(p, W_down=2.5 * p["W_down"]), "leaky_relu")[0] - base
    np.testing.assert_allclose(b3, 2.5 * b1, rtol=0, atol=1e-12)
    q = dict(p, phi1=np.full_like(p["phi1"], 50.0))   # every A1 > 0
    H = q["x"] @ q["W_down"]
    lin = (H * q["omega1"] + q["phi1"]) @ q["W_up"]
    np.testing.assert_allclose(_fwd_a(q, "leaky_relu")[0] - base, lin, rtol=0, atol=1e-10)


def test_gelu_tends_to_identity_and_zero():
    """GELU(a) -> a for large a and -> 0 for very negative a (the 1-layer
    branch becomes linear, then vanishes)."""
    p = _tiny(seed=41)
    W0 = dict(p, W_up=np.zeros_like(p["W_up"]))
    base = _fwd_a(W0, "gelu")[0]
    H = p["x"] @ p["W_down"]
    q = dict(p, phi1=np.full_like(p["phi1"], 40.0))
    np.testing.assert_allclose(_fwd_a(q, "gelu")[0] - base, (H * q["omega1"] + 40.0) @ q["W_up"],
                               rtol=0, atol=1e-10)
    q = dict(p, phi1=np.full_like(p["phi1"], -40.0))
    np.testing.assert_allclose(_fwd_a(q, "gelu")[0] - base, 0.0, rtol=0, atol=1e-12)



def test_slopes_keep_relative_accuracy_in_the_tails():
    """Where tanh saturates and in GELU's lower tail the slopes are tiny, and
    a saturated unit's gradient is that tiny number times dC.  Pinned against
    bounds from analysis rather than a second evaluation of the same formula:
    1 - tanh(a)^2 = 1 / cosh(a)^2, and the Mills-ratio bounds of the normal
    tail, phi(a) / |a| (1 - 1 / a^2) < Phi(a) < phi(a) / |a| for a < 0, which
    bracket GELU = a Phi(a) and its slope Phi(a) + a phi(a)."""
    a = np.array([2.0, 5.0, 8.0, 9.5, 12.0])
    for s in (1.0, -1.0):
        np.testing.assert_allclose(oracle.activation_slope("tanh", s * a), np.cosh(a) ** -2.0, rtol=1e-5, atol=0)
    a = np.array([-4.0, -6.0, -8.0, -10.0, -20.0])
    dens = np.exp(-0.5 * a * a) / math.sqrt(2.0 * math.pi)
    lo, hi = dens / np.abs(a) * (1.0 - 1.0 / (a * a)), dens / np.abs(a)
    cdf = oracle.activation_value("gelu", a) / a
    assert np.all(lo < cdf) and np.all(cdf < hi), (lo, cdf, hi)
    d = oracle.activation_slope("gelu", a)
    assert np.all(lo + a * dens < d) and np.all(d < hi + a * dens)

# ------------------------------------------------------------ grouped layers --

def _block_diagonal(p, G, layers=2):
    """The grouped layer's parameters as one rank-G r layer: M and W_up block
    diagonal (zeros off the blocks), everything else as is.  For the 3-layer
    form each of the two stacked mixing matrices is made block diagonal."""
    R = p["W_down"].shape[1]
    r, dg = R // G, p["W"].shape[1] // G
    L = 2 if layers == 3 else 1
    Mb = np.zeros((L, R, R))
    Ub = np.zeros((R, G * dg))
    for g in range(G):
        for l in range(L):
            Mb[l, g * r:(g + 1) * r, g * r:(g + 1) * r] = p["M"][l, g] if layers == 3 else p["M"][g]
        Ub[g * r:(g + 1) * r, g * dg:(g + 1) * dg] = p["W_up"][g * r:(g + 1) * r]
    return (Mb if layers == 3 else Mb[0]), Ub


@pytest.mark.parametrize("act", ["cosnet", "gelu_m", "tanh", "cosnet3"])
def test_grouped_layer_is_block_diagonal_single_layer(act):
    """G branches on G column blocks of one x equal one rank-G r branch whose
    M and W_up are block diagonal: same y, dx, dW, db, dW_down and vector
    gradients; dM and dW_up are the diagonal blocks of the single layer's."""
    G = 3
    layers = oracle.ACTIVATIONS[act][1]
    q = inp.draw_projection("grp", 7, 10, 3 * 6, 4, "f32", 43, bias_std=0.5, groups=G, layers=layers)
    p = {k: v.astype(np.float64) for k, v in q.arrays.items()}
    Mb, Ub = _block_diagonal(p, G, layers)
    args = (p["W_down"], p["omega1"], p["phi1"])
    Yg, Hg = oracle.forward_grouped(p["x"], p["W"], p["b"], *args, p["M"], p["omega2"], p["phi2"], p["W_up"], G,
                                    activation=act)
    Ys, Hs = oracle.forward(p["x"], p["W"], p["b"], *args, Mb, p["omega2"], p["phi2"], Ub, activation=act)
    np.testing.assert_allclose(Yg, Ys, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Hg, Hs, rtol=0, atol=1e-12)
    gg = oracle.backward_grouped(p["dy"], p["x"], p["W"], *args, p["M"], p["omega2"], p["phi2"], p["W_up"], G,
                                 activation=act)
    gs = oracle.backward(p["dy"], p["x"], p["W"], *args, Mb, p["omega2"], p["phi2"], Ub, activation=act)
    for k in ("dx", "dW", "db", "dW_down", "domega1", "dphi1", "domega2", "dphi2"):
        if gs[k] is None:
            assert gg[k] is None, k
            continue
        np.testing.assert_allclose(gg[k], gs[k], rtol=0, atol=1e-12, err_msg=k)
    r, dg = 4, 6
    for g in range(G):
        np.testing.assert_allclose(gg["dW_up"][g * r:(g + 1) * r], gs["dW_up"][g * r:(g + 1) * r, g * dg:(g + 1) * dg],
                                   rtol=0, atol=1e-12)
        if gs["dM"] is not None and layers == 3:
            for l in range(2):
                np.testing.assert_allclose(gg["dM"][l, g], gs["dM"][l, g * r:(g + 1) * r, g * r:(g + 1) * r],
                                           rtol=0, atol=1e-12)
        elif gs["dM"] is not None:
            np.testing.assert_allclose(gg["dM"][g], gs["dM"][g * r:(g + 1) * r, g * r:(g + 1) * r], rtol=0, atol=1e-12)


def test_grouped_layer_with_one_group_is_the_layer():
    q = inp.draw_projection("grp1", 6, 9, 8, 3, "f32", 47, bias_std=0.5)
    p = {k: v.astype(np.float64) for k, v in q.arrays.items()}
    a = (p["W_down"], p["omega1"], p["phi1"], p["M"], p["omega2"], p["phi2"], p["W_up"])
    Y1, _ = oracle.forward_grouped(p["x"], p["W"], p["b"], *a, 1)
    Y0, _ = oracle.forward(p["x"], p["W"], p["b"], *a)
    np.testing.assert_array_equal(Y1, Y0)
    g1 = oracle.backward_grouped(p["dy"], p["x"], p["W"], *a, 1)
    g0 = oracle.backward(p["dy"], p["x"], p["W"], *a)
    for k in GRADS:
        np.testing.assert_array_equal(g1[k], g0[k])


def test_grouped_gradients_match_central_differences():
    G = 2
    q = inp.draw_projection("grpfd", 4, 5, 2 * 3, 2, "f32", 53, bias_std=0.5, groups=G)
    p = {k: v.astype(np.float64) for k, v in q.arrays.items()}
    names = ("W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up")

    def loss(qq):
        Y, _ = oracle.forward_grouped(qq["x"], qq["W"], qq["b"], *(qq[n] for n in names), G)
        return float(np.sum(qq["dy"] * Y))

    g = oracle.backward_grouped(p["dy"], p["x"], p["W"], *(p[n] for n in names), G)
    pairs = {"x": "dx", "W": "dW", "b": "db", "W_down": "dW_down", "M": "dM", "W_up": "dW_up",
             "omega1": "domega1", "phi1": "dphi1", "omega2": "domega2", "phi2": "dphi2"}
    for pn, gn in pairs.items():
        fd = np.zeros_like(p[pn])
        for idx in np.ndindex(p[pn].shape):
            qp, qm = dict(p), dict(p)
            qp[pn] = p[pn].copy()
            qm[pn] = p[pn].copy()
            qp[pn][idx] += 1e-6
            qm[pn][idx] -= 1e-6
            fd[idx] = (loss(qp) - loss(qm)) / 2e-6
        assert np.max(np.abs(fd - g[gn])) <= 1e-6 * max(1.0, float(np.max(np.abs(g[gn])))), gn


# ---------------------------------------------------- 3-layer CosNet -------
# (Table 5, last row.)  Closed forms where the third layer degenerates.

def _fwd3(p):
    return _fwd_a(p, "cosnet3")


def _bwd3(p):
    return _bwd_a(p, "cosnet3")


@pytest.mark.parametrize("which", ["M2", "omega3"])
def test_three_layer_constant_third_input(which):
    """The second mixing matrix, or the third frequency, at zero makes the
    third layer's input constant: sigma = cos(p3) in every row, so y = x W +
    b + cos(p3) W_up and every gradient below the third layer is exactly 0
    (dM[0], dW_down, the first two frequency / phase pairs); with M' = 0 the
    third frequency gets no gradient either (H3 = 0)."""
    p = _tiny(seed=61, layers=3)
    if which == "M2":
        p["M"][1] = 0.0
    else:
        p["omega2"][1] = 0.0
    Y, _ = _fwd3(p)
    np.testing.assert_allclose(Y, p["x"] @ p["W"] + p["b"] + np.cos(p["phi2"][1]) @ p["W_up"], rtol=0, atol=1e-12)
    g = _bwd3(p)
    for k in ("dW_down", "domega1", "dphi1"):
        assert np.all(g[k] == 0), k
    assert np.all(g["dM"][0] == 0) and np.all(g["domega2"][0] == 0) and np.all(g["dphi2"][0] == 0)
    dC3 = p["dy"] @ p["W_up"].T
    np.testing.assert_allclose(g["dphi2"][1], np.sum(-np.sin(p["phi2"][1]) * dC3, axis=0), rtol=0, atol=1e-12)
    np.testing.assert_allclose(g["dx"], p["dy"] @ p["W"].T, rtol=0, atol=1e-12)
    if which == "M2":
        assert np.all(g["domega2"][1] == 0)


def test_three_layer_evenness_of_the_last_cosine():
    """(w3, p3) -> (-w3, -p3) leaves y and every gradient outside the third
    pair unchanged and flips the sign of dw3 and dp3."""
    p = _tiny(seed=67, layers=3)
    q = {k: v.copy() for k, v in p.items()}
    q["omega2"][1] *= -1.0
    q["phi2"][1] *= -1.0
    np.testing.assert_allclose(_fwd3(p)[0], _fwd3(q)[0], rtol=0, atol=1e-12)
    a, b = _bwd3(p), _bwd3(q)
    for k in ("dx", "dW", "dW_down", "dW_up", "domega1", "dphi1"):
        np.testing.assert_allclose(a[k], b[k], rtol=0, atol=1e-12, err_msg=k)
    np.testing.assert_allclose(a["dM"], b["dM"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(a["domega2"][0], b["domega2"][0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(a["domega2"][1], -b["domega2"][1], rtol=0, atol=1e-12)
    np.testing.assert_allclose(a["dphi2"][1], -b["dphi2"][1], rtol=0, atol=1e-12)


def test_three_layer_with_identity_tail_is_not_the_two_layer_form():
    """The third layer is a real extra cosine: with M' = I, w3 = 1, p3 = 0
    the 3-layer output is cos(C2), the cosine of the 2-layer output."""
    p = _tiny(seed=71, layers=3)
    r = p["M"].shape[-1]
    p["M"][1] = np.eye(r)
    p["omega2"][1] = 1.0
    p["phi2"][1] = 0.0
    q = dict(p, M=p["M"][0], omega2=p["omega2"][0], phi2=p["phi2"][0])
    H = p["x"] @ p["W_down"]
    c2 = oracle.branch_forward(H, "cosnet", q["omega1"], q["phi1"], q["M"], q["omega2"], q["phi2"])["out"]
    c3 = oracle.branch_forward(H, "cosnet3", p["omega1"], p["phi1"], p["M"], p["omega2"], p["phi2"])["out"]
    np.testing.assert_allclose(c3, np.cos(c2), rtol=0, atol=1e-12)
