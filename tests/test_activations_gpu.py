"""Parity of the bottleneck activation variants through the C ABI against the
fp64 oracle: single cosine, tanh, LeakyReLU and GELU, each as one application
and (except cosine, whose two-application form is the CosNet covered by
test_parity_gpu.py) as two applications with the mixing matrix M, and the
3-layer CosNet (two mixing matrices; more of it in test_cosnet3_gpu.py).

Same metric and bounds as test_parity_gpu.py, against the plain oracle.  On
the bf16 path the kernels take the mixing operand (C1 in H2 = C1 M, dH2 in
dC1 = dH2 M^T) and the operands of dM as high + low bf16 pairs, so A2 is
float32-accurate: LeakyReLU's sign decision on A2 and GELU's slope, whose
relative size grows like |a| for negative a, see the same values the oracle
computes.  Every seeded LeakyReLU case keeps its pre-activations clear of the
band where float32 and float64 can disagree on the sign (kink_margin > 1).
"""

import numpy as np
import pytest

from paper_2603_06492_amd import inputs as inp
from paper_2603_06492_amd import noble

from _parity import OUTPUTS, TOL, kink_margin, oracle_outputs, parity_report

pytestmark = pytest.mark.gpu

VARIANTS = sorted(a for a in noble.ACTIVATIONS if a != "cosnet")
CASES = [
    # id, T, d_in, d_out, r, dtype, seed
    ("bf16_ragged_r40", 300, 200, 264, 40, "bf16", 204),
    ("bf16_r128_multitile", 777, 512, 384, 128, "bf16", 205),
    ("f32_ragged_r24", 333, 96, 136, 24, "f32", 204),
]
SECOND = ("dM", "domega2", "dphi2")


def _say(*a):
    print(*a, flush=True)


def _run(p, act, **kw):
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    dp = DeviceProblem(p, canary=True, activation=act, **kw)
    dp.fwd()
    dp.bwd()
    return dp


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("act", VARIANTS)
def test_activation_parity(act, case):
    name, T, di, do, r, dt, seed = case
    # LeakyReLU: the seed is stepped (deterministically) until no
    # pre-activation lies in the kink band, as in test_fuzz_gpu.py
    for attempt in range(50 if act.startswith("leaky") else 1):
        p = inp.draw_projection(name, T, di, do, r, dt, seed=seed + 1000 * attempt, bias_std=0.5,
                                layers=max(2, noble.layers(act)))
        if not act.startswith("leaky") or kink_margin(p, act) > 1.0:
            break
    else:
        pytest.fail("no draw clears the LeakyReLU kink band")
    _say(f"[activation] {act} {name}: T={T} d_in={di} d_out={do} r={r} {dt} seed={seed + 1000 * attempt}")
    dp = _run(p, act)
    got = dp.outputs()
    ref = oracle_outputs(p, activation=act)
    rep = parity_report(got, ref)
    _say(rep)
    want = set(OUTPUTS) - (set() if noble.two_layers(act) else set(SECOND))
    assert set(rep) == want
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert dp.guards_intact(), "write outside an output buffer"


@pytest.mark.parametrize("act", [a for a in VARIANTS if not noble.two_layers(a)])
def test_one_layer_ignores_and_zeroes_second_layer(act):
    """Passing M, omega2, phi2 changes nothing (bit for bit) and the given
    dM, domega2, dphi2 buffers come back exactly zero."""
    import torch
    p = inp.draw_projection("one", 257, 128, 136, 32, "bf16", seed=206, bias_std=0.5)
    _say(f"[activation] {act}: second-layer buffers")
    a = _run(p, act)
    b = _run(p, act, pass_unused=True)
    torch.cuda.synchronize()
    assert bool((a.y.view(torch.int16) == b.y.view(torch.int16)).all())
    assert bool((a.g["dx"].view(torch.int16) == b.g["dx"].view(torch.int16)).all())
    for n in ("dW", "dW_down", "dW_up"):
        assert bool((a.g[n] == b.g[n]).all()), n
    for n in SECOND:
        assert a.g[n] is None
        assert bool((b.g[n] == 0).all()), n
    assert b.guards_intact()


@pytest.mark.parametrize("act", ["gelu_m", "tanh"])
def test_activation_full_size_block(act):
    """One projection of the 1.5B block at full size (T = 8192, 2048 -> 2048,
    r = 128) with a variant activation: sampled rows of y, dx, dW, every rank
    gradient in full."""
    p = inp.draw_workload_projection("llm1p5b_block_r128", 1)
    _say(f"[activation] full {act} {p.name}: T={p.T} d_in={p.d_in} d_out={p.d_out} r={p.r}")
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, 1, 255, 256, p.T - 1], rng.integers(0, p.T, 24)]))
    dw_rows = np.unique(np.concatenate([[0, p.d_in - 1], rng.integers(0, p.d_in, 8)]))
    dp = _run(p, act)
    got = dp.outputs(rows=rows, dw_rows=dw_rows)
    ok = dp.guards_intact()
    del dp
    ref = oracle_outputs(p, rows=rows, dw_rows=dw_rows, activation=act)
    rep = parity_report(got, ref)
    _say(rep)
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)
    assert ok


SATURATED = [("tanh", 9.0), ("tanh_m", 9.0), ("gelu", -6.5), ("gelu_m", -6.5)]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("act,shift", SATURATED, ids=[a for a, _ in SATURATED])
def test_saturated_units_keep_relative_gradient_accuracy(act, shift, dt):
    """Every other rank column gets a phase that puts its unit deep in the
    flat part of tanh (|a| near 9, slope near 1e-7) or in GELU's lower tail
    (a near -6.5).  At T = 1 the phase gradient of a column is f'(A) dC of
    that one element, so it is compared element by element, relative to its
    own size: a slope taken as 1 - t^2 from a rounded tanh, or a normal
    distribution function taken as 1 + erf, loses most of its digits there
    while the row-normalised metric above does not see it.  Columns whose dC
    cancels (sum of |terms| over 1e3 times |dC|) are left out."""
    T, di, do, r = 1, 96, 160, 64
    _say(f"[saturated] {act} {dt}: T={T} d_in={di} d_out={do} r={r} shift={shift}")
    p = inp.draw_projection(f"sat_{act}", T, di, do, r, dt, seed=515, bias_std=0.5)
    two = noble.two_layers(act)
    k = "phi2" if two else "phi1"
    sat = np.arange(r) % 2 == 0
    sign = np.where(np.arange(r) % 4 == 0, 1.0, -1.0) if act.startswith("tanh") else 1.0
    p.arrays[k] = np.where(sat, sign * shift, p.arrays[k]).astype(np.float32)
    ref = oracle_outputs(p, activation=act)
    got = _run(p, act).outputs()
    a = {n: np.asarray(v, dtype=np.float64) for n, v in p.arrays.items() if v is not None}
    terms = np.abs(a["dy"][0])[None, :] * np.abs(a["W_up"])
    dC = a["W_up"] @ a["dy"][0]
    keep = sat & (terms.sum(axis=1) < 1e3 * np.abs(dC))
    assert keep.sum() >= r // 4
    want, have = ref["d" + k][keep], np.asarray(got["d" + k], dtype=np.float64)[keep]
    rel = np.abs(have - want) / np.abs(want)
    _say(f"  {keep.sum()} saturated columns, |slope dC| from {np.abs(want).min():.2e}, max rel err {rel.max():.2e}")
    assert np.all(np.abs(want) > 0)
    assert rel.max() <= {"bf16": 1e-2, "f32": 1e-4}[dt], rel.max()
