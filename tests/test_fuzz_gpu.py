"""Seeded random shapes through the C ABI against the fp64 oracle: token
counts from 1 to 700, widths that are any multiple of 8, ranks up to 256
(bf16) / 128 (f32 and the 3-layer CosNet), 1 to 4 groups, every activation,
both storage types.

Every case is compared with the plain oracle.  A LeakyReLU case is redrawn
(deterministically) until no pre-activation lies in the band where float32
and float64 can take different sides of the kink.

FIXED holds cases of a wider one-off sweep that came nearest the bound
before the mixing and gradient operands became high + low bf16 pairs (a
4-group tanh_m layer over 256 tokens, whose dW_down rows cancel), and the
single-token float32 case of test_f32_single_token_conditioning."""

import numpy as np
import pytest

from paper_2603_06492_amd import inputs as inp
from paper_2603_06492_amd import noble

from _parity import OUTPUTS, TOL, kink_margin, oracle_outputs, parity_report

pytestmark = pytest.mark.gpu


def _cases(n=24, seed=2026, acts=None, rmax_bf16=256, tag=""):
    rng = np.random.default_rng(seed)
    acts = sorted(a for a in noble.ACTIVATIONS if a != "cosnet3") if acts is None else acts
    out = []
    for i in range(n):
        dt = "bf16" if i % 4 else "f32"
        G = int(rng.choice([1, 1, 2, 3, 4]))
        r = 8 * int(rng.integers(1, (rmax_bf16 // 8 if dt == "bf16" else 16) + 1))
        T = int(rng.choice([1, 2, 31, 33, 64, 127, 129, 255, 300, 511, 700]))
        d_in = 8 * int(rng.integers(1, 65))
        d_out = 8 * G * int(rng.integers(1, 65 // G + 1))
        act = acts[i % len(acts)]
        out.append((f"c{tag}{i}_{dt}_T{T}_{d_in}x{d_out}_r{r}_g{G}_{act}", T, d_in, d_out, r, G, dt, act,
                    500 + i))
    return out


FIXED = [
    ("fixed_bf16_T256_192x160_r8_g4_tanh_m", 256, 192, 160, 8, 4, "bf16", "tanh_m", 749),
    ("fixed_bf16_T256_96x128_r16_g4_tanh_m", 256, 96, 128, 16, 4, "bf16", "tanh_m", 727),
]
# the 3-layer CosNet (r <= 128 on both paths) over shapes of its own
CASES = _cases() + _cases(8, 2027, ["cosnet3"], 128, "l3_") + FIXED
# A single float32 token whose dW_up row is the relative error of one tanh
# value near zero: plain float32 evaluation misses the bound there
# (tests/test_conditioning.py), so the row metric is expected to fail.
COND = ("cond_f32_T1_40x352_r64_g4_tanh", 1, 40, 352, 64, 4, "f32", "tanh", 20166)
CASES.append(pytest.param(COND, marks=pytest.mark.xfail(
    reason="float32 conditioning: a float32 evaluation of the layer misses the 1e-4 row bound on this "
           "single-token case (tests/test_conditioning.py)", strict=False)))


def _case_id(c):
    return (c.values[0] if hasattr(c, "values") else c)[0]


@pytest.mark.parametrize("case", CASES, ids=[_case_id(c) for c in CASES])
def test_fuzz_parity(case):
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    name, T, d_in, d_out, r, G, dt, act, seed = case
    for attempt in range(50):
        p = inp.draw_projection(name, T, d_in, d_out, r, dt, seed=seed + 1000 * attempt, bias_std=0.5, groups=G,
                                layers=max(2, noble.layers(act)))
        if not act.startswith("leaky") or kink_margin(p, act) > 1.0:
            break
    else:
        pytest.fail("no draw clears the LeakyReLU kink band")
    print(f"[fuzz] {name} seed={seed + 1000 * attempt}", flush=True)
    dp = DeviceProblem(p, canary=True, activation=act)
    dp.fwd()
    dp.bwd()
    got = dp.outputs()
    rep = parity_report(got, oracle_outputs(p, activation=act))
    print(rep, flush=True)
    second = {"dM", "domega2", "dphi2"}
    assert set(rep) == set(OUTPUTS) - (set() if noble.two_layers(act) else second)
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert dp.guards_intact(), "write outside an output buffer"
