"""Seeded random shapes through the C ABI against the fp64 oracle: token
counts from 1 to 700, widths that are any multiple of 8, ranks up to 256
(bf16) / 128 (f32), 1 to 4 groups, every activation, both storage types.

The comparison follows the readings the targeted tests use: bf16
two-application forms and single-token bf16 cases are compared with the
oracle that rounds the mixing operand C1 to bf16 as the kernels do, and a
LeakyReLU case is redrawn (deterministically) until no pre-activation lies
in the band where float32 and float64 can take different sides of the
kink."""

import numpy as np
import pytest

from paper_2603_06492_amd import inputs as inp
from paper_2603_06492_amd import noble

from _parity import OUTPUTS, TOL, kink_margin, oracle_outputs, parity_report, round_bf16_f64

pytestmark = pytest.mark.gpu


def _cases(n=24, seed=2026):
    rng = np.random.default_rng(seed)
    acts = sorted(noble.ACTIVATIONS)
    out = []
    for i in range(n):
        dt = "bf16" if i % 4 else "f32"
        G = int(rng.choice([1, 1, 2, 3, 4]))
        r = 8 * int(rng.integers(1, (32 if dt == "bf16" else 16) + 1))
        T = int(rng.choice([1, 2, 31, 33, 64, 127, 129, 255, 300, 511, 700]))
        d_in = 8 * int(rng.integers(1, 65))
        d_out = 8 * G * int(rng.integers(1, 65 // G + 1))
        act = acts[i % len(acts)]
        out.append((f"c{i}_{dt}_T{T}_{d_in}x{d_out}_r{r}_g{G}_{act}", T, d_in, d_out, r, G, dt, act, 500 + i))
    return out


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fuzz_parity(case):
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    name, T, d_in, d_out, r, G, dt, act, seed = case
    mix = round_bf16_f64 if dt == "bf16" and (noble.two_layers(act) or T == 1) else None
    for attempt in range(50):
        p = inp.draw_projection(name, T, d_in, d_out, r, dt, seed=seed + 1000 * attempt, bias_std=0.5, groups=G)
        if not act.startswith("leaky") or kink_margin(p, act, mix) > 1.0:
            break
    else:
        pytest.fail("no draw clears the LeakyReLU kink band")
    print(f"[fuzz] {name} seed={seed + 1000 * attempt}", flush=True)
    dp = DeviceProblem(p, canary=True, activation=act)
    dp.fwd()
    dp.bwd()
    got = dp.outputs()
    rep = parity_report(got, oracle_outputs(p, activation=act, mix_round=mix))
    print(rep, flush=True)
    second = {"dM", "domega2", "dphi2"}
    assert set(rep) == set(OUTPUTS) - (set() if noble.two_layers(act) else second)
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert dp.guards_intact(), "write outside an output buffer"
