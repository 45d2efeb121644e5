"""noble_linear_fwd_static (the forward on the library's static device
scratch, for callers that cannot allocate) against noble_linear_fwd on the
same inputs: y and the reserve H bit for bit, on two calls in a row whose
second is smaller (the array keeps the first call's contents)."""

import numpy as np
import pytest

from paper_2603_06492_amd import inputs as inp
from paper_2603_06492_amd import noble

pytestmark = pytest.mark.gpu

CASES = [
    # id, T, d_in, d_out, r, groups, dtype, activation
    ("bf16_r128_T2500", 2500, 512, 384, 128, 1, "bf16", "cosnet"),
    ("bf16_g3_r40_T300", 300, 200, 264, 40, 3, "bf16", "gelu_m"),
    ("f32_r24_T333", 333, 96, 136, 24, 1, "f32", "cosnet"),
]


def _say(*a):
    print(*a, flush=True)


def test_static_forward_matches_forward_on_calls_in_a_row():
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    for (name, T, di, do, r, G, dt, act) in CASES:
        _say(f"[no-alloc] {name}: T={T} d_in={di} d_out={do} r={r} groups={G} {dt} {act}")
        p = inp.draw_projection(name, T, di, do, r, dt, seed=41, bias_std=0.5, groups=G)
        dp = DeviceProblem(p, canary=True, activation=act)
        dp.fwd()
        t = dp.t
        y2 = torch.full_like(dp.y, float("nan"))
        res2 = torch.zeros_like(dp.reserve)
        noble.noble_linear_fwd_static(t["x"], t["W"], t["b"], t["W_down"], t["omega1"], t["phi1"], t["M"],
                                      t["omega2"], t["phi2"], t["W_up"], y2, res2,
                                      activation=noble.activation_code(act), groups=G)
        torch.cuda.synchronize()
        view = torch.int16 if dp.y.dtype == torch.bfloat16 else torch.int32
        assert bool((dp.y.view(view) == y2.view(view)).all()), name
        nres = T * G * r * 4
        assert bool((dp.reserve[:nres] == res2[:nres]).all()), name
        assert dp.guards_intact()
        # the inference form (no reserve) gives the same y
        y3 = torch.full_like(dp.y, float("nan"))
        noble.noble_linear_fwd_static(t["x"], t["W"], t["b"], t["W_down"], t["omega1"], t["phi1"], t["M"],
                                      t["omega2"], t["phi2"], t["W_up"], y3, None,
                                      activation=noble.activation_code(act), groups=G)
        torch.cuda.synchronize()
        assert bool((dp.y.view(view) == y3.view(view)).all()), name
