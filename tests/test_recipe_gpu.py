"""The recipe's device fill and the inference-only forward on the GPU, through
the C ABI: noble_init_params against the CPU statement of the same draws
(oracle/recipe.py), and a forward with a NULL reserve against the normal one."""

import numpy as np
import pytest

from oracle import recipe as rec
from paper_2603_06492_amd import inputs as inp
from paper_2603_06492_amd import noble

pytestmark = pytest.mark.gpu

NAMES = ("W", "b", "W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up")


def _say(*a):
    print(*a, flush=True)


def _alloc(d_in, d_out, r, dt):
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    sd = torch.bfloat16 if dt == "bf16" else torch.float32
    f32 = torch.float32
    shapes = dict(W=((d_in, d_out), sd), b=((d_out,), f32), W_down=((d_in, r), sd), omega1=((r,), f32),
                  phi1=((r,), f32), M=((r, r), sd), omega2=((r,), f32), phi2=((r,), f32), W_up=((r, d_out), sd))
    return {k: torch.full(s, float("nan"), dtype=t, device="cuda") for k, (s, t) in shapes.items()}


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("shape", [(200, 264, 40), (2048, 2048, 128)])
def test_init_params_match_cpu_draws(dt, shape):
    """Every value equals the CPU statement of the draw (Philox4x32-10 words,
    the documented uniform / Box-Muller maps in double, rounding to float32
    and bf16); at most a handful may differ by one unit in the last place
    where the device and host double-precision log / cos land on opposite
    sides of a rounding boundary."""
    import torch
    d_in, d_out, r = shape
    seed = 0x1234_5678_9ABC
    _say(f"[recipe] init {dt} d_in={d_in} d_out={d_out} r={r}")
    t = _alloc(d_in, d_out, r, dt)
    noble.noble_init_params(*(t[k] for k in NAMES), seed=seed)
    torch.cuda.synchronize()
    want = rec.init_values(d_in, d_out, r, seed, dtype=dt)
    for k in NAMES:
        got = t[k].float().cpu().numpy()
        w = want[k]
        assert got.shape == w.shape, k
        diff = got != w
        if diff.any():
            ulp = np.spacing(np.abs(w[diff]).astype(np.float32)) * (2 ** 16 if dt == "bf16" and k in
                                                                      ("W", "W_down", "M", "W_up") else 1)
            assert np.all(np.abs(got[diff] - w[diff]) <= ulp), k
            assert diff.sum() <= 4, (k, int(diff.sum()))


def test_init_params_reproducible_and_seeded():
    import torch
    a, b = _alloc(256, 128, 16, "bf16"), _alloc(256, 128, 16, "bf16")
    c = _alloc(256, 128, 16, "bf16")
    noble.noble_init_params(*(a[k] for k in NAMES), seed=7)
    noble.noble_init_params(*(b[k] for k in NAMES), seed=7)
    noble.noble_init_params(*(c[k] for k in NAMES), seed=8)
    torch.cuda.synchronize()
    for k in NAMES:
        assert bool((a[k] == b[k]).all()), k
    for k in ("W", "W_down", "M", "W_up", "omega1", "phi1"):
        assert not bool((a[k] == c[k]).all()), k


def test_init_params_skips_null_tensors():
    import torch
    t = _alloc(64, 64, 8, "f32")
    noble.noble_init_params(t["W"], None, None, None, None, None, None, None, t["W_up"], seed=1)
    torch.cuda.synchronize()
    assert not bool(torch.isnan(t["W"]).any()) and not bool(torch.isnan(t["W_up"]).any())
    for k in ("b", "W_down", "omega1", "phi1", "M", "omega2", "phi2"):
        assert bool(torch.isnan(t[k]).all()), k


@pytest.mark.parametrize("dt,act", [("bf16", "cosnet"), ("bf16", "gelu"), ("f32", "cosnet")])
def test_inference_forward_without_reserve(dt, act):
    """reserve = NULL: y is bit for bit the y of the forward that keeps H."""
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    p = inp.draw_projection("infer", 300, 200, 264, 40, dt, seed=31, bias_std=0.5)
    _say(f"[recipe] inference forward {dt} {act}")
    dp = DeviceProblem(p, activation=act)
    dp.fwd()
    y_train = dp.y.clone()
    dp.y.fill_(float("nan"))
    t = dp.t
    noble.noble_linear_fwd(t["x"], t["W"], t["b"], t["W_down"], t["omega1"], t["phi1"], t["M"], t["omega2"],
                           t["phi2"], t["W_up"], dp.y, None, dp.scratch, activation=dp.act)
    torch.cuda.synchronize()
    iv = torch.int16 if dt == "bf16" else torch.int32
    assert bool((dp.y.view(iv) == y_train.view(iv)).all())
