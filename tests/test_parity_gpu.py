"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Metric per output tensor: max over rows of max_j |gpu - ref| / (max_j |ref| + 1e-6);
bound 2e-2 for bf16 operands with float32 accumulation, 1e-4 for float32.
Small cases are compared element by element; the full-size workloads (the
launch configuration bench.py times) on sampled rows of y, dx and dW and in
full for every rank-r gradient.
"""

import numpy as np
import pytest

from paper_2603_06492_amd import inputs as inp

from _parity import OUTPUTS, TOL, oracle_outputs, parity_report

pytestmark = pytest.mark.gpu


def _torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    return torch


def _run(p, **kw):
    from paper_2603_06492_amd.runner import DeviceProblem
    _torch_gpu()
    dp = DeviceProblem(p, canary=True, **kw)
    dp.fwd()
    dp.bwd()
    return dp


def _say(*a):
    print(*a, flush=True)


SMALL = [
    # id, T, d_in, d_out, r, dtype, bias_std
    ("bf16_ragged_r40", 300, 200, 264, 40, "bf16", 0.5),
    ("bf16_r128_multitile", 777, 512, 384, 128, "bf16", 0.5),
    ("bf16_r8_T129", 129, 64, 72, 8, "bf16", 0.5),
    ("bf16_r64_T1", 1, 256, 128, 64, "bf16", 0.5),
    ("bf16_r32_T127", 127, 128, 128, 32, "bf16", 0.0),
    ("bf16_r64_T2500_splitK", 2500, 1024, 256, 64, "bf16", 0.5),
    # narrow layers over many tokens: dW split into 16 and 8 K pieces whose
    # float32 partials the reduction sums
    ("bf16_r32_T8192_dW16", 8192, 256, 264, 32, "bf16", 0.5),
    ("bf16_r64_T4096_dW8", 4096, 256, 256, 64, "bf16", 0.5),
    ("f32_r24_T4096_dW16", 4096, 128, 136, 24, "f32", 0.5),

    ("f32_ragged_r24", 333, 96, 136, 24, "f32", 0.5),
    ("f32_r128", 200, 160, 96, 128, "f32", 0.5),
    ("f32_r72", 65, 40, 48, 72, "f32", 0.5),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_cases_elementwise(case):
    name, T, di, do, r, dt, bstd = case
    _say(f"[parity] {name}: T={T} d_in={di} d_out={do} r={r} {dt}")
    p = inp.draw_projection(name, T, di, do, r, dt, seed=101, bias_std=bstd)
    dp = _run(p)
    got = dp.outputs()
    ref = oracle_outputs(p)
    rep = parity_report(got, ref)
    _say(rep)
    assert set(rep) == set(OUTPUTS)
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert dp.guards_intact(), "write outside an output buffer"


def test_tiny_fp32_workload():
    """64 -> 64, r = 8, T = 256 in float32 (the small workload), b = 0."""
    p = inp.draw_workload_projection("tiny_fp32", 0)
    _say(f"[parity] tiny_fp32 T={p.T}")
    dp = _run(p)
    rep = parity_report(dp.outputs(), oracle_outputs(p))
    _say(rep)
    for k, e in rep.items():
        assert e <= TOL["f32"], (k, e)
    assert dp.guards_intact()


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_plain_linear_r0(dt):
    p = inp.draw_projection("plain", 333, 136, 200, 16, dt, seed=7, bias_std=0.5)
    _say(f"[parity] plain r=0 {dt}")
    dp = _run(p, branch=False)
    rep = parity_report(dp.outputs(), oracle_outputs(p, branch=False), names=("y", "dx", "dW", "db"))
    _say(rep)
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert dp.guards_intact()


def test_no_bias_no_db():
    p = inp.draw_projection("nobias", 200, 128, 192, 32, "bf16", seed=8, bias_std=0.0)
    _say("[parity] no bias, no db")
    dp = _run(p, with_bias=False, with_db=False)
    got = dp.outputs()
    assert got["db"] is None
    rep = parity_report(got, oracle_outputs(p, with_bias=False))
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)


def test_zero_tokens():
    torch = _torch_gpu()
    from paper_2603_06492_amd.runner import DeviceProblem
    p = inp.draw_projection("empty", 0, 64, 64, 16, "bf16", seed=9)
    _say("[parity] T = 0")
    dp = DeviceProblem(p)
    for g in dp.g.values():
        if g is not None and g.numel():
            g.fill_(float("nan"))
    dp.fwd()
    dp.bwd()
    torch.cuda.synchronize()
    for n, g in dp.g.items():
        if g is not None and n != "dx":
            assert bool((g == 0).all()), n


def test_zero_up_projection_matches_plain_bitwise():
    """W_up = 0: the branch is exactly zero, y and dx equal the r = 0 run bit
    for bit (up to the sign of zero) and the branch gradients are exact zeros."""
    torch = _torch_gpu()
    p = inp.draw_projection("wup0", 300, 256, 200, 64, "bf16", seed=10, bias_std=0.5)
    p.arrays["W_up"][:] = 0
    _say("[parity] W_up = 0")
    a = _run(p)
    b = _run(p, branch=False)
    torch.cuda.synchronize()
    ya, yb = a.y.float(), b.y.float()
    assert bool((ya == yb).all())
    assert bool((a.g["dx"].float() == b.g["dx"].float()).all())
    for n in ("dW_down", "dM", "domega1", "dphi1", "domega2", "dphi2"):
        assert bool((a.g[n] == 0).all()), n
    rep = parity_report(a.outputs(), oracle_outputs(p))
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)


@pytest.mark.parametrize("which", ["omega2", "omega1", "M"])
def test_degenerate_chain(which):
    """omega2 = 0 or M = 0 make the branch a constant row; omega1 = 0 makes the
    first cosine constant.  The gradients the chain rule makes exactly zero
    must come out exactly zero."""
    torch = _torch_gpu()
    p = inp.draw_projection("degen", 257, 128, 136, 32, "bf16", seed=11, bias_std=0.5)
    p.arrays[which][:] = 0
    _say(f"[parity] {which} = 0")
    dp = _run(p)
    torch.cuda.synchronize()
    zeros = {"omega2": ("dM", "domega1", "dphi1", "dW_down"),
             "omega1": ("dW_down",),
             "M": ("domega1", "dphi1", "dW_down")}[which]
    for n in zeros:
        assert bool((dp.g[n] == 0).all()), n
    got, ref = dp.outputs(), oracle_outputs(p)
    rep = parity_report(got, ref)
    _say(rep)
    # With omega1 = 0 every token has the same C2 row, so row q of dW_up is
    # C2[q] sum(dy): its row error is the relative error of one cosine value,
    # which the float32-accurate mixing product keeps small near its zeros.
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)


def test_backward_repeatable():
    """y, dx, dW and the rank gradients dW_down, dM, dW_up are reproducible
    bit for bit: no float atomics in their paths; a split product (here dW
    and the rank products, both in two pieces) sums its partials in a fixed
    order.  db and the frequency / phase gradients are summed with float
    atomics in a varying order: two runs must agree far inside the
    tolerance."""
    p = inp.draw_projection("rep", 1000, 512, 256, 64, "bf16", seed=12, bias_std=0.5)
    _say("[parity] repeatability")
    dp = _run(p)
    first = dp.outputs()
    dp.fwd()
    dp.bwd()
    second = dp.outputs()
    for k in ("y", "dx", "dW", "dW_down", "dM", "dW_up"):
        assert np.array_equal(first[k], second[k]), k
    rep = parity_report(second, first)
    for k, e in rep.items():
        assert e <= TOL["bf16"] / 10, (k, e)


def test_pending_hip_error_of_the_caller():
    """A failed HIP call of the caller's, pending in the thread's last-error
    state, is not taken for a failure of the library's launches: the calls
    succeed, and y, dx and dW are bit for bit those of a clean run."""
    import ctypes
    _torch_gpu()
    hip = ctypes.CDLL("libamdhip64.so")
    p = inp.draw_projection("pending", 300, 256, 264, 40, "bf16", seed=14, bias_std=0.5)
    _say("[parity] pending caller error")
    dp = _run(p)
    clean = dp.outputs()
    assert hip.hipGetLastError() == 0
    assert hip.hipSetDevice(ctypes.c_int(1 << 20)) != 0   # an ordinal no box has
    try:
        dp.fwd()
        dp.bwd()
    finally:
        hip.hipGetLastError()   # clear it: torch checks the state after its own launches
    again = dp.outputs()
    for k in ("y", "dx", "dW"):
        assert np.array_equal(clean[k], again[k]), k


def test_autograd_function():
    torch = _torch_gpu()
    from paper_2603_06492_amd.noble import NobleLinearFunction
    p = inp.draw_projection("autograd", 96, 64, 80, 16, "f32", seed=13, bias_std=0.5)
    _say("[parity] autograd Function")
    t = {k: torch.from_numpy(v).cuda().requires_grad_(True) for k, v in p.arrays.items() if k != "dy"}
    y = NobleLinearFunction.apply(t["x"], t["W"], t["b"], t["W_down"], t["omega1"], t["phi1"], t["M"],
                                  t["omega2"], t["phi2"], t["W_up"])
    y.backward(torch.from_numpy(p["dy"]).cuda())
    ref = oracle_outputs(p)
    got = {"y": y.detach().cpu().double().numpy()}
    names = {"x": "dx", "W": "dW", "b": "db", "W_down": "dW_down", "M": "dM", "W_up": "dW_up",
             "omega1": "domega1", "phi1": "dphi1", "omega2": "domega2", "phi2": "dphi2"}
    for k, n in names.items():
        got[n] = t[k].grad.detach().cpu().double().numpy()
    rep = parity_report(got, ref)
    for k, e in rep.items():
        assert e <= TOL["f32"], (k, e)


# ----------------------------------------------------- full-size workloads ----

FULL = [("llm250m_r64", 0), ("llm250m_r64", 1),
        ("llm1p5b_block_r128", 0), ("llm1p5b_block_r128", 1), ("llm1p5b_block_r128", 2),
        ("llm1p5b_block_r128", 3),
        ("vitb_ffn_r32", 0), ("vitb_ffn_r32", 1),
        ("llm1p5b_stack4_r128", 0), ("llm1p5b_stack4_r128", 4), ("llm1p5b_stack4_r128", 5)]


def _sample(n, extra, seed):
    base = [0, 1, 31, 32, 127, 128, 255, 256, n // 2, n - 2, n - 1]
    rng = np.random.default_rng(seed)
    return np.unique(np.clip(np.concatenate([base, rng.integers(0, n, extra)]), 0, n - 1))


@pytest.mark.parametrize("wl,idx", FULL, ids=[f"{w}-{inp.WORKLOADS[w]['projections'][i][0]}" for w, i in FULL])
def test_full_size_workloads(wl, idx):
    p = inp.draw_workload_projection(wl, idx)
    _say(f"[parity] full {p.name}: T={p.T} d_in={p.d_in} d_out={p.d_out} r={p.r}")
    rows = _sample(p.T, 24, 1)
    dw_rows = _sample(p.d_in, 8, 2)
    dp = _run(p)
    got = dp.outputs(rows=rows, dw_rows=dw_rows)
    ok = dp.guards_intact()
    del dp
    ref = oracle_outputs(p, rows=rows, dw_rows=dw_rows)
    rep = parity_report(got, ref)
    _say(rep)
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)
    assert ok


def test_buffers_past_2gib():
    """x and dx of 2.16 GB (T = 2^20 + 4133 tokens, d_in = 1024): every
    device offset past the 2^31-byte mark is formed in 64 bits before it
    reaches a 32-bit buffer offset.  x and dy repeat a seeded block of 65537
    rows (drawing 10^9 values would take minutes); 2^20 is not a multiple of
    65537, so a read wrapped by 2^31 bytes (2^20 rows) would land on a
    different row.  Rows on both sides of byte 2^31 of x and dx are compared
    with the oracle, with dW on sampled columns and the rank gradients in
    full."""
    T, di, do, r, period = (1 << 20) + 4133, 1024, 256, 64, 65537
    base = inp.draw_projection("bf16_past_2gib", period, di, do, r, "bf16", seed=131, bias_std=0.5)
    arrays = dict(base.arrays)
    for k in ("x", "dy"):
        arrays[k] = np.resize(base.arrays[k], (T, base.arrays[k].shape[1]))   # row t = block row t % period
    p = inp.Projection("bf16_past_2gib", T, di, do, r, "bf16", arrays)
    assert p.arrays["x"].size * 2 > (1 << 31)
    _say(f"[parity] past 2 GiB: T={T} d_in={di} d_out={do} r={r}")
    edge = 1 << 20
    rows = np.unique(np.concatenate([_sample(T, 16, 3), np.arange(edge - 3, edge + 3)]))
    dw_rows = _sample(di, 8, 4)
    dp = _run(p)
    got = dp.outputs(rows=rows, dw_rows=dw_rows)
    ok = dp.guards_intact()
    del dp
    ref = oracle_outputs(p, rows=rows, dw_rows=dw_rows)
    rep = parity_report(got, ref)
    _say(rep)
    assert set(rep) == set(OUTPUTS)
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)
    assert ok


WIDEST = [("bf16_max_d_in", 1 << 20, 16), ("bf16_max_d_out", 16, 1 << 20)]


@pytest.mark.parametrize("case", WIDEST, ids=[c[0] for c in WIDEST])
def test_maximum_widths(case):
    """The widest layers the ABI accepts (d = 2^20; T = 40, r = 8): K = 2^20
    in the forward GEMM or the backward's dx, 4096 tiles in the other
    products.  Element by element against the oracle by the row metric.
    dW_down = x^T dH has 2^20 rows of 40-term sums, and its worst row cancels
    to a seventh of the typical row size: one bf16 dH operand would move it
    by 2.4% of that row, the high + low pair keeps it at float32 accuracy."""
    name, di, do = case
    T, r = 40, 8
    _say(f"[parity] {name}: T={T} d_in={di} d_out={do} r={r}")
    p = inp.draw_projection(name, T, di, do, r, "bf16", seed=101, bias_std=0.5)
    dp = _run(p)
    got = dp.outputs()
    ok = dp.guards_intact()
    del dp
    ref = oracle_outputs(p)
    rep = parity_report(got, ref)
    _say(rep)
    assert set(rep) == set(OUTPUTS)
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)
    assert ok
