"""Parity of grouped layers (several output column blocks of one x, each with
its own branch: Q, K and V) and of ranks above 128 (up to 256, two 128-rank
tiles per group) through the C ABI against the fp64 oracle.  Same metric and
bounds as test_parity_gpu.py; every output is guarded by canary bands."""

import numpy as np
import pytest

from paper_2603_06492_amd import inputs as inp

from _parity import OUTPUTS, TOL, oracle_outputs, parity_report

pytestmark = pytest.mark.gpu

CASES = [
    # id, T, d_in, d_out, r, groups, dtype
    ("bf16_g3_r40_ragged", 300, 200, 264, 40, 3, "bf16"),
    ("bf16_g3_r128_multitile", 777, 512, 384, 128, 3, "bf16"),
    ("bf16_g2_r64_T1", 1, 256, 256, 64, 2, "bf16"),
    ("bf16_g4_r16_T129", 129, 64, 96, 16, 4, "bf16"),
    ("bf16_r256", 300, 264, 200, 256, 1, "bf16"),
    ("bf16_r200_T129", 129, 128, 136, 200, 1, "bf16"),
    ("bf16_r136", 200, 128, 128, 136, 1, "bf16"),
    ("bf16_g2_r256", 257, 256, 272, 256, 2, "bf16"),
    ("f32_g2_r24", 333, 96, 144, 24, 2, "f32"),
    ("f32_g3_r8", 65, 40, 72, 8, 3, "f32"),
]


def _say(*a):
    print(*a, flush=True)


def _run(p, **kw):
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    dp = DeviceProblem(p, canary=True, **kw)
    dp.fwd()
    dp.bwd()
    return dp


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_grouped_and_wide_rank_parity(case):
    name, T, di, do, r, G, dt = case
    _say(f"[groups] {name}: T={T} d_in={di} d_out={do} r={r} groups={G} {dt}")
    p = inp.draw_projection(name, T, di, do, r, dt, seed=301, bias_std=0.5, groups=G)
    dp = _run(p)
    got = dp.outputs()
    # A single token makes row q of dW_up one C2 value times dy (and row i of
    # dM one C1 value times dH2): the row metric is then the relative error
    # of one cosine, which the float32-accurate mixing product keeps small
    # near the cosine's zeros too.
    rep = parity_report(got, oracle_outputs(p))
    _say(rep)
    assert set(rep) == set(OUTPUTS)
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert dp.guards_intact(), "write outside an output buffer"


@pytest.mark.parametrize("act", ["gelu_m", "tanh", "cos"])
def test_grouped_activation_variants(act):
    """A 3-group layer with r = 256 tiles absent (r = 40) and a 1-group r = 256
    layer, with variant activations (two-application forms compared with the
    plain oracle, as in test_activations_gpu.py)."""
    for (T, di, do, r, G) in ((300, 200, 264, 40, 3), (300, 264, 200, 256, 1)):
        _say(f"[groups] {act}: T={T} d_in={di} d_out={do} r={r} groups={G}")
        p = inp.draw_projection("grp_act", T, di, do, r, "bf16", seed=302, bias_std=0.5, groups=G)
        dp = _run(p, activation=act)
        rep = parity_report(dp.outputs(), oracle_outputs(p, activation=act))
        _say(rep)
        for k, e in rep.items():
            assert e <= TOL["bf16"], (k, e)
        assert dp.guards_intact()


def _sample(n, extra, seed):
    base = [0, 1, 31, 32, 127, 128, 255, 256, n // 2, n - 2, n - 1]
    rng = np.random.default_rng(seed)
    return np.unique(np.clip(np.concatenate([base, rng.integers(0, n, extra)]), 0, n - 1))


@pytest.mark.parametrize("shape", [
    # name, T, d_in, d_out, r, groups
    ("qkv_grouped_T32768", 32768, 2048, 6144, 128, 3),   # Q, K, V of the four-block stack, one call
    ("o_r256_T8192", 8192, 2048, 2048, 256, 1),           # the 1.5B block's O projection at r = 256
], ids=lambda s: s[0])
def test_full_size_grouped_and_r256(shape):
    name, T, di, do, r, G = shape
    p = inp.draw_projection(name, T, di, do, r, "bf16", seed=303, groups=G)
    _say(f"[groups] full {name}: T={T} d_in={di} d_out={do} r={r} groups={G}")
    rows, dw_rows = _sample(T, 24, 1), _sample(di, 8, 2)
    dp = _run(p)
    got = dp.outputs(rows=rows, dw_rows=dw_rows)
    ok = dp.guards_intact()
    del dp
    rep = parity_report(got, oracle_outputs(p, rows=rows, dw_rows=dw_rows))
    _say(rep)
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)
    assert ok


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_two_dimensional_grids(dt):
    """T = 2^21 + 4133 tokens, four groups of r = 8: the launches whose
    workgroup count grows with T pass the 65536 workgroups of one grid row
    (bf16: 65668 projection workgroups and 262664 branch workgroups; f32:
    65666 chain workgroups per group), so workgroups past the first row, and
    the surplus of the last one, are exercised.  y and dx on sampled rows
    (both ends and the first row boundaries), every weight gradient in full."""
    T, di, do, r, G = (1 << 21) + 4133, 32, 64, 8, 4
    name = f"{dt}_g4_r8_T{T}"
    _say(f"[groups] {name}: T={T} d_in={di} d_out={do} r={r} groups={G} {dt}")
    p = inp.draw_projection(name, T, di, do, r, dt, seed=305, bias_std=0.5, groups=G)
    # first tokens of the second grid row: branch (32-token blocks x G),
    # f32 chain (32-token blocks), projection (128-token blocks x G jobs)
    edges = np.array([32 * 65536 // G, 32 * 65536, 65536 % -(-T // 128) * 128])
    rows = np.unique(np.concatenate([_sample(T, 24, 5), edges - 1, edges]))
    dp = _run(p)
    got = dp.outputs(rows=rows)
    ok = dp.guards_intact()
    del dp
    rep = parity_report(got, oracle_outputs(p, rows=rows))
    _say(rep)
    assert set(rep) == set(OUTPUTS)
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert ok
