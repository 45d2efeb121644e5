"""The 3-layer CosNet (last row of Table 5) through the C ABI against the fp64
oracle: grouped layers, a full-size projection of the 1.5B block with sampled
rows, T = 0, the device initialisation of its stacked parameters, and the
autograd module.  Same metric and bounds as test_parity_gpu.py.

The stacked layout: M [2, (G,) r, r] holds the two mixing matrices and
omega2, phi2 [2, G r] the second and third layers' frequency / phase, and so
do the gradients dM, domega2, dphi2."""

import numpy as np
import pytest

from oracle import recipe as rec
from paper_2603_06492_amd import inputs as inp
from paper_2603_06492_amd import noble

from _parity import TOL, oracle_outputs, parity_report

pytestmark = pytest.mark.gpu

ACT = "cosnet3"


def _say(*a):
    print(*a, flush=True)


def _run(p, **kw):
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    dp = DeviceProblem(p, canary=True, activation=ACT, **kw)
    dp.fwd()
    dp.bwd()
    return dp


GROUPED = [
    # id, T, d_in, d_out, r, G, dtype, seed
    ("bf16_G3_r40", 300, 200, 264, 40, 3, "bf16", 301),
    ("bf16_G2_r128", 515, 256, 512, 128, 2, "bf16", 302),
    ("f32_G4_r16", 129, 64, 256, 16, 4, "f32", 303),
]


@pytest.mark.parametrize("case", GROUPED, ids=[c[0] for c in GROUPED])
def test_cosnet3_grouped_parity(case):
    name, T, di, do, r, G, dt, seed = case
    _say(f"[cosnet3] grouped {name}: T={T} d_in={di} d_out={do} r={r} G={G} {dt} seed={seed}")
    p = inp.draw_projection(name, T, di, do, r, dt, seed=seed, bias_std=0.5, groups=G, layers=3)
    dp = _run(p)
    got = dp.outputs()
    ref = oracle_outputs(p, activation=ACT)
    rep = parity_report(got, ref)
    _say(rep)
    assert got["dM"].shape == (2, G, r, r) and got["domega2"].shape == (2, G * r)
    for k, e in rep.items():
        assert e <= TOL[dt], (k, e)
    assert dp.guards_intact(), "write outside an output buffer"


def test_cosnet3_full_size_projection():
    """The square attention projection of the 1.5B block at full size
    (T = 8192, 2048 -> 2048, r = 128): sampled rows of y, dx and dW, every
    rank gradient in full."""
    p = inp.draw_workload_projection("llm1p5b_block_r128", 1, layers=3)
    _say(f"[cosnet3] full {p.name}: T={p.T} d_in={p.d_in} d_out={p.d_out} r={p.r}")
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([[0, 1, 255, 256, p.T - 1], rng.integers(0, p.T, 24)]))
    dw_rows = np.unique(np.concatenate([[0, p.d_in - 1], rng.integers(0, p.d_in, 8)]))
    dp = _run(p)
    got = dp.outputs(rows=rows, dw_rows=dw_rows)
    ok = dp.guards_intact()
    del dp
    ref = oracle_outputs(p, rows=rows, dw_rows=dw_rows, activation=ACT)
    rep = parity_report(got, ref)
    _say(rep)
    for k, e in rep.items():
        assert e <= TOL["bf16"], (k, e)
    assert ok


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_cosnet3_no_tokens_zeroes_gradients(dt):
    import torch
    p = inp.draw_projection("empty", 0, 64, 128, 16, dt, seed=304, layers=3)
    _say(f"[cosnet3] T=0 {dt}")
    from paper_2603_06492_amd.runner import DeviceProblem
    dp = DeviceProblem(p, canary=True, activation=ACT)
    for g in dp.g.values():
        if g is not None and g.dtype == torch.float32:
            g.fill_(float("nan"))
    dp.fwd()
    dp.bwd()
    torch.cuda.synchronize()
    for n in ("dW", "db", "dW_down", "dM", "dW_up", "domega1", "dphi1", "domega2", "dphi2"):
        assert bool((dp.g[n] == 0).all()), n
    assert dp.g["dM"].shape == (2, 16, 16) and dp.g["dphi2"].shape == (2, 16)
    assert dp.guards_intact()


@pytest.mark.parametrize("G", [1, 3])
def test_cosnet3_init_params_match_cpu_draws(G):
    """noble_init_params fills the stacked M and omega2 / phi2 as the
    continuation of their streams (oracle.recipe.init_values, layers = 3)."""
    import torch
    d_in, d_out, r = 200, 264, 40
    sd, f32 = torch.bfloat16, torch.float32
    R = G * r
    M = (2, r, r) if G == 1 else (2, G, r, r)
    shapes = dict(W=((d_in, d_out), sd), b=((d_out,), f32), W_down=((d_in, R), sd), omega1=((R,), f32),
                  phi1=((R,), f32), M=(M, sd), omega2=((2, R), f32), phi2=((2, R), f32),
                  W_up=((R, d_out // G), sd))
    _say(f"[cosnet3] init G={G}")
    t = {k: torch.full(s, float("nan"), dtype=ty, device="cuda") for k, (s, ty) in shapes.items()}
    names = ("W", "b", "W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up")
    noble.noble_init_params(*(t[k] for k in names), seed=77, groups=G, activation=ACT)
    torch.cuda.synchronize()
    want = rec.init_values(d_in, d_out, r, 77, dtype="bf16", groups=G, layers=3)
    for k in names:
        got = t[k].float().cpu().numpy()
        w = want[k]
        assert got.shape == w.shape, k
        diff = got != w
        if diff.any():
            ulp = np.spacing(np.abs(w[diff]).astype(np.float32)) * (2 ** 16 if k in ("W", "W_down", "M", "W_up")
                                                                     else 1)
            assert np.all(np.abs(got[diff] - w[diff]) <= ulp), k
            assert diff.sum() <= 4, (k, int(diff.sum()))


def test_cosnet3_module_gradients():
    """NobleLinear(activation="cosnet3"): autograd through the library gives
    the oracle's gradients for the module's own initialised parameters."""
    import torch
    from paper_2603_06492_amd.noble import NobleLinear
    _say("[cosnet3] module")
    T, di, do, r = 200, 128, 192, 32
    m = NobleLinear(di, do, r, dtype=torch.float32, activation=ACT, seed=5)
    # a visible branch: W_up's init scale is small by design
    with torch.no_grad():
        m.W_up.normal_(0.0, 0.2)
        m.b.normal_(0.0, 0.5)
    assert m.M.shape == (2, r, r) and m.omega2.shape == (2, r)
    g = torch.Generator().manual_seed(11)
    x = torch.randn(T, di, generator=g).cuda().requires_grad_(True)
    dy = torch.randn(T, do, generator=g).cuda()
    y = m(x)
    y.backward(dy)
    torch.cuda.synchronize()

    class P:
        pass

    p = P()
    p.d_in, p.d_out, p.r, p.groups = di, do, r, 1
    arr = {k: getattr(m, k).detach().cpu().numpy() for k in
           ("W", "b", "W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up")}
    arr["x"] = x.detach().cpu().numpy()
    arr["dy"] = dy.cpu().numpy()
    p.arrays = arr
    ref = oracle_outputs(p, activation=ACT)
    got = {"y": y.detach().cpu().numpy(), "dx": x.grad.cpu().numpy()}
    for k in ("W", "b", "W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up"):
        gk = {"omega1": "domega1", "phi1": "dphi1", "omega2": "domega2", "phi2": "dphi2"}.get(k, "d" + k)
        got[gk] = getattr(m, k).grad.cpu().numpy()
    rep = parity_report(got, ref)
    _say(rep)
    assert len(rep) == 11
    for k, e in rep.items():
        assert e <= TOL["f32"], (k, e)
