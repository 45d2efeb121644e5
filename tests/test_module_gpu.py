"""noble.NobleLinear, the torch.nn.Module around the C ABI: its parameters
start at the recipe's documented draws, its forward / backward through the
autograd Function match the oracle for inputs with leading batch dimensions,
its optimizer groups carry the recipe's multipliers, and a few SGD steps with
them reduce a loss."""

import numpy as np
import pytest

import oracle
from oracle import recipe as rec
from paper_2603_06492_amd import noble

from _parity import TOL, parity_report

pytestmark = pytest.mark.gpu

NAMES = ("W", "b", "W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up")


def _host(t):
    return None if t is None else t.detach().float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("act,G,r", [("cosnet", 1, 40), ("gelu", 1, 40), ("cosnet", 3, 16), ("cosnet", 1, 0)])
def test_module_matches_oracle(act, G, r):
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    d_in, d_out = 200, 264
    print(f"[module] {act} groups={G} r={r}", flush=True)
    m = noble.NobleLinear(d_in, d_out, r, activation=act, groups=G, seed=11)
    torch.cuda.synchronize()
    # initial values: the recipe's draws (storage tensors rounded to bf16)
    want = rec.init_values(d_in, d_out, r, 11, dtype="bf16", groups=G)
    for n in NAMES:
        t = getattr(m, n, None)
        if t is None or n not in want:
            continue
        got = t.detach().float().cpu().numpy()
        close = np.isclose(got, want[n], rtol=2 ** -7, atol=0)   # at most one bf16 step apart
        assert close.all() and (got != want[n]).sum() <= 4, n
    # forward / backward with leading dimensions [2, 75, d_in]
    g = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randn(2, 75, d_in, device="cuda", generator=g).to(torch.bfloat16).requires_grad_(True)
    dy = torch.randn(2, 75, d_out, device="cuda", generator=g).to(torch.bfloat16)
    # a non-zero W_up so that the branch is visible (the init's alpha = 0.01 is tiny)
    if r > 0:
        with torch.no_grad():
            m.W_up.copy_(torch.randn(m.W_up.shape, device="cuda", generator=g) / np.sqrt(r))
    y = m(x)
    y.backward(dy)
    torch.cuda.synchronize()
    p = {n: _host(getattr(m, n, None)) for n in NAMES}
    X = _host(x).reshape(-1, d_in)
    DY = _host(dy).reshape(-1, d_out)
    if r == 0:
        Y = X @ p["W"] + p["b"]
        ref = {"y": Y, "dx": DY @ p["W"].T, "dW": X.T @ DY, "db": DY.sum(0)}
    else:
        args = (p["W_down"], p["omega1"], p["phi1"], p["M"], p["omega2"], p["phi2"], p["W_up"])
        if G > 1:
            Y, _ = oracle.forward_grouped(X, p["W"], p["b"], *args, G, activation=act)
            ref = oracle.backward_grouped(DY, X, p["W"], *args, G, activation=act)
        else:
            Y, _ = oracle.forward(X, p["W"], p["b"], *args, activation=act)
            ref = oracle.backward(DY, X, p["W"], *args, activation=act)
        ref["y"] = Y
    got = {"y": _host(y).reshape(-1, d_out), "dx": _host(x.grad).reshape(-1, d_in)}
    for n, gn in (("W", "dW"), ("b", "db"), ("W_down", "dW_down"), ("M", "dM"), ("W_up", "dW_up"),
                  ("omega1", "domega1"), ("phi1", "dphi1"), ("omega2", "domega2"), ("phi2", "dphi2")):
        t = getattr(m, n, None)
        if t is not None and t.grad is not None:
            got[gn] = _host(t.grad)
    rep = parity_report(got, ref)
    print(rep, flush=True)
    assert {"y", "dx", "dW", "db"} <= set(rep)
    for k, e in rep.items():
        # bf16 parameter gradients are rounded to bf16 by the module
        assert e <= TOL["bf16"], (k, e)


@pytest.mark.parametrize("act,G,r", [("cosnet", 1, 40), ("tanh", 2, 24), ("cosnet", 1, 0)])
def test_module_inference_forward(act, G, r):
    """Under no_grad (or with nothing requiring a gradient) the module runs
    the forward without the reserve: y is bit for bit the y of the forward
    that records the graph."""
    import torch
    print(f"[module] inference {act} groups={G} r={r}", flush=True)
    m = noble.NobleLinear(136, 144, r, activation=act, groups=G, seed=13)
    g = torch.Generator(device="cuda").manual_seed(7)
    if r > 0:
        with torch.no_grad():
            m.W_up.copy_(torch.randn(m.W_up.shape, device="cuda", generator=g) / np.sqrt(r))
    x = torch.randn(3, 41, 136, device="cuda", generator=g).to(torch.bfloat16)
    y_grad = m(x)
    assert y_grad.requires_grad
    with torch.no_grad():
        y_nograd = m(x)
    m.requires_grad_(False)
    y_frozen = m(x)
    torch.cuda.synchronize()
    assert not y_nograd.requires_grad and not y_frozen.requires_grad
    assert y_nograd.shape == (3, 41, 144)
    for y in (y_nograd, y_frozen):
        assert bool((y.view(torch.int16) == y_grad.detach().view(torch.int16)).all())


def test_module_param_groups_and_training_steps():
    import torch
    d_in, d_out, r = 256, 256, 32
    m = noble.NobleLinear(d_in, d_out, r, seed=2, dtype=torch.float32)
    groups = m.param_groups(1e-2)
    lr = {g["name"]: g["lr"] for g in groups}
    mult = rec.lr_multipliers(d_in, d_out, r)
    for k in ("W", "b", "W_down", "W_up", "M", "omega", "phi"):
        assert lr[k] == pytest.approx(1e-2 * mult[k], rel=1e-12), k
    opt = torch.optim.SGD(groups, lr=1e-2)
    g = torch.Generator(device="cuda").manual_seed(9)
    x = torch.randn(512, d_in, device="cuda", generator=g)
    target = torch.randn(512, d_out, device="cuda", generator=g)
    losses = []
    for _ in range(20):
        opt.zero_grad()
        loss = ((m(x) - target) ** 2).mean()
        loss.backward()
        opt.step()
        losses.append(float(loss.detach()))
    print("[module] losses", losses[0], losses[-1], flush=True)
    assert np.isfinite(losses).all() and losses[-1] < losses[0]
