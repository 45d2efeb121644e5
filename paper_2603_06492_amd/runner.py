"""Device-resident problem holder: uploads one projection's inputs, owns the
outputs and work buffers, and calls the libnoble forward/backward through the
binding.  Used by the tests and by bench.py; it does no arithmetic itself."""

from __future__ import annotations

from typing import Dict, Optional

import numpy as np

from . import noble
from .inputs import STORAGE, Projection

GRAD_NAMES = ("dx", "dW", "db", "dW_down", "dM", "dW_up", "domega1", "dphi1", "domega2", "dphi2")
GUARD = 4096  # elements of canary before and after every output


def _torch():
    import torch
    return torch


class DeviceProblem:
    """One NOBLE linear problem resident in HBM.

    ``canary=True`` surrounds every output with guard bands filled with a NaN
    pattern, so out-of-bounds writes can be detected with ``guards_intact``.
    ``branch=False`` runs the same shapes as a plain linear (r = 0).
    ``x_from`` reads x from that problem's device tensor (the same values:
    projections that share their block's input).
    ``activation`` names the bottleneck activation (noble.ACTIVATIONS).  For a
    one-application activation, M, omega2, phi2 and their gradients are passed
    as None unless ``pass_unused`` (then the gradients must come back zero).
    """

    def __init__(self, p: Projection, device: str = "cuda", *, with_bias: bool = True,
                 with_db: bool = True, branch: bool = True, canary: bool = False,
                 inputs_from: Optional["DeviceProblem"] = None, activation: str = "cosnet",
                 pass_unused: bool = False, x_from: Optional["DeviceProblem"] = None):
        torch = _torch()
        if not torch.cuda.is_available():
            raise RuntimeError("DeviceProblem needs a GPU")
        self.p = p
        self.device = device
        self.sdt = torch.bfloat16 if p.dtype == "bf16" else torch.float32
        self.code = noble.NOBLE_BF16 if p.dtype == "bf16" else noble.NOBLE_F32
        self.r = p.r if branch else 0
        self.G = getattr(p, "groups", 1) if branch else 1
        self.canary = canary
        self.activation = activation
        self.act = noble.activation_code(activation)
        unused = () if noble.two_layers(activation) or pass_unused else ("M", "omega2", "phi2")
        self.guards = []
        self.t: Dict[str, object] = {}
        if inputs_from is not None:
            self.t.update(inputs_from.t)
        else:
            for k, v in p.device_arrays().items():
                if k == "x" and x_from is not None:
                    # the same device tensor as x_from's (a shared block input)
                    assert tuple(x_from.t["x"].shape) == v.shape
                    self.t["x"] = x_from.t["x"]
                    continue
                if k in STORAGE and p.dtype == "bf16":
                    t = torch.from_numpy(v.view(np.int16)).to(device).view(torch.bfloat16)
                else:
                    t = torch.from_numpy(v).to(device)
                self.t[k] = t.contiguous()
        if not with_bias:
            self.t["b"] = None
        if self.r == 0:
            for k in ("W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up"):
                self.t[k] = None
        for k in unused:
            self.t[k] = None
        T, di, do, r = p.T, p.d_in, p.d_out, self.r
        G = self.G
        R, dog = G * r, do // G
        f32 = torch.float32
        self.y = self._out((T, do), self.sdt)
        self.g = {
            "dx": self._out((T, di), self.sdt),
            "dW": self._out((di, do), f32),
            "db": self._out((do,), f32) if with_db else None,
        }
        if r > 0:
            mshape = (r, r) if G == 1 else (G, r, r)
            v2 = (R,)
            if noble.layers(activation) == 3:   # stacked second and third layers
                mshape, v2 = (2,) + mshape, (2, R)
            for n, s in (("dW_down", (di, R)), ("dM", mshape), ("dW_up", (R, dog)), ("domega1", (R,)),
                         ("dphi1", (R,)), ("domega2", v2), ("dphi2", v2)):
                self.g[n] = self._out(s, f32)
            for n in unused:
                self.g["d" + n] = None
        else:
            for n in ("dW_down", "dM", "dW_up", "domega1", "dphi1", "domega2", "dphi2"):
                self.g[n] = None
        res, scr = noble.noble_linear_workspace_size(T, di, do, r, self.code, self.act, G)
        self.reserve = torch.empty(max(res, 16), dtype=torch.uint8, device=device)
        self.scratch = torch.empty(max(scr, 16), dtype=torch.uint8, device=device)

    def _out(self, shape, dtype):
        torch = _torch()
        n = int(np.prod(shape))
        if not self.canary:
            return torch.empty(shape, dtype=dtype, device=self.device)
        buf = torch.empty(n + 2 * GUARD, dtype=dtype, device=self.device)
        buf.view(torch.int16 if dtype == torch.bfloat16 else torch.int32).fill_(-1)  # NaN pattern
        self.guards.append(buf)
        return buf[GUARD:GUARD + n].view(shape)

    def guards_intact(self) -> bool:
        torch = _torch()
        for buf in self.guards:
            bits = buf.view(torch.int16 if buf.dtype == torch.bfloat16 else torch.int32)
            if not (bool((bits[:GUARD] == -1).all()) and bool((bits[-GUARD:] == -1).all())):
                return False
        return True

    def fwd(self, stream=None):
        t = self.t
        noble.noble_linear_fwd(t["x"], t["W"], t["b"], t["W_down"], t["omega1"], t["phi1"], t["M"],
                               t["omega2"], t["phi2"], t["W_up"], self.y, self.reserve, self.scratch,
                               stream=stream, activation=self.act, groups=self.G)

    def bwd(self, stream=None):
        t, g = self.t, self.g
        noble.noble_linear_bwd(t["dy"], t["x"], t["W"], t["W_down"], t["omega1"], t["phi1"], t["M"],
                               t["omega2"], t["phi2"], t["W_up"], self.reserve,
                               g["dx"], g["dW"], g["db"], g["dW_down"], g["dM"], g["dW_up"],
                               g["domega1"], g["dphi1"], g["domega2"], g["dphi2"], self.scratch,
                               stream=stream, activation=self.act, groups=self.G)

    def outputs(self, rows: Optional[np.ndarray] = None, dw_rows: Optional[np.ndarray] = None):
        """Host float64 copies of y and every gradient (optionally row-sampled)."""
        torch = _torch()
        torch.cuda.synchronize()

        def host(t, sel=None):
            if t is None:
                return None
            if sel is not None:
                t = t[torch.as_tensor(sel, device=t.device)]
            return t.float().cpu().numpy().astype(np.float64)

        out = {"y": host(self.y, rows)}
        for n in GRAD_NAMES:
            sel = rows if n == "dx" else (dw_rows if n == "dW" else None)
            out[n] = host(self.g[n], sel)
        return out
