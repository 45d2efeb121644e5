"""Plain fp64 CPU oracle for the NOBLE-CosNet augmented linear layer.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The HIP
product path never does, and this module imports nothing from it.

What it computes (the paper, arXiv 2603.06492):

* Forward, §3.1 Eq. (1): ``f(x) = x W + b + sigma(x W_down) W_up`` with
  ``W: [d_in, d_out]``, ``W_down: [d_in, r]``, ``W_up: [r, d_out]``; rows of
  ``x`` are tokens (the paper writes ``x W``, a row-vector convention).
* sigma, §3.2 Eq. (2) and its restatement in App. A ("CosNet Architecture"):
  ``h1 = cos(w1 * h + p1)``, ``h2 = mix(h1, M)``, ``sigma(h) = cos(w2 * h2 + p2)``
  with four separate length-r vectors (frequency and phase per dimension,
  §3.2) and an r x r mixing matrix ``M``.
* Backward: the paper prints no gradient formulas.  They follow from the
  forward by the chain rule, using d cos(u)/du = -sin(u) (the derivative the
  paper names in §6, "Why Cosine Activations?").

Readings where the paper is silent or ambiguous:

* Orientation of M.  Eq. (2) and App. A write ``M h1`` for a column vector.  In
  the row-batch form used here that is ``C1 @ M.T``; this oracle instead uses
  ``H2 = C1 @ M`` with M stored ``[r_in, r_out]``, the ``(cos(...)) M`` form
  of the row-batch layer statement.  Both parametrise the same function
  class (M.T is just another learned matrix).  A hand-worked example with a
  non-symmetric M (tests/golden/hand_examples.json) pins the choice.
* No branch scale (Eq. (1) has none; alpha in §3.3 is an init scale only).
* ``b`` is optional (``None`` means no bias, ``db`` is then still returned as
  the column sum of ``dy``, i.e. the gradient a bias would receive).

Everything is evaluated in float64 on whatever values it is handed; callers pass
the exact values the device sees (bf16-rounded storage tensors upcast to
float64).  There is no blocking, fusion or reordering beyond the equations.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "cosnet_forward",
    "cosnet_backward",
    "forward",
    "backward",
    "branch_param_shapes",
]


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def cosnet_forward(H, omega1, phi1, M, omega2, phi2):
    """sigma of §3.2 Eq. (2) (App. A), applied to every row of ``H: [T, r]``.

    Returns the intermediates by name: A1, C1, H2, A2, C2 (all ``[T, r]``).
    """
    H = _f64(H)
    A1 = H * _f64(omega1) + _f64(phi1)          # w1 (.) h + p1
    C1 = np.cos(A1)                              # h1 = cos(.)
    H2 = C1 @ _f64(M)                            # h2 = h1 mixed by M (row form)
    A2 = H2 * _f64(omega2) + _f64(phi2)          # w2 (.) h2 + p2
    C2 = np.cos(A2)                              # sigma(h) = cos(.)
    return {"A1": A1, "C1": C1, "H2": H2, "A2": A2, "C2": C2}


def forward(x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up):
    """Eq. (1) with sigma = CosNet.  Rows of ``x`` are independent tokens, so
    passing a subset of rows of ``x`` yields exactly those rows of ``Y``.

    Returns ``(Y, H)`` where ``H = x @ W_down`` is the bottleneck input.
    """
    x = _f64(x)
    H = x @ _f64(W_down)
    C2 = cosnet_forward(H, omega1, phi1, M, omega2, phi2)["C2"]
    Y = x @ _f64(W) + C2 @ _f64(W_up)
    if b is not None:
        Y = Y + _f64(b)
    return Y, H


def cosnet_backward(dC2, H, omega1, phi1, M, omega2, phi2):
    """Chain rule through sigma for ``L`` with ``dL/dC2 = dC2`` (rows = tokens).

    Recomputes the forward chain from ``H``.  Returns dH, dM, domega1, dphi1,
    domega2, dphi2 and the recomputed C2.
    """
    dC2 = _f64(dC2)
    H = _f64(H)
    w1, w2 = _f64(omega1), _f64(omega2)
    f = cosnet_forward(H, omega1, phi1, M, omega2, phi2)
    dA2 = -np.sin(f["A2"]) * dC2                 # d cos(A2) = -sin(A2) dA2
    domega2 = np.sum(dA2 * f["H2"], axis=0)      # A2 = w2 (.) H2 + p2
    dphi2 = np.sum(dA2, axis=0)
    dH2 = dA2 * w2
    dM = f["C1"].T @ dH2                         # H2 = C1 @ M
    dC1 = dH2 @ _f64(M).T
    dA1 = -np.sin(f["A1"]) * dC1                 # C1 = cos(A1)
    domega1 = np.sum(dA1 * H, axis=0)            # A1 = w1 (.) H + p1
    dphi1 = np.sum(dA1, axis=0)
    dH = dA1 * w1
    return {
        "dH": dH,
        "dM": dM,
        "domega1": domega1,
        "dphi1": dphi1,
        "domega2": domega2,
        "dphi2": dphi2,
        "C2": f["C2"],
    }


def backward(dy, x, W, W_down, omega1, phi1, M, omega2, phi2, W_up,
             dx_rows=None, dW_rows=None):
    """Gradients of ``L = sum(dy * Y)`` with respect to every input of Eq. (1).

    Returns a dict with dx, dW, db, dW_down, dM, dW_up, domega1, dphi1,
    domega2, dphi2.  ``dx_rows`` / ``dW_rows`` (index arrays) restrict the two
    large products to the listed rows of dx and dW; every other gradient is
    always complete.  Row selection does not change any value.
    """
    dy = _f64(dy)
    x = _f64(x)
    W = _f64(W)
    D = _f64(W_down)
    U = _f64(W_up)
    H = x @ D
    dC2 = dy @ U.T                               # Y = ... + C2 @ W_up
    cb = cosnet_backward(dC2, H, omega1, phi1, M, omega2, phi2)
    dH = cb["dH"]
    out = {
        "dW_up": cb["C2"].T @ dy,
        "dW_down": x.T @ dH,                     # H = x @ W_down
        "db": np.sum(dy, axis=0),
        "dM": cb["dM"],
        "domega1": cb["domega1"],
        "dphi1": cb["dphi1"],
        "domega2": cb["domega2"],
        "dphi2": cb["dphi2"],
    }
    if dW_rows is None:
        out["dW"] = x.T @ dy                     # Y = x @ W + ...
    else:
        out["dW"] = x[:, dW_rows].T @ dy
    if dx_rows is None:
        out["dx"] = dy @ W.T + dH @ D.T          # x enters through W and W_down
    else:
        out["dx"] = dy[dx_rows] @ W.T + dH[dx_rows] @ D.T
    return out


def branch_param_shapes(d_in, d_out, r):
    """Shapes of the parameters the branch adds to one linear layer (§3.1,
    §3.2): W_down, W_up, M and the four per-dimension frequency/phase
    vectors."""
    return {
        "W_down": (d_in, r),
        "W_up": (r, d_out),
        "M": (r, r),
        "omega1": (r,),
        "phi1": (r,),
        "omega2": (r,),
        "phi2": (r,),
    }
