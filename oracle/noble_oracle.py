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
  paper names in §5, "Why Cosine Activations?").

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
    "ACTIVATIONS",
    "LEAKY_SLOPE",
    "activation_value",
    "activation_slope",
    "branch_forward",
    "branch_backward",
    "cosnet_forward",
    "cosnet_backward",
    "forward",
    "backward",
    "branch_param_shapes",
    "forward_grouped",
    "backward_grouped",
]

# The bottleneck activations of the ablation in §4.4 (Table 5): each nonlinearity
# as a single activation and as the 2-layer sandwich with the mixing matrix M
# between two applications (the CosNet form of Eq. (2)).  name -> (f, layers).
# Readings (the paper names the activations but not their parameters): every
# layer keeps the per-dimension affine w (.) h + p of Eq. (2) before f, so
# w = 1, p = 0 gives the bare activation; LeakyReLU has negative slope 0.01 and
# GELU is the exact form x Phi(x) (the common library defaults).
ACTIVATIONS = {
    "cosnet": ("cos", 2),
    "cos": ("cos", 1),
    "tanh": ("tanh", 1),
    "tanh_m": ("tanh", 2),
    "leaky_relu": ("leaky_relu", 1),
    "leaky_relu_m": ("leaky_relu", 2),
    "gelu": ("gelu", 1),
    "gelu_m": ("gelu", 2),
    "cosnet3": ("cos", 3),
}
LEAKY_SLOPE = 0.01
# The 3-layer CosNet (last row of Table 5; §5 "CosNet Architecture
# Evolution": three or more layers).  Reading: a third cosine application
# after a second r x r mixing matrix, with its own per-dimension frequency
# and phase, the same pattern that links the first two:
#     A3 = w3 (.) (C2 M') + p3,  C3 = cos(A3),  sigma(h) = C3.
# Its parameters travel stacked with the second layer's: M is [2, r, r]
# (M[0] between layers 1 and 2, M[1] between 2 and 3; [2, G, r, r] for a
# grouped layer), omega2 and phi2 are [2, r] (row 0 layer 2, row 1 layer 3),
# and so are the gradients dM, domega2, dphi2.


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def _phi_cdf(a):
    """Standard normal CDF, 0.5 (1 + erf(a / sqrt 2)), evaluated as
    0.5 erfc(-a / sqrt 2), the same function without the cancellation of
    1 + erf in the lower tail."""
    from scipy.special import erfc
    return 0.5 * erfc(-a / np.sqrt(2.0))


def activation_value(f, a):
    """f(a) elementwise for f in cos, tanh, leaky_relu, gelu."""
    a = _f64(a)
    if f == "cos":
        return np.cos(a)
    if f == "tanh":
        return np.tanh(a)
    if f == "leaky_relu":
        return np.where(a > 0, a, LEAKY_SLOPE * a)
    if f == "gelu":
        return a * _phi_cdf(a)
    raise ValueError(f"unknown activation {f!r}")


def activation_slope(f, a):
    """f'(a) elementwise.  d cos = -sin; d tanh = 1 - tanh^2; LeakyReLU's slope
    is 1 for a > 0 and LEAKY_SLOPE otherwise; d (a Phi(a)) = Phi(a) + a phi(a)
    with phi the standard normal density."""
    a = _f64(a)
    if f == "cos":
        return -np.sin(a)
    if f == "tanh":
        return 1.0 - np.tanh(a) ** 2
    if f == "leaky_relu":
        return np.where(a > 0, 1.0, LEAKY_SLOPE)
    if f == "gelu":
        return _phi_cdf(a) + a * np.exp(-0.5 * a * a) / np.sqrt(2.0 * np.pi)
    raise ValueError(f"unknown activation {f!r}")


def _third_layer(M, omega2, phi2):
    """Split the stacked parameters of the 3-layer form: (M, w2, p2) of the
    second layer and (M', w3, p3) of the third."""
    M, omega2, phi2 = _f64(M), _f64(omega2), _f64(phi2)
    return (M[0], omega2[0], phi2[0]), (M[1], omega2[1], phi2[1])


def branch_forward(H, activation, omega1, phi1, M=None, omega2=None, phi2=None):
    """The bottleneck nonlinearity sigma applied to every row of ``H: [T, r]``.

    2-layer forms (Eq. (2) for cosine):  A1 = w1 (.) H + p1, C1 = f(A1),
    H2 = C1 M, A2 = w2 (.) H2 + p2, C2 = f(A2).  1-layer forms stop at
    C2 = C1 = f(A1) and ignore M, w2, p2.  The 3-layer form continues with
    H3 = C2 M', A3 = w3 (.) H3 + p3, C3 = f(A3) (parameters stacked, see
    ACTIVATIONS).  Returns the intermediates by name; "out" is sigma(H).
    """
    f, layers = ACTIVATIONS[activation]
    H = _f64(H)
    if layers == 3:
        (M, omega2, phi2), third = _third_layer(M, omega2, phi2)
    A1 = H * _f64(omega1) + _f64(phi1)          # w1 (.) h + p1
    C1 = activation_value(f, A1)                 # h1 = f(.)
    if layers == 1:
        return {"A1": A1, "C1": C1, "C2": C1, "out": C1}
    H2 = C1 @ _f64(M)                            # h2 = h1 mixed by M (row form)
    A2 = H2 * _f64(omega2) + _f64(phi2)          # w2 (.) h2 + p2
    C2 = activation_value(f, A2)                 # sigma(h) = f(.)
    fw = {"A1": A1, "C1": C1, "H2": H2, "A2": A2, "C2": C2, "out": C2}
    if layers == 3:
        M3, w3, p3 = third
        H3 = C2 @ M3                             # the second layer's output mixed by M'
        A3 = H3 * w3 + p3                        # w3 (.) h3 + p3
        C3 = activation_value(f, A3)
        fw.update(H3=H3, A3=A3, C3=C3, out=C3)
    return fw


def cosnet_forward(H, omega1, phi1, M, omega2, phi2):
    """sigma of §3.2 Eq. (2) (App. A), applied to every row of ``H: [T, r]``.

    Returns the intermediates by name: A1, C1, H2, A2, C2 (all ``[T, r]``).
    """
    return branch_forward(H, "cosnet", omega1, phi1, M, omega2, phi2)


def forward(x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, activation="cosnet"):
    """Eq. (1) with sigma = the named bottleneck activation (CosNet by
    default).  Rows of ``x`` are independent tokens, so passing a subset of
    rows of ``x`` yields exactly those rows of ``Y``.

    Returns ``(Y, H)`` where ``H = x @ W_down`` is the bottleneck input.
    """
    x = _f64(x)
    H = x @ _f64(W_down)
    C2 = branch_forward(H, activation, omega1, phi1, M, omega2, phi2)["out"]
    Y = x @ _f64(W) + C2 @ _f64(W_up)
    if b is not None:
        Y = Y + _f64(b)
    return Y, H


def branch_backward(dC2, H, activation, omega1, phi1, M=None, omega2=None, phi2=None):
    """Chain rule through sigma for ``L`` with ``dL/d sigma = dC2`` (rows =
    tokens).

    Recomputes the forward chain from ``H``.  Returns dH, domega1, dphi1, the
    recomputed sigma(H) ("out") and, for 2-layer forms, dM, domega2, dphi2
    (None otherwise; stacked [2, ...] for the 3-layer form).
    """
    f, layers = ACTIVATIONS[activation]
    dC2 = _f64(dC2)
    H = _f64(H)
    w1 = _f64(omega1)
    fw = branch_forward(H, activation, omega1, phi1, M, omega2, phi2)
    out = {"dM": None, "domega2": None, "dphi2": None, "out": fw["out"]}
    if layers == 3:
        # the third layer first; dC2 becomes the gradient of the middle C2
        (M, omega2, phi2), (M3, w3, p3) = _third_layer(M, omega2, phi2)
        dA3 = activation_slope(f, fw["A3"]) * dC2    # C3 = f(A3)
        domega3 = np.sum(dA3 * fw["H3"], axis=0)     # A3 = w3 (.) H3 + p3
        dphi3 = np.sum(dA3, axis=0)
        dH3 = dA3 * w3
        dM3 = fw["C2"].T @ dH3                       # H3 = C2 @ M'
        dC2 = dH3 @ M3.T
    if layers >= 2:
        dA2 = activation_slope(f, fw["A2"]) * dC2    # C2 = f(A2)
        out["domega2"] = np.sum(dA2 * fw["H2"], axis=0)   # A2 = w2 (.) H2 + p2
        out["dphi2"] = np.sum(dA2, axis=0)
        dH2 = dA2 * _f64(omega2)
        out["dM"] = fw["C1"].T @ dH2                 # H2 = C1 @ M
        dC1 = dH2 @ _f64(M).T
    else:
        dC1 = dC2                                    # C2 = C1
    dA1 = activation_slope(f, fw["A1"]) * dC1        # C1 = f(A1)
    out["domega1"] = np.sum(dA1 * H, axis=0)         # A1 = w1 (.) H + p1
    out["dphi1"] = np.sum(dA1, axis=0)
    out["dH"] = dA1 * w1
    if layers == 3:
        out["dM"] = np.stack([out["dM"], dM3])
        out["domega2"] = np.stack([out["domega2"], domega3])
        out["dphi2"] = np.stack([out["dphi2"], dphi3])
    return out


def cosnet_backward(dC2, H, omega1, phi1, M, omega2, phi2):
    """Chain rule through sigma for ``L`` with ``dL/dC2 = dC2`` (rows = tokens).

    Recomputes the forward chain from ``H``.  Returns dH, dM, domega1, dphi1,
    domega2, dphi2 and the recomputed C2.
    """
    return branch_backward(dC2, H, "cosnet", omega1, phi1, M, omega2, phi2)


def backward(dy, x, W, W_down, omega1, phi1, M, omega2, phi2, W_up,
             dx_rows=None, dW_rows=None, activation="cosnet"):
    """Gradients of ``L = sum(dy * Y)`` with respect to every input of Eq. (1).

    Returns a dict with dx, dW, db, dW_down, dM, dW_up, domega1, dphi1,
    domega2, dphi2 (dM, domega2, dphi2 are None for 1-layer activations).
    ``dx_rows`` / ``dW_rows`` (index arrays) restrict the two large products
    to the listed rows of dx and dW; every other gradient is always complete.
    Row selection does not change any value.
    """
    dy = _f64(dy)
    x = _f64(x)
    W = _f64(W)
    D = _f64(W_down)
    U = _f64(W_up)
    H = x @ D
    dC2 = dy @ U.T                               # Y = ... + C2 @ W_up
    cb = branch_backward(dC2, H, activation, omega1, phi1, M, omega2, phi2)
    dH = cb["dH"]
    out = {
        "dW_up": cb["out"].T @ dy,
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


# ------------------------------------------------------------ grouped layers --
# NOBLE puts a branch on every linear projection, Q, K and V included
# (§4.1.1).  When Q, K and V are computed as one product of the shared x, the
# layer's d_out columns form G equal blocks, and block g is a layer of its own:
#     y[:, g] = x W[:, g] + b[g] + sigma_g(x W_down[:, g]) W_up[g]
# with W_down's column block g (r columns), M[g], the vectors' entries
# g r .. g r + r - 1 and W_up's row block g ([G r, d_out / G]).


def _group_views(G, d_out, R, W_down, omega1, phi1, M, omega2, phi2, W_up, g, layers=2):
    r, dg = R // G, d_out // G
    rs = slice(g * r, (g + 1) * r)
    pick = lambda v: None if v is None else _f64(v)[..., rs]     # stacked [2, R] vectors too
    if M is None or G == 1:
        Mg = _f64(M)
    else:
        Mg = _f64(M)[:, g] if layers == 3 else _f64(M)[g]       # [2, G, r, r] or [G, r, r]
    return (slice(g * dg, (g + 1) * dg), _f64(W_down)[:, rs], pick(omega1), pick(phi1), Mg, pick(omega2),
            pick(phi2), _f64(W_up)[rs])


def forward_grouped(x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, groups,
                    activation="cosnet"):
    """Eq. (1) for each of ``groups`` column blocks sharing x.  Returns
    ``(Y, H)`` with H = x W_down ([T, G r])."""
    W = _f64(W)
    G, d_out, R = int(groups), W.shape[1], _f64(W_down).shape[1]
    Ys = []
    for g in range(G):
        cs, Dg, w1, p1, Mg, w2, p2, Ug = _group_views(G, d_out, R, W_down, omega1, phi1, M, omega2, phi2, W_up, g,
                                                      ACTIVATIONS[activation][1])
        Y, _ = forward(x, W[:, cs], None if b is None else _f64(b)[cs], Dg, w1, p1, Mg, w2, p2, Ug,
                       activation=activation)
        Ys.append(Y)
    return np.concatenate(Ys, axis=1), _f64(x) @ _f64(W_down)


def backward_grouped(dy, x, W, W_down, omega1, phi1, M, omega2, phi2, W_up, groups,
                     dx_rows=None, dW_rows=None, activation="cosnet"):
    """Gradients of L = sum(dy * Y) for the grouped layer: each block's
    backward on its columns of dy; dx, which every block reaches through x,
    is the sum of the blocks' dx, every other gradient is the blocks'
    gradients side by side (dM stacked [G, r, r], or [r, r] for G = 1; for
    the 3-layer form [2, G, r, r] and domega2, dphi2 [2, G r])."""
    W, dy = _f64(W), _f64(dy)
    G, d_out, R = int(groups), W.shape[1], _f64(W_down).shape[1]
    layers = ACTIVATIONS[activation][1]
    parts = []
    for g in range(G):
        cs, Dg, w1, p1, Mg, w2, p2, Ug = _group_views(G, d_out, R, W_down, omega1, phi1, M, omega2, phi2, W_up, g,
                                                      layers)
        parts.append(backward(dy[:, cs], x, W[:, cs], Dg, w1, p1, Mg, w2, p2, Ug, dx_rows=dx_rows,
                              dW_rows=dW_rows, activation=activation))
    cat = lambda k, ax: None if parts[0][k] is None else np.concatenate([q[k] for q in parts], axis=ax)
    out = {"dx": sum(q["dx"] for q in parts), "dW": cat("dW", 1), "db": cat("db", 0),
           "dW_down": cat("dW_down", 1), "dW_up": cat("dW_up", 0)}
    for k in ("domega1", "dphi1", "domega2", "dphi2"):
        out[k] = cat(k, -1)
    if parts[0]["dM"] is None:
        out["dM"] = None
    else:
        out["dM"] = parts[0]["dM"] if G == 1 else np.stack([q["dM"] for q in parts], axis=1 if layers == 3 else 0)
    return out
