"""Parity metric and oracle references for the GPU tests (test helpers only)."""

from __future__ import annotations

import numpy as np

import oracle

# max over rows of max_j |gpu - ref| / (max_j |ref| + 1e-6): bf16 operands with
# float32 accumulation, and the float32 path
TOL = {"bf16": 2e-2, "f32": 1e-4}
OUTPUTS = ("y", "dx", "dW", "db", "dW_down", "dM", "dW_up", "domega1", "dphi1", "domega2", "dphi2")


def row_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    gpu = np.atleast_2d(np.asarray(gpu, dtype=np.float64))
    ref = np.atleast_2d(np.asarray(ref, dtype=np.float64))
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    denom = np.max(np.abs(ref), axis=1) + 1e-6
    return float(np.max(np.max(np.abs(gpu - ref), axis=1) / denom))


def oracle_outputs(p, *, with_bias=True, branch=True, rows=None, dw_rows=None, activation="cosnet"):
    """fp64 oracle y and gradients for projection ``p`` (optionally row-sampled)."""
    a = p.arrays
    if branch:
        br = {k: a[k] for k in ("W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up")}
    else:
        z = np.zeros
        br = {"W_down": z((p.d_in, 0)), "omega1": z(0), "phi1": z(0), "M": z((0, 0)),
              "omega2": z(0), "phi2": z(0), "W_up": z((0, p.d_out))}
    b = a["b"] if with_bias else None
    x = a["x"] if rows is None else a["x"][rows]
    G = getattr(p, "groups", 1)
    if branch and G > 1:
        Y, _ = oracle.forward_grouped(x, a["W"], b, br["W_down"], br["omega1"], br["phi1"], br["M"],
                                      br["omega2"], br["phi2"], br["W_up"], G, activation=activation)
        g = oracle.backward_grouped(a["dy"], a["x"], a["W"], br["W_down"], br["omega1"], br["phi1"], br["M"],
                                    br["omega2"], br["phi2"], br["W_up"], G, dx_rows=rows, dW_rows=dw_rows,
                                    activation=activation)
        g["y"] = Y
        return g
    Y, _ = oracle.forward(x, a["W"], b, br["W_down"], br["omega1"], br["phi1"], br["M"],
                          br["omega2"], br["phi2"], br["W_up"], activation=activation)
    g = oracle.backward(a["dy"], a["x"], a["W"], br["W_down"], br["omega1"], br["phi1"], br["M"],
                        br["omega2"], br["phi2"], br["W_up"], dx_rows=rows, dW_rows=dw_rows,
                        activation=activation)
    g["y"] = Y
    return g


def parity_report(gpu: dict, ref: dict, names=OUTPUTS) -> dict:
    return {n: row_err(gpu[n], ref[n]) for n in names if gpu.get(n) is not None and ref.get(n) is not None}


def kink_margin(p, activation, rel=1e-5):
    """Smallest |A| / band over the pre-activations A1 (and A2) of the
    LeakyReLU forms, band = rel * (|w| max_t |h| + |p|) per rank column (h the
    column that w scales).  Below 1 an element sits where float32 and float64
    can take different branches of the kink; a parity case needs > 1.  The
    kernels compute H = x W_down and H2 = C1 M to float32 accuracy (the
    mixing operand as a three-part bf16 split), so A1 and A2 carry float32
    rounding only.  Grouped layers are checked group by group."""
    a = {k: (None if v is None else np.asarray(v, dtype=np.float64)) for k, v in p.arrays.items()}
    G = getattr(p, "groups", 1)
    r = p.r
    H = a["x"] @ a["W_down"]

    def margin(A, h, w, ph):
        band = rel * (np.abs(w) * np.max(np.abs(h), axis=0) + np.abs(ph))
        return float(np.min(np.abs(A) / band))

    m = np.inf
    for g in range(G):
        cs = slice(g * r, (g + 1) * r)
        Mg = a["M"] if G == 1 else a["M"][g]
        fw = oracle.branch_forward(H[:, cs], activation, a["omega1"][cs], a["phi1"][cs], Mg, a["omega2"][cs],
                                   a["phi2"][cs])
        m = min(m, margin(fw["A1"], H[:, cs], a["omega1"][cs], a["phi1"][cs]))
        if "A2" in fw:
            m = min(m, margin(fw["A2"], fw["H2"], a["omega2"][cs], a["phi2"][cs]))
    return m
