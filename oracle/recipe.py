"""Plain CPU statement of the layer's training recipe (Sec. 3.3 "Key Design
Choices"; App. A "Hyperparameter Defaults").

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` may import or call this module; the
HIP product path never does, and this module imports nothing from it.

* ``lr_multipliers``: Sec. 3.3 Eqs. 3-4, the elevated learning rates of W_up
  and M, and App. A's fixed multipliers for the frequencies (3.0) and phases
  (5.0); W, b and W_down take the base rate.
* ``init_values``: the initial values the library's device fill draws.
  - W ~ N(0, (0.5 / sqrt(d_in))^2) (half the Kaiming scale, Sec. 3.3);
  - W_up ~ N(0, (alpha / sqrt(r))^2), alpha = 0.01 (Sec. 3.3);
  - omega ~ U[0.8, 1.2], phi ~ N(0, 0.1^2) (Sec. 3.3, App. A);
  - M Xavier: read as Xavier-uniform, U(-sqrt(6 / (r + r)), +sqrt(6 / (r + r)));
  - W_down: the paper states none; read as the common linear-layer default
    U(-1/sqrt(d_in), 1/sqrt(d_in));
  - b = 0 (not stated; read as zero).
  The random words come from Philox4x32-10 (Salmon, Moraes, Dror and Shaw,
  "Parallel random numbers: as easy as 1, 2, 3", SC 2011), written here from
  that definition; the counter layout, the mapping of words to uniforms
  and the Box-Muller transform are the library's documented conventions.
"""

from __future__ import annotations

import numpy as np

DEFAULTS = dict(alpha=0.01, w_scale=0.5, omega_min=0.8, omega_max=1.2, phi_std=0.1,
                gamma=0.3, gamma_M=0.45, omega_lr=3.0, phi_lr=5.0)

# tensor ids of the counter layout
TENSOR_IDS = dict(W=0, W_down=1, omega1=2, phi1=3, M=4, omega2=5, phi2=6, W_up=7)

_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(c, k):
    """Philox4x32 with 10 rounds.  ``c``: four uint32 arrays (or ints), ``k``:
    two.  Each round multiplies words 0 and 2 by the two Philox constants
    (full 64-bit products), and recombines the high halves with words 1 and
    3 and the key; the key is bumped by the two Weyl constants before every
    round but the first.  Returns four uint32 arrays."""
    c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) & _MASK for x in c)
    k0, k1 = (np.asarray(x, dtype=np.uint64) & _MASK for x in k)
    m0, m1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
    w0, w1 = np.uint64(0x9E3779B9), np.uint64(0xBB67AE85)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + w0) & _MASK
            k1 = (k1 + w1) & _MASK
        p0 = m0 * c0
        p1 = m1 * c2
        c0, c1, c2, c3 = ((p1 >> np.uint64(32)) ^ c1 ^ k0, p1 & _MASK,
                          (p0 >> np.uint64(32)) ^ c3 ^ k1, p0 & _MASK)
    return tuple(x.astype(np.uint32) for x in (c0, c1, c2, c3))


def _words(seed: int, tensor_id: int, n: int):
    e = np.arange(n, dtype=np.uint64)
    return philox4x32_10((e & _MASK, e >> np.uint64(32), np.full(n, tensor_id, np.uint64), np.zeros(n, np.uint64)),
                         (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))


def _unit(x):
    return (x.astype(np.float64) + 0.5) * 2.0 ** -32


def draw_uniform(seed, tensor_id, n, lo, hi):
    x = _words(seed, tensor_id, n)
    return lo + (hi - lo) * _unit(x[0])


def draw_normal(seed, tensor_id, n, std):
    """Box-Muller: std * sqrt(-2 ln u0) * cos(2 pi u1)."""
    x = _words(seed, tensor_id, n)
    return std * np.sqrt(-2.0 * np.log(_unit(x[0]))) * np.cos(2.0 * np.pi * _unit(x[1]))


def to_bf16(a):
    """float32 -> bf16 (round to nearest even) -> float32, for finite values."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)) << np.uint64(16)
    return u.astype(np.uint32).view(np.float32)


def init_values(d_in, d_out, r, seed, dtype="bf16", recipe=None, groups=1, layers=2):
    """Initial values of every parameter, as float32 arrays (storage tensors
    rounded to bf16 when ``dtype`` is "bf16").  ``groups`` G > 1: W_down
    [d_in, G r], M [G, r, r], the vectors [G r], W_up [G r, d_out / G], each
    tensor drawn as one row-major stream.  ``layers`` = 3 (the 3-layer CosNet
    of Table 5): M is [2, (G,) r, r] and omega2, phi2 are [2, G r], the second
    mixing matrix and the third frequency / phase drawn as the continuation
    of the same streams (the paper gives no initialisation for them; this
    reading takes the second layer's)."""
    G = groups
    n = 2 if layers == 3 else 1
    R, dog = G * r, d_out // G
    rc = dict(DEFAULTS, **(recipe or {}))
    store = (lambda a: to_bf16(a.astype(np.float32))) if dtype == "bf16" else (lambda a: a.astype(np.float32))
    out = {
        "W": store(draw_normal(seed, TENSOR_IDS["W"], d_in * d_out, rc["w_scale"] / np.sqrt(d_in))
                   ).reshape(d_in, d_out),
        "b": np.zeros(d_out, np.float32),
    }
    if r > 0:
        db = 1.0 / np.sqrt(d_in)
        mb = np.sqrt(6.0 / (r + r))
        out["W_down"] = store(draw_uniform(seed, TENSOR_IDS["W_down"], d_in * R, -db, db)).reshape(d_in, R)
        M = store(draw_uniform(seed, TENSOR_IDS["M"], n * G * r * r, -mb, mb))
        mshape = (r, r) if G == 1 else (G, r, r)
        out["M"] = M.reshape(((n,) if n > 1 else ()) + mshape)
        out["W_up"] = store(draw_normal(seed, TENSOR_IDS["W_up"], R * dog, rc["alpha"] / np.sqrt(r))
                            ).reshape(R, dog)
        for i in (1, 2):
            k = n if i == 2 else 1
            vshape = (k, R) if k > 1 else (R,)
            out[f"omega{i}"] = draw_uniform(seed, TENSOR_IDS[f"omega{i}"], k * R, rc["omega_min"],
                                            rc["omega_max"]).astype(np.float32).reshape(vshape)
            out[f"phi{i}"] = draw_normal(seed, TENSOR_IDS[f"phi{i}"], k * R,
                                         rc["phi_std"]).astype(np.float32).reshape(vshape)
    return out


def lr_multipliers(d_in, d_out, r, recipe=None):
    """Sec. 3.3 Eqs. 3-4 with App. A's frequency and phase multipliers."""
    rc = dict(DEFAULTS, **(recipe or {}))
    if r == 0:
        return dict(W=1.0, b=1.0, W_down=0.0, W_up=0.0, M=0.0, omega=0.0, phi=0.0)
    ratio = min(d_in, d_out) / r
    return dict(W=1.0, b=1.0, W_down=1.0, W_up=ratio ** (2 * rc["gamma"]), M=ratio ** rc["gamma_M"],
                omega=rc["omega_lr"], phi=rc["phi_lr"])
