"""Seeded synthetic inputs for the NOBLE-CosNet linear layer.

This module only draws random numbers and rounds them to the storage type the
device uses.  It holds none of the layer's arithmetic, so both the device path
(tests, bench) and the fp64 oracle can be fed from it without sharing code.

Recipe (one projection, one ``numpy.random.Generator(PCG64(seed))``):

* draw order: x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, dy
* x ~ N(0, 1) [T, d_in];  dy ~ N(0, 1) [T, d_out]
* W ~ N(0, w_var) [d_in, d_out], W_down ~ N(0, d_var) [d_in, r]
  (w_var = d_var = 1/d_in: variance 1/fan-in)
* M ~ N(0, m_var) [r, r], W_up ~ N(0, u_var) [r, d_out] (m_var = u_var = 1/r)
* omega = 1 + 0.1 N(0, 1), phi ~ U(0, 2 pi) per rank (both cosines)
* b ~ N(0, 1) * bias_std (bias_std = 0 gives the b = 0 of the workloads)

Samples are drawn in float32.  For the bf16 path the storage tensors
(x, W, W_down, M, W_up, dy) are rounded to bf16 with round-to-nearest-even;
b, omega and phi stay float32.  The float32 arrays returned hold exactly the
values the device sees.

The frequency/phase distributions deliberately differ from the training init
of §3.3 (omega ~ U[0.8, 1.2], phi ~ N(0, 0.1^2)) so that the cosine arguments
cover full periods and the branch contributes visibly to y.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

STORAGE = ("x", "W", "W_down", "M", "W_up", "dy")
FP32_PARAMS = ("b", "omega1", "phi1", "omega2", "phi2")


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even.

    Inputs are finite (no NaN handling needed for synthetic draws)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_bf16(a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(bf16_bits(a))


@dataclasses.dataclass
class Projection:
    """One NOBLE linear problem: shapes, dtype and the exact input values."""

    name: str
    T: int
    d_in: int
    d_out: int
    r: int                          # rank of each group's branch
    dtype: str                      # "bf16" or "f32" (storage type)
    arrays: Dict[str, np.ndarray]   # float32 arrays of exactly the device values
    groups: int = 1                 # output column groups sharing x, one branch each

    def __getitem__(self, k):
        return self.arrays[k]

    def device_arrays(self) -> Dict[str, np.ndarray]:
        """Arrays in device storage format: bf16 bits (uint16) for storage
        tensors on the bf16 path, float32 otherwise."""
        out = {}
        for k, v in self.arrays.items():
            if self.dtype == "bf16" and k in STORAGE:
                out[k] = bf16_bits(v)
            else:
                out[k] = np.ascontiguousarray(v, dtype=np.float32)
        return out


def draw_projection(name: str, T: int, d_in: int, d_out: int, r: int,
                    dtype: str = "bf16", seed: int = 0, *,
                    w_var: Optional[float] = None, d_var: Optional[float] = None,
                    m_var: Optional[float] = None, u_var: Optional[float] = None,
                    bias_std: float = 0.0, groups: int = 1, layers: int = 2) -> Projection:
    """Seeded inputs of one layer.  ``groups`` G > 1 gives the grouped layout:
    W_down [d_in, G r], M [G, r, r], frequency / phase vectors [G r] and
    W_up [G r, d_out / G]; G = 1 draws exactly the single-layer arrays.
    ``layers`` = 3 (the 3-layer CosNet) draws the mixing matrices and the
    second frequency / phase pair stacked: M [2, r, r] ([2, G, r, r]),
    omega2 and phi2 [2, G r], in the same draw order."""
    if dtype not in ("bf16", "f32"):
        raise ValueError(f"dtype must be 'bf16' or 'f32', got {dtype!r}")
    w_var = 1.0 / d_in if w_var is None else w_var
    d_var = 1.0 / d_in if d_var is None else d_var
    rr = max(r, 1)
    m_var = 1.0 / rr if m_var is None else m_var
    u_var = 1.0 / rr if u_var is None else u_var
    rng = np.random.Generator(np.random.PCG64(seed))
    f32 = np.float32

    def normal(shape, var):
        a = rng.standard_normal(shape, dtype=f32)
        if var != 1.0:
            a *= f32(math.sqrt(var))
        return a

    G = int(groups)
    if G < 1 or d_out % G:
        raise ValueError(f"d_out ({d_out}) must split into {G} groups")
    R = G * r

    def freq(n=None):
        shape = R if n is None else (n, R)
        return (f32(1.0) + f32(0.1) * rng.standard_normal(shape, dtype=f32)).astype(f32)

    def phase(n=None):
        shape = R if n is None else (n, R)
        return (rng.random(shape, dtype=f32) * f32(2.0 * math.pi)).astype(f32)

    stack = (2,) if layers == 3 else ()

    a = {}
    a["x"] = normal((T, d_in), 1.0)
    a["W"] = normal((d_in, d_out), w_var)
    a["b"] = (rng.standard_normal(d_out, dtype=f32) * f32(bias_std)).astype(f32)
    a["W_down"] = normal((d_in, R), d_var)
    a["omega1"] = freq()
    a["phi1"] = phase()
    a["M"] = normal(stack + ((r, r) if G == 1 else (G, r, r)), m_var)
    a["omega2"] = freq(2 if layers == 3 else None)
    a["phi2"] = phase(2 if layers == 3 else None)
    a["W_up"] = normal((R, d_out // G), u_var)
    a["dy"] = normal((T, d_out), 1.0)
    if dtype == "bf16":
        for k in STORAGE:
            a[k] = round_bf16(a[k])
    return Projection(name, T, d_in, d_out, r, dtype, a, G)


# ---------------------------------------------------------------------------
# Workloads: the layer shapes of the paper's models (§4.1.1 Base 250M and
# Large 1.5B LLMs, §4.2 ViT), one GPU's share of tokens.
# ---------------------------------------------------------------------------

WORKLOADS: Dict[str, dict] = {
    # tiny fp32 case; the oracle finishes it in milliseconds
    "tiny_fp32": dict(T=256, r=8, dtype="f32",
                      projections=[("proj", 64, 64)],
                      var=dict(w_var=1 / 64, d_var=1 / 64, m_var=1 / 8, u_var=1 / 64)),
    # 250M-LLM layer: 8 x 1024 tokens per GPU, d = 1024, r = 64
    "llm250m_r64": dict(T=8192, r=64, dtype="bf16",
                        projections=[("qkv", 1024, 3072), ("ffn_up", 1024, 4096)]),
    # 1.5B-LLM block: 8 x 1024 tokens, d = 2048, r = 128, four projections
    "llm1p5b_block_r128": dict(T=8192, r=128, dtype="bf16",
                               projections=[("qkv", 2048, 6144), ("o", 2048, 2048),
                                            ("ffn_up", 2048, 8192), ("ffn_down", 8192, 2048)]),
    # ViT-B-width layer: 128 images x 197 tokens, d = 768, r = 32
    "vitb_ffn_r32": dict(T=25216, r=32, dtype="bf16",
                         projections=[("ffn_up", 768, 3072), ("ffn_down", 3072, 768)]),
    # four 1.5B-style blocks, six projections each, 16 x 2048 tokens; Q, K
    # and V of a block read the same block input (K and V reuse Q's x)
    "llm1p5b_stack4_r128": dict(T=32768, r=128, dtype="bf16",
                                share_x={6 * blk + j: 6 * blk for blk in range(4) for j in (1, 2)},
                                projections=[(f"b{blk}_{p}", di, do)
                                             for blk in range(4)
                                             for (p, di, do) in (("q", 2048, 2048), ("k", 2048, 2048),
                                                                 ("v", 2048, 2048), ("o", 2048, 2048),
                                                                 ("ffn_up", 2048, 8192),
                                                                 ("ffn_down", 8192, 2048))]),
    # the same four blocks with Q, K and V as one grouped call per block (one
    # shared x, three branches): four projections per block
    "llm1p5b_stack4_r128_gqkv": dict(T=32768, r=128, dtype="bf16",
                                     projections=[(f"b{blk}_{p}", di, do, g)
                                                  for blk in range(4)
                                                  for (p, di, do, g) in (("qkv", 2048, 6144, 3),
                                                                         ("o", 2048, 2048, 1),
                                                                         ("ffn_up", 2048, 8192, 1),
                                                                         ("ffn_down", 8192, 2048, 1))]),
}


def _proj(entry):
    """(name, d_in, d_out, groups) of a workload's projection entry."""
    return (entry[0], entry[1], entry[2], entry[3] if len(entry) > 3 else 1)


def workload_shapes(name: str) -> List[Tuple[str, int, int, int, int]]:
    """[(projection name, T, d_in, d_out, r)] of a workload (r per group)."""
    w = WORKLOADS[name]
    return [(p, w["T"], di, do, w["r"]) for (p, di, do, _) in map(_proj, w["projections"])]


def workload_x_source(name: str) -> List[int]:
    """For each projection of a workload, the index of the projection whose x
    it reads (itself, or the Q projection of its block for K and V)."""
    w = WORKLOADS[name]
    share = w.get("share_x", {})
    return [share.get(i, i) for i in range(len(w["projections"]))]


def draw_x(T: int, d_in: int, dtype: str, seed: int) -> np.ndarray:
    """The x that draw_projection(..., seed) draws first, alone."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal((T, d_in), dtype=np.float32)
    return round_bf16(x) if dtype == "bf16" else x


def workload_groups(name: str) -> List[int]:
    """Branch groups of each projection of a workload."""
    return [_proj(e)[3] for e in WORKLOADS[name]["projections"]]


def draw_workload_projection(name: str, index: int, seed: int = 0, T: Optional[int] = None,
                             **overrides) -> Projection:
    """Projection ``index`` of workload ``name`` drawn with seed ``seed + index``.
    A projection that shares its block's input (workload_x_source) has the
    x of its source projection instead of its own first draw.

    ``T`` overrides the token count (a prefix sample of the workload's rows is
    not the same draw; use the full T for full-size checks)."""
    w = WORKLOADS[name]
    p, di, do, G = _proj(w["projections"][index])
    kw = dict(w.get("var", {}))
    kw.update(overrides)
    kw.setdefault("groups", G)
    TT = w["T"] if T is None else T
    proj = draw_projection(f"{name}/{p}", TT, di, do, w["r"], w["dtype"], seed + index, **kw)
    src = workload_x_source(name)[index]
    if src != index:
        proj.arrays["x"] = draw_x(TT, di, w["dtype"], seed + src)
    return proj
