"""Python binding of libnoble (include/noble.h): argument marshalling only.

Every step of the layer runs in the HIP kernels of ``libnoble.so``; this module
only checks tensors, passes their device pointers and the current HIP stream,
and turns status codes into exceptions.  There is no fallback: if the library
is not built, or the device is not gfx950, calls raise.

Functions keep the C names: ``noble_linear_workspace_size``,
``noble_linear_fwd_scratch_size``,
``noble_linear_fwd``, ``noble_linear_bwd``, ``noble_status_string``, and the
training-recipe calls ``noble_recipe_defaults``, ``noble_lr_multipliers``,
``noble_init_params`` (plus ``param_groups``, which only arranges the
multipliers into optimizer parameter groups).
``NobleLinearFunction`` wraps the pair as a ``torch.autograd.Function``.

``activation`` (keyword of the calls) is a noble_activation code or one of the
names in ``ACTIVATIONS``; the default is the CosNet.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libnoble.so")

NOBLE_BF16 = 0
NOBLE_F32 = 1
# NOBLE_ABI_VERSION of include/noble.h that the structures below mirror
ABI_VERSION = 5

STATUS = {
    0: "NOBLE_OK",
    1: "NOBLE_ERR_NULL_ARG",
    2: "NOBLE_ERR_BAD_SHAPE",
    3: "NOBLE_ERR_BAD_DTYPE",
    4: "NOBLE_ERR_MISALIGNED",
    5: "NOBLE_ERR_WORKSPACE_TOO_SMALL",
    6: "NOBLE_ERR_UNSUPPORTED_DEVICE",
    7: "NOBLE_ERR_HIP",
    8: "NOBLE_ERR_BAD_ACTIVATION",
}

# noble_activation codes by name.
ACTIVATIONS = {
    "cosnet": 0,
    "cos": 1,
    "tanh": 2,
    "tanh_m": 3,
    "leaky_relu": 4,
    "leaky_relu_m": 5,
    "gelu": 6,
    "gelu_m": 7,
    "cosnet3": 8,
}
# applications of the nonlinearity per activation (mixing matrices: one fewer)
LAYERS = {"cosnet": 2, "cos": 1, "tanh": 1, "tanh_m": 2, "leaky_relu": 1, "leaky_relu_m": 2, "gelu": 1,
          "gelu_m": 2, "cosnet3": 3}
TWO_LAYER = {n for n, k in LAYERS.items() if k >= 2}


def activation_code(activation) -> int:
    """noble_activation code of a name (or of a code, returned as is)."""
    if isinstance(activation, str):
        if activation not in ACTIVATIONS:
            raise ValueError(f"unknown activation {activation!r}; expected one of {sorted(ACTIVATIONS)}")
        return ACTIVATIONS[activation]
    return int(activation)


def layers(activation) -> int:
    """Applications of the nonlinearity: 1, 2 (CosNet and the _m names) or 3
    (the 3-layer CosNet)."""
    code = activation_code(activation)
    for n, c in ACTIVATIONS.items():
        if c == code:
            return LAYERS[n]
    raise ValueError(f"unknown activation code {code}")


def two_layers(activation) -> bool:
    """True for the forms with a mixing matrix M (two or three layers)."""
    return layers(activation) >= 2


class NobleError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {noble_status_string(status)}")


class noble_linear_desc(ctypes.Structure):
    _fields_ = [
        ("T", ctypes.c_int64),
        ("d_in", ctypes.c_int64),
        ("d_out", ctypes.c_int64),
        ("r", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
        ("activation", ctypes.c_int32),
        ("groups", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class noble_recipe(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in
                ("alpha", "w_scale", "omega_min", "omega_max", "phi_std", "gamma", "gamma_M", "omega_lr", "phi_lr")]


class noble_lr_mults(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("W", "b", "W_down", "W_up", "M", "omega", "phi")]


_lib = None
_vp = ctypes.c_void_p


def lib() -> ctypes.CDLL:
    """The loaded libnoble.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(or python -m paper_2603_06492_amd._build)")
        L = ctypes.CDLL(LIB_PATH)
        L.noble_status_string.restype = ctypes.c_char_p
        L.noble_status_string.argtypes = [ctypes.c_int]
        L.noble_abi_version.restype = ctypes.c_int
        L.noble_abi_version.argtypes = []
        if L.noble_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has C ABI version {L.noble_abi_version()}, the binding expects "
                               f"{ABI_VERSION}: rebuild it")
        L.noble_linear_workspace_size.restype = ctypes.c_int
        L.noble_linear_workspace_size.argtypes = [ctypes.POINTER(noble_linear_desc),
                                                  ctypes.POINTER(ctypes.c_size_t),
                                                  ctypes.POINTER(ctypes.c_size_t)]
        L.noble_linear_fwd_static.restype = ctypes.c_int
        L.noble_linear_fwd_static.argtypes = [ctypes.POINTER(noble_linear_desc)] + [ctypes.c_void_p] * 13
        L.noble_profile_next_wgrad.restype = ctypes.c_int
        L.noble_profile_next_wgrad.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)]
        L.noble_linear_fwd_scratch_size.restype = ctypes.c_int
        L.noble_linear_fwd_scratch_size.argtypes = [ctypes.POINTER(noble_linear_desc),
                                                    ctypes.POINTER(ctypes.c_size_t)]
        L.noble_linear_fwd.restype = ctypes.c_int
        L.noble_linear_fwd.argtypes = [ctypes.POINTER(noble_linear_desc)] + [_vp] * 13 + [ctypes.c_size_t, _vp]
        L.noble_linear_bwd.restype = ctypes.c_int
        L.noble_linear_bwd.argtypes = [ctypes.POINTER(noble_linear_desc)] + [_vp] * 22 + [ctypes.c_size_t, _vp]
        L.noble_recipe_defaults.restype = None
        L.noble_recipe_defaults.argtypes = [ctypes.POINTER(noble_recipe)]
        L.noble_lr_multipliers.restype = ctypes.c_int
        L.noble_lr_multipliers.argtypes = [ctypes.POINTER(noble_linear_desc), ctypes.POINTER(noble_recipe),
                                           ctypes.POINTER(noble_lr_mults)]
        L.noble_init_params.restype = ctypes.c_int
        L.noble_init_params.argtypes = [ctypes.POINTER(noble_linear_desc), ctypes.POINTER(noble_recipe),
                                        ctypes.c_uint64] + [_vp] * 10
        _lib = L
    return _lib


def noble_status_string(status: int) -> str:
    return lib().noble_status_string(int(status)).decode()


def make_desc(T: int, d_in: int, d_out: int, r: int, dtype: int, activation=0, groups: int = 1) -> noble_linear_desc:
    return noble_linear_desc(int(T), int(d_in), int(d_out), int(r), int(dtype), activation_code(activation),
                             int(groups), 0)


def noble_profile_next_wgrad(start_event: int, stop_event: int, workgroups=None) -> None:
    """The calling thread's next backward records these hipEvent_t handles
    around its weight-gradient launch and, given a ctypes.c_int64,
    stores that launch's workgroup count in it (instrumentation)."""
    lib().noble_profile_next_wgrad(ctypes.c_void_p(start_event), ctypes.c_void_p(stop_event),
                                   None if workgroups is None else ctypes.byref(workgroups))


def noble_linear_fwd_scratch_size(T: int, d_in: int, d_out: int, r: int, dtype: int,
                                  activation=0, groups: int = 1) -> int:
    """Scratch bytes of the forward alone (r: rank per group)."""
    d = make_desc(T, d_in, d_out, r, dtype, activation, groups)
    scr = ctypes.c_size_t(0)
    st = lib().noble_linear_fwd_scratch_size(ctypes.byref(d), ctypes.byref(scr))
    if st != 0:
        raise NobleError(st, "noble_linear_fwd_scratch_size")
    return scr.value


def noble_linear_workspace_size(T: int, d_in: int, d_out: int, r: int, dtype: int,
                                activation=0, groups: int = 1) -> Tuple[int, int]:
    """(reserve_bytes, scratch_bytes) for the problem (r: rank per group)."""
    d = make_desc(T, d_in, d_out, r, dtype, activation, groups)
    res, scr = ctypes.c_size_t(0), ctypes.c_size_t(0)
    st = lib().noble_linear_workspace_size(ctypes.byref(d), ctypes.byref(res), ctypes.byref(scr))
    if st != 0:
        raise NobleError(st, "noble_linear_workspace_size")
    return res.value, scr.value


# ----------------------------------------------------------------- tensors --

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return NOBLE_BF16
    if t.dtype == torch.float32:
        return NOBLE_F32
    raise TypeError(f"storage tensors must be bfloat16 or float32, got {t.dtype}")


def _ptr(t, name: str, dtype=None, shape=None, device=None) -> Optional[int]:
    if t is None:
        return None
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the call runs on {device}: all tensors must share one device")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr() or None


def _stream(stream, device) -> Optional[int]:
    """The stream handle of ``stream`` (default: torch's current stream of
    ``device``), which must belong to ``device``."""
    torch = _torch()
    s = torch.cuda.current_stream(device) if stream is None else stream
    if s.device != device:
        raise ValueError(f"stream belongs to {s.device}, the tensors to {device}")
    return s.cuda_stream or None


def _on(device):
    """Context making ``device`` current: the library launches on the
    current HIP device."""
    return _torch().cuda.device(device)


def _branch_shapes(d_in, d_out, R, groups, activation=0):
    """Shapes of W_down, the [R] vectors, M, the second-layer vectors (vec2)
    and W_up for ``groups`` groups of total rank R (M is [r, r] for one group,
    [G, r, r] otherwise; the 3-layer form stacks two of each: M [2, ...],
    omega2 / phi2 [2, R])."""
    G = int(groups)
    if R % G or d_out % G:
        raise ValueError(f"d_out ({d_out}) and the total rank ({R}) must divide into {G} groups")
    r = R // G
    M = (r, r) if G == 1 else (G, r, r)
    three = layers(activation) == 3
    return dict(W_down=(d_in, R), vec=(R,), M=(2,) + M if three else M, vec2=(2, R) if three else (R,),
                W_up=(R, d_out // G)), r


def noble_linear_fwd(x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, scratch,
                     stream=None, activation=0, groups: int = 1) -> None:
    """Enqueue the forward on ``stream`` (default: torch's current stream).

    Storage tensors (x, W, W_down, M, W_up, y) share one dtype (bf16 or f32);
    b, omega*, phi* are float32.  reserve/scratch are byte (uint8) tensors of
    at least the sizes from noble_linear_workspace_size.  With r = 0 pass None
    for the branch tensors; one-application activations do not read M,
    omega2, phi2 (None allowed).  ``groups`` > 1: W_down [d_in, G r], M
    [G, r, r], the vectors [G r], W_up [G r, d_out / G] (one branch per block
    of d_out / G output columns).
    """
    torch = _torch()
    T, d_in = x.shape
    d_out = W.shape[1]
    R = 0 if W_down is None else W_down.shape[1]
    sh, r = _branch_shapes(d_in, d_out, R, groups, activation)
    dt = _dtype_code(x)
    sd = x.dtype
    f32 = torch.float32
    d = make_desc(T, d_in, d_out, r, dt, activation, groups)
    dev = x.device
    args = [
        _ptr(x, "x", sd, (T, d_in), dev), _ptr(W, "W", sd, (d_in, d_out), dev), _ptr(b, "b", f32, (d_out,), dev),
        _ptr(W_down, "W_down", sd, sh["W_down"], dev), _ptr(omega1, "omega1", f32, sh["vec"], dev),
        _ptr(phi1, "phi1", f32, sh["vec"], dev), _ptr(M, "M", sd, sh["M"], dev),
        _ptr(omega2, "omega2", f32, sh["vec2"], dev), _ptr(phi2, "phi2", f32, sh["vec2"], dev),
        _ptr(W_up, "W_up", sd, sh["W_up"], dev), _ptr(y, "y", sd, (T, d_out), dev),
        _ptr(reserve, "reserve", device=dev), _ptr(scratch, "scratch", device=dev),
    ]
    nbytes = 0 if scratch is None else scratch.numel() * scratch.element_size()
    with _on(dev):
        st = lib().noble_linear_fwd(ctypes.byref(d), *args, nbytes, _stream(stream, dev))
    if st != 0:
        raise NobleError(st, "noble_linear_fwd")


def noble_linear_fwd_static(x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve,
                            stream=None, activation=0, groups: int = 1) -> None:
    """noble_linear_fwd without a scratch argument: the library's own static
    device scratch (for callers that cannot allocate; see include/noble.h)."""
    torch = _torch()
    T, d_in = x.shape
    d_out = W.shape[1]
    R = 0 if W_down is None else W_down.shape[1]
    sh, r = _branch_shapes(d_in, d_out, R, groups, activation)
    sd, f32, dev = x.dtype, torch.float32, x.device
    d = make_desc(T, d_in, d_out, r, _dtype_code(x), activation, groups)
    args = [
        _ptr(x, "x", sd, (T, d_in), dev), _ptr(W, "W", sd, (d_in, d_out), dev), _ptr(b, "b", f32, (d_out,), dev),
        _ptr(W_down, "W_down", sd, sh["W_down"], dev), _ptr(omega1, "omega1", f32, sh["vec"], dev),
        _ptr(phi1, "phi1", f32, sh["vec"], dev), _ptr(M, "M", sd, sh["M"], dev),
        _ptr(omega2, "omega2", f32, sh["vec2"], dev), _ptr(phi2, "phi2", f32, sh["vec2"], dev),
        _ptr(W_up, "W_up", sd, sh["W_up"], dev), _ptr(y, "y", sd, (T, d_out), dev),
        _ptr(reserve, "reserve", device=dev),
    ]
    with _on(dev):
        st = lib().noble_linear_fwd_static(ctypes.byref(d), *args, _stream(stream, dev))
    if st != 0:
        raise NobleError(st, "noble_linear_fwd_static")


def noble_linear_bwd(dy, x, W, W_down, omega1, phi1, M, omega2, phi2, W_up, reserve,
                     dx, dW, db, dW_down, dM, dW_up, domega1, dphi1, domega2, dphi2, scratch,
                     stream=None, activation=0, groups: int = 1) -> None:
    """Enqueue the backward on ``stream``; overwrites every gradient tensor.

    dx has the storage dtype; dW, db (optional), dW_down, dM, dW_up and the
    four frequency/phase gradients are float32.  One-application activations
    accept None for M, omega2, phi2, dM, domega2 and dphi2 (given gradient
    tensors are set to zero).
    """
    torch = _torch()
    T, d_in = x.shape
    d_out = W.shape[1]
    R = 0 if W_down is None else W_down.shape[1]
    sh, r = _branch_shapes(d_in, d_out, R, groups, activation)
    dt = _dtype_code(x)
    sd = x.dtype
    f32 = torch.float32
    d = make_desc(T, d_in, d_out, r, dt, activation, groups)
    v, v2 = sh["vec"], sh["vec2"]
    dev = x.device
    args = [
        _ptr(dy, "dy", sd, (T, d_out), dev), _ptr(x, "x", sd, (T, d_in), dev), _ptr(W, "W", sd, (d_in, d_out), dev),
        _ptr(W_down, "W_down", sd, sh["W_down"], dev), _ptr(omega1, "omega1", f32, v, dev),
        _ptr(phi1, "phi1", f32, v, dev), _ptr(M, "M", sd, sh["M"], dev), _ptr(omega2, "omega2", f32, v2, dev),
        _ptr(phi2, "phi2", f32, v2, dev), _ptr(W_up, "W_up", sd, sh["W_up"], dev),
        _ptr(reserve, "reserve", device=dev),
        _ptr(dx, "dx", sd, (T, d_in), dev), _ptr(dW, "dW", f32, (d_in, d_out), dev),
        _ptr(db, "db", f32, (d_out,), dev),
        _ptr(dW_down, "dW_down", f32, sh["W_down"], dev), _ptr(dM, "dM", f32, sh["M"], dev),
        _ptr(dW_up, "dW_up", f32, sh["W_up"], dev),
        _ptr(domega1, "domega1", f32, v, dev), _ptr(dphi1, "dphi1", f32, v, dev),
        _ptr(domega2, "domega2", f32, v2, dev), _ptr(dphi2, "dphi2", f32, v2, dev),
        _ptr(scratch, "scratch", device=dev),
    ]
    nbytes = 0 if scratch is None else scratch.numel() * scratch.element_size()
    with _on(dev):
        st = lib().noble_linear_bwd(ctypes.byref(d), *args, nbytes, _stream(stream, dev))
    if st != 0:
        raise NobleError(st, "noble_linear_bwd")


# --------------------------------------------------------- training recipe --

def noble_recipe_defaults(**overrides) -> noble_recipe:
    """The recipe defaults (Sec. 3.3, App. A), with keyword overrides."""
    rc = noble_recipe()
    lib().noble_recipe_defaults(ctypes.byref(rc))
    for k, v in overrides.items():
        if k not in dict(noble_recipe._fields_):
            raise TypeError(f"unknown recipe field {k!r}")
        setattr(rc, k, float(v))
    return rc


def noble_lr_multipliers(d_in: int, d_out: int, r: int, recipe: Optional[noble_recipe] = None,
                         groups: int = 1) -> dict:
    """Learning-rate multipliers of W, b, W_down, W_up, M, omega, phi."""
    rc = noble_recipe_defaults() if recipe is None else recipe
    d = make_desc(0, d_in, d_out, r, NOBLE_BF16, 0, groups)
    out = noble_lr_mults()
    st = lib().noble_lr_multipliers(ctypes.byref(d), ctypes.byref(rc), ctypes.byref(out))
    if st != 0:
        raise NobleError(st, "noble_lr_multipliers")
    return {n: getattr(out, n) for n, _ in noble_lr_mults._fields_}


def noble_init_params(W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, seed: int,
                      recipe: Optional[noble_recipe] = None, stream=None, groups: int = 1,
                      activation=0) -> None:
    """Fill the layer's parameter tensors on the device from ``seed``
    (None skips a tensor).  Storage tensors share one dtype (bf16 or f32);
    the 3-layer form's M, omega2, phi2 are its stacked [2, ...] tensors."""
    torch = _torch()
    rc = noble_recipe_defaults() if recipe is None else recipe
    d_in, d_out = W.shape
    R = 0
    for t, dim in ((W_down, 1), (W_up, 0), (omega1, 0), (phi1, 0), (omega2, -1), (phi2, -1)):
        if t is not None:
            R = t.shape[dim]
            break
    if R == 0 and M is not None:
        R = M.shape[-1] * groups
    sh, r = _branch_shapes(d_in, d_out, R, groups, activation)
    dt = _dtype_code(W)
    sd, f32 = W.dtype, torch.float32
    d = make_desc(0, d_in, d_out, r, dt, activation, groups)
    v, v2 = sh["vec"], sh["vec2"]
    dev = W.device
    args = [_ptr(W, "W", sd, (d_in, d_out), dev), _ptr(b, "b", f32, (d_out,), dev),
            _ptr(W_down, "W_down", sd, sh["W_down"], dev), _ptr(omega1, "omega1", f32, v, dev),
            _ptr(phi1, "phi1", f32, v, dev), _ptr(M, "M", sd, sh["M"], dev), _ptr(omega2, "omega2", f32, v2, dev),
            _ptr(phi2, "phi2", f32, v2, dev), _ptr(W_up, "W_up", sd, sh["W_up"], dev)]
    with _on(dev):
        st = lib().noble_init_params(ctypes.byref(d), ctypes.byref(rc), int(seed) & (2 ** 64 - 1), *args,
                                     _stream(stream, dev))
    if st != 0:
        raise NobleError(st, "noble_init_params")


def param_groups(params: dict, lr: float, d_in: int, d_out: int, r: int,
                 recipe: Optional[noble_recipe] = None) -> list:
    """Optimizer parameter groups for one layer: ``params`` maps the names
    W, b, W_down, omega1, phi1, M, omega2, phi2, W_up to tensors (missing or
    None entries are left out); each group's ``lr`` is ``lr`` times the
    layer's multiplier from noble_lr_multipliers."""
    m = noble_lr_multipliers(d_in, d_out, r, recipe)
    which = {"W": "W", "b": "b", "W_down": "W_down", "W_up": "W_up", "M": "M",
             "omega1": "omega", "omega2": "omega", "phi1": "phi", "phi2": "phi"}
    groups = {}
    for name, t in params.items():
        if t is None:
            continue
        if name not in which:
            raise KeyError(f"unknown parameter name {name!r}")
        key = which[name]
        groups.setdefault(key, []).append(t)
    return [{"params": ts, "lr": lr * m[key], "name": key} for key, ts in groups.items()]


# ------------------------------------------------------------ conveniences --

def alloc_workspace(T, d_in, d_out, r, dtype_code, device="cuda", groups: int = 1, forward_only=False,
                    activation=0):
    """(reserve, scratch) uint8 tensors of the required sizes; with
    ``forward_only`` the scratch covers the forward alone."""
    torch = _torch()
    res, scr = noble_linear_workspace_size(T, d_in, d_out, r, dtype_code, activation, groups=groups)
    if forward_only:
        scr = noble_linear_fwd_scratch_size(T, d_in, d_out, r, dtype_code, activation, groups=groups)
    return (torch.empty(max(res, 16), dtype=torch.uint8, device=device),
            torch.empty(max(scr, 16), dtype=torch.uint8, device=device))


def _make_function():
    torch = _torch()

    class NobleLinearFunction(torch.autograd.Function):
        """y = x W + b + sigma(x W_down) W_up with the libnoble kernels, sigma
        the CosNet or another bottleneck activation (``activation``, not
        differentiated), optionally grouped (``groups``).  One-application
        activations take None for M, omega2, phi2.  Parameter gradients are
        computed in float32 and returned in each parameter's dtype."""

        @staticmethod
        def forward(ctx, x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, activation=0, groups=1):
            T, d_in = x.shape
            d_out, R = W.shape[1], W_down.shape[1]
            r = R // groups
            dt = _dtype_code(x)
            act = activation_code(activation)
            reserve, scratch = alloc_workspace(T, d_in, d_out, r, dt, x.device, groups=groups, forward_only=True,
                                               activation=act)
            y = torch.empty((T, d_out), dtype=x.dtype, device=x.device)
            noble_linear_fwd(x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, scratch,
                             activation=act, groups=groups)
            ctx.save_for_backward(x, W, W_down, omega1, phi1, M, omega2, phi2, W_up, reserve)
            ctx.has_bias = b is not None
            ctx.act = act
            ctx.groups = groups
            return y

        @staticmethod
        def backward(ctx, dy):
            x, W, W_down, omega1, phi1, M, omega2, phi2, W_up, reserve = ctx.saved_tensors
            T, d_in = x.shape
            d_out, R = W.shape[1], W_down.shape[1]
            G = ctx.groups
            sh, r = _branch_shapes(d_in, d_out, R, G, ctx.act)
            dev, f32 = x.device, torch.float32
            two = two_layers(ctx.act)
            dy = dy.contiguous().to(x.dtype)
            _, scratch = alloc_workspace(T, d_in, d_out, r, _dtype_code(x), dev, groups=G, activation=ctx.act)
            dx = torch.empty_like(x)
            g = {n: torch.empty(s, dtype=f32, device=dev) for n, s in (
                ("dW", (d_in, d_out)), ("db", (d_out,)), ("dW_down", sh["W_down"]), ("dM", sh["M"]),
                ("dW_up", sh["W_up"]), ("domega1", sh["vec"]), ("dphi1", sh["vec"]), ("domega2", sh["vec2"]),
                ("dphi2", sh["vec2"]))}
            if not two:
                g["dM"] = g["domega2"] = g["dphi2"] = None
            noble_linear_bwd(dy, x, W, W_down, omega1, phi1, M, omega2, phi2, W_up, reserve,
                             dx, g["dW"], g["db"], g["dW_down"], g["dM"], g["dW_up"],
                             g["domega1"], g["dphi1"], g["domega2"], g["dphi2"], scratch, activation=ctx.act,
                             groups=G)
            dM = g["dM"].to(M.dtype) if (two and M is not None) else None
            cast = lambda gr, p: None if p is None or gr is None else gr.to(p.dtype)
            return (dx, g["dW"].to(W.dtype), g["db"] if ctx.has_bias else None, g["dW_down"].to(W_down.dtype),
                    cast(g["domega1"], omega1), cast(g["dphi1"], phi1), dM, cast(g["domega2"], omega2),
                    cast(g["dphi2"], phi2), g["dW_up"].to(W_up.dtype), None, None)

    return NobleLinearFunction


def _make_module():
    torch = _torch()
    Function = __getattr__("NobleLinearFunction")

    class NobleLinear(torch.nn.Module):
        """A linear layer with the NOBLE branch, parameters initialised by the
        paper's recipe (noble_init_params) and its learning-rate multipliers
        available as optimizer groups (param_groups).  Input [..., d_in] in
        the storage dtype; any leading dimensions are tokens.  The storage
        parameters (W, W_down, M, W_up) have the storage dtype; b and the
        frequency / phase vectors are float32.  r = 0 is the plain layer."""

        def __init__(self, d_in, d_out, r, *, bias=True, dtype=None, device="cuda", activation="cosnet",
                     groups=1, seed=0, recipe=None):
            super().__init__()
            dtype = torch.bfloat16 if dtype is None else dtype
            if dtype not in (torch.bfloat16, torch.float32):
                raise TypeError("dtype must be torch.bfloat16 or torch.float32")
            self.d_in, self.d_out, self.r, self.groups = int(d_in), int(d_out), int(r), int(groups)
            self.activation = activation
            self.recipe = recipe
            R = self.groups * self.r
            sh, _ = _branch_shapes(self.d_in, self.d_out, R, self.groups, activation)
            f32 = torch.float32
            P = lambda shape, dt: torch.nn.Parameter(torch.empty(shape, dtype=dt, device=device))
            self.W = P((self.d_in, self.d_out), dtype)
            self.b = P((self.d_out,), f32) if bias else None
            two = two_layers(activation)
            if self.r > 0:
                self.W_down = P(sh["W_down"], dtype)
                self.omega1 = P(sh["vec"], f32)
                self.phi1 = P(sh["vec"], f32)
                self.M = P(sh["M"], dtype) if two else None
                self.omega2 = P(sh["vec2"], f32) if two else None
                self.phi2 = P(sh["vec2"], f32) if two else None
                self.W_up = P(sh["W_up"], dtype)
            self.reset_parameters(seed)

        def _branch(self):
            if self.r == 0:
                return (None,) * 7
            return (self.W_down, self.omega1, self.phi1, self.M, self.omega2, self.phi2, self.W_up)

        @torch.no_grad()
        def reset_parameters(self, seed=0):
            noble_init_params(self.W, self.b, *self._branch(), seed=seed, recipe=self.recipe, groups=self.groups,
                              activation=self.activation)

        def _infer(self, x2):
            # Nothing to differentiate: the forward without the reserve, so H
            # is neither written nor kept.
            T = x2.shape[0]
            _, scratch = alloc_workspace(T, self.d_in, self.d_out, self.r, _dtype_code(x2), x2.device,
                                         groups=self.groups, forward_only=True,
                                         activation=activation_code(self.activation))
            y = torch.empty((T, self.d_out), dtype=x2.dtype, device=x2.device)
            noble_linear_fwd(x2, self.W, self.b, *self._branch(), y, None, scratch,
                             activation=activation_code(self.activation), groups=self.groups)
            return y

        def param_groups(self, lr):
            """Optimizer parameter groups with the layer's learning-rate
            multipliers (Sec. 3.3 Eqs. 3-4, App. A)."""
            names = ("W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up")
            params = {"W": self.W, "b": self.b}
            params.update({n: t for n, t in zip(names, self._branch())})
            return param_groups(params, lr, self.d_in, self.d_out // self.groups, self.r, self.recipe)

        def forward(self, x):
            lead = x.shape[:-1]
            x2 = x.reshape(-1, self.d_in).contiguous()
            if not torch.is_grad_enabled() or not (x2.requires_grad or any(p.requires_grad for p in self.parameters())):
                return self._infer(x2).reshape(*lead, self.d_out)
            if self.r == 0:
                # plain layer: the same library call with no branch
                y = Function.apply(x2, self.W, self.b, torch.empty((self.d_in, 0), dtype=x.dtype, device=x.device),
                                   None, None, None, None, None, torch.empty((0, self.d_out), dtype=x.dtype,
                                                                               device=x.device), 0, 1)
            else:
                y = Function.apply(x2, self.W, self.b, *self._branch(), activation_code(self.activation),
                                   self.groups)
            return y.reshape(*lead, self.d_out)

    return NobleLinear


def __getattr__(name):
    makers = {"NobleLinearFunction": _make_function, "NobleLinear": _make_module}
    if name in makers:
        obj = makers[name]()
        globals()[name] = obj
        return obj
    raise AttributeError(name)
