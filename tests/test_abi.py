"""C ABI of libnoble on the CPU: the library loads, exports every function
include/noble.h declares, sizes workspaces, and rejects bad arguments before
any HIP call.  Every fwd/bwd call here carries exactly one defect that the
validation catches, so nothing can reach a device."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2603_06492_amd import noble

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "noble.h")

OK, NULL, SHAPE, DTYPE, MISAL, WS, BADACT = 0, 1, 2, 3, 4, 5, 8

# fake, 16-byte aligned addresses: never dereferenced because every call below
# fails validation first
FAKE = [0x100000 + 0x1000 * i for i in range(32)]


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(noble_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    names = _declared_functions()
    assert set(names) == {"noble_linear_workspace_size", "noble_linear_fwd_scratch_size", "noble_linear_fwd",
                          "noble_linear_bwd", "noble_profile_next_wgrad", "noble_linear_fwd_static",
                          "noble_status_string", "noble_abi_version", "noble_recipe_defaults",
                          "noble_lr_multipliers", "noble_init_params"}
    L = noble.lib()
    for n in names:
        assert hasattr(L, n), n
    assert L.noble_abi_version() == 5 == noble.ABI_VERSION


def test_status_strings():
    for code, name in noble.STATUS.items():
        assert noble.noble_status_string(code).startswith(name)
    assert "UNKNOWN" in noble.noble_status_string(99)


def _ws(T, di, do, r, dt, groups=1, act=0):
    d = noble.make_desc(T, di, do, r, dt, act, groups)
    a, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    st = noble.lib().noble_linear_workspace_size(ctypes.byref(d), ctypes.byref(a), ctypes.byref(b))
    return st, a.value, b.value


def _proj_split(T, K, J=1):
    """K pieces of the bf16 rank projection run as J jobs (group, 128-rank
    block): workgroups of 128 tokens until 256 are in flight, at least 4
    chunks of 64 per piece, at most 8 pieces."""
    blocks, nkc, s = -(-T // 128), -(-K // 64), 1
    while blocks * s * J < 256 and 2 * s * 4 <= nkc and 2 * s <= 8:
        s *= 2
    return s


def _align(n):
    return -(-n // 256) * 256


def _split_partials(tiles, nk, mn):
    """K split of one weight-gradient product: waves of 256 workgroups x K
    chunks of 64 (1.7 us each) plus (2S + 1) passes over the float32
    partials at 5 TB/s; a split must beat the best so far by 3%."""
    best, bs, s = 0.0, 1, 1
    while s <= 16:
        if s > 1 and s * 8 > nk:
            break
        waves = -(-(tiles * s) // 256)
        cost = waves * (nk / s) * 1.7 + ((2.0 * s + 1) * mn * 4 / 5.0e6 if s > 1 else 0.0)
        if s == 1 or cost < best * 0.97:
            best, bs = cost, s
        s *= 2
    return bs


def _copies(R, nvec=4):
    """bf16 backward: 8 copies of the four frequency / phase gradient vectors
    (six for the 3-layer form)."""
    return _align(nvec * 8 * R * 4)


def _makespan(groups):
    """List scheduling of (count, K chunks) workgroup groups, in launch order,
    on 256 CUs: each workgroup costs 12 + 1.45 x chunks, dispatched one at a
    time to the CU that frees first."""
    import heapq
    cu, end = [0.0] * 256, 0.0
    for n, ch in groups:
        for _ in range(n):
            t = heapq.heappop(cu) + (12.0 + 1.45 * ch)
            heapq.heappush(cu, t)
            end = max(end, t)
    return end


def _rank_parts(di, do, r, groups, hl, nm=1):
    """Float32 elements of one K piece of the rank products' partials:
    (folded, unfolded).  On the bf16 path (hl = 2) dW_down = x^T [dH_hi |
    dH_lo] ([d_in, 2 R]) and dM_g = [C1_hi | C1_lo]_g^T [dH2_hi | dH2_lo]_g
    ([2 r, 2 r]; nm = 2 such products per group for the 3-layer form) are
    stored for any split and folded by the reduction; dW_up [r, d_out / G]
    per group is stored only when split."""
    R, dog = groups * r, do // groups
    return di * hl * R + nm * groups * (hl * r) ** 2, groups * r * dog


def _wgrad_split(T, di, do, r, bk, tile=256, groups=1, hl=2, nm=1):
    """K pieces of dW in the weight-gradient launch.  r = 0: dW alone
    (_split_partials).  r > 0: dW and the rank products (dW_down, dW_up and
    dM, counted whatever the activation) together, minimising the makespan
    plus the partial traffic at 5 MB/us ((2 S + 1) x the output bytes of
    each stored product, S its pieces); both splits from 2^a 3^b up to 16
    with at least 8 K chunks per piece.  Returns (dW split, rank split)."""
    nk = -(-T // bk) if T > 0 else 0
    if nk == 0:
        return 1, 1
    cd = lambda a, b: -(-a // b)
    tiles = cd(di, tile) * cd(do, tile)
    if r == 0:
        return _split_partials(tiles, nk, di * do), 1
    G, R, dog = groups, groups * r, do // groups
    # rank products in launch order; bf16 products of at most 128 rows split
    # each K chunk between the workgroup's two halves (half the chunk time)
    kp = lambda m: tile == 256 and m <= 128
    rank = [(cd(di, tile) * cd(hl * R, tile), kp(di))]
    for _ in range(G):
        rank += [(cd(r, tile) * cd(dog, tile), kp(r)), (nm * cd(hl * r, tile) ** 2, kp(hl * r))]
    folded, unfolded = _rank_parts(di, do, r, groups, hl, nm)
    best, pick = None, (1, 1)
    cands = (1, 2, 3, 4, 6, 8, 12, 16)
    for sw in cands:
        if sw > 1 and sw * 8 > nk:
            break
        for sr in cands:
            if sr > 1 and sr * 8 > nk:
                break
            fp = (max(sr, 1) if hl == 2 else (sr if sr > 1 else 0))
            up = sr if sr > 1 else 0
            traffic = 4.0 * (((2.0 * fp + 1) * folded if fp else 0.0) + ((2.0 * up + 1) * unfolded if up else 0.0))
            t = (_makespan([(tiles * sw, cd(nk, sw))] + [(n * sr, cd(nk, sr) / (2.0 if h else 1.0)) for n, h in rank])
                 + ((2.0 * sw + 1) * di * do * 4 / 5.0e6 if sw > 1 else 0.0)
                 + traffic / 5.0e6)
            if best is None or t < best:
                best, pick = t, (sw, sr)
    return pick


def _wgrad_bytes(T, di, do, r, bk, tile=256, groups=1, hl=2, nm=1):
    """Split-K partials of the weight gradients: dW's region, then one
    region for the rank products (see _rank_parts).  Output tiles are 256
    square on the bf16 path (hl = 2), 128 on the float32 path (hl = 1)."""
    sw, sr = _wgrad_split(T, di, do, r, bk, tile, groups, hl, nm)
    folded, unfolded = _rank_parts(di, do, r, groups, hl, nm)
    fp = max(sr, 1) if hl == 2 else (sr if sr > 1 else 0)
    rank = fp * folded + (sr * unfolded if sr > 1 else 0)
    return (_align(sw * di * do * 4) if sw > 1 else 0) + (_align(rank * 4) if r > 0 and T > 0 and rank else 0)


def _branch_scratch(T, di, do, r, G=1, bf16=True, three=False):
    """Rank-side scratch: C2 [T, R], the bf16 projection partials, then C1,
    dH2, dH [T, hl R] (and the 3-layer form's middle C2 and dH3) and the
    bf16 copies of the frequency / phase gradients."""
    R, es, hl = G * r, (2 if bf16 else 4), (2 if bf16 else 1)
    if r == 0:
        return 0
    part = 0
    if bf16:
        J = G * -(-r // 128)
        S = max(_proj_split(T, di, J), _proj_split(T, do // G, J))
        part = _align(S * T * R * 4)
    nreg, nvec = (5, 6) if three else (3, 4)
    return _align(T * R * es) + part + nreg * _align(hl * T * R * es) + (_copies(R, nvec) if bf16 else 0)


def test_workspace_sizes():
    # forward part first (C2, the bf16 projection partials), then C1, dH2 and
    # dH as high + low bf16 pairs, the copies, and the float32 partials of the
    # weight-gradient products
    st, res, scr = _ws(8192, 2048, 2048, 128, noble.NOBLE_BF16)
    assert _proj_split(8192, 2048) == 4
    assert st == OK and res == 4 * 8192 * 128
    assert scr == (8192 * 128 * 2 + 4 * 8192 * 128 * 4 + 3 * 2 * 8192 * 128 * 2 + _copies(128)
                   + _wgrad_bytes(8192, 2048, 2048, 128, 64))
    st, res, scr = _ws(8192, 2048, 8192, 128, noble.NOBLE_BF16)
    assert st == OK and scr == _branch_scratch(8192, 2048, 8192, 128) + _wgrad_bytes(8192, 2048, 8192, 128, 64)
    st, res, scr = _ws(300, 64, 1024, 40, noble.NOBLE_BF16)
    S = max(_proj_split(300, 64), _proj_split(300, 1024))
    # 5 K chunks: no split, but dW_down and dM store their high + low products
    assert _wgrad_split(300, 64, 1024, 40, 64) == (1, 1)
    assert _wgrad_bytes(300, 64, 1024, 40, 64) == _align((64 * 80 + 80 * 80) * 4)
    assert S == 4 and st == OK
    assert scr == (_align(300 * 40 * 2) + _align(S * 300 * 40 * 4) + 3 * _align(2 * 300 * 40 * 2) + _copies(40)
                   + _align((64 * 80 + 80 * 80) * 4))
    st, res, scr = _ws(256, 64, 64, 8, noble.NOBLE_F32)
    assert st == OK and res == 4 * 256 * 8 and scr == 4 * 256 * 8 * 4
    # float32 tiles are 128 square: 64 tiles of 1024 x 1024 split dW in 4
    # (with 256 tiles it would be 16)
    st, res, scr = _ws(8192, 1024, 1024, 0, noble.NOBLE_F32)
    assert _wgrad_bytes(8192, 1024, 1024, 0, 32, tile=256, hl=1) == 16 * 1024 * 1024 * 4
    assert st == OK and scr == _wgrad_bytes(8192, 1024, 1024, 0, 32, tile=128, hl=1) == 4 * 1024 * 1024 * 4
    st, res, scr = _ws(1000, 64, 64, 0, noble.NOBLE_BF16)
    assert st == OK and res == 0 and scr == _wgrad_bytes(1000, 64, 64, 0, 64) == 2 * 64 * 64 * 4
    st, res, scr = _ws(200, 64, 64, 0, noble.NOBLE_BF16)
    assert st == OK and res == 0 and scr == 0
    # a plain layer still needs the dW partials when it splits
    st, res, scr = _ws(8192, 2048, 2048, 0, noble.NOBLE_BF16)
    assert st == OK and res == 0 and scr == 4 * 2048 * 2048 * 4
    st, res, scr = _ws(0, 64, 64, 32, noble.NOBLE_BF16)
    assert st == OK and res == 0
    # each region of the scratch is 256-byte aligned
    st, res, scr = _ws(3, 64, 64, 8, noble.NOBLE_BF16)
    assert st == OK and scr == 256 + 256 + 3 * 256 + _copies(8) + _align((64 * 16 + 16 * 16) * 4)
    assert noble.lib().noble_linear_workspace_size(None, None, None) == NULL


def _fws(T, di, do, r, dt, groups=1):
    d = noble.make_desc(T, di, do, r, dt, 0, groups)
    b = ctypes.c_size_t(0)
    st = noble.lib().noble_linear_fwd_scratch_size(ctypes.byref(d), ctypes.byref(b))
    return st, b.value


def test_forward_scratch_is_the_prefix():
    """The forward needs only C2 and (bf16) the projection partials: the
    prefix of the full scratch, tens of MB less at the block's shapes."""
    for (T, di, do, r, G, dt) in ((8192, 2048, 2048, 128, 1, noble.NOBLE_BF16),
                                  (8192, 2048, 6144, 128, 3, noble.NOBLE_BF16),
                                  (256, 64, 64, 8, 1, noble.NOBLE_F32), (300, 64, 1024, 40, 1, noble.NOBLE_BF16)):
        st, f = _fws(T, di, do, r, dt, G)
        st2, _, full = _ws(T, di, do, r, dt, G)
        R, bf = G * r, dt == noble.NOBLE_BF16
        part = 0
        if bf:
            J = G * -(-r // 128)
            part = _align(max(_proj_split(T, di, J), _proj_split(T, do // G, J)) * T * R * 4)
        assert st == st2 == OK and f == _align(T * R * (2 if bf else 4)) + part and f < full
    assert _fws(8192, 2048, 2048, 0, noble.NOBLE_BF16) == (OK, 0)
    assert _fws(16, 12, 64, 8, noble.NOBLE_BF16)[0] == SHAPE
    assert noble.lib().noble_linear_fwd_scratch_size(None, None) == NULL


@pytest.mark.parametrize("di,do,r,G,split", [
    (2048, 6144, 128, 1, (1, 1)),   # QKV: 192 dW tiles, the rank problems fill the other 64 CUs
    (2048, 2048, 128, 1, (3, 3)),   # square: 3 dW pieces and 3 rank pieces in one wave
    (2048, 8192, 128, 1, (1, 6)),   # FFN up: one wave of dW, the rank problems split 6 ways after it
    (8192, 2048, 128, 1, (1, 6)),   # FFN down
    (2048, 6144, 128, 3, (1, 1)),   # grouped Q/K/V
    (2048, 2048, 0, 1, (4, 1)),     # the plain square layer: dW alone, 4 pieces
])
def test_weight_gradient_plan_of_the_block(di, do, r, G, split):
    """The dW and rank splits the library plans at T = 8192 (visible in the
    scratch size, which holds both products' partials) match the independent
    one-at-a-time scheduler of _wgrad_split."""
    T = 8192
    assert _wgrad_split(T, di, do, r, 64, 256, G) == split
    st, _, scr = _ws(T, di, do, r, noble.NOBLE_BF16, G)
    assert st == OK and scr == _branch_scratch(T, di, do, r, G) + _wgrad_bytes(T, di, do, r, 64, 256, G)


def test_workspace_sizes_grouped_and_rank_256():
    """Grouped layers size every rank-side region by R = G r, and the
    projection's split counts one job per (group, 128-rank block)."""
    T, di, do, r, G = 8192, 2048, 6144, 128, 3
    st, res, scr = _ws(T, di, do, r, noble.NOBLE_BF16, G)
    R = G * r
    S = max(_proj_split(T, di, G), _proj_split(T, do // G, G))
    assert S == 2   # 64 token blocks x 3 jobs = 192 < 256 workgroups: split K in two
    assert st == OK and res == 4 * T * R
    assert scr == (T * R * 2 + _align(S * T * R * 4) + 3 * 2 * T * R * 2 + _copies(R)
                   + _wgrad_bytes(T, di, do, r, 64, groups=G))
    T, di, do, r = 300, 264, 200, 256
    st, res, scr = _ws(T, di, do, r, noble.NOBLE_BF16)
    S = max(_proj_split(T, di, 2), _proj_split(T, do, 2))
    assert st == OK and res == 4 * T * r
    assert scr == (_align(T * r * 2) + _align(S * T * r * 4) + 3 * _align(2 * T * r * 2) + _copies(r)
                   + _wgrad_bytes(T, di, do, r, 64))


@pytest.mark.parametrize("shape,code", [
    ((-1, 64, 64, 8), SHAPE), ((16, 0, 64, 8), SHAPE), ((16, 12, 64, 8), SHAPE),
    ((16, 64, 60, 8), SHAPE), ((16, 64, 64, 4), SHAPE), ((16, 64, 64, 12), SHAPE),
    ((16, 64, 64, 136), OK), ((16, 64, 64, 256), OK), ((16, 64, 64, 264), SHAPE),
    ((16, 64, 64, -8), SHAPE), ((16, 64, 64, 128), OK),
    ((16, 64, 64, 0), OK), ((1 << 31, 64, 64, 8), SHAPE),
])
def test_shape_validation(shape, code):
    assert _ws(*shape, noble.NOBLE_BF16)[0] == code


def test_f32_rank_limit():
    assert _ws(16, 64, 64, 128, noble.NOBLE_F32)[0] == OK
    assert _ws(16, 64, 64, 136, noble.NOBLE_F32)[0] == SHAPE


TMAX = (1 << 31) - 4096


@pytest.mark.parametrize("shape,dtype,code", [
    # the forward at the largest T: 8388592 token tiles of 256 (bf16, 512
    # threads each) fit one dispatch once, not twice; float32 tiles of 128
    # (256 threads) likewise
    ((TMAX, 8, 256, 8), noble.NOBLE_BF16, OK), ((TMAX, 8, 264, 8), noble.NOBLE_BF16, SHAPE),
    ((TMAX + 1, 8, 8, 0), noble.NOBLE_BF16, SHAPE),
    ((TMAX, 8, 128, 8), noble.NOBLE_F32, OK), ((TMAX, 8, 136, 8), noble.NOBLE_F32, SHAPE),
    ((TMAX, 264, 8, 8), noble.NOBLE_BF16, SHAPE),   # dx
    # dW: 2^20 x (2^19 - 256) is 8384512 tiles, 2^20 x 2^19 is 8388608
    ((1, 1 << 20, (1 << 19) - 256, 0), noble.NOBLE_BF16, OK),
    ((1, 1 << 20, 1 << 19, 0), noble.NOBLE_BF16, SHAPE),
    ((0, 1 << 20, 1 << 20, 0), noble.NOBLE_BF16, SHAPE),
    ((16, 1 << 20, 1 << 20, 0), noble.NOBLE_F32, SHAPE),
    ((16, 1 << 20, (1 << 18) - 128, 0), noble.NOBLE_F32, OK),   # 16769024 tiles of 128
    ((16, 1 << 20, 1 << 18, 0), noble.NOBLE_F32, SHAPE),          # 16777216
])
def test_launch_grid_limits(shape, dtype, code):
    """A dispatch counts its work-items in 32 bits: a call whose GEMM
    launch would pass 2^32 - 1 is rejected (only layers far beyond a GPU's
    memory come near).  The rank-side launches, whose workgroup count grows
    with T, run on two-dimensional grids and set no limit of their own."""
    assert _ws(*shape, dtype)[0] == code


@pytest.mark.parametrize("do,groups,code", [
    (96, 3, OK), (96, 4, OK), (104, 4, SHAPE), (128, 4, OK), (64, 0, OK), (64, 1, OK), (80, 5, SHAPE),
    (64, -1, SHAPE), (72, 3, OK), (64, 3, SHAPE),
])
def test_group_validation(do, groups, code):
    """1 to 4 groups (0 counts as 1), d_out / G a multiple of 8."""
    assert _ws(16, 64, do, 16, noble.NOBLE_BF16, groups)[0] == code


def test_dtype_validation():
    assert _ws(16, 64, 64, 8, 2)[0] == DTYPE
    assert _ws(16, 64, 64, 8, -1)[0] == DTYPE


def _fwd(desc, ptrs, scratch_bytes):
    return noble.lib().noble_linear_fwd(ctypes.byref(desc), *ptrs, scratch_bytes, None)


def _bwd(desc, ptrs, scratch_bytes):
    return noble.lib().noble_linear_bwd(ctypes.byref(desc), *ptrs, scratch_bytes, None)


FWD_ARGS = ["x", "W", "b", "W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up", "y", "reserve", "scratch"]
BWD_ARGS = ["dy", "x", "W", "W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up", "reserve", "dx", "dW",
            "db", "dW_down", "dM", "dW_up", "domega1", "dphi1", "domega2", "dphi2", "scratch"]
NULLABLE = {"b", "db"}
FWD_NULLABLE = NULLABLE | {"reserve"}   # NULL reserve: inference-only forward


@pytest.mark.parametrize("which", FWD_ARGS)
def test_fwd_rejects_null_and_misaligned(which):
    d = noble.make_desc(64, 64, 64, 16, noble.NOBLE_BF16)
    _, scr = noble.noble_linear_workspace_size(64, 64, 64, 16, noble.NOBLE_BF16)
    ptrs = list(FAKE[:len(FWD_ARGS)])
    i = FWD_ARGS.index(which)
    if which not in FWD_NULLABLE:
        ptrs[i] = None
        assert _fwd(d, ptrs, scr) == NULL
    ptrs[i] = FAKE[i] + 4
    assert _fwd(d, ptrs, scr) == MISAL


@pytest.mark.parametrize("which", BWD_ARGS)
def test_bwd_rejects_null_and_misaligned(which):
    d = noble.make_desc(64, 64, 64, 16, noble.NOBLE_F32)
    _, scr = noble.noble_linear_workspace_size(64, 64, 64, 16, noble.NOBLE_F32)
    ptrs = list(FAKE[:len(BWD_ARGS)])
    i = BWD_ARGS.index(which)
    if which not in NULLABLE:
        ptrs[i] = None
        assert _bwd(d, ptrs, scr) == NULL
    ptrs[i] = FAKE[i] + 8
    assert _bwd(d, ptrs, scr) == MISAL


def test_workspace_too_small():
    d = noble.make_desc(64, 64, 64, 16, noble.NOBLE_BF16)
    _, scr = noble.noble_linear_workspace_size(64, 64, 64, 16, noble.NOBLE_BF16)
    fscr = noble.noble_linear_fwd_scratch_size(64, 64, 64, 16, noble.NOBLE_BF16)
    assert 0 < fscr < scr
    assert _fwd(d, FAKE[:13], fscr - 1) == WS
    assert _bwd(d, FAKE[:22], scr - 256) == WS


def test_bad_desc_rejected_by_fwd_and_bwd():
    for d, code in ((noble.make_desc(64, 64, 64, 16, 7), DTYPE), (noble.make_desc(64, 64, 64, 20, 0), SHAPE)):
        assert _fwd(d, FAKE[:13], 1 << 30) == code
        assert _bwd(d, FAKE[:22], 1 << 30) == code
    assert noble.lib().noble_linear_fwd(None, *FAKE[:13], 0, None) == NULL


def test_plain_linear_branch_pointers_unchecked():
    """With r = 0 the branch pointers are ignored (may be NULL); a NULL x is
    still rejected, proving validation ran past them."""
    d = noble.make_desc(64, 64, 64, 0, noble.NOBLE_BF16)
    ptrs = list(FAKE[:13])
    for k in ("W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up", "reserve", "scratch"):
        ptrs[FWD_ARGS.index(k)] = None
    ptrs[0] = None
    assert _fwd(d, ptrs, 0) == NULL


def test_plain_backward_needs_scratch_when_dW_splits():
    """r = 0 with 1000 tokens splits dW over K, so the backward needs the
    partials scratch even without a branch: NULL or short scratch is rejected
    before any HIP call."""
    d = noble.make_desc(1000, 64, 64, 0, noble.NOBLE_BF16)
    _, scr = noble.noble_linear_workspace_size(1000, 64, 64, 0, noble.NOBLE_BF16)
    assert scr > 0
    ptrs = list(FAKE[:22])
    for k in ("W_down", "omega1", "phi1", "M", "omega2", "phi2", "W_up", "reserve", "dW_down", "dM", "dW_up",
              "domega1", "dphi1", "domega2", "dphi2"):
        ptrs[BWD_ARGS.index(k)] = None
    ptrs[BWD_ARGS.index("scratch")] = None
    assert _bwd(d, ptrs, scr) == NULL
    ptrs[BWD_ARGS.index("scratch")] = FAKE[21]
    assert _bwd(d, ptrs, scr - 256) == WS


# ----------------------------------------------------------- activations --

def _header_enum(prefix):
    src = open(HEADER).read()
    return {m.group(1): int(m.group(2)) for m in re.finditer(prefix + r"([A-Z_0-9]+)\s*=\s*(\d+)", src)}


def test_activation_codes_match_header_and_oracle():
    """The binding's names and codes are the header's enum, and name the same
    (f, applications) pairs as the oracle's activation table."""
    import oracle
    hdr = _header_enum("NOBLE_ACT_")
    assert {k.lower(): v for k, v in hdr.items()} == noble.ACTIVATIONS
    assert set(noble.ACTIVATIONS) == set(oracle.ACTIVATIONS)
    for name, (_, layers) in oracle.ACTIVATIONS.items():
        assert noble.layers(name) == layers, name
        assert noble.two_layers(name) == (layers >= 2), name
    assert _header_enum("NOBLE_ERR_")["BAD_ACTIVATION"] == BADACT


@pytest.mark.parametrize("act", [-1, 9, 1 << 20])
def test_bad_activation_rejected(act):
    d = noble.make_desc(64, 64, 64, 16, noble.NOBLE_BF16, act)
    a, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert noble.lib().noble_linear_workspace_size(ctypes.byref(d), ctypes.byref(a), ctypes.byref(b)) == BADACT
    assert _fwd(d, FAKE[:13], 1 << 30) == BADACT
    assert _bwd(d, FAKE[:22], 1 << 30) == BADACT
    with pytest.raises(ValueError):
        noble.activation_code("relu")


def test_workspace_depends_only_on_the_three_layer_form():
    """Every one- and two-application activation shares one size; the
    3-layer form adds the middle C2 and dH3 regions, two more copies of the
    gradient vectors (bf16) and its second dM product's partials."""
    for dt in (noble.NOBLE_BF16, noble.NOBLE_F32):
        sizes = {noble.noble_linear_workspace_size(300, 64, 1024, 40, dt, a) for a in noble.ACTIVATIONS
                 if a != "cosnet3"}
        assert len(sizes) == 1
        three = noble.noble_linear_workspace_size(300, 64, 1024, 40, dt, "cosnet3")
        assert three[0] == sizes.pop()[0] and three[1] > 0
    for (T, di, do, r, G) in ((300, 64, 1024, 40, 1), (8192, 2048, 6144, 128, 3), (8192, 2048, 8192, 128, 1)):
        bf = _branch_scratch(T, di, do, r, G, True, True) + _wgrad_bytes(T, di, do, r, 64, 256, G, 2, 2)
        assert _ws(T, di, do, r, noble.NOBLE_BF16, G, 8) == (OK, 4 * T * G * r, bf)
        f32 = _branch_scratch(T, di, do, r, G, False, True) + _wgrad_bytes(T, di, do, r, 32, 128, G, 1, 2)
        assert _ws(T, di, do, r, noble.NOBLE_F32, G, 8) == (OK, 4 * T * G * r, f32)
    # both mixing matrices stay in LDS: r <= 128 on either path
    assert _ws(16, 64, 64, 128, noble.NOBLE_BF16, 1, 8)[0] == OK
    assert _ws(16, 64, 64, 136, noble.NOBLE_BF16, 1, 8)[0] == SHAPE


ONE = [a for a in noble.ACTIVATIONS if not noble.two_layers(a)]
TWO = [a for a in noble.ACTIVATIONS if noble.two_layers(a)]


@pytest.mark.parametrize("act", ONE)
def test_one_layer_second_layer_pointers_optional(act):
    """One application reads no M, omega2, phi2 and writes no dM, domega2,
    dphi2: NULL passes their checks (a misaligned pointer checked after them
    is what fails), a misaligned one is still rejected."""
    d = noble.make_desc(64, 64, 64, 16, noble.NOBLE_BF16, act)
    _, scr = noble.noble_linear_workspace_size(64, 64, 64, 16, noble.NOBLE_BF16, act)
    ptrs = list(FAKE[:13])
    for k in ("M", "omega2", "phi2"):
        ptrs[FWD_ARGS.index(k)] = None
    ptrs[FWD_ARGS.index("reserve")] = FAKE[0] + 4
    assert _fwd(d, ptrs, scr) == MISAL
    ptrs[FWD_ARGS.index("reserve")] = FAKE[0]
    ptrs[FWD_ARGS.index("M")] = FAKE[0] + 4
    assert _fwd(d, ptrs, scr) == MISAL
    ptrs = list(FAKE[:22])
    for k in ("M", "omega2", "phi2", "dM", "domega2", "dphi2"):
        ptrs[BWD_ARGS.index(k)] = None
    ptrs[BWD_ARGS.index("scratch")] = FAKE[0] + 4
    assert _bwd(d, ptrs, scr) == MISAL
    ptrs[BWD_ARGS.index("scratch")] = FAKE[0]
    ptrs[BWD_ARGS.index("dM")] = FAKE[0] + 8
    assert _bwd(d, ptrs, scr) == MISAL


@pytest.mark.parametrize("act", TWO)
def test_two_layer_second_layer_pointers_required(act):
    d = noble.make_desc(64, 64, 64, 16, noble.NOBLE_F32, act)
    _, scr = noble.noble_linear_workspace_size(64, 64, 64, 16, noble.NOBLE_F32, act)
    for k in ("M", "omega2", "phi2"):
        ptrs = list(FAKE[:13])
        ptrs[FWD_ARGS.index(k)] = None
        assert _fwd(d, ptrs, scr) == NULL, k
    for k in ("M", "omega2", "phi2", "dM", "domega2", "dphi2"):
        ptrs = list(FAKE[:22])
        ptrs[BWD_ARGS.index(k)] = None
        assert _bwd(d, ptrs, scr) == NULL, k


def test_reserved_field_must_be_zero():
    d = noble.make_desc(16, 64, 64, 8, noble.NOBLE_BF16)
    d.reserved = 1
    a, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert noble.lib().noble_linear_workspace_size(ctypes.byref(d), ctypes.byref(a), ctypes.byref(b)) == SHAPE
    assert _fwd(d, FAKE[:13], 1 << 30) == SHAPE


def test_workspace_queries_from_many_threads():
    """The weight-gradient plan behind the scratch size is cached per thread
    (eight entries): many threads querying more shapes than a cache holds,
    in different orders, get the single-threaded answers."""
    from concurrent.futures import ThreadPoolExecutor
    shapes = [(T, di, do, r, G) for T in (1000, 8192, 40000) for (di, do, r, G) in
              ((2048, 6144, 128, 3), (2048, 2048, 128, 1), (8192, 2048, 64, 1), (512, 384, 0, 1))]
    want = {s: _ws(*s[:4], noble.NOBLE_BF16, s[4]) for s in shapes}

    def worker(seed):
        rng = np.random.default_rng(seed)
        bad = 0
        for _ in range(300):
            s = shapes[rng.integers(len(shapes))]
            bad += _ws(*s[:4], noble.NOBLE_BF16, s[4]) != want[s]
        return bad

    with ThreadPoolExecutor(8) as ex:
        assert sum(ex.map(worker, range(16))) == 0


def test_static_forward_rejects_before_any_hip_call():
    """noble_linear_fwd_static checks like noble_linear_fwd and rejects a
    layer whose forward scratch exceeds the static array
    (NOBLE_STATIC_SCRATCH_BYTES, 64 MiB) with NOBLE_ERR_WORKSPACE_TOO_SMALL;
    none of these calls reaches the device."""
    L = noble.lib()
    limit = 64 << 20
    fits, big = 80000, 90000
    assert _fws(fits, 2048, 2048, 128, noble.NOBLE_BF16)[1] <= limit < _fws(big, 2048, 2048, 128, noble.NOBLE_BF16)[1]
    d = noble.make_desc(big, 2048, 2048, 128, noble.NOBLE_BF16)
    assert L.noble_linear_fwd_static(ctypes.byref(d), *FAKE[:12], None) == WS
    d = noble.make_desc(64, 64, 64, 16, noble.NOBLE_BF16)
    ptrs = list(FAKE[:12])
    ptrs[0] = None
    assert L.noble_linear_fwd_static(ctypes.byref(d), *ptrs, None) == NULL
    ptrs = list(FAKE[:12])
    ptrs[3] = FAKE[3] + 8
    assert L.noble_linear_fwd_static(ctypes.byref(d), *ptrs, None) == MISAL
    assert L.noble_linear_fwd_static(None, *FAKE[:12], None) == NULL
    d = noble.make_desc(64, 64, 64, 20, noble.NOBLE_BF16)
    assert L.noble_linear_fwd_static(ctypes.byref(d), *FAKE[:12], None) == SHAPE
