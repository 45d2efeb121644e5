// NOBLE-CosNet linear layer kernels for gfx950: the zero fill used before the
// atomically reduced gradients, and the float32-path chain kernels (the bf16
// path uses the fused branch kernels of noble_skinny.hpp).
//
// Forward (Eq. 1 with the CosNet of Eq. 2):
//   fwd_chain_kernel : H = x W_down (MFMA), C1 = cos(H w1 + p1), H2 = C1 M
//                      (MFMA from LDS), C2 = cos(H2 w2 + p2).  Writes H (f32,
//                      the reserve) and C2 (storage type, scratch).
//   gemm_kernel      : y = [x | C2] [W ; W_up] + b  (the rank-r up-projection
//                      is a K-extension of the main product).
// Backward (chain rule, cosines recomputed from H):
//   bwd_chain_kernel : dC2 = dy W_up^T (MFMA), then the chain backwards with
//                      both r x r mixings on MFMA; writes C1, C2, dH2, dH
//                      (scratch) and reduces dw/dp with wave shuffles and one
//                      atomic per column per wave.
//   gemm_kernel      : dx = [dy | dH] [W^T ; W_down^T]      (K-extension)
//   gemm_kernel      : dW = x^T dy, dW_down = x^T dH, dW_up = C2^T dy,
//                      dM = C1^T dH2 as one grouped launch with split-K over
//                      tokens; db = column sums of dy, taken from the dy tiles
//                      the dW problem already stages.
// The chain kernels are instantiated per bottleneck activation (cos, tanh,
// LeakyReLU, GELU) and for the one-application form C2 = f(H w1 + p1), which
// has no M and therefore no mixing products and no dM.
#pragma once

#include "noble_act.hpp"
#include "noble_gemm.hpp"
#include "noble_tiles.hpp"

namespace noble {

// ------------------------------------------------------------- launch grids --

// A dispatch counts its work-items in 32 bits per grid dimension.  The
// launches whose workgroup count grows with T (the chain, projection and
// branch kernels: up to 2^28 workgroups at the largest T) therefore run on
// rows of kGridRow workgroups: workgroup b sits at (b % kGridRow, b /
// kGridRow), and the surplus of the last row exits on entry.
constexpr int kGridRow = 65536;
__device__ __forceinline__ int64_t flat_block() { return (int64_t)blockIdx.y * gridDim.x + blockIdx.x; }

// ---------------------------------------------------------------- zero fill --

constexpr int kMaxZero = 24;
struct ZeroList {
    float* ptr[kMaxZero];
    int64_t n[kMaxZero];
    int count;
};

__global__ __launch_bounds__(256) void zero_kernel(ZeroList z) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int s = 0; s < z.count; ++s) {
        float* p = z.ptr[s];
        const int64_t n = z.n[s];
        const int64_t n4 = n >> 2;
        for (int64_t i = gid; i < n4; i += stride)
            reinterpret_cast<f32x4*>(p)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int64_t i = (n4 << 2) + gid; i < n; i += stride) p[i] = 0.f;
    }
}

// Split-K partial sums: out[i] = sum over p < S of part[p * n + i], for up to
// kMaxZero float arrays.  A folded array sums, besides the slices, two or
// four blocks of each slice: its partial products were computed over
// operands split into high and low bf16 parts, laid side by side.  With
// out = [rows][F] (F = fw[s]):
//  - fold bit 0 (columns): a slice row holds 2F values, out[i][j] adds
//    elements j and F + j of it;
//  - fold bit 1 (rows): a slice holds 2 rows blocks, out[i][j] adds rows i
//    and rows + i.
struct ReduceList {
    const float* part[kMaxZero];
    float* out[kMaxZero];
    int64_t n[kMaxZero];
    int S[kMaxZero];
    int fw[kMaxZero];          // folded arrays: the output row width F (a multiple of 4)
    int fold[kMaxZero];        // 0, or the fold bits above
    int first[kMaxZero + 1];   // array s owns blocks first[s] .. first[s + 1] - 1
    int count;
};

constexpr int kMaxReduceSlices = 16;

// out[i] = part[i] + part[n + i] + ... + part[(S - 1) n + i] for each array,
// every array on its own range of blocks.  The S loads of an element are
// issued together (S is at most kMaxReduceSlices) and added in slice order:
// a loop that waits on each slice in turn makes the few-element arrays
// (the frequency / phase copies) a chain of dependent L2 round trips.
// Folded arrays add, per slice, the fold blocks of the element in a fixed
// order (high-high, high-low, low-high, low-low).
__global__ __launch_bounds__(256) void reduce_kernel(ReduceList z) {
    int s = 0;
    while (s + 1 < z.count && (int)blockIdx.x >= z.first[s + 1]) ++s;
    const float* p = z.part[s];
    float* o = z.out[s];
    const int64_t n = z.n[s];
    const int S = z.S[s];
    const int64_t stride = (int64_t)(z.first[s + 1] - z.first[s]) * blockDim.x;
    const int64_t gid = (int64_t)(blockIdx.x - z.first[s]) * blockDim.x + threadIdx.x;
    const int64_t n4 = n >> 2;
    const int fold = z.fold[s];
    if (fold != 0) {
        const int64_t F = z.fw[s], rows = n / F;
        const int64_t pw = (fold & 1) ? 2 * F : F;                 // slice row width
        const int64_t sstride = ((fold & 2) ? 2 * rows : rows) * pw;
        const int64_t col_off = (fold & 1) ? F : 0, row_off = (fold & 2) ? rows * pw : 0;
        for (int64_t i = gid; i < n4; i += stride) {
            const int64_t e = 4 * i, row = e / F, col = e - row * F;
            const float* q = p + row * pw + col;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            for (int sl = 0; sl < S; ++sl, q += sstride) {
                f32x4 v[4];
                v[0] = *reinterpret_cast<const f32x4*>(q);
                v[1] = (fold & 1) ? *reinterpret_cast<const f32x4*>(q + col_off) : f32x4{0.f, 0.f, 0.f, 0.f};
                v[2] = (fold & 2) ? *reinterpret_cast<const f32x4*>(q + row_off) : f32x4{0.f, 0.f, 0.f, 0.f};
                v[3] = (fold == 3) ? *reinterpret_cast<const f32x4*>(q + row_off + col_off)
                                   : f32x4{0.f, 0.f, 0.f, 0.f};
                acc += v[0];
                acc += v[1];
                acc += v[2];
                acc += v[3];
            }
            reinterpret_cast<f32x4*>(o)[i] = acc;
        }
        return;
    }
    for (int64_t i = gid; i < n4; i += stride) {
        f32x4 v[kMaxReduceSlices];
#pragma unroll
        for (int q = 0; q < kMaxReduceSlices; ++q)
            if (q < S) v[q] = reinterpret_cast<const f32x4*>(p + q * n)[i];
        f32x4 acc = v[0];
#pragma unroll
        for (int q = 1; q < kMaxReduceSlices; ++q)
            if (q < S) acc += v[q];
        reinterpret_cast<f32x4*>(o)[i] = acc;
    }
    for (int64_t i = (n4 << 2) + gid; i < n; i += stride) {
        float v[kMaxReduceSlices];
#pragma unroll
        for (int q = 0; q < kMaxReduceSlices; ++q)
            if (q < S) v[q] = p[q * n + i];
        float acc = v[0];
#pragma unroll
        for (int q = 1; q < kMaxReduceSlices; ++q)
            if (q < S) acc += v[q];
        o[i] = acc;
    }
}

// ------------------------------------------------------------- chain kernels --

struct ChainArgs {
    Operand A;          // fwd: x [T, d_in];  bwd: dy [T, d_out]   (K-major)
    Operand B;          // fwd: W_down [d_in, r] (MN-major);  bwd: W_up as W_up^T (K-major)
    const char* M;      // [r, r] storage type
    const char* M2;     // 3-layer form: the second mixing matrix [r, r]
    const float* w1;
    const float* p1;
    const float* w2;
    const float* p2;
    const float* w3;    // 3-layer form
    const float* p3;
    float* H;           // reserve [T, r]: written by fwd, read by bwd
    char* C1s;          // scratch [T, r] storage type (bwd)
    char* C2s;          // scratch [T, r] storage type: the branch output (C2, or C3)
    char* dH2s;         // scratch [T, r] storage type (bwd)
    char* dHs;          // scratch [T, r] storage type (bwd)
    char* C2ms;         // scratch [T, r] storage type (bwd, 3-layer form): the middle C2
    char* dH3s;         // scratch [T, r] storage type (bwd, 3-layer form)
    float* dw1;
    float* dp1;
    float* dw2;
    float* dp2;
    float* dw3;         // 3-layer form
    float* dp3;
    int T, r, nk;
    int ldr;            // row stride of H and of the scratch arrays (G r for grouped layers)
};

constexpr int kChainRows = 32;  // tokens per workgroup in the chain kernels

template <typename E, int RP>
struct ChainShape {
    static constexpr int BK = Elt<E>::BK;
    static constexpr int NKB = RP / BK;     // K chunks of the r x r mixing
    static constexpr int TN = RP / 32;      // 16-wide tiles per wave (waves 2 x 2)
    static constexpr int MAIN = 2 * (kChainRows + RP) * kRowBytes;
    static constexpr int MIX = NKB * (kChainRows + RP) * kRowBytes;
    static constexpr int LDS = MAIN > MIX ? MAIN : MIX;
    static_assert(RP % BK == 0, "RP must be a multiple of the K chunk");
};

// Element (row, col) of a kChainRows x RP operand tile laid out as NKB K chunks.
template <typename E>
__device__ __forceinline__ int tile_elem_off(int row, int col, int rows) {
    constexpr int BK = Elt<E>::BK, VEC = Elt<E>::VEC;
    return (col / BK) * rows * kRowBytes + lds_off(row, (col % BK) / VEC) + (col % VEC) * (int)sizeof(E);
}

// Stage the r x r matrix M as the B operand of a mixing product, all K chunks.
// KMAJ = false: B(k, n) = M[k][n] (for C1 M).  KMAJ = true: B(k, n) = M[n][k]
// (for dH2 M^T).
template <typename E, int RP, bool KMAJ>
__device__ __forceinline__ void stage_mix_matrix(const char* M, int r, char* dst, int tid) {
    Operand om;
    om.s[0].ptr = M;
    om.s[0].ld = r;
    om.s[0].klen = r;
    om.s[1] = om.s[0];
    om.nk1 = 1 << 30;
    om.rows = r;
#pragma unroll
    for (int kb = 0; kb < ChainShape<E, RP>::NKB; ++kb) {
        Stage<E, RP, KMAJ> st;
        st.load(om, 0, kb, tid);
        st.store(dst + kb * RP * kRowBytes, tid);
    }
}

// Sum over the 16-row slab of a wave, per column; lanes 0..15 return the total.
__device__ __forceinline__ float wave_colsum(float x) {
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

// f(acc w + p) of the wave's tile as the A operand of the next mixing
// product (element type E in LDS), or, with `out`, stored to the [T, ldr]
// array out.
template <typename E, int TN, Act F>
__device__ __forceinline__ void chain_apply(const f32x4 (&acc)[1][TN], const float* w, const float* p, int r, int wm0,
                                            int wn0, int r16, int g, int m0, int T, int ldr, char* tile, char* out) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = wn0 + 16 * j + r16;
        const bool cv = col < r;
        const float ww = cv ? w[col] : 0.f, pp = cv ? p[col] : 0.f;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = wm0 + 4 * g + v, grow = m0 + row;
            const float c = cv ? act_value<F, false>(acc[0][j][v] * ww + pp) : 0.f;
            if (tile)
                *reinterpret_cast<E*>(tile + tile_elem_off<E>(row, col, kChainRows)) = to_elt<E>(c);
            else if (cv && grow < T)
                reinterpret_cast<E*>(out)[(int64_t)grow * ldr + col] = to_elt<E>(c);
        }
    }
}

// acc = the tile in LDS (A operand, all NKB K chunks) times the staged M.
template <typename E, int RP>
__device__ __forceinline__ void chain_mix(const char* Cb, const char* Mb, int wm0, int wn0, int lane,
                                          f32x4 (&acc)[1][ChainShape<E, RP>::TN]) {
    using S = ChainShape<E, RP>;
#pragma unroll
    for (int j = 0; j < S::TN; ++j) acc[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < S::NKB; ++kb)
        mma_chunk<E, 1, S::TN>(Cb + kb * kChainRows * kRowBytes, Mb + kb * RP * kRowBytes, wm0, wn0, lane, acc);
}

// Forward chain for activation F with L applications: L = 2 with M between
// them (CosNet for F = Cos), L = 1 (C2 = f(H w1 + p1); M, w2, p2 unused),
// L = 3 with M2 between the second and third (the 3-layer CosNet).
template <typename E, int RP, Act F, int L>
__global__ __launch_bounds__(kThreads) void fwd_chain_kernel(ChainArgs a) {
    using S = ChainShape<E, RP>;
    constexpr int TN = S::TN;
    __shared__ __attribute__((aligned(16))) char lds[S::LDS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r16 = lane & 15, g = lane >> 4;
    const int wm0 = (wave >> 1) * 16, wn0 = (wave & 1) * (RP / 2);
    const int64_t wg = flat_block();
    if (wg * kChainRows >= a.T) return;
    const int m0 = (int)wg * kChainRows;
    const int r = a.r;

    f32x4 acc[1][TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    mainloop<E, kChainRows, RP, 2, 2, true, false>(a.A, a.B, m0, 0, 0, a.nk, lds, acc);

    char* Cb = lds;
    char* Mb = lds + S::NKB * kChainRows * kRowBytes;
    if constexpr (L >= 2) stage_mix_matrix<E, RP, false>(a.M, r, Mb, tid);

    // H -> reserve
    if (a.H) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = wn0 + 16 * j + r16;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int grow = m0 + wm0 + 4 * g + v;
                if (col < r && grow < a.T) a.H[(int64_t)grow * a.ldr + col] = acc[0][j][v];
            }
        }
    }
    // C1 = f(H w1 + p1) -> LDS (A operand of the mixing), or straight to the
    // output for one application
    chain_apply<E, TN, F>(acc, a.w1, a.p1, r, wm0, wn0, r16, g, m0, a.T, a.ldr, L >= 2 ? Cb : nullptr, a.C2s);
    if constexpr (L == 1) return;
    __syncthreads();
    f32x4 mix[1][TN];
    chain_mix<E, RP>(Cb, Mb, wm0, wn0, lane, mix);   // H2 = C1 M
    if constexpr (L == 3) {
        __syncthreads();   // every wave is done with C1 and M in LDS
        stage_mix_matrix<E, RP, false>(a.M2, r, Mb, tid);
        chain_apply<E, TN, F>(mix, a.w2, a.p2, r, wm0, wn0, r16, g, m0, a.T, a.ldr, Cb, nullptr);   // C2 -> LDS
        __syncthreads();
        chain_mix<E, RP>(Cb, Mb, wm0, wn0, lane, mix);   // H3 = C2 M2
        // C3 = f(H3 w3 + p3) -> scratch
        chain_apply<E, TN, F>(mix, a.w3, a.p3, r, wm0, wn0, r16, g, m0, a.T, a.ldr, nullptr, a.C2s);
    } else {
        // C2 = f(H2 w2 + p2) -> scratch
        chain_apply<E, TN, F>(mix, a.w2, a.p2, r, wm0, wn0, r16, g, m0, a.T, a.ldr, nullptr, a.C2s);
    }
}

// One layer of the backward through A = acc w + p, C = f(A), for the wave's
// tile: with the output gradient dC (registers), dA = f'(A) dC, the column
// sums of dA acc and dA are added to dw and dp, dA w goes to LDS (the A
// operand of the next gradient mixing product) and to dst; C = f(A) goes to
// cdst (when given).
template <typename E, int TN, Act F>
__device__ __forceinline__ void chain_back_layer(const f32x4 (&acc)[1][TN], const f32x4 (&dC)[1][TN], const float* w,
                                                 const float* p, float* dw, float* dp, int r, int wm0, int wn0, int r16,
                                                 int g, int m0, int T, int ldr, char* tile, char* dst, char* cdst) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = wn0 + 16 * j + r16;
        const bool cv = col < r;
        const float ww = cv ? w[col] : 0.f, pp = cv ? p[col] : 0.f;
        float sw = 0.f, sp = 0.f;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = wm0 + 4 * g + v, grow = m0 + row;
            const bool ok = cv && grow < T;
            float f = 0.f, d = 0.f;
            if (cv) act_value_slope<F, false>(acc[0][j][v] * ww + pp, f, d);
            const float da = ok ? d * dC[0][j][v] : 0.f;
            sw += da * acc[0][j][v];
            sp += da;
            const E dh = to_elt<E>(da * ww);
            *reinterpret_cast<E*>(tile + tile_elem_off<E>(row, col, kChainRows)) = dh;
            if (ok) {
                if (cdst) reinterpret_cast<E*>(cdst)[(int64_t)grow * ldr + col] = to_elt<E>(f);
                reinterpret_cast<E*>(dst)[(int64_t)grow * ldr + col] = dh;
            }
        }
        sw = wave_colsum(sw);
        sp = wave_colsum(sp);
        if (g == 0 && cv) {
            unsafeAtomicAdd(dw + col, sw);
            unsafeAtomicAdd(dp + col, sp);
        }
    }
}

// Backward chain, same forms as fwd_chain_kernel.  The one-application form
// writes C2 and dH only.
template <typename E, int RP, Act F, int L>
__global__ __launch_bounds__(kThreads) void bwd_chain_kernel(ChainArgs a) {
    using S = ChainShape<E, RP>;
    constexpr int TN = S::TN;
    __shared__ __attribute__((aligned(16))) char lds[S::LDS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r16 = lane & 15, g = lane >> 4;
    const int wm0 = (wave >> 1) * 16, wn0 = (wave & 1) * (RP / 2);
    const int64_t wg = flat_block();
    if (wg * kChainRows >= a.T) return;
    const int m0 = (int)wg * kChainRows;
    const int r = a.r;

    // the output's gradient dy W_up^T
    f32x4 dc2[1][TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) dc2[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    mainloop<E, kChainRows, RP, 2, 2, true, true>(a.A, a.B, m0, 0, 0, a.nk, lds, dc2);

    char* Cb = lds;
    char* Mb = lds + S::NKB * kChainRows * kRowBytes;
    if constexpr (L >= 2) stage_mix_matrix<E, RP, false>(a.M, r, Mb, tid);

    // Recompute A1 = H w1 + p1 and C1 = f(A1) (-> LDS and scratch, or to the
    // output for one application); keep H and f'(A1).
    float hr[TN][4], d1[TN][4];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = wn0 + 16 * j + r16;
        const bool cv = col < r;
        const float w = cv ? a.w1[col] : 0.f, p = cv ? a.p1[col] : 0.f;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = wm0 + 4 * g + v, grow = m0 + row;
            const bool ok = cv && grow < a.T;
            const float h = ok ? a.H[(int64_t)grow * a.ldr + col] : 0.f;
            float f = 0.f, d = 0.f;
            if (cv) act_value_slope<F, false>(h * w + p, f, d);
            hr[j][v] = h;
            d1[j][v] = d;
            const E c1 = to_elt<E>(f);
            if constexpr (L >= 2) {
                *reinterpret_cast<E*>(Cb + tile_elem_off<E>(row, col, kChainRows)) = c1;
                if (ok) reinterpret_cast<E*>(a.C1s)[(int64_t)grow * a.ldr + col] = c1;
            } else if (ok) {
                reinterpret_cast<E*>(a.C2s)[(int64_t)grow * a.ldr + col] = c1;
            }
        }
    }

    // dC1: the output's gradient itself (one application), or back through
    // the mixing layers
    f32x4 dc1[1][TN];
    if constexpr (L == 1) {
#pragma unroll
        for (int j = 0; j < TN; ++j) dc1[0][j] = dc2[0][j];
    } else {
        __syncthreads();
        f32x4 h2[1][TN];
        chain_mix<E, RP>(Cb, Mb, wm0, wn0, lane, h2);   // H2 = C1 M
        __syncthreads();  // every wave is done with C1 and M in LDS

        f32x4 dcm[1][TN];   // gradient of C2
        if constexpr (L == 3) {
            // C2 = f(H2 w2 + p2) -> LDS and scratch (the middle layer's C2)
            stage_mix_matrix<E, RP, false>(a.M2, r, Mb, tid);
            chain_apply<E, TN, F>(h2, a.w2, a.p2, r, wm0, wn0, r16, g, m0, a.T, a.ldr, Cb, nullptr);
            chain_apply<E, TN, F>(h2, a.w2, a.p2, r, wm0, wn0, r16, g, m0, a.T, a.ldr, nullptr, a.C2ms);
            __syncthreads();
            f32x4 h3[1][TN];
            chain_mix<E, RP>(Cb, Mb, wm0, wn0, lane, h3);   // H3 = C2 M2
            __syncthreads();
            stage_mix_matrix<E, RP, true>(a.M2, r, Mb, tid);
            // C3 -> output; dA3 = f'(A3) dC3; dw3, dp3; dH3 -> LDS and scratch
            chain_back_layer<E, TN, F>(h3, dc2, a.w3, a.p3, a.dw3, a.dp3, r, wm0, wn0, r16, g, m0, a.T, a.ldr, Cb,
                                       a.dH3s, a.C2s);
            __syncthreads();
            chain_mix<E, RP>(Cb, Mb, wm0, wn0, lane, dcm);   // dC2 = dH3 M2^T
            __syncthreads();
            stage_mix_matrix<E, RP, true>(a.M, r, Mb, tid);
            // C2 was stored above; dA2, dH2
            chain_back_layer<E, TN, F>(h2, dcm, a.w2, a.p2, a.dw2, a.dp2, r, wm0, wn0, r16, g, m0, a.T, a.ldr, Cb,
                                       a.dH2s, nullptr);
        } else {
            stage_mix_matrix<E, RP, true>(a.M, r, Mb, tid);
            // C2 -> output; dA2 = f'(A2) dC2; dw2, dp2; dH2 -> LDS and scratch
            chain_back_layer<E, TN, F>(h2, dc2, a.w2, a.p2, a.dw2, a.dp2, r, wm0, wn0, r16, g, m0, a.T, a.ldr, Cb,
                                       a.dH2s, a.C2s);
        }
        __syncthreads();
        chain_mix<E, RP>(Cb, Mb, wm0, wn0, lane, dc1);   // dC1 = dH2 M^T
    }

    // dA1 = f'(A1) dC1; dw1 += dA1 H, dp1 += dA1; dH = dA1 w1 -> scratch
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = wn0 + 16 * j + r16;
        const bool cv = col < r;
        const float w = cv ? a.w1[col] : 0.f;
        float sw = 0.f, sp = 0.f;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int grow = m0 + wm0 + 4 * g + v;
            const bool ok = cv && grow < a.T;
            const float da1 = ok ? d1[j][v] * dc1[0][j][v] : 0.f;
            sw += da1 * hr[j][v];
            sp += da1;
            if (ok) reinterpret_cast<E*>(a.dHs)[(int64_t)grow * a.ldr + col] = to_elt<E>(da1 * w);
        }
        sw = wave_colsum(sw);
        sp = wave_colsum(sp);
        if (g == 0 && cv) {
            unsafeAtomicAdd(a.dw1 + col, sw);
            unsafeAtomicAdd(a.dp1 + col, sp);
        }
    }
}

}  // namespace noble
