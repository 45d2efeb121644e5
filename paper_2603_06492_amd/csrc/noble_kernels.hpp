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

constexpr int kMaxZero = 16;
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
    const float* w1;
    const float* p1;
    const float* w2;
    const float* p2;
    float* H;           // reserve [T, r]: written by fwd, read by bwd
    char* C1s;          // scratch [T, r] storage type (bwd)
    char* C2s;          // scratch [T, r] storage type
    char* dH2s;         // scratch [T, r] storage type (bwd)
    char* dHs;          // scratch [T, r] storage type (bwd)
    float* dw1;
    float* dp1;
    float* dw2;
    float* dp2;
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

// Forward chain for activation F; L2 = two applications with M between them
// (CosNet for F = Cos), otherwise C2 = f(H w1 + p1) and M, w2, p2 are unused.
template <typename E, int RP, Act F, bool L2>
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
    if constexpr (L2) stage_mix_matrix<E, RP, false>(a.M, r, Mb, tid);

    // H -> reserve; C1 = f(H w1 + p1) -> LDS (A operand of the mixing), or
    // straight to C2 for one application
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = wn0 + 16 * j + r16;
        const bool cv = col < r;
        const float w = cv ? a.w1[col] : 0.f, p = cv ? a.p1[col] : 0.f;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = wm0 + 4 * g + v, grow = m0 + row;
            const float h = acc[0][j][v];
            if (a.H && cv && grow < a.T) a.H[(int64_t)grow * a.ldr + col] = h;
            const float c1 = cv ? act_value<F, false>(h * w + p) : 0.f;
            if constexpr (L2)
                *reinterpret_cast<E*>(Cb + tile_elem_off<E>(row, col, kChainRows)) = to_elt<E>(c1);
            else if (cv && grow < a.T)
                reinterpret_cast<E*>(a.C2s)[(int64_t)grow * a.ldr + col] = to_elt<E>(c1);
        }
    }
    if constexpr (!L2) return;
    __syncthreads();

    f32x4 mix[1][TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) mix[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < S::NKB; ++kb)
        mma_chunk<E, 1, TN>(Cb + kb * kChainRows * kRowBytes, Mb + kb * RP * kRowBytes, wm0, wn0, lane, mix);

    // C2 = f(H2 w2 + p2) -> scratch
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = wn0 + 16 * j + r16;
        if (col >= r) continue;
        const float w = a.w2[col], p = a.p2[col];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int grow = m0 + wm0 + 4 * g + v;
            if (grow < a.T)
                reinterpret_cast<E*>(a.C2s)[(int64_t)grow * a.ldr + col] =
                    to_elt<E>(act_value<F, false>(mix[0][j][v] * w + p));
        }
    }
}

// Backward chain, same forms as fwd_chain_kernel.  The one-application form
// writes C2 and dH only.
template <typename E, int RP, Act F, bool L2>
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

    // dC2 = dy W_up^T
    f32x4 dc2[1][TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) dc2[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    mainloop<E, kChainRows, RP, 2, 2, true, true>(a.A, a.B, m0, 0, 0, a.nk, lds, dc2);

    char* Cb = lds;
    char* Mb = lds + S::NKB * kChainRows * kRowBytes;
    if constexpr (L2) stage_mix_matrix<E, RP, false>(a.M, r, Mb, tid);

    // Recompute A1 = H w1 + p1 and C1 = f(A1) (-> LDS and scratch, or to C2
    // for one application); keep H and f'(A1).
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
            if constexpr (L2) {
                *reinterpret_cast<E*>(Cb + tile_elem_off<E>(row, col, kChainRows)) = c1;
                if (ok) reinterpret_cast<E*>(a.C1s)[(int64_t)grow * a.ldr + col] = c1;
            } else if (ok) {
                reinterpret_cast<E*>(a.C2s)[(int64_t)grow * a.ldr + col] = c1;
            }
        }
    }

    // dC1: dC2 itself (one application) or dH2 M^T (two)
    f32x4 dc1[1][TN];
    if constexpr (!L2) {
#pragma unroll
        for (int j = 0; j < TN; ++j) dc1[0][j] = dc2[0][j];
    } else {
        __syncthreads();

        // H2 = C1 M
        f32x4 h2[1][TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) h2[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < S::NKB; ++kb)
            mma_chunk<E, 1, TN>(Cb + kb * kChainRows * kRowBytes, Mb + kb * RP * kRowBytes, wm0, wn0, lane, h2);
        __syncthreads();  // every wave is done with C1 and M in LDS

        stage_mix_matrix<E, RP, true>(a.M, r, Mb, tid);

        // A2 = H2 w2 + p2; C2 = f(A2) -> scratch; dA2 = f'(A2) dC2;
        // dw2 += dA2 H2, dp2 += dA2; dH2 = dA2 w2 -> LDS and scratch.
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = wn0 + 16 * j + r16;
            const bool cv = col < r;
            const float w = cv ? a.w2[col] : 0.f, p = cv ? a.p2[col] : 0.f;
            float sw = 0.f, sp = 0.f;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = wm0 + 4 * g + v, grow = m0 + row;
                const bool ok = cv && grow < a.T;
                float f = 0.f, d = 0.f;
                if (cv) act_value_slope<F, false>(h2[0][j][v] * w + p, f, d);
                const float da2 = ok ? d * dc2[0][j][v] : 0.f;
                sw += da2 * h2[0][j][v];
                sp += da2;
                const E dh2 = to_elt<E>(da2 * w);
                *reinterpret_cast<E*>(Cb + tile_elem_off<E>(row, col, kChainRows)) = dh2;
                if (ok) {
                    reinterpret_cast<E*>(a.C2s)[(int64_t)grow * a.ldr + col] = to_elt<E>(f);
                    reinterpret_cast<E*>(a.dH2s)[(int64_t)grow * a.ldr + col] = dh2;
                }
            }
            sw = wave_colsum(sw);
            sp = wave_colsum(sp);
            if (g == 0 && cv) {
                unsafeAtomicAdd(a.dw2 + col, sw);
                unsafeAtomicAdd(a.dp2 + col, sp);
            }
        }
        __syncthreads();

#pragma unroll
        for (int j = 0; j < TN; ++j) dc1[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < S::NKB; ++kb)
            mma_chunk<E, 1, TN>(Cb + kb * kChainRows * kRowBytes, Mb + kb * RP * kRowBytes, wm0, wn0, lane, dc1);
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
