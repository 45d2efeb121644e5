// Grouped MFMA GEMM for gfx950 used by every large product of the layer:
//   forward  y  = [x | C2] [W ; W_up] + b       (A K-major, B MN-major)
//   backward dx = [dy | dH] [W^T ; W_down^T]      (A K-major, B K-major)
//   backward dW, dW_down, dW_up, dM over tokens (A MN-major, B MN-major)
//
// Workgroup tile BM x BN (256 x 256 for the large products), four wave64 in a
// 2 x 2 grid, each wave owning a (BM/2) x (BN/2) block of 32 x 32 MFMA tiles
// (v_mfma_f32_32x32x16_bf16; 4 x v_mfma_f32_32x32x2f32 per 16-byte chunk on
// the float32 path).  Operand tiles go global -> registers -> LDS (two LDS
// stages, the global loads of chunk k+2 in flight while chunk k is multiplied),
// transposed in registers when the operand is MN-contiguous in HBM.
#pragma once

#include <type_traits>

#include "noble_tiles.hpp"

namespace noble {

typedef float f32x16 __attribute__((ext_vector_type(16)));

template <typename E> __device__ __forceinline__ void mma32(f32x16& c, const u32x4& a, const u32x4& b);
template <> __device__ __forceinline__ void mma32<uint16_t>(f32x16& c, const u32x4& a, const u32x4& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <> __device__ __forceinline__ void mma32<float>(f32x16& c, const u32x4& a, const u32x4& b) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[q]), __uint_as_float(b[q]), c, 0, 0, 0);
}

struct GemmProblem {
    Operand A, B;
    void* C;
    int64_t ldc;
    const float* bias;  // per output column, added by K piece 0 (nullable)
    float* bsum;        // column sums of B over K, atomically added (nullable)
    int M, N;
    int nk;             // K chunks (both segments)
    int split;          // K pieces: with atomic, added into C; else piece p
                        // stores its partial at C + p * pstride elements
    int tiles_m, tiles_n;
    int tile_begin;     // first block index of this problem
    int nblocks;        // tiles_m * tiles_n * split
    int out_f32;        // C holds float (1) or the storage type (0)
    int atomic;         // atomicAdd into a zeroed float C
    int kpair;          // bf16 path, M <= 128, no bsum: the two M halves of the
                        // workgroup's waves split each K chunk instead
    int npair;          // bf16 path: 256 x 128 output tiles, the waves of the
                        // two N halves splitting each K chunk (no bsum)
    int pad2_;
    int64_t pstride;    // elements between the partials of consecutive pieces
};

constexpr int kMaxProblems = 14;   // weight gradients of a 4-group 3-layer CosNet: dW, dW_down, 4 x (dW_up, dM, dM')
struct GemmBatch {
    GemmProblem p[kMaxProblems];
    int count;
    int pad_;
};

// Tiles of a problem in "column groups" of kGroupM tile rows, so the blocks an
// XCD runs together share A row panels and B column panels in its L2.
constexpr int kGroupM = 4;

template <typename E, int BM, int BN, bool AK, bool BKM, bool HAS_BSUM>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(GemmBatch batch) {
    constexpr int TM = BM / 64, TN = BN / 64;  // 32x32 tiles per wave (waves 2 x 2)
    constexpr int STAGE = (BM + BN) * kRowBytes;
    __shared__ __attribute__((aligned(16))) char lds[2 * STAGE];

    const int bid = blockIdx.x;
    int q = 0;
#pragma unroll
    for (int t = 1; t < kMaxProblems; ++t)
        if (t < batch.count && bid >= batch.p[t].tile_begin) q = t;
    const GemmProblem& P = batch.p[q];

    // XCD-aware order: consecutive block ids land on different XCDs (round
    // robin over 8), so give each XCD a contiguous range of the problem's tiles.
    int L = bid - P.tile_begin;
    if ((P.nblocks & 7) == 0) L = (L & 7) * (P.nblocks >> 3) + (L >> 3);
    const int ntiles = P.tiles_m * P.tiles_n;
    const int piece = L / ntiles;
    const int tile = L - piece * ntiles;
    const int span = kGroupM * P.tiles_n;
    const int grp = tile / span, in = tile - grp * span;
    const int first_m = grp * kGroupM;
    const int gsz = min(P.tiles_m - first_m, kGroupM);
    const int tm = first_m + in % gsz, tn = in / gsz;
    const int m0 = tm * BM, n0 = tn * BN;
    const int kc0 = (int)((int64_t)P.nk * piece / P.split);
    const int kc1 = (int)((int64_t)P.nk * (piece + 1) / P.split);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm0 = (wave >> 1) * (BM / 2), wn0 = (wave & 1) * (BN / 2);
    const int r32 = lane & 31, h = lane >> 5;

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const bool do_bsum = (P.bsum != nullptr) && tm == 0 && (wave >> 1) == 0;
    float bs[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) bs[j] = 0.f;

    if (kc0 < kc1) {
        // Registers hold chunk kc + 1 while chunk kc is multiplied from LDS;
        // during K step s the part s of chunk kc + 1 is written to the other
        // LDS stage and part s of chunk kc + 2 is requested from memory.
        Stage<E, BM, AK> sa;
        Stage<E, BN, BKM> sb;
        sa.load(P.A, m0, kc0, tid);
        sb.load(P.B, n0, kc0, tid);
        sa.store(lds, tid);
        sb.store(lds + BM * kRowBytes, tid);
        if (kc0 + 1 < kc1) {
            sa.load(P.A, m0, kc0 + 1, tid);
            sb.load(P.B, n0, kc0 + 1, tid);
        }
        __syncthreads();
        // Fragment (i, s) of a wave: rows w0 + 32i + l%32, K step s (chunk
        // 2s + l/32).  With the row swizzle of lds_off its byte offset is
        // (base ^ s<<5 ^ (i&1)<<6) + 4096 i, base = lds_off(w0 + l%32, l/32).
        const uint32_t baseA = (uint32_t)lds_off(wm0 + r32, h);
        const uint32_t baseB = (uint32_t)lds_off(wn0 + r32, h);
        // One K chunk; MORE: chunk kc + 1 exists, MORE2: kc + 2 exists,
        // BS: accumulate column sums of B.  All compile-time, so the steady
        // state is one branch-free block.
        auto chunk = [&](int kc, auto more_c, auto more2_c, auto bs_c) {
            constexpr bool MORE = decltype(more_c)::value, MORE2 = decltype(more2_c)::value;
            constexpr bool BS = decltype(bs_c)::value;
            const char* ldsA = lds + ((kc - kc0) & 1) * STAGE;
            const char* ldsB = ldsA + BM * kRowBytes;
            char* nxt = lds + (((kc - kc0) & 1) ^ 1) * STAGE;
            u32x4 a[2][TM], b[2][TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[0][i] = *reinterpret_cast<const u32x4*>(ldsA + ((baseA ^ ((i & 1) << 6)) + 4096 * i));
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[0][j] = *reinterpret_cast<const u32x4*>(ldsB + ((baseB ^ ((j & 1) << 6)) + 4096 * j));
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int cb = s & 1, nb = cb ^ 1;
                if (s + 1 < 4) {
                    const uint32_t xs = (uint32_t)(s + 1) << 5;
#pragma unroll
                    for (int i = 0; i < TM; ++i)
                        a[nb][i] = *reinterpret_cast<const u32x4*>(ldsA + ((baseA ^ xs ^ ((i & 1) << 6)) + 4096 * i));
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        b[nb][j] = *reinterpret_cast<const u32x4*>(ldsB + ((baseB ^ xs ^ ((j & 1) << 6)) + 4096 * j));
                }
                if constexpr (BS) {
#pragma unroll
                    for (int j = 0; j < TN; ++j)
#pragma unroll
                        for (int w = 0; w < 4; ++w) {
                            if constexpr (sizeof(E) == 2)
                                bs[j] += bf2f(b[cb][j][w] & 0xffffu) + bf2f(b[cb][j][w] >> 16);
                            else
                                bs[j] += __uint_as_float(b[cb][j][w]);
                        }
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) mma32<E>(acc[i][j], a[cb][i], b[cb][j]);
                if constexpr (MORE) {
                    sa.template store_part<4>(nxt, tid, s);
                    sb.template store_part<4>(nxt + BM * kRowBytes, tid, s);
                    if constexpr (MORE2) {
                        sa.template load_part<4>(P.A, m0, kc + 2, tid, s);
                        sb.template load_part<4>(P.B, n0, kc + 2, tid, s);
                    }
                }
                // Keep each step's staging in its step: the loads of chunk
                // kc + 2 then have a whole chunk of MFMA work to land.
                __builtin_amdgcn_sched_barrier(0);
            }
            __syncthreads();
        };
        auto run = [&](auto bs_c) {
            using T_ = std::true_type;
            using F_ = std::false_type;
            int kc = kc0;
            for (; kc + 2 < kc1; ++kc) chunk(kc, T_{}, T_{}, bs_c);
            if (kc + 1 < kc1) chunk(kc++, T_{}, F_{}, bs_c);
            chunk(kc, F_{}, F_{}, bs_c);
        };
        if constexpr (HAS_BSUM) {
            if (do_bsum)
                run(std::true_type{});
            else
                run(std::false_type{});
        } else {
            run(std::false_type{});
        }
    }

    if (do_bsum) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const float s = bs[j] + __shfl_xor(bs[j], 32);
            const int col = n0 + wn0 + 32 * j + r32;
            if (h == 0 && col < P.N) unsafeAtomicAdd(P.bsum + col, s);
        }
    }

    // Output element v of acc[i][j] in lane l sits at row
    // 32i + 8(v/4) + 4(l/32) + v%4, column 32j + l%32 of the wave block.
    // Stores go through a buffer resource that ends at row M, so rows past
    // the end are dropped by the hardware; columns past N get an offset past
    // the end.  The store mode is uniform: branch once, outside the loops.
    const bool add_bias = (P.bias != nullptr) && piece == 0;
    const int es = P.out_f32 ? 4 : (int)sizeof(E);
    const __amdgpu_buffer_rsrc_t rc =
        make_rsrc(static_cast<const char*>(P.C) + (piece * P.pstride + (int64_t)m0 * P.ldc) * es,
                  (int64_t)(P.M - m0) * P.ldc * es);
    uint32_t voff[TM][TN];
    float bcol[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn0 + 32 * j + r32;
        bcol[j] = (add_bias && col < P.N) ? P.bias[col] : 0.f;
#pragma unroll
        for (int i = 0; i < TM; ++i)
            voff[i][j] = col < P.N ? (uint32_t)(((int64_t)(wm0 + 32 * i + 4 * h) * P.ldc + col) * es) : kOOB;
    }
    auto epilogue = [&](auto store) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    store(acc[i][j][v] + bcol[j], voff[i][j],
                          (uint32_t)((int64_t)(8 * (v >> 2) + (v & 3)) * P.ldc * es));
    };
    if (P.atomic)
        epilogue([&](float val, uint32_t vo, uint32_t so) {
            __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(val, rc, vo, so, 0);
        });
    else if (P.out_f32)
        epilogue([&](float val, uint32_t vo, uint32_t so) {
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), rc, vo, so, 0);
        });
    else if constexpr (sizeof(E) == 2)
        epilogue([&](float val, uint32_t vo, uint32_t so) {
            __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf(val), rc, vo, so, 0);
        });
}

}  // namespace noble
