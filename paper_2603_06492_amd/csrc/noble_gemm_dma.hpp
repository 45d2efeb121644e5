// bf16 grouped MFMA GEMM for gfx950 with direct-to-LDS operand loads.
//
// Same problems and epilogue as gemm_kernel (noble_gemm.hpp), but operand
// tiles never pass through VGPRs: buffer_load_dwordx4 ... lds writes each
// lane's 16 bytes to LDS at (M0 base + 16 * lane).  Every operand keeps its
// HBM orientation in LDS:
//  - K-major tiles (rows of x, dy, W as W^T rows, C2, dH): [256 rows][128 B],
//    16-byte chunk c of row r stored at physical chunk c ^ ((r ^ r/8) & 7);
//    MFMA fragments come from ds_read_b128.
//  - MN-major tiles (W in the forward, x and dy in the weight gradients):
//    [64 k][512 B], 16-byte segment s of k-row k stored at physical segment
//    s ^ 4(k & 3); fragments come from two ds_read_b64_tr_b16, each of which
//    transposes a 4 (k) x 16 (m or n) block across a 16-lane group.
// The swizzles make every fragment read pass cover the 64 LDS banks once.
// Two LDS stages: the loads of chunk k+1 are issued before chunk k is
// multiplied; fragment reads of the next K step are interleaved one-to-one
// with the MFMAs of the current one.
#pragma once

#include <type_traits>

#include "noble_gemm.hpp"
#include "noble_tiles.hpp"

namespace noble {

typedef short s16x4 __attribute__((ext_vector_type(4)));
#define NOBLE_LDS(p) ((__attribute__((address_space(3))) void*)(p))

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor words (base, stride 0, num_records, gfx9 format word).
__device__ __forceinline__ i32x4 make_desc(const char* base, int64_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const int n = bytes <= 0 ? 0 : (bytes >= 0x7fffffff ? 0x7fffffff : (int)bytes);
    i32x4 d;
    d[0] = (int)(uint32_t)a;
    d[1] = (int)((uint32_t)(a >> 32) & 0xffffu);
    d[2] = n;
    d[3] = 0x00020000;
    return d;
}

// 16 bytes per lane from the buffer into LDS at lds_dst + 16 * lane.  Issued
// from asm: the compiler then does not treat later LDS reads of the other
// stage as depending on this load; the kernel waits on vmcnt itself before
// the barrier that publishes the stage.
__device__ __forceinline__ void dma16(i32x4 desc, char* lds_dst, uint32_t voff, uint32_t soff) {
    const uint32_t m0 = (uint32_t)reinterpret_cast<uintptr_t>(NOBLE_LDS(lds_dst));
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "buffer_load_dwordx4 %1, %2, %3 offen lds"
        :
        : "s"(m0), "v"(voff), "s"(desc), "s"(soff)
        : "memory", "m0");
}

__device__ __forceinline__ uint64_t ds_read_tr(const char* p) {
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
    return __builtin_bit_cast(uint64_t, v);
}

// Issue the loads of one 256-row operand tile (one 64-element K chunk) into
// `dst` (32 KB): 32 instructions of 1 KB shared by NW waves.
template <bool KMAJ, int NW>
__device__ __forceinline__ void dma_tile(const Operand& op, int row0, int kc, char* dst, int wave, int lane) {
    constexpr int ES = 2, PERW = 32 / NW;
    const bool second = kc >= op.nk1;
    const char* ptr = second ? op.s[1].ptr : op.s[0].ptr;
    const int64_t ld = second ? op.s[1].ld : op.s[0].ld;
    const int klen = second ? op.s[1].klen : op.s[0].klen;
    const int k0 = (second ? kc - op.nk1 : kc) * 64;
    if constexpr (KMAJ) {
        // block b = NW i + wave holds rows 8b .. 8b+7; lane p -> row 8b + p/8,
        // physical chunk p%8 = logical chunk (p%8) ^ swz(row), where
        // swz(row) = (row ^ row/8) & 7 = (p/8) ^ (b & 7).
        const i32x4 rs = make_desc(ptr + (int64_t)row0 * ld * ES, (int64_t)(op.rows - row0) * ld * ES);
        const int rr = lane >> 3;
#pragma unroll
        for (int i = 0; i < PERW; ++i) {
            const int b = NW * i + wave;
            const int c = (lane & 7) ^ rr ^ (b & 7);
            const int k = k0 + c * 8;
            const uint32_t vo = k < klen ? (uint32_t)(((int64_t)rr * ld + k) * ES) : kOOB;
            dma16(rs, dst + b * 1024, vo, (uint32_t)((int64_t)8 * b * ld * ES));
        }
    } else {
        // instruction i of wave w holds k-rows 2(NW i + w) and the next; lane p
        // -> k-row kr = 2(NW i + w) + p/32, physical segment p%32 holds logical
        // segment (p%32) ^ 4(kr & 3)
        const i32x4 rs = make_desc(ptr + (int64_t)k0 * ld * ES, (int64_t)(klen - k0) * ld * ES);
        const int kq = lane >> 5;
        const int seg = (lane & 31) ^ (4 * ((2 * wave + kq) & 3));
        const int col = row0 + 8 * seg;
        const uint32_t vo = col < op.rows ? (uint32_t)(((int64_t)kq * ld + col) * ES) : kOOB;
#pragma unroll
        for (int i = 0; i < PERW; ++i) {
            const int kr = 2 * (NW * i + wave);
            dma16(rs, dst + kr * 512, vo, (uint32_t)((int64_t)kr * ld * ES));
        }
    }
}

// s_waitcnt with only the vector-memory count constrained (gfx9 encoding).
template <int VM>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(VM >= 0 && VM < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

// MFMA fragment reads (32 x 32 x 16 bf16) of a wave whose block starts at
// row/column w0 of the tile (w0 a multiple of 64).
//  K-major: fragment (i, s) at (kbase ^ s<<5 ^ (i&1)<<6) + 4096 i; with
//  swz(row) = (row ^ row/8) & 7 a 16-lane pass of ds_read_b128 (16
//  consecutive rows, one logical chunk) covers all 64 banks.
//  MN-major: half t of fragment (i, s) at mbase + col[i] + (16 s + 4 t) 512,
//  col[i] = 64 ((w0/32 + i) ^ c), c = (lane % 16) / 4.
template <bool KMAJ, int T>
struct FragAddr {
    uint32_t base;
    uint32_t col[T];
    __device__ __forceinline__ FragAddr(int w0, int lane) {
        if constexpr (KMAJ) {
            const int r32 = lane & 31, h = lane >> 5;
            base = (uint32_t)((w0 + r32) * 128 + ((h ^ (r32 & 7) ^ (r32 >> 3)) << 4));
        } else {
            const int g = lane >> 4, j = lane & 15, c = j >> 2;
            const int x = 2 * (g & 1) + ((j & 3) >> 1);
            base = (uint32_t)((8 * (g >> 1) + c) * 512 + 16 * x + 8 * (j & 1));
#pragma unroll
            for (int i = 0; i < T; ++i) col[i] = (uint32_t)(64 * (((w0 >> 5) + i) ^ c));
        }
    }
    __device__ __forceinline__ u32x4 read(const char* tile, int i, int s) const {
        if constexpr (KMAJ) {
            return *reinterpret_cast<const u32x4*>(tile + ((base ^ ((uint32_t)s << 5) ^ ((uint32_t)(i & 1) << 6)) +
                                                           4096u * i));
        } else {
            const char* p = tile + (base + col[i] + 512u * 16 * s);
            const uint64_t lo = ds_read_tr(p);
            const uint64_t hi = ds_read_tr(p + 4 * 512);
            u32x4 v;
            v[0] = (uint32_t)lo;
            v[1] = (uint32_t)(lo >> 32);
            v[2] = (uint32_t)hi;
            v[3] = (uint32_t)(hi >> 32);
            return v;
        }
    }
};

constexpr int kDmaWM = 2, kDmaWN = 4, kDmaThreads = 64 * kDmaWM * kDmaWN;

// Cache policy of the epilogue's plain stores: non-temporal (the NT bit of
// the buffer instruction's cache-policy operand).  The product is bound by
// the MFMAs, so its output can go to HBM while it runs; stored with the
// default policy it stays dirty in the memory-side cache and is written back
// while the next kernel, often a bandwidth-bound rank projection, reads its
// own operand.  Measured on the 1.5B-style block step: 3-4% less time.
constexpr int kStoreNT = 2;

// TAG only separates launch sites in profiles (1: the plain r = 0 forward);
// the code is the same.
template <bool AK, bool BKM, bool HAS_BSUM, int TAG>
__global__ __launch_bounds__(kDmaThreads, 1) void gemm_bf16_kernel(GemmBatch batch) {
    constexpr int BM = 256, BN = 256, NW = kDmaWM * kDmaWN;
    constexpr int WTM = BM / kDmaWM, WTN = BN / kDmaWN;   // wave tile 128 x 64
    constexpr int TM = WTM / 32, TN = WTN / 32;
    constexpr int TILE = 256 * 128;   // bytes of one operand tile per stage
    constexpr int STAGE = 2 * TILE;
    // Two stages as two objects, so the compiler can tell the stage being
    // filled by DMA from the one being read.
    __shared__ __attribute__((aligned(1024))) char lds0[STAGE];
    __shared__ __attribute__((aligned(1024))) char lds1[STAGE];

    const int bid = blockIdx.x;
    int q = 0;
#pragma unroll
    for (int t = 1; t < kMaxProblems; ++t)
        if (t < batch.count && bid >= batch.p[t].tile_begin) q = t;
    const GemmProblem& P = batch.p[q];

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
    const bool kpair = P.kpair != 0, npair = P.npair != 0;
    const int m0 = tm * BM, n0 = tn * (npair ? BN / 2 : BN);
    const int kc0 = (int)((int64_t)P.nk * piece / P.split);
    const int kc1 = (int)((int64_t)P.nk * (piece + 1) / P.split);

    // The wave index is uniform; say so, so DMA offsets and LDS bases stay
    // in SGPRs.
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // Wave w takes M half w / 4 and N quarter (w % 4) ^ 2 (w / 4).  Waves w and
    // w + 4 share a SIMD, and this way they differ in both the M half and the
    // N half: a tile that is only half inside M or N (the rank-r products,
    // r <= 128) leaves every SIMD one live wave instead of idling two SIMDs.
    // A problem with M <= 128 (`kpair`: W_up's gradient, r rows) instead gives
    // both halves the rows 0..127: half w / 4 takes K steps 2 (w / 4) and
    // 2 (w / 4) + 1 of every chunk, and the second half's sums are added to
    // the first's through LDS at the end, so the half-empty tile costs about
    // half the MFMA time.  `npair` tiles are 256 x 128 (twice the tiles of a
    // launch that would under-fill the CUs): the wave that would take N
    // quarter q >= 2 takes quarter q - 2 and K steps 2 and 3, its partner
    // (same M half, quarter q - 2) steps 0 and 1, with the same hand-over.
    const int khalf = wave / kDmaWN;
    const int qw = (wave % kDmaWN) ^ (khalf * (kDmaWN / 2));
    const int wm0 = kpair ? 0 : khalf * WTM, wn0 = (npair ? (qw & 1) : qw) * WTN;
    const bool split2 = kpair || npair;               // a K-split pair of waves per output block
    const int kh = kpair ? khalf : (npair ? qw >> 1 : 0);   // this wave's K half
    static_assert(kDmaWM == 2, "the N-quarter swizzle pairs two M halves");
    const int r32 = lane & 31, h = lane >> 5;

    // A wave whose block lies wholly outside the problem only loads its share
    // of the operand tiles and meets the barriers: the same stages and the
    // same barrier sequence (one after the first chunk's loads, one per chunk)
    // as the loop below, without fragment reads, MFMAs or stores.  Kept apart
    // from that loop: a test inside it slowed the full tiles by 2-4%.
    // B rows of an npair tile stop at its 128 columns (the rest read nothing).
    auto b_operand = [&]() {
        Operand o = P.B;
        if (npair) o.rows = min(o.rows, n0 + BN / 2);
        return o;
    };
    if (m0 + wm0 >= P.M || n0 + wn0 >= P.N) {
        if (kc0 < kc1) {
            const Operand opA = P.A, opB = b_operand();
            dma_tile<AK, NW>(opA, m0, kc0, lds0, wave, lane);
            dma_tile<BKM, NW>(opB, n0, kc0, lds0 + TILE, wave, lane);
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            for (int kc = kc0; kc < kc1; ++kc) {
                char* nxt = ((kc - kc0) & 1) ? lds0 : lds1;
                if (kc + 1 < kc1) {
                    dma_tile<AK, NW>(opA, m0, kc + 1, nxt, wave, lane);
                    dma_tile<BKM, NW>(opB, n0, kc + 1, nxt + TILE, wave, lane);
                }
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                __syncthreads();
            }
        }
        if (split2) __syncthreads();   // the hand-over of the second half's sums
        return;
    }

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // db's column sums ride on the B fragments of the waves of M half 0.  The
    // tiles of one column block share them out: tile row tm sums its own
    // contiguous share of the K chunks, so that no tile row carries all of
    // that work (a launch ends with its slowest tile).
    const bool do_bsum = HAS_BSUM && (P.bsum != nullptr) && wm0 == 0 && !split2;
    float bs[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) bs[j] = 0.f;

    if (kc0 < kc1) {
        const FragAddr<AK, TM> fa(wm0, lane);
        const FragAddr<BKM, TN> fb(wn0, lane);
        // Local copies of the operand descriptions: read once from the kernel
        // arguments instead of once per chunk.
        const Operand opA = P.A, opB = b_operand();
        dma_tile<AK, NW>(opA, m0, kc0, lds0, wave, lane);
        dma_tile<BKM, NW>(opB, n0, kc0, lds0 + TILE, wave, lane);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();

        // Multiply chunk kc from `cur` while chunk kc + 1 streams into `nxt`:
        // all four K steps, or (NS = 2, kpair) the two of this wave's half.
        auto chunk = [&](int kc, const char* cur, char* nxt, auto bs_c, auto ns_c) __attribute__((always_inline)) {
            constexpr bool BS = decltype(bs_c)::value;
            constexpr int NS = decltype(ns_c)::value;
            const int sb = NS == 4 ? 0 : 2 * kh;
            const char* ldsA = cur;
            const char* ldsB = cur + TILE;
            if (kc + 1 < kc1) {
                dma_tile<AK, NW>(opA, m0, kc + 1, nxt, wave, lane);
                dma_tile<BKM, NW>(opB, n0, kc + 1, nxt + TILE, wave, lane);
            }
            // Fragments of K step s + 1 are read while the MFMAs of step s run:
            // one LDS read issued per MFMA (schedule pinned below).
            constexpr int NREAD = TM * (AK ? 1 : 2) + TN * (BKM ? 1 : 2);
            constexpr int NMFMA = TM * TN;
            u32x4 a[2][TM], b[2][TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) a[0][i] = fa.read(ldsA, i, sb);
#pragma unroll
            for (int j = 0; j < TN; ++j) b[0][j] = fb.read(ldsB, j, sb);
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const int cb = s & 1, nb = cb ^ 1;
                __builtin_amdgcn_sched_barrier(0);
                if (s + 1 < NS) {
#pragma unroll
                    for (int i = 0; i < TM; ++i) a[nb][i] = fa.read(ldsA, i, sb + s + 1);
#pragma unroll
                    for (int j = 0; j < TN; ++j) b[nb][j] = fb.read(ldsB, j, sb + s + 1);
                }
                if constexpr (BS) {
#pragma unroll
                    for (int j = 0; j < TN; ++j)
#pragma unroll
                        for (int w = 0; w < 4; ++w) bs[j] += bf2f(b[cb][j][w] & 0xffffu) + bf2f(b[cb][j][w] >> 16);
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) mma32<uint16_t>(acc[i][j], a[cb][i], b[cb][j]);
                if (s + 1 < NS) {
#pragma unroll
                    for (int qq = 0; qq < NMFMA; ++qq) {
                        if (qq < NREAD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                   // MFMA
                    }
                }
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
        };
        auto run = [&](auto bs_c, auto ns_c) __attribute__((always_inline)) {
            int kc = kc0;
            for (; kc + 1 < kc1; kc += 2) {
                chunk(kc, lds0, lds1, bs_c, ns_c);
                chunk(kc + 1, lds1, lds0, bs_c, ns_c);
            }
            if (kc < kc1) chunk(kc, lds0, lds1, bs_c, ns_c);
        };
        // chunks [b, e) of the piece (chunk kc uses stage (kc - kc0) % 2)
        auto run_range = [&](int b, int e, auto bs_c) __attribute__((always_inline)) {
            using Four = std::integral_constant<int, 4>;
            int kc = b;
            if (kc < e && ((kc - kc0) & 1)) chunk(kc++, lds1, lds0, bs_c, Four{});
            for (; kc + 1 < e; kc += 2) {
                chunk(kc, lds0, lds1, bs_c, Four{});
                chunk(kc + 1, lds1, lds0, bs_c, Four{});
            }
            if (kc < e) chunk(kc, lds0, lds1, bs_c, Four{});
        };
        using Four = std::integral_constant<int, 4>;
        using Two = std::integral_constant<int, 2>;
        if (split2)
            run(std::false_type{}, Two{});
        else if constexpr (HAS_BSUM) {
            if (do_bsum) {
                const int n = kc1 - kc0;
                const int sb = kc0 + (int)((int64_t)n * tm / P.tiles_m), se = kc0 + (int)((int64_t)n * (tm + 1) / P.tiles_m);
                run_range(kc0, sb, std::false_type{});
                run_range(sb, se, std::true_type{});
                run_range(se, kc1, std::false_type{});
            } else {
                run(std::false_type{}, Four{});
            }
        } else {
            run(std::false_type{}, Four{});
        }
    }

    if (split2) {
        // Hand-over: the waves of the second K half store their sums in the
        // (now idle) operand stages, 32 KB per output block (kpair: per N
        // quarter; npair: per M half and N quarter), lane-interleaved 16-byte
        // vectors; the first K half adds them.  The last chunk's barrier has
        // retired every fragment read of the stages.
        const int reg = kpair ? wn0 / WTN : 2 * khalf + (qw & 1);
        char* hand = (reg < 2 ? lds0 : lds1) + (reg & 1) * (STAGE / 2);
        static_assert(TM * TN * 16 * 4 * 64 == STAGE / 2, "one wave's sums fill half a stage");
        if (kh == 1) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int v4 = 0; v4 < 4; ++v4) {
                        f32x4 t;
#pragma unroll
                        for (int e = 0; e < 4; ++e) t[e] = acc[i][j][4 * v4 + e];
                        *reinterpret_cast<f32x4*>(hand + (((i * TN + j) * 4 + v4) * 64 + lane) * 16) = t;
                    }
        }
        __syncthreads();
        if (kh == 1) return;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v4 = 0; v4 < 4; ++v4) {
                    const f32x4 t = *reinterpret_cast<const f32x4*>(hand + (((i * TN + j) * 4 + v4) * 64 + lane) * 16);
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[i][j][4 * v4 + e] += t[e];
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
    const bool add_bias = (P.bias != nullptr) && piece == 0;
    const int es = P.out_f32 ? 4 : 2;
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
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), rc, vo, so, kStoreNT);
        });
    else
        epilogue([&](float val, uint32_t vo, uint32_t so) {
            __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf(val), rc, vo, so, kStoreNT);
        });
}

}  // namespace noble
