// The rank-r side of the layer, bf16 path, on gfx950, in two steps:
//
//   proj_kernel:        the rank projection, H = x W_down (forward) or
//                       dC2 = dy W_up^T (backward), as a split-K MFMA product:
//                       a workgroup owns 128 tokens x all 128 (padded) ranks
//                       and one of S pieces of K, and writes its float32
//                       partial sum to scratch.  Streaming 128 tokens against
//                       the rank operand (instead of 32) cuts the L2 traffic of
//                       that operand four-fold; the K split keeps every CU busy.
//   branch_fwd_kernel:  per token, H = the sum of the S partials, then the
//                       CosNet chain C1 = cos(H w1 + p1), H2 = C1 M (MFMA),
//                       C2 = cos(H2 w2 + p2).  Writes H (float32, the reserve)
//                       and C2 (bf16, scratch).
//   branch_bwd_kernel:  dC2 = the sum of the partials, then the chain backwards
//                       from the saved H: C1, sin A1, H2 = C1 M, C2, sin A2,
//                       dA2 = -sin(A2) dC2, dH2 = dA2 w2, dC1 = dH2 M^T (MFMA),
//                       dA1 = -sin(A1) dC1, dH = dA1 w1.  Writes C1, C2, dH2, dH
//                       (bf16 scratch, operands of the weight-gradient products)
//                       and reduces dw1, dp1, dw2, dp2 over its tokens with wave
//                       shuffles, then one float atomic per column.
//   Both chain kernels also take the other bottleneck activations (tanh,
//   LeakyReLU, GELU in place of cos; see noble_act.hpp) and the
//   one-application form C2 = f(H w1 + p1), which skips M and the second
//   frequency/phase pair.
//
// The chain kernels run 32 tokens x one group's ranks per workgroup: four
// waves (r <= 128) or eight (r <= 256), each owning 32 rank columns.  M [r, r]
// is loaded into LDS once per workgroup as 128 x 128 tiles in its HBM
// orientation [r_in][r_out]; C1 M reads it with ds_read_b64_tr_b16 and
// dH2 M^T with ds_read_b128.
//
// Grouped layers (several output column blocks of one x, each with its own
// branch, e.g. Q, K and V): the rank side is stored token-major as [T, G r];
// the projection runs one job per (group, 128-rank block) and the chain one
// workgroup per (token block, group).
#pragma once

#include "noble_gemm_dma.hpp"
#include "noble_kernels.hpp"

namespace noble {

constexpr int kSkRows = 32;     // tokens per chain workgroup
constexpr int kSkN = 128;       // rank columns of one M tile
constexpr int kSkM = kSkN * kSkN * 2;     // one M tile, 128 x 128 bf16
constexpr int kSkC = kSkRows * kSkN * 2;  // 32 x 128 bf16 of the C1 / dH2 operand tile
constexpr int kSkMaxNT = 2;               // ranks up to 2 x 128 per group
// LDS of a chain workgroup with L - 1 mixing matrices of NT x NT M tiles
// and two 32 x 128 NT operand tiles: the high and low bf16 parts of the
// mixing operand (C1, C2, dH2 or dH3).  The 3-layer form runs at NT = 1.
template <int NT, int L = 2>
constexpr int sk_lds() {
    return (L == 3 ? 2 : 1) * NT * NT * kSkM + 2 * NT * kSkC;
}
static_assert(sk_lds<kSkMaxNT>() <= 160 * 1024, "chain LDS exceeds a CU's 160 KB");
static_assert(sk_lds<1, 3>() <= 160 * 1024, "chain LDS exceeds a CU's 160 KB");

// A float32 value as the sum of two bf16 values (round to nearest even
// twice): hi carries the leading 8 significant bits, lo the next 8.  hi + lo
// equals v to about 2^-17 relative, so an MFMA product over the pair is
// float32-accurate where one bf16 operand would carry 2^-9.
struct BfPair {
    uint16_t hi, lo;
};
__device__ __forceinline__ BfPair bf_split(float v) {
    const uint32_t hi = f2bf(v);
    return BfPair{(uint16_t)hi, (uint16_t)f2bf(v - bf2f(hi))};
}
// Three parts: hi and mid as bf_split gives them (hi + mid is its pair), lo
// the bf16 rounding of what remains.  hi + mid + lo equals v to about 2^-27
// relative, below float32's own rounding, so a product over the three parts
// is as accurate as a float32 product.  Each subtraction is exact in
// float32 (the remainder has at most 16 significant bits).
struct BfTriple {
    uint16_t hi, mid, lo;
};
__device__ __forceinline__ BfTriple bf_split3(float v) {
    const uint32_t hi = f2bf(v);
    const float r1 = v - bf2f(hi);
    const uint32_t mid = f2bf(r1);
    return BfTriple{(uint16_t)hi, (uint16_t)mid, (uint16_t)f2bf(r1 - bf2f(mid))};
}

constexpr int kPjRows = 128;                 // tokens per projection workgroup
constexpr int kPjThreads = 512;              // eight waves: 4 token blocks x 2 rank halves
constexpr int kPjStages = 4;                 // LDS ring depth
constexpr int kPjA = kPjRows * 128;          // A bytes per stage (128 rows x 64 K)
constexpr int kPjB = kSkN * 128;             // B bytes per stage (16 KB either layout)
constexpr int kPjStage = kPjA + kPjB;
constexpr int kPjLoads = 4;                  // DMA instructions per wave per K chunk
constexpr int kPjMinChunks = 4;              // 64-element K chunks per piece, at least
constexpr int kPjMaxSplit = 8;
constexpr int kPjMaxJobs = 8;                // (group, 128-rank block) pairs per launch

// One block of at most 128 rank columns of the projection: A [T, K] K-major
// (x in the forward, a group's column block of dy in the backward) times B
// (W_down's column block [K, n] MN-major, or W_up's row block [n, K] K-major),
// written to partial columns c0 .. c0 + n - 1 (n = B.rows).
struct ProjJob {
    Operand A;
    Operand B;
    int c0, pad_;
};

struct ProjArgs {
    ProjJob job[kPjMaxJobs];
    float* P;           // partials [S][T][ldp] float32
    int64_t pstride;    // T * ldp
    int T, ldp, nk, S;  // nk: 64-element K chunks (the same for every job)
    int J, pad_;        // jobs
    ZeroList z;         // float arrays to clear on the side (the backward's
                        // atomically accumulated gradients)
};

// G groups of r ranks, stored token-major with row stride R = G r: group g
// owns columns g r .. g r + r - 1 of H, C1, C2, dH2, dH and of the partials,
// rows g r .. of the frequency / phase vectors and M + g r r.
struct BranchArgs {
    const float* P;       // projection partials [S][T][R]
    int64_t pstride;
    const uint16_t* M;    // [G][r][r]
    const uint16_t* M2;   // 3-layer form: the second mixing matrices [G][r][r]
    const float* w1;      // [R]
    const float* p1;
    const float* w2;
    const float* p2;
    const float* w3;      // 3-layer form: the third frequency / phase [R]
    const float* p3;
    float* H;             // reserve [T, R] float32 (NULL in an inference forward)
    uint16_t* C1s;        // scratch (backward), see branch_bwd_kernel
    uint16_t* C2s;        // scratch [T, R] bf16: the branch output (C2, or C3 in the 3-layer form)
    uint16_t* dH2s;       // scratch (backward)
    uint16_t* dHs;        // scratch (backward)
    uint16_t* C2ms;       // scratch (backward, 3-layer form): the middle layer's C2 pairs
    uint16_t* dH3s;       // scratch (backward, 3-layer form): dH3 pairs
    float* dw1;           // [R]
    float* dp1;
    float* dw2;
    float* dp2;
    float* dw3;           // 3-layer form
    float* dp3;
    // Backward: when set, the frequency / phase gradients are added into
    // kChainCopies zeroed copies [2 L][kChainCopies][R] (dw1, dp1, dw2, dp2,
    // dw3, dp3), copy = workgroup % kChainCopies, instead of into dw1 ..; a
    // reduction sums the copies afterwards.  Fewer workgroups then add into
    // one address, which float atomics serialise on.
    float* copies;
    int T, r, S, G, R, pad_;
};

constexpr int kChainCopies = 8;


// One 64-element K chunk of the projection operands: 4 DMA instructions per
// wave (two for A, two for B).
template <bool BKM>
__device__ __forceinline__ void proj_dma(const Operand& A, const Operand& B, int row0, int kc, char* st, int wave,
                                         int lane) {
    constexpr int ES = 2;
    const int k0 = kc * 64;
    // K-major tiles store logical 16-byte chunk c of row q at physical chunk
    // c ^ swz(q), swz(q) = (q ^ q/8) & 7, so a 16-row pass of ds_read_b128
    // covers all banks.  128 rows x 128 B: block b = 8i + w holds rows
    // 8b .. 8b+7; lane p -> row 8b + p/8, and swz = (p/8) ^ w.
    auto kmajor = [&](const Operand& op, int64_t row_base, char* dst) {
        const int64_t ld = op.s[0].ld;
        const i32x4 rs = make_desc(op.s[0].ptr + row_base * ld * ES, (int64_t)(op.rows - row_base) * ld * ES);
        const int rr = lane >> 3, c = (lane & 7) ^ rr ^ wave;
        const int k = k0 + c * 8;
        const uint32_t vo = k < op.s[0].klen ? (uint32_t)(((int64_t)rr * ld + k) * ES) : kOOB;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int b = 8 * i + wave;
            dma16(rs, dst + b * 1024, vo, (uint32_t)((int64_t)8 * b * ld * ES));
        }
    };
    kmajor(A, row0, st);
    char* dst = st + kPjA;
    if constexpr (BKM) {
        kmajor(B, 0, dst);
    } else {
        // 64 k-rows x 256 B, block b = 8i + w holds k-rows 4b .. 4b+3; lane p ->
        // k-row 4b + p/16, physical segment p%16 holding logical (p%16) ^ 4(p/16)
        const Operand& op = B;
        const int64_t ld = op.s[0].ld;
        const int klen = op.s[0].klen;
        const i32x4 rs = make_desc(op.s[0].ptr + (int64_t)k0 * ld * ES, (int64_t)(klen - k0) * ld * ES);
        const int kq = lane >> 4;
        const int seg = (lane & 15) ^ (4 * kq);
        const int col = 8 * seg;
        const uint32_t vo = col < op.rows ? (uint32_t)(((int64_t)kq * ld + col) * ES) : kOOB;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int b = 8 * i + wave;
            dma16(rs, dst + b * 1024, vo, (uint32_t)((int64_t)4 * b * ld * ES));
        }
    }
}

// M [r, r] into LDS as NT x NT tiles of [128 r_in][256 B]; tile i NT + j
// holds M[128 i .., 128 j ..], and 16-byte segment s of tile row p sits at
// physical segment s ^ 4(p & 3).  Rows / columns past r read as zero.
template <int NT>
__device__ __forceinline__ void m_dma(const uint16_t* M, int r, char* dst, int wave, int lane) {
    constexpr int NW = 4 * NT;   // waves of the workgroup
    const i32x4 rs = make_desc(reinterpret_cast<const char*>(M), (int64_t)r * r * 2);
    const int kq = lane >> 4;
    const int seg = (lane & 15) ^ (4 * kq);
#pragma unroll
    for (int ti = 0; ti < NT; ++ti)
#pragma unroll
        for (int tj = 0; tj < NT; ++tj) {
            const int col = 128 * tj + 8 * seg;
            const uint32_t vo = col < r ? (uint32_t)(((int64_t)(128 * ti + kq) * r + col) * 2) : kOOB;
            char* tile = dst + (ti * NT + tj) * kSkM;
#pragma unroll
            for (int i = 0; i < 32 / NW; ++i) {
                const int b = NW * i + wave;   // tile rows 4b .. 4b+3
                dma16(rs, tile + b * 1024, vo, (uint32_t)((int64_t)4 * b * r * 2));
            }
        }
}

// Transposed 8-row read of a [k][256 B] tile (16-byte segments swizzled by
// 4(k & 3)): lane l receives the column 32 w + l % 32 for k rows
// 8 (l / 32) .. +7 of K step s.
__device__ __forceinline__ uint32_t tr_base(int w, int lane) {
    const int g = lane >> 4, j = lane & 15, c = j >> 2;
    const int x = 2 * (g & 1) + ((j & 3) >> 1);
    return (uint32_t)((8 * (g >> 1) + c) * 256 + 64 * (w ^ c) + 16 * x + 8 * (j & 1));
}
__device__ __forceinline__ u32x4 tr_read8(const char* tile, uint32_t base, int s) {
    const char* p = tile + base + 256u * 16 * s;
    const uint64_t lo = ds_read_tr(p);
    const uint64_t hi = ds_read_tr(p + 4 * 256);
    u32x4 v;
    v[0] = (uint32_t)lo;
    v[1] = (uint32_t)(lo >> 32);
    v[2] = (uint32_t)hi;
    v[3] = (uint32_t)(hi >> 32);
    return v;
}

// Byte offset of element (row, col) of the 32 x 128 NT bf16 operand tile,
// laid out K-major as 64-column chunks of [32 rows][128 B], chunk c of row
// stored at c ^ swz(row).
__device__ __forceinline__ int ctile_off(int row, int col) {
    return (col >> 6) * 4096 + row * 128 + ((((col >> 3) & 7) ^ ((row ^ (row >> 3)) & 7)) << 4) + (col & 7) * 2;
}

// acc (one 32x32 block per wave, columns 32 w .. of the 128 NT) over the K
// steps of a [32 x 128 NT] operand held as two tiles in LDS (A, K-major: its
// high bf16 part at `chi`, its low part at `clo`) times M (TRANS_M = false:
// B(k, n) = M[k][n]) or M^T (B(k, n) = M[n][k]), M held as NT x NT tiles.
// Each K step issues two MFMAs on the same M fragment, high part first.
template <bool TRANS_M, int NT>
__device__ __forceinline__ void mix_mma(const char* chi, const char* clo, const char* mt, int wave, int lane,
                                        f32x16& acc) {
    const int r32 = lane & 31, h = lane >> 5;
    const int wl = wave & 3, nb = wave >> 2;   // 32-column block within tile column nb
    const uint32_t tb = tr_base(wl, lane);
    const int p = 32 * wl + r32;   // tile row of M for the M^T product
#pragma unroll
    for (int kb = 0; kb < NT; ++kb) {
        const char* tile = mt + (TRANS_M ? nb * NT + kb : kb * NT + nb) * kSkM;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const int ql = 2 * s + h;     // 8-element K group of this lane within the tile
            const int q = 16 * kb + ql;   // ... within the whole rank
            const uint32_t ao = (uint32_t)((q >> 3) * 4096 + r32 * 128 + ((((q & 7) ^ (r32 & 7) ^ (r32 >> 3))) << 4));
            const u32x4 ah = *reinterpret_cast<const u32x4*>(chi + ao);
            const u32x4 al = *reinterpret_cast<const u32x4*>(clo + ao);
            u32x4 bv;
            if constexpr (!TRANS_M)
                bv = tr_read8(tile, tb, s);
            else
                bv = *reinterpret_cast<const u32x4*>(tile + p * 256 + ((ql ^ (4 * (p & 3))) << 4));
            mma32<uint16_t>(acc, ah, bv);
            mma32<uint16_t>(acc, al, bv);
        }
    }
}

// One more pass of the same product over a third operand tile `c` (the low
// part of a three-part split), accumulated into acc.
template <bool TRANS_M, int NT>
__device__ __forceinline__ void mix_mma1(const char* c, const char* mt, int wave, int lane, f32x16& acc) {
    const int r32 = lane & 31, h = lane >> 5;
    const int wl = wave & 3, nb = wave >> 2;
    const uint32_t tb = tr_base(wl, lane);
    const int p = 32 * wl + r32;
#pragma unroll
    for (int kb = 0; kb < NT; ++kb) {
        const char* tile = mt + (TRANS_M ? nb * NT + kb : kb * NT + nb) * kSkM;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const int ql = 2 * s + h;
            const int q = 16 * kb + ql;
            const u32x4 av = *reinterpret_cast<const u32x4*>(c + (q >> 3) * 4096 + r32 * 128 +
                                                             ((((q & 7) ^ (r32 & 7) ^ (r32 >> 3))) << 4));
            u32x4 bv;
            if constexpr (!TRANS_M)
                bv = tr_read8(tile, tb, s);
            else
                bv = *reinterpret_cast<const u32x4*>(tile + p * 256 + ((ql ^ (4 * (p & 3))) << 4));
            mma32<uint16_t>(acc, av, bv);
        }
    }
}

// Split-K rank projection.  Workgroup g: token block g % blocks, K piece
// (g / blocks) % S, job g / (blocks S).  Wave w owns rows 32 (w / 2) .. +31
// and rank columns 64 (w % 2) .. +63 of the job's 128 x 128 tile (two
// 32x32x16 MFMAs per K step).
template <bool BKM>
__global__ __launch_bounds__(kPjThreads, 1) void proj_kernel(ProjArgs a) {
    __shared__ __attribute__((aligned(1024))) char lds[kPjStages * kPjStage];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r32 = lane & 31, h = lane >> 5;
    const int blocks = (a.T + kPjRows - 1) / kPjRows;
    const int64_t wg = flat_block(), nb = (int64_t)blocks * a.S * a.J;
    if (wg >= nb) return;
    const int ji = (int)(wg / (blocks * a.S));
    const int rem = (int)(wg - (int64_t)ji * blocks * a.S);
    const int piece = rem / blocks;
    const int row0 = (rem - piece * blocks) * kPjRows;
    const ProjJob& jb = a.job[ji];
    const int kc0 = (int)((int64_t)a.nk * piece / a.S), kc1 = (int)((int64_t)a.nk * (piece + 1) / a.S);
    const int wr = wave >> 1, wc = wave & 1;

    // A rows 32 wr + r32: swz = (r32 & 7) ^ (r32 >> 3) ^ 4(wr & 1)
    const uint32_t fa = (uint32_t)((32 * wr + r32) * 128 + ((h ^ (r32 & 7) ^ (r32 >> 3) ^ (4 * (wr & 1))) << 4));
    uint32_t fb[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        if constexpr (BKM)   // W_up rows 64 wc + 32 j + r32: swz = (r32 & 7) ^ (r32 >> 3) ^ 4(j & 1)
            fb[j] = (uint32_t)((64 * wc + 32 * j + r32) * 128 + ((h ^ (r32 & 7) ^ (r32 >> 3) ^ (4 * (j & 1))) << 4));
        else
            fb[j] = tr_base(2 * wc + j, lane);
    }
    f32x16 acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;

    const int n = kc1 - kc0;
#pragma unroll
    for (int c = 0; c < kPjStages - 1; ++c)
        if (c < n) proj_dma<BKM>(jb.A, jb.B, row0, kc0 + c, lds + c * kPjStage, wave, lane);

    // The zeroing rides on the projection: every workgroup clears a strided
    // share while its first loads are in flight.
    {
        const int64_t stride = nb * kPjThreads;
        const int64_t gid = wg * kPjThreads + tid;
        for (int s = 0; s < a.z.count; ++s) {
            float* p = a.z.ptr[s];
            const int64_t cnt = a.z.n[s];
            const int64_t n4 = cnt >> 2;
            for (int64_t i = gid; i < n4; i += stride)
                reinterpret_cast<f32x4*>(p)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            for (int64_t i = (n4 << 2) + gid; i < cnt; i += stride) p[i] = 0.f;
        }
    }
    for (int i = 0; i < n; ++i) {
        // chunk i has landed once at most (stages - 2) later chunks are in flight
        const int ahead = min(n - 1 - i, kPjStages - 2);
        if (ahead >= 2)
            wait_vmcnt<2 * kPjLoads>();
        else if (ahead == 1)
            wait_vmcnt<kPjLoads>();
        else
            wait_vmcnt<0>();
        __syncthreads();
        if (i + kPjStages - 1 < n)
            proj_dma<BKM>(jb.A, jb.B, row0, kc0 + i + kPjStages - 1,
                          lds + ((i + kPjStages - 1) % kPjStages) * kPjStage, wave, lane);
        const char* st = lds + (i % kPjStages) * kPjStage;
        const char* sb = st + kPjA;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const u32x4 av = *reinterpret_cast<const u32x4*>(st + (fa ^ ((uint32_t)s << 5)));
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                u32x4 bv;
                if constexpr (BKM)
                    bv = *reinterpret_cast<const u32x4*>(sb + (fb[j] ^ ((uint32_t)s << 5)));
                else
                    bv = tr_read8(sb, fb[j], s);
                mma32<uint16_t>(acc[j], av, bv);
            }
        }
    }

    // acc[j][v]: row 32 wr + 8(v/4) + 4h + v%4, column c0 + 64 wc + 32 j + r32;
    // rows past T are dropped by the buffer range check, columns past the
    // job's width by the kOOB offset
    const int ldp = a.ldp, n_cols = jb.B.rows;
    const __amdgpu_buffer_rsrc_t rp =
        make_rsrc(reinterpret_cast<const char*>(a.P + piece * a.pstride + jb.c0) + (int64_t)row0 * ldp * 4,
                  (int64_t)(a.T - row0) * ldp * 4);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int col = 64 * wc + 32 * j + r32;
        const uint32_t vo = col < n_cols ? (uint32_t)(((32 * wr + 4 * h) * ldp + col) * 4) : kOOB;
#pragma unroll
        for (int v = 0; v < 16; ++v)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[j][v]), rp, vo,
                                                  (uint32_t)((8 * (v >> 2) + (v & 3)) * ldp * 4), 0);
    }
}

// acc[v] = sum over the S partials of token row0 + 8(v/4) + 4h + v%4, rank
// column c0 + col of the group (zero past T or past the group's r).  The
// partials are loaded four at a time, all loads of a batch issued before any
// is used, so S <= 4 costs one memory round trip; the sum keeps the order
// partial 0, 1, 2, ...  Slots past S read through a zero-length buffer (no
// memory access, value 0), which leaves the sum unchanged.
__device__ __forceinline__ void sum_partials(const BranchArgs& a, int row0, int c0, int col, int h, f32x16& acc) {
    constexpr int kBatch = 4;
    const int R = a.R;
    const uint32_t vo = col < a.r ? (uint32_t)(((4 * h) * R + col) * 4) : kOOB;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.f;
    for (int s0 = 0; s0 < a.S; s0 += kBatch) {
        float x[kBatch][16];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const bool live = s0 + i < a.S;
            const __amdgpu_buffer_rsrc_t rp =
                make_rsrc(reinterpret_cast<const char*>(a.P + (live ? (s0 + i) * a.pstride : 0) + c0) +
                              (int64_t)row0 * R * 4,
                          live ? (int64_t)(a.T - row0) * R * 4 : 0);
#pragma unroll
            for (int v = 0; v < 16; ++v)
                x[i][v] = __uint_as_float(
                    __builtin_amdgcn_raw_buffer_load_b32(rp, vo, (uint32_t)((8 * (v >> 2) + (v & 3)) * R * 4), 0));
        }
#pragma unroll
        for (int i = 0; i < kBatch; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[v] += x[i][v];
    }
}

// Sum over the 32 rows of a wave's block, per column (lanes l and l ^ 32
// hold the same column); every lane returns the column total.
__device__ __forceinline__ float block_colsum(const float (&x)[16]) {
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) s += x[v];
    return s + __shfl_xor(s, 32);
}

// Workgroup b of a chain launch: token block b / G, group b % G.  Wave w
// owns rank column 32 w + lane % 32 of the group (NT = 1: 4 waves, 128 ranks;
// NT = 2: 8 waves, 256 ranks).
struct ChainPos {
    int row0, g, c0;
};
__device__ __forceinline__ ChainPos chain_pos(const BranchArgs& a) {
    const int64_t wg = flat_block();
    const int tb = (int)(wg / a.G);
    const int g = (int)(wg - (int64_t)tb * a.G);
    return ChainPos{tb * kSkRows, g, g * a.r};
}
// False for the surplus workgroups of the last grid row.
__device__ __forceinline__ bool chain_live(const BranchArgs& a) {
    return flat_block() < (int64_t)((a.T + kSkRows - 1) / kSkRows) * a.G;
}

// Buffer resource over a token-major array with row stride `ld` elements
// (element size es), from token row0 and column c0: offsets (row * ld + col)
// * es.  Rows past T fall past its end.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* base, int T, int row0, int64_t ld,
                                                            int64_t c0, int es) {
    return make_rsrc(reinterpret_cast<const char*>(base) + ((int64_t)row0 * ld + c0) * es,
                     (int64_t)(T - row0) * ld * es);
}
// The group's columns of a [T, R] array.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t group_rsrc(const void* base, const BranchArgs& a, const ChainPos& q,
                                                             int es) {
    return rows_rsrc(base, a.T, q.row0, a.R, q.c0, es);
}

// The wave's 32 x 32 block of P M (TRANS = false) or P M^T (TRANS = true)
// for a float32 operand P held in registers (the lane's 16 values at rows
// 8(v/4) + 4h + v%4, column col): P goes to the operand tiles in three bf16
// parts (two passes), so the product is as accurate as a float32 one.
// Leaves the tiles free (a barrier after the last read).
template <bool TRANS, int NT>
__device__ __forceinline__ void mix3(const float (&pv)[16], char* chi, char* clo, const char* mt, int wave, int lane,
                                     int col, f32x16& acc) {
    const int h = lane >> 5;
    uint16_t lo[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int row = 8 * (v >> 2) + 4 * h + (v & 3);
        const BfTriple t = bf_split3(pv[v]);
        *reinterpret_cast<uint16_t*>(chi + ctile_off(row, col)) = t.hi;
        *reinterpret_cast<uint16_t*>(clo + ctile_off(row, col)) = t.mid;
        lo[v] = t.lo;
        acc[v] = 0.f;
    }
    __syncthreads();
    mix_mma<TRANS, NT>(chi, clo, mt, wave, lane, acc);
    __syncthreads();   // every wave is done with the high part
#pragma unroll
    for (int v = 0; v < 16; ++v)
        *reinterpret_cast<uint16_t*>(chi + ctile_off(8 * (v >> 2) + 4 * h + (v & 3), col)) = lo[v];
    __syncthreads();
    mix_mma1<TRANS, NT>(chi, mt, wave, lane, acc);
    __syncthreads();   // done reading the tiles
}

// Forward chain.  L = 2: the two-application form with M (CosNet for F =
// Cos); L = 1: C2 = f(H w1 + p1), M, w2, p2 not read; L = 3 (the 3-layer
// CosNet): C3 = f((C2 M') w3 + p3) after the second layer, M' = a.M2.  Each
// mixing operand (C1, and C2 in the 3-layer form) enters the MFMAs as three
// bf16 parts (bf_split3: high and middle parts from the two operand tiles,
// then the low part from the first tile again), so every mixing product is
// as accurate as a float32 one and the cosine arguments carry float32
// rounding only.
template <Act F, int L, int NT>
__global__ __launch_bounds__(kThreads * NT, 1) void branch_fwd_kernel(BranchArgs a) {
    static_assert(L != 3 || NT == 1, "the 3-layer form holds both mixing matrices in LDS at r <= 128");
    __shared__ __attribute__((aligned(1024))) char lds[sk_lds<NT, L>()];
    char* mt = lds;
    char* mt2 = mt + NT * NT * kSkM;   // 3-layer form
    char* chi = mt + (L == 3 ? 2 : 1) * NT * NT * kSkM;
    char* clo = chi + NT * kSkC;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r32 = lane & 31, h = lane >> 5;
    if (!chain_live(a)) return;
    const ChainPos q = chain_pos(a);
    const int r = a.r, R = a.R;

    // M (and M') land while the partials are summed
    if constexpr (L >= 2) m_dma<NT>(a.M + (int64_t)q.g * r * r, r, mt, wave, lane);
    if constexpr (L == 3) m_dma<NT>(a.M2 + (int64_t)q.g * r * r, r, mt2, wave, lane);
    // acc[v]: token row0 + 8(v/4) + 4h + v%4, rank column 32 wave + r32 of the group
    const int col = 32 * wave + r32;
    f32x16 acc;
    sum_partials(a, q.row0, q.c0, col, h, acc);

    const bool cv = col < r;
    const float w1 = cv ? a.w1[q.c0 + col] : 0.f, p1 = cv ? a.p1[q.c0 + col] : 0.f;
    const __amdgpu_buffer_rsrc_t rh = group_rsrc(a.H, a, q, 4);
    const __amdgpu_buffer_rsrc_t rc = group_rsrc(a.C2s, a, q, 2);
    const uint32_t vo4 = cv ? (uint32_t)(((4 * h) * R + col) * 4) : kOOB;
    const uint32_t vo2 = cv ? (uint32_t)(((4 * h) * R + col) * 2) : kOOB;
    auto soff = [&](int v, int es) { return (uint32_t)((8 * (v >> 2) + (v & 3)) * R * es); };
    const bool keep_h = a.H != nullptr;   // NULL: inference-only forward
    // H is read again only by the backward, after every other projection's
    // forward: it is stored non-temporal, so that it does not linger dirty in
    // the memory-side cache.
    // Stores count in vmcnt: in the mixing forms H is stored after the
    // barrier, whose wait for M would otherwise also wait for them.
    auto store_h = [&]() {
        if (keep_h)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[v]), rh, vo4, soff(v, 4), kStoreNT);
    };
    float c1[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) c1[v] = cv ? act_value<F, true>(acc[v] * w1 + p1) : 0.f;
    if constexpr (L == 1) {
        store_h();
#pragma unroll
        for (int v = 0; v < 16; ++v)
            __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf(c1[v]), rc, vo2, soff(v, 2), 0);
        return;
    }
    const float w2 = cv ? a.w2[q.c0 + col] : 0.f, p2 = cv ? a.p2[q.c0 + col] : 0.f;
    wait_vmcnt<0>();   // this wave's part of M (and M') has landed
    store_h();
    f32x16 h2;
    mix3<false, NT>(c1, chi, clo, mt, wave, lane, col, h2);   // H2 = C1 M (its first barrier publishes M)
    float c2[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) c2[v] = cv ? act_value<F, true>(h2[v] * w2 + p2) : 0.f;
    if constexpr (L == 3) {
        const float w3 = cv ? a.w3[q.c0 + col] : 0.f, p3 = cv ? a.p3[q.c0 + col] : 0.f;
        f32x16 h3;
        mix3<false, NT>(c2, chi, clo, mt2, wave, lane, col, h3);   // H3 = C2 M'
#pragma unroll
        for (int v = 0; v < 16; ++v) c2[v] = cv ? act_value<F, true>(h3[v] * w3 + p3) : 0.f;
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf(c2[v]), rc, vo2, soff(v, 2), 0);
}

// Backward chain, same forms as branch_fwd_kernel.  The one-application form
// writes C2 and dH only (no C1, dH2 and no second frequency/phase).
//
// Scratch layouts (operands of the weight-gradient products, each a high +
// low bf16 pair so that those products are float32-accurate):
//  - C1 and dH2 (and in the 3-layer form the middle C2 and dH3): [T][G][2 r],
//    group g's high part in columns 2 g r .. 2 g r + r - 1 and its low part
//    in the next r (row stride 2 R);
//  - dH: [T][2 R], the high part of all groups in columns 0 .. R - 1, the
//    low part in R .. 2 R - 1 (the dx product reads only the high part);
//  - the branch output (C2, or C3): [T][R], one bf16 value (the operand of
//    dW_up).
// The recomputed mixing products take their float32 operand in three
// parts, as the forward does (so the cosine arguments are the forward's);
// the gradient mixing products (dC1 = dH2 M^T, dC2 = dH3 M'^T) take theirs as
// a high + low pair.
template <Act F, int L, int NT>
__global__ __launch_bounds__(kThreads * NT, 1) void branch_bwd_kernel(BranchArgs a) {
    static_assert(L != 3 || NT == 1, "the 3-layer form holds both mixing matrices in LDS at r <= 128");
    __shared__ __attribute__((aligned(1024))) char lds[sk_lds<NT, L>()];
    char* mt = lds;
    char* mt2 = mt + NT * NT * kSkM;   // 3-layer form
    char* chi = mt + (L == 3 ? 2 : 1) * NT * NT * kSkM;
    char* clo = chi + NT * kSkC;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r32 = lane & 31, h = lane >> 5;
    if (!chain_live(a)) return;
    const ChainPos q = chain_pos(a);
    const int r = a.r, R = a.R;
    // targets of the frequency / phase gradient sums
    float* gw1 = a.dw1;
    float* gp1 = a.dp1;
    float* gw2 = a.dw2;
    float* gp2 = a.dp2;
    float* gw3 = a.dw3;
    float* gp3 = a.dp3;
    if (a.copies) {
        float* c = a.copies + (flat_block() % kChainCopies) * R;
        const int64_t arr = (int64_t)kChainCopies * R;
        gw1 = c;
        gp1 = c + arr;
        gw2 = c + 2 * arr;
        gp2 = c + 3 * arr;
        gw3 = c + 4 * arr;
        gp3 = c + 5 * arr;
    }

    if constexpr (L >= 2) m_dma<NT>(a.M + (int64_t)q.g * r * r, r, mt, wave, lane);
    if constexpr (L == 3) m_dma<NT>(a.M2 + (int64_t)q.g * r * r, r, mt2, wave, lane);
    const int col = 32 * wave + r32;
    const bool cv = col < r;
    const int gc = q.c0 + col;   // column of the [R] vectors
    const int64_t rows_left = a.T - q.row0;
    const __amdgpu_buffer_rsrc_t rh = group_rsrc(a.H, a, q, 4);
    const __amdgpu_buffer_rsrc_t rc2 = group_rsrc(a.C2s, a, q, 2);
    // dH [T][2R]: high part at column gc, low part at R + gc
    const __amdgpu_buffer_rsrc_t rdh = rows_rsrc(a.dHs, a.T, q.row0, 2 * (int64_t)R, q.c0, 2);
    const uint32_t vo4 = cv ? (uint32_t)(((4 * h) * R + col) * 4) : kOOB;
    const uint32_t vo2 = cv ? (uint32_t)(((4 * h) * R + col) * 2) : kOOB;
    const uint32_t vw2 = cv ? (uint32_t)(((4 * h) * 2 * R + col) * 2) : kOOB;   // row stride 2R
    auto soff = [&](int v, int es) { return (uint32_t)((8 * (v >> 2) + (v & 3)) * R * es); };
    auto soffw = [&](int v) { return (uint32_t)((8 * (v >> 2) + (v & 3)) * 2 * R * 2); };
    const uint32_t lo_off = (uint32_t)r * 2;   // [T][G][2r] pairs: bytes from the high part to the low part
    // the group's pair columns of a [T][G][2r] array start at 2 c0
    auto pair_rsrc = [&](const uint16_t* base) {
        return rows_rsrc(base, a.T, q.row0, 2 * (int64_t)R, 2 * (int64_t)q.c0, 2);
    };
    auto store_pair = [&](__amdgpu_buffer_rsrc_t rs, int v, uint16_t hi, uint16_t lo) {
        __builtin_amdgcn_raw_buffer_store_b16(hi, rs, vw2, soffw(v), 0);
        __builtin_amdgcn_raw_buffer_store_b16(lo, rs, vw2 + lo_off, soffw(v), 0);
    };
    auto row_of = [&](int v) { return 8 * (v >> 2) + 4 * h + (v & 3); };

    // H from the reserve (rows past T and columns past r read as zero),
    // issued before the partial sums so that both arrive in one round trip
    float hr[16], d1[16];
#pragma unroll
    for (int v = 0; v < 16; ++v)
        hr[v] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rh, vo4, soff(v, 4), 0));
    f32x16 dc2;
    sum_partials(a, q.row0, q.c0, col, h, dc2);   // the output's gradient dy W_up^T
    // A1 = H w1 + p1, keep f'(A1)
    const float w1 = cv ? a.w1[gc] : 0.f, p1 = cv ? a.p1[gc] : 0.f;
    float c1[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        float f = 0.f, d = 0.f;
        if (cv) act_value_slope<F, true>(hr[v] * w1 + p1, f, d);
        d1[v] = d;
        c1[v] = f;
    }

    // dC1: the output's gradient itself (one application), or back through
    // the mixing layers
    f32x16 dc1;
    if constexpr (L == 1) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf(c1[v]), rc2, vo2, soff(v, 2), 0);   // C2 = C1
            dc1[v] = dc2[v];
        }
    } else {
        const float w2 = cv ? a.w2[gc] : 0.f, p2 = cv ? a.p2[gc] : 0.f;
        const __amdgpu_buffer_rsrc_t rc1 = pair_rsrc(a.C1s), rdh2 = pair_rsrc(a.dH2s);
        wait_vmcnt<0>();   // this wave's part of M (and M') has landed
        // C1's pair (for dM) to scratch; the barrier in mix3 publishes M
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const BfPair c = bf_split(c1[v]);
            store_pair(rc1, v, c.hi, c.lo);
        }
        f32x16 h2;
        mix3<false, NT>(c1, chi, clo, mt, wave, lane, col, h2);   // H2 = C1 M
        // A2 = H2 w2 + p2: C2 = f(A2), keep f'(A2)
        float c2[16], d2[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            float f = 0.f, d = 0.f;
            if (cv) act_value_slope<F, true>(h2[v] * w2 + p2, f, d);
            c2[v] = f;
            d2[v] = d;
        }
        f32x16 dcm;   // gradient of C2
        if constexpr (L == 2) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf(c2[v]), rc2, vo2, soff(v, 2), 0);
                dcm[v] = dc2[v];
            }
        } else {
            // the third layer: H3 = C2 M', A3 = H3 w3 + p3, C3 = f(A3);
            // dA3 = f'(A3) dC3, dH3 = dA3 w3, dC2 = dH3 M'^T
            const float w3 = cv ? a.w3[gc] : 0.f, p3 = cv ? a.p3[gc] : 0.f;
            const __amdgpu_buffer_rsrc_t rc2m = pair_rsrc(a.C2ms), rdh3 = pair_rsrc(a.dH3s);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const BfPair c = bf_split(c2[v]);
                store_pair(rc2m, v, c.hi, c.lo);
            }
            f32x16 h3;
            mix3<false, NT>(c2, chi, clo, mt2, wave, lane, col, h3);
            float da3h3[16], da3[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const bool ok = cv && row_of(v) < rows_left;
                float f = 0.f, d = 0.f;
                if (cv) act_value_slope<F, true>(h3[v] * w3 + p3, f, d);
                __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf(f), rc2, vo2, soff(v, 2), 0);
                const float g = ok ? d * dc2[v] : 0.f;
                da3[v] = g;
                da3h3[v] = g * h3[v];
                const BfPair dh3 = bf_split(g * w3);
                *reinterpret_cast<uint16_t*>(chi + ctile_off(row_of(v), col)) = dh3.hi;
                *reinterpret_cast<uint16_t*>(clo + ctile_off(row_of(v), col)) = dh3.lo;
                store_pair(rdh3, v, dh3.hi, dh3.lo);
            }
            {
                const float sw = block_colsum(da3h3), sp = block_colsum(da3);
                if (h == 0 && cv) {
                    unsafeAtomicAdd(gw3 + gc, sw);
                    unsafeAtomicAdd(gp3 + gc, sp);
                }
            }
            __syncthreads();   // dH3 tiles complete
#pragma unroll
            for (int v = 0; v < 16; ++v) dcm[v] = 0.f;
            mix_mma<true, NT>(chi, clo, mt2, wave, lane, dcm);   // dC2 = dH3 M'^T
            __syncthreads();                                      // done reading the dH3 tiles
        }

        // dA2 = f'(A2) dC2, dH2 = dA2 w2
        float da2h2[16], da2[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const bool ok = cv && row_of(v) < rows_left;
            const float g = ok ? d2[v] * dcm[v] : 0.f;
            da2[v] = g;
            da2h2[v] = g * h2[v];
            const BfPair dh2 = bf_split(g * w2);
            *reinterpret_cast<uint16_t*>(chi + ctile_off(row_of(v), col)) = dh2.hi;
            *reinterpret_cast<uint16_t*>(clo + ctile_off(row_of(v), col)) = dh2.lo;
            store_pair(rdh2, v, dh2.hi, dh2.lo);
        }
        {
            const float sw = block_colsum(da2h2), sp = block_colsum(da2);
            if (h == 0 && cv) {
                unsafeAtomicAdd(gw2 + gc, sw);
                unsafeAtomicAdd(gp2 + gc, sp);
            }
        }
        __syncthreads();   // dH2 tiles complete

#pragma unroll
        for (int v = 0; v < 16; ++v) dc1[v] = 0.f;
        mix_mma<true, NT>(chi, clo, mt, wave, lane, dc1);   // dC1 = dH2 M^T
    }

    // dA1 = f'(A1) dC1; dw1 += dA1 H, dp1 += dA1; dH = dA1 w1
    float da1h[16], da1[16];
    const uint32_t dh_lo = (uint32_t)R * 2;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const bool ok = cv && row_of(v) < rows_left;
        const float g = ok ? d1[v] * dc1[v] : 0.f;
        da1[v] = g;
        da1h[v] = g * hr[v];
        const BfPair dh = bf_split(g * w1);
        __builtin_amdgcn_raw_buffer_store_b16(dh.hi, rdh, vw2, soffw(v), 0);
        __builtin_amdgcn_raw_buffer_store_b16(dh.lo, rdh, vw2 + dh_lo, soffw(v), 0);
    }
    const float sw = block_colsum(da1h), sp = block_colsum(da1);
    if (h == 0 && cv) {
        unsafeAtomicAdd(gw1 + gc, sw);
        unsafeAtomicAdd(gp1 + gc, sp);
    }
}

}  // namespace noble
