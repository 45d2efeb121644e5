// Device building blocks shared by every NOBLE kernel on gfx950 (CDNA4):
// LDS tile layout, global->LDS staging for both operand orientations, and the
// 16x16 MFMA step.
//
// Tiles are staged through LDS as "rows x 128 bytes": each row of an operand
// tile (a row of A, or a column of B) holds one K-chunk of 128 bytes (64 bf16 or
// 32 f32) as eight 16-byte chunks.  The chunk index is XOR-swizzled with the
// row so that both the row-wise stores and the MFMA fragment loads (16 rows at
// one chunk) spread over all LDS banks.  Operands stored MN-contiguous in HBM
// (W in the forward, x^T and dy in the weight gradients) are transposed in
// registers while staging, so the MFMA loop is the same for every layout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace noble {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;   // four wave64 per workgroup
constexpr int kRowBytes = 128;  // bytes of one LDS tile row (one K chunk)

// Element traits: VEC elements per 16-byte vector, BK elements per K chunk.
template <typename E> struct Elt;
template <> struct Elt<uint16_t> { static constexpr int VEC = 8; static constexpr int BK = 64; };
template <> struct Elt<float> { static constexpr int VEC = 4; static constexpr int BK = 32; };

__device__ __forceinline__ int lds_off(int row, int chunk) {
    return row * kRowBytes + ((chunk ^ ((row ^ (row >> 3)) & 7)) << 4);
}

// bf16 <-> f32 (bf16 kept as raw uint16 bits).  Round to nearest even.
__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }
__device__ __forceinline__ uint32_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
template <typename E> __device__ __forceinline__ E to_elt(float f);
template <> __device__ __forceinline__ uint16_t to_elt<uint16_t>(float f) { return (uint16_t)f2bf(f); }
template <> __device__ __forceinline__ float to_elt<float>(float f) { return f; }

// One K segment of an operand.  Element (row, k) of a K-major operand is at
// ptr[row * ld + k]; of an MN-major operand at ptr[k * ld + row].
struct Seg {
    const char* ptr;
    int64_t ld;
    int klen;   // valid K extent of the segment (elements)
    int pad_;
};

// An operand made of up to two K segments (the second one is the K-extension
// that appends the rank-r branch to a main product).  K chunks [0, nk1) come
// from segment 0, the rest from segment 1, each starting at its own k = 0.
struct Operand {
    Seg s[2];
    int nk1;
    int rows;   // valid extent along M (operand A) or N (operand B)
};

// Raw buffer resource over [base, base + bytes).  Loads at offsets at or past
// the end return zero, which is how tile edges and K tails are zero-filled
// without branches.  Offsets inside one tile stay below 2^31.
constexpr uint32_t kOOB = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const char* base, int64_t bytes) {
    const int n = bytes <= 0 ? 0 : (bytes >= 0x7fffffff ? 0x7fffffff : (int)bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), (short)0, n, 0x00020000);
}
__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0);
}

// Global -> registers -> LDS staging of one R-row operand tile for one K chunk.
template <typename E, int R, bool KMAJ>
struct Stage {
    static constexpr int VEC = Elt<E>::VEC;
    static constexpr int BK = Elt<E>::BK;
    static constexpr int ES = (int)sizeof(E);
    static constexpr int NB = R / VEC;                     // MN-major: vector columns
    static constexpr int UNITS = KMAJ ? R * 8 : 8 * NB;     // 16B chunks or VECxVEC blocks
    static constexpr int PER = (UNITS + kThreads - 1) / kThreads;
    static constexpr int NREG = KMAJ ? PER : PER * VEC;
    u32x4 v[NREG];

    __device__ __forceinline__ void load(const Operand& op, int row0, int kc, int tid) {
        const bool second = kc >= op.nk1;
        const char* ptr = second ? op.s[1].ptr : op.s[0].ptr;
        const int64_t ld = second ? op.s[1].ld : op.s[0].ld;
        const int klen = second ? op.s[1].klen : op.s[0].klen;
        const int k0 = (second ? kc - op.nk1 : kc) * BK;
        if constexpr (KMAJ) {
            // Tile rows row0.. of a [rows, ld] matrix; thread t loads rows
            // t/8 + 32i, chunk t%8.  Rows past the matrix fall past the end.
            static_assert(kThreads % 8 == 0 && (UNITS % kThreads == 0), "whole passes");
            const __amdgpu_buffer_rsrc_t rs =
                make_rsrc(ptr + (int64_t)row0 * ld * ES, (int64_t)(op.rows - row0) * ld * ES);
            const int r = tid >> 3, k = k0 + (tid & 7) * VEC;
            const uint32_t vo = k < klen ? (uint32_t)(((int64_t)r * ld + k) * ES) : kOOB;
#pragma unroll
            for (int i = 0; i < PER; ++i)
                v[i] = buf_load16(rs, vo, (uint32_t)((int64_t)i * (kThreads / 8) * ld * ES));
        } else {
            // K rows k0.. of a [klen, ld] matrix; VEC rows of one VEC-wide column
            // block per thread.  K rows past the end fall past the end.
            const __amdgpu_buffer_rsrc_t rs =
                make_rsrc(ptr + (int64_t)k0 * ld * ES, (int64_t)(klen - k0) * ld * ES);
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int u = tid + i * kThreads;
                const int kb = u / NB, nb = u % NB;
                const int col = row0 + nb * VEC;
                const bool ok = ((UNITS % kThreads == 0) || u < UNITS) && col < op.rows;
                const uint32_t vo = ok ? (uint32_t)(((int64_t)kb * VEC * ld + col) * ES) : kOOB;
#pragma unroll
                for (int e = 0; e < VEC; ++e) v[i * VEC + e] = buf_load16(rs, vo, (uint32_t)((int64_t)e * ld * ES));
            }
        }
    }

    __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int u = tid + i * kThreads;
            if (!((UNITS % kThreads == 0) || u < UNITS)) continue;
            if constexpr (KMAJ) {
                *reinterpret_cast<u32x4*>(lds + lds_off(u >> 3, u & 7)) = v[i];
            } else {
                const int kb = u / NB, nb = u % NB;
                if constexpr (VEC == 8) {
                    // 8x8 bf16 transpose: out[n] holds k = 0..7 of column n.
#pragma unroll
                    for (int n = 0; n < 8; ++n) {
                        u32x4 o;
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const uint32_t lo = v[i * 8 + 2 * j][n >> 1];
                            const uint32_t hi = v[i * 8 + 2 * j + 1][n >> 1];
                            o[j] = (n & 1) ? ((lo >> 16) | (hi & 0xffff0000u))
                                           : ((lo & 0xffffu) | (hi << 16));
                        }
                        *reinterpret_cast<u32x4*>(lds + lds_off(nb * 8 + n, kb)) = o;
                    }
                } else {
#pragma unroll
                    for (int n = 0; n < 4; ++n) {
                        u32x4 o;
#pragma unroll
                        for (int j = 0; j < 4; ++j) o[j] = v[i * 4 + j][n];
                        *reinterpret_cast<u32x4*>(lds + lds_off(nb * 4 + n, kb)) = o;
                    }
                }
            }
        }
    }

    // Split staging for software pipelining: part p of NP.  K-major operands
    // split their loads and stores evenly.  MN-major operands (a VEC x VEC
    // transpose per thread needs all VEC rows) store everything and reload
    // everything in part 0, which leaves the reload a whole K chunk of cover.
    template <int NP>
    __device__ __forceinline__ void load_part(const Operand& op, int row0, int kc, int tid, int p) {
        static_assert(PER % NP == 0 || !KMAJ, "even split");
        if constexpr (KMAJ) {
            const bool second = kc >= op.nk1;
            const char* ptr = second ? op.s[1].ptr : op.s[0].ptr;
            const int64_t ld = second ? op.s[1].ld : op.s[0].ld;
            const int klen = second ? op.s[1].klen : op.s[0].klen;
            const int k0 = (second ? kc - op.nk1 : kc) * BK;
            const __amdgpu_buffer_rsrc_t rs =
                make_rsrc(ptr + (int64_t)row0 * ld * ES, (int64_t)(op.rows - row0) * ld * ES);
            const int r = tid >> 3, k = k0 + (tid & 7) * VEC;
            const uint32_t vo = k < klen ? (uint32_t)(((int64_t)r * ld + k) * ES) : kOOB;
#pragma unroll
            for (int i = p * (PER / NP); i < (p + 1) * (PER / NP); ++i)
                v[i] = buf_load16(rs, vo, (uint32_t)((int64_t)i * (kThreads / 8) * ld * ES));
        } else {
            if (p == 0) load(op, row0, kc, tid);
        }
    }

    template <int NP>
    __device__ __forceinline__ void store_part(char* lds, int tid, int p) const {
        if constexpr (KMAJ) {
#pragma unroll
            for (int i = p * (PER / NP); i < (p + 1) * (PER / NP); ++i) {
                const int u = tid + i * kThreads;
                *reinterpret_cast<u32x4*>(lds + lds_off(u >> 3, u & 7)) = v[i];
            }
        } else {
            if (p != 0) return;
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int u = tid + i * kThreads;
                if (!((UNITS % kThreads == 0) || u < UNITS)) continue;
                const int kb = u / NB, nb = u % NB;
#pragma unroll
                for (int n = 0; n < VEC; ++n) {
                    u32x4 o;
                    if constexpr (VEC == 8) {
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const uint32_t lo = v[i * 8 + 2 * j][n >> 1];
                            const uint32_t hi = v[i * 8 + 2 * j + 1][n >> 1];
                            o[j] = (n & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
                        }
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j) o[j] = v[i * 4 + j][n];
                    }
                    *reinterpret_cast<u32x4*>(lds + lds_off(nb * VEC + n, kb)) = o;
                }
            }
        }
    }
};

// One 16x16 output tile += A_frag (16 x 32 bf16 | 16 x 16 f32) * B_frag.
// Lane l supplies row (l % 16) and the 16-byte chunk (l / 16) of the K step.
template <typename E> __device__ __forceinline__ void mma(f32x4& c, const u32x4& a, const u32x4& b);
template <> __device__ __forceinline__ void mma<uint16_t>(f32x4& c, const u32x4& a, const u32x4& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <> __device__ __forceinline__ void mma<float>(f32x4& c, const u32x4& a, const u32x4& b) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[q]), __uint_as_float(b[q]), c, 0, 0, 0);
}

// acc[i][j] += A(rows wm0+16i..) * B(rows wn0+16j..) over one 128-byte K chunk
// held in LDS.  Output element (v) of acc[i][j] in lane l is
// C[wm0 + 16i + 4*(l/16) + v][wn0 + 16j + l%16].
template <typename E, int TM, int TN>
__device__ __forceinline__ void mma_chunk(const char* ldsA, const char* ldsB, int wm0, int wn0,
                                          int lane, f32x4 (&acc)[TM][TN]) {
    const int r16 = lane & 15, g = lane >> 4;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        u32x4 a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
            a[i] = *reinterpret_cast<const u32x4*>(ldsA + lds_off(wm0 + 16 * i + r16, 4 * s + g));
#pragma unroll
        for (int j = 0; j < TN; ++j)
            b[j] = *reinterpret_cast<const u32x4*>(ldsB + lds_off(wn0 + 16 * j + r16, 4 * s + g));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) mma<E>(acc[i][j], a[i], b[j]);
    }
}

// Double-buffered main loop over K chunks [kc0, kc1) of a BM x BN tile whose
// top-left output is (m0, n0).  Four waves as WM x WN.  `lds` must hold
// 2 * (BM + BN) * 128 bytes.  On return every wave has passed a barrier after
// its last LDS read, so the caller may reuse `lds`.
template <typename E, int BM, int BN, int WM, int WN, bool AK, bool BKM>
__device__ __forceinline__ void mainloop(const Operand& A, const Operand& B, int m0, int n0,
                                         int kc0, int kc1, char* lds,
                                         f32x4 (&acc)[BM / WM / 16][BN / WN / 16]) {
    static_assert(WM * WN == 4, "four waves");
    constexpr int TM = BM / WM / 16, TN = BN / WN / 16;
    constexpr int STAGE = (BM + BN) * kRowBytes;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm0 = (wave / WN) * (BM / WM), wn0 = (wave % WN) * (BN / WN);
    if (kc0 >= kc1) return;
    Stage<E, BM, AK> sa;
    Stage<E, BN, BKM> sb;
    sa.load(A, m0, kc0, tid);
    sb.load(B, n0, kc0, tid);
    sa.store(lds, tid);
    sb.store(lds + BM * kRowBytes, tid);
    __syncthreads();
    for (int kc = kc0; kc < kc1; ++kc) {
        char* cur = lds + ((kc - kc0) & 1) * STAGE;
        char* nxt = lds + (((kc - kc0) & 1) ^ 1) * STAGE;
        const bool more = kc + 1 < kc1;
        if (more) {
            sa.load(A, m0, kc + 1, tid);
            sb.load(B, n0, kc + 1, tid);
        }
        mma_chunk<E, TM, TN>(cur, cur + BM * kRowBytes, wm0, wn0, lane, acc);
        if (more) {
            sa.store(nxt, tid);
            sb.store(nxt + BM * kRowBytes, tid);
        }
        __syncthreads();
    }
}

}  // namespace noble
