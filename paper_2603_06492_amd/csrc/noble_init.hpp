// Parameter initialisation of the layer's training recipe (Sec. 3.3 and the
// defaults of App. A) as one device fill.
//
// Random numbers come from Philox4x32-10, the counter-based generator of
// Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2,
// 3" (SC 2011): ten rounds of two 32x32 -> 64-bit multiplications mixed with
// the key, the key bumped by two Weyl constants between rounds.  Element e of
// tensor t takes the block at counter (e mod 2^32, e / 2^32, t, 0), so every
// value depends only on (seed, t, e), never on the launch shape.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace noble {

struct Philox4 {
    uint32_t x[4];
};

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                                 uint32_t k1) {
    constexpr uint32_t kMul0 = 0xD2511F53u, kMul1 = 0xCD9E8D57u;
    constexpr uint32_t kWeyl0 = 0x9E3779B9u, kWeyl1 = 0xBB67AE85u;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += kWeyl0;
            k1 += kWeyl1;
        }
        const uint64_t p0 = (uint64_t)kMul0 * c0;
        const uint64_t p1 = (uint64_t)kMul1 * c2;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    return Philox4{{c0, c1, c2, c3}};
}

// One tensor of the fill: kind 0 = normal N(0, a^2), 1 = uniform [a, b],
// 2 = zeros.  bf16 = 1 stores bf16 (nearest even), else float32.
struct InitTensor {
    void* ptr;
    int64_t n;
    double a, b;
    int kind, bf16, tensor_id, pad_;
};

constexpr int kMaxInit = 9;

struct InitList {
    InitTensor t[kMaxInit];
    int count;
    uint32_t k0, k1;
};

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__global__ __launch_bounds__(256) void init_kernel(InitList L) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int i = 0; i < L.count; ++i) {
        const InitTensor t = L.t[i];
        for (int64_t e = gid; e < t.n; e += stride) {
            double v = 0.0;
            if (t.kind != 2) {
                const Philox4 r = philox4x32_10((uint32_t)e, (uint32_t)((uint64_t)e >> 32), (uint32_t)t.tensor_id,
                                                0u, L.k0, L.k1);
                const double u0 = ((double)r.x[0] + 0.5) * 0x1p-32;
                if (t.kind == 1) {
                    v = t.a + (t.b - t.a) * u0;
                } else {
                    const double u1 = ((double)r.x[1] + 0.5) * 0x1p-32;
                    v = t.a * sqrt(-2.0 * log(u0)) * cos(6.283185307179586 * u1);
                }
            }
            const float f = (float)v;
            if (t.bf16)
                static_cast<uint16_t*>(t.ptr)[e] = f32_to_bf16_rne(f);
            else
                static_cast<float*>(t.ptr)[e] = f;
        }
    }
}

}  // namespace noble
