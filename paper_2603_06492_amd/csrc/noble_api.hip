// libnoble: C ABI of the NOBLE-CosNet linear layer (include/noble.h).
//
// Host side: argument validation (complete before any HIP call), workspace
// layout, launch planning (tile choice, split-K) and kernel launches on the
// caller's stream.  The library is stateless apart from a per-device cache of
// the architecture check and a per-thread cache of weight-gradient plans.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <functional>
#include <map>
#include <vector>

#include "noble.h"
#include "noble_gemm_dma.hpp"
#include "noble_init.hpp"
#include "noble_kernels.hpp"
#include "noble_skinny.hpp"

using namespace noble;

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 20;
constexpr int kMaxGroups = 4;
constexpr int64_t kMaxTokens = (int64_t(1) << 31) - 4096;
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

noble_status check_desc(const noble_linear_desc* d) {
    if (!d) return NOBLE_ERR_NULL_ARG;
    if (d->dtype != NOBLE_BF16 && d->dtype != NOBLE_F32) return NOBLE_ERR_BAD_DTYPE;
    if (d->activation < NOBLE_ACT_COSNET || d->activation > NOBLE_ACT_COSNET3) return NOBLE_ERR_BAD_ACTIVATION;
    if (d->reserved != 0) return NOBLE_ERR_BAD_SHAPE;
    if (d->T < 0 || d->T > kMaxTokens) return NOBLE_ERR_BAD_SHAPE;
    if (d->d_in < 8 || d->d_in % 8 || d->d_in > kMaxDim) return NOBLE_ERR_BAD_SHAPE;
    if (d->d_out < 8 || d->d_out % 8 || d->d_out > kMaxDim) return NOBLE_ERR_BAD_SHAPE;
    const int64_t rmax = d->dtype == NOBLE_BF16 ? 256 : 128;
    if (d->r < 0 || (d->r > 0 && (d->r < 8 || d->r % 8 || d->r > rmax))) return NOBLE_ERR_BAD_SHAPE;
    // the 3-layer form keeps both mixing matrices in LDS: r <= 128
    if (d->activation == NOBLE_ACT_COSNET3 && d->r > 128) return NOBLE_ERR_BAD_SHAPE;
    if (d->groups < 0 || d->groups > kMaxGroups) return NOBLE_ERR_BAD_SHAPE;
    const int64_t G = d->groups > 0 ? d->groups : 1;
    if (d->d_out % (8 * G)) return NOBLE_ERR_BAD_SHAPE;
    return NOBLE_OK;
}

// Groups of output columns, each with its own branch (0 counts as 1).
int ngroups(const noble_linear_desc* d) { return d->groups > 0 ? d->groups : 1; }
// Total rank G r: the width of H and of the rank-side scratch arrays.
int64_t rank_total(const noble_linear_desc* d) { return ngroups(d) * d->r; }
// Output columns of one group.
int64_t group_dout(const noble_linear_desc* d) { return d->d_out / ngroups(d); }
// 128-rank blocks of one group.
int rank_blocks(const noble_linear_desc* d) { return (int)((d->r + kSkN - 1) / kSkN); }

size_t elt_size(const noble_linear_desc* d) { return d->dtype == NOBLE_BF16 ? 2 : 4; }

// Function and number of applications of a noble_activation.
Act act_fn(int a) {
    switch (a) {
        case NOBLE_ACT_TANH:
        case NOBLE_ACT_TANH_M: return Act::Tanh;
        case NOBLE_ACT_LEAKY_RELU:
        case NOBLE_ACT_LEAKY_RELU_M: return Act::Leaky;
        case NOBLE_ACT_GELU:
        case NOBLE_ACT_GELU_M: return Act::Gelu;
        default: return Act::Cos;
    }
}
// Applications of the activation: 1 (single), 2 (with M between, the
// CosNet), 3 (the 3-layer CosNet, M and M').
int act_layers(int a) {
    if (a == NOBLE_ACT_COSNET3) return 3;
    return a == NOBLE_ACT_COSNET || a == NOBLE_ACT_TANH_M || a == NOBLE_ACT_LEAKY_RELU_M || a == NOBLE_ACT_GELU_M
               ? 2
               : 1;
}
bool act_two_layers(int a) { return act_layers(a) >= 2; }

// Calls fn.template operator()<F, L>() for the activation `a` (L its
// applications).
template <typename Fn>
noble_status with_act(int a, Fn&& fn) {
    const int L = act_layers(a);
    switch (act_fn(a)) {
        case Act::Cos:
            return L == 3 ? fn.template operator()<Act::Cos, 3>()
                          : (L == 2 ? fn.template operator()<Act::Cos, 2>() : fn.template operator()<Act::Cos, 1>());
        case Act::Tanh:
            return L == 2 ? fn.template operator()<Act::Tanh, 2>() : fn.template operator()<Act::Tanh, 1>();
        case Act::Leaky:
            return L == 2 ? fn.template operator()<Act::Leaky, 2>() : fn.template operator()<Act::Leaky, 1>();
        case Act::Gelu:
            return L == 2 ? fn.template operator()<Act::Gelu, 2>() : fn.template operator()<Act::Gelu, 1>();
    }
    return NOBLE_ERR_BAD_ACTIVATION;
}

// Pieces of K for the bf16 rank projection [T, K] x [K, r] run as J jobs
// (group, 128-rank block): enough workgroups of 128 tokens to cover the CUs,
// at least kPjMinChunks K chunks per piece, at most kPjMaxSplit pieces.
int proj_split(int64_t T, int64_t K, int J) {
    const int64_t blocks = (T + kPjRows - 1) / kPjRows;
    const int64_t nkc = (K + 63) / 64;
    int s = 1;
    while (blocks * s * J < 256 && 2 * s * kPjMinChunks <= nkc && 2 * s <= kPjMaxSplit) s *= 2;
    return s;
}
int proj_jobs(const noble_linear_desc* d) { return ngroups(d) * rank_blocks(d); }

// Scratch layout, each part 256-byte aligned.  The forward's part comes
// first, so that a forward-only call needs just that prefix:
//  - C2 [T, R] storage type;
//  - bf16: the float32 projection partials [S][T][R] for the larger split of
//    the forward and backward projections;
// then the backward's:
//  - C1, dH2, dH [T, hl R] storage type, hl = 2 on the bf16 path (each value
//    as a high + low bf16 pair, see branch_bwd_kernel), 1 on the float32
//    path; the 3-layer form adds the middle C2 and dH3 alike;
//  - bf16: the copies of the frequency / phase gradients;
//  - the float32 split-K partials of the weight-gradient products.
// The 3-layer form's extra regions and products make its sizes larger than
// the other activations' (which share one size).
int hilo(const noble_linear_desc* d) { return d->dtype == NOBLE_BF16 ? 2 : 1; }
size_t scratch_region(const noble_linear_desc* d) {
    return align_up((size_t)d->T * rank_total(d) * elt_size(d));
}
size_t scratch_region_w(const noble_linear_desc* d) {
    return align_up((size_t)hilo(d) * d->T * rank_total(d) * elt_size(d));
}
size_t partial_need(const noble_linear_desc* d) {
    if (d->r == 0 || d->dtype != NOBLE_BF16) return 0;
    const int J = proj_jobs(d);
    const int s = std::max(proj_split(d->T, d->d_in, J), proj_split(d->T, group_dout(d), J));
    return align_up((size_t)s * d->T * rank_total(d) * 4);
}
bool three_layers(const noble_linear_desc* d) { return d->activation == NOBLE_ACT_COSNET3; }
// [T, hl R] regions of the backward: C1, dH2, dH (and C2, dH3).
int bwd_regions(const noble_linear_desc* d) { return three_layers(d) ? 5 : 3; }
// bf16 backward: kChainCopies copies of the frequency / phase gradient
// vectors, [2 L][kChainCopies][R] float32 (four vectors, six for three layers).
int nvec(const noble_linear_desc* d) { return three_layers(d) ? 6 : 4; }
size_t copies_need(const noble_linear_desc* d) {
    if (d->r == 0 || d->dtype != NOBLE_BF16) return 0;
    return align_up((size_t)nvec(d) * kChainCopies * rank_total(d) * 4);
}
size_t wgrad_need(const noble_linear_desc* d);
size_t fwd_scratch_need(const noble_linear_desc* d) {
    return d->r > 0 ? scratch_region(d) + partial_need(d) : 0;
}
size_t scratch_need(const noble_linear_desc* d) {
    return (d->r > 0 ? fwd_scratch_need(d) + bwd_regions(d) * scratch_region_w(d) + copies_need(d) : 0) +
           wgrad_need(d);
}
size_t reserve_need(const noble_linear_desc* d) { return (size_t)d->T * rank_total(d) * 4; }

// A required buffer: non-NULL and 16-byte aligned, unless it holds no bytes.
noble_status need(const void* p, bool nonempty) {
    if (!p) return nonempty ? NOBLE_ERR_NULL_ARG : NOBLE_OK;
    return aligned16(p) ? NOBLE_OK : NOBLE_ERR_MISALIGNED;
}
noble_status optional(const void* p) { return (!p || aligned16(p)) ? NOBLE_OK : NOBLE_ERR_MISALIGNED; }

#define NOBLE_TRY(expr)                              \
    do {                                             \
        noble_status s_ = (expr);                    \
        if (s_ != NOBLE_OK) return s_;               \
    } while (0)

// gfx950 check, cached per device ordinal (0 unknown, 1 ok, 2 unsupported).
std::atomic<int> g_arch_ok[256];

noble_status check_device(int* dev_out = nullptr) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return NOBLE_ERR_HIP;
    if (dev_out) *dev_out = dev;
    if (dev < 0 || dev >= 256) return NOBLE_ERR_UNSUPPORTED_DEVICE;
    int s = g_arch_ok[dev].load(std::memory_order_relaxed);
    if (s == 0) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return NOBLE_ERR_HIP;
        s = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
        g_arch_ok[dev].store(s, std::memory_order_relaxed);
    }
    return s == 1 ? NOBLE_OK : NOBLE_ERR_UNSUPPORTED_DEVICE;
}

// Launch of a kernel that takes one argument struct, with the status of this
// launch itself (the thread's last-error state would also carry, and clear,
// an earlier failure of the caller's).
template <typename Arg>
noble_status launch(void (*kernel)(Arg), dim3 grid, dim3 block, hipStream_t st, const Arg& arg) {
    void* argv[] = {const_cast<Arg*>(&arg)};
    return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, 0, st) == hipSuccess
               ? NOBLE_OK
               : NOBLE_ERR_HIP;
}

int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Scratch of noble_linear_fwd_static: a file-scope device array, one copy per
// GPU the library runs on, held until the process ends.  Host code never
// passes this name to a kernel (in host code it is only a stand-in for the
// device symbol): each device's address comes from hipGetSymbolAddress,
// taken once per device with that device current, and cached here.
constexpr size_t kStaticScratchBytes = NOBLE_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) char g_static_scratch[kStaticScratchBytes];
std::atomic<void*> g_static_scratch_addr[256];

// Device address of g_static_scratch on the current device `dev`.
noble_status static_scratch(int dev, void** out) {
    void* p = g_static_scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_static_scratch)) != hipSuccess || !p) return NOBLE_ERR_HIP;
        g_static_scratch_addr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return NOBLE_OK;
}

// Events of noble_profile_next_wgrad, one pair per host thread, consumed by
// that thread's next backward with a weight-gradient launch.
thread_local hipEvent_t t_wgrad_ev0 = nullptr, t_wgrad_ev1 = nullptr;
thread_local int64_t* t_wgrad_wgs = nullptr;

// Grid of a launch of n workgroups on rows of kGridRow (see flat_block).
dim3 flat_grid(int64_t n) {
    return n <= kGridRow ? dim3((unsigned)n) : dim3(kGridRow, (unsigned)((n + kGridRow - 1) / kGridRow));
}

Seg seg(const void* p, int64_t ld, int64_t klen) {
    Seg s;
    s.ptr = static_cast<const char*>(p);
    s.ld = ld;
    s.klen = (int)klen;
    s.pad_ = 0;
    return s;
}

Operand operand1(Seg s0, int64_t rows) {
    Operand o;
    o.s[0] = s0;
    o.s[1] = s0;
    o.nk1 = 1 << 30;
    o.rows = (int)rows;
    return o;
}

// Two-segment operand: K chunks [0, nk1) from s0 (K extent K0, chunk BK), then s1.
Operand operand2(Seg s0, Seg s1, int nk1, int64_t rows) {
    Operand o;
    o.s[0] = s0;
    o.s[1] = s1;
    o.nk1 = nk1;
    o.rows = (int)rows;
    return o;
}

// Square output tile of the large products: 256 on the bf16 path; 128 on
// the float32 path, which serves small layers (a 256 tile of a 64 x 64
// output would leave one wave doing 16 times the needed work on one CU).
template <typename E>
constexpr int gemm_tile() {
    return sizeof(E) == 2 ? 256 : 128;
}
int gemm_tile_of(const noble_linear_desc* d) {
    return d->dtype == NOBLE_BF16 ? gemm_tile<uint16_t>() : gemm_tile<float>();
}

// Largest workgroup count of one GEMM launch: a dispatch counts its
// work-items in 32 bits.
int64_t max_gemm_blocks(const noble_linear_desc* d) {
    return (int64_t)UINT32_MAX / (d->dtype == NOBLE_BF16 ? kDmaThreads : kThreads);
}

// bf16 products (256-square tiles) of at most 128 rows without column sums
// split each K chunk between the two M halves of the workgroup's waves
// (gemm_bf16_kernel), which takes about half the MFMA time of a full tile.
bool kpair_tile(int tile, int64_t M, bool bsum) { return tile == 256 && M <= 128 && !bsum; }

// A bf16 launch of 256 x 256 tiles that fills its last wave of 256 CUs
// poorly runs as 256 x 128 `npair` tiles (gemm_bf16_kernel): chosen when
// their waves, weighted by kHalfTileCost, are fewer.  A half tile does half
// the MFMA work but loads three quarters of the operand bytes per chunk;
// measured on the 250M and ViT layers it costs about 0.8 of a full tile
// (so 2 waves of full tiles beat 3 of half tiles, 1 of half tiles beats 1 of
// full ones).
constexpr double kHalfTileCost = 0.8;
bool npair_pays(int64_t full_blocks, int64_t half_blocks) {
    const int64_t wf = (full_blocks + 255) / 256, wh = (half_blocks + 255) / 256;
    return half_blocks < (1 << 22) && (double)wh * kHalfTileCost < 0.95 * (double)wf;
}

struct Batch {
    GemmBatch b{};
    int blocks = 0;
    int tile = 256;      // square output tile
    bool npair = false;  // bf16: 256 x 128 tiles (set before adding problems)
    // With `partials`, each of the `split` pieces stores its float32 partial
    // [M][ldc] at partials + piece * M * ldc (also for split = 1); without,
    // split > 1 pieces add atomically into C.
    void add(const Operand& A, const Operand& B, int M, int N, int nk, void* C, int64_t ldc, bool out_f32,
             const float* bias, float* bsum, int split, float* partials = nullptr) {
        GemmProblem& p = b.p[b.count++];
        p.A = A;
        p.B = B;
        p.C = partials ? partials : C;
        p.pstride = partials ? (int64_t)M * ldc : 0;
        p.ldc = ldc;
        p.bias = bias;
        p.bsum = bsum;
        p.M = M;
        p.N = N;
        p.nk = nk;
        p.split = split;
        p.tiles_m = cdiv(M, tile);
        p.tiles_n = cdiv(N, npair ? tile / 2 : tile);
        p.tile_begin = blocks;
        p.nblocks = p.tiles_m * p.tiles_n * split;
        p.out_f32 = out_f32 ? 1 : 0;
        p.atomic = split > 1 && !partials ? 1 : 0;
        p.npair = npair ? 1 : 0;
        p.kpair = !npair && kpair_tile(tile, M, bsum != nullptr) ? 1 : 0;
        blocks += p.nblocks;
    }
};

// Makespan of a grouped launch, in microseconds of the cost model: its
// workgroups, given as (count, K chunks each) in launch order, are dispatched
// in that order to whichever of the 256 CUs frees first (one 256 x 256
// workgroup per CU).  A workgroup costs kWgFixed plus kWgChunk per 64-token
// chunk (fit to the measured time of the forward GEMM against K: prologue,
// epilogue stores and ramp are about 12 us per tile, a chunk 1.45 us).
double launch_makespan(const std::vector<std::pair<int, double>>& wgs) {
    constexpr double kWgFixed = 12.0, kWgChunk = 1.45;
    // CU free times with their multiplicities.  The workgroups of one group
    // are identical, so handing all the CUs that free first to as many of
    // them at once gives the same schedule as one at a time, in a handful of
    // steps: the planner runs on every call.
    std::map<double, int> free_at{{0.0, 256}};
    double end = 0.0;
    for (const auto& g : wgs) {
        const double d = kWgFixed + kWgChunk * g.second;
        for (int n = g.first; n > 0;) {
            const auto it = free_at.begin();
            const double t = it->first;
            const int k = std::min(n, it->second);
            if ((it->second -= k) == 0) free_at.erase(it);
            free_at[t + d] += k;
            end = std::max(end, t + d);
            n -= k;
        }
    }
    return end;
}

// K split of one weight-gradient product (K = T tokens) whose pieces store
// float32 partials that a reduction sums afterwards.  Cost model: the longest
// CU's share of 64-element K chunks (waves of 256 workgroups) plus the partial
// traffic (S writes, S reads, one result write).  A split must beat the
// unsplit cost by 3% and keep the launch within `cap` workgroups.
int choose_split_partials(int tiles, int nk, int64_t MN, int64_t cap) {
    constexpr double kChunkUs = 1.7;          // one K chunk of a 256 x 256 tile
    constexpr double kBytesPerUs = 5.0e6;     // HBM rate of the partials
    double best = 0;
    int bs = 1;
    for (int s = 1; s <= kMaxReduceSlices; s *= 2) {   // reduce_kernel sums at most that many
        if (s > 1 && (s * 8 > nk || (int64_t)tiles * s > cap)) break;
        const double waves = (double)((int64_t)tiles * s + 255) / 256;
        const double cost = (int)waves * ((double)nk / s) * kChunkUs + (s > 1 ? (2.0 * s + 1) * MN * 4 / kBytesPerUs : 0);
        if (s == 1 || cost < best * 0.97) {
            best = cost;
            bs = s;
        }
    }
    return bs;
}

// K splits of the weight-gradient launch (K = T tokens).  The pieces of
// every product (dW, and the rank products dW_down, dW_up, dM) store float32
// partials that reduce_kernel sums in piece order.  Float atomics were used
// for the rank products before: they are device-scope, so the eight XCDs'
// adds meet beyond their L2s, and they cost about 1 MB of output per us.
//  - r = 0: dW alone, choose_split_partials.
//  - r > 0: both splits together (the rank problems share dW's launch and
//    can fill the CUs that a smaller dW split leaves), minimising the
//    launch's makespan under the list-scheduling model above plus the dW
//    partial traffic of both products ((2 S + 1) x their output bytes at
//    5 MB per us).  Candidates are 2^a 3^b up to 16 with at least 8 K
//    chunks per piece: the model is flat near its optimum, and a coarse set
//    keeps its choice off near-ties.  dM is counted whatever the activation,
//    so that the workspace does not depend on it.
struct WgradPlan {
    int split;      // K pieces of dW
    int rank;       // K pieces of the rank products
    size_t bytes;        // dW partials
    size_t rank_bytes;   // rank-product partials: [S][d_in][hl R] (dW_down), then per group
                         // [S][r][d_out/G] (dW_up, only when split) and [S][hl r][hl r] (dM)
};

// Elements of one K piece of the rank products' float32 partials.  On the
// bf16 path dW_down and dM are products over high + low bf16 operand pairs
// (hl = 2): their partials are stored for any split, folded by the
// reduction; dW_up is stored only when split.
struct RankParts {
    int64_t folded;     // dW_down and dM, per piece
    int64_t unfolded;   // dW_up, per piece
};
// dM products per group: 1, or 2 for the 3-layer form (counted for every
// other activation too, so that their sizes agree).
int64_t n_mix(const noble_linear_desc* d) { return three_layers(d) ? 2 : 1; }
RankParts rank_parts(const noble_linear_desc* d) {
    const int64_t hl = hilo(d), G = ngroups(d), r = d->r, R = rank_total(d), dog = group_dout(d);
    return RankParts{d->d_in * hl * R + n_mix(d) * G * hl * r * hl * r, G * r * dog};
}
// Pieces of partials stored for the folded and the unfolded rank products.
int64_t rank_folded_pieces(const noble_linear_desc* d, int rank) {
    return hilo(d) == 2 ? std::max(rank, 1) : (rank > 1 ? rank : 0);
}

WgradPlan plan_wgrad_uncached(const noble_linear_desc* d) {
    WgradPlan w{1, 1, 0, 0};
    const bool bf = d->dtype == NOBLE_BF16;
    const int bk = bf ? Elt<uint16_t>::BK : Elt<float>::BK, tile = gemm_tile_of(d);
    const int64_t T = d->T, din = d->d_in, dout = d->d_out, r = d->r;
    const int nkT = T > 0 ? cdiv(T, bk) : 0;
    if (nkT == 0) return w;
    const int tiles = cdiv(din, tile) * cdiv(dout, tile);
    const int64_t MN = din * dout;
    if (r == 0) {
        w.split = choose_split_partials(tiles, nkT, MN, max_gemm_blocks(d));
    } else {
        constexpr double kPartialBytesPerUs = 5.0e6;
        const int64_t R = rank_total(d), dog = group_dout(d), hl = hilo(d);
        const int G = ngroups(d);
        // the rank products in launch order (dW_down, then per group dW_up
        // and dM): tiles and whether they run as kpair tiles (half the chunk time)
        std::vector<std::pair<int, bool>> rank;
        rank.push_back({cdiv(din, tile) * cdiv(hl * R, tile), kpair_tile(tile, din, false)});
        for (int g = 0; g < G; ++g) {
            rank.push_back({cdiv(r, tile) * cdiv(dog, tile), kpair_tile(tile, r, false)});
            rank.push_back({(int)n_mix(d) * cdiv(hl * r, tile) * cdiv(hl * r, tile), kpair_tile(tile, hl * r, false)});
        }
        int rank_tiles = 0;
        for (const auto& e : rank) rank_tiles += e.first;
        const RankParts rp = rank_parts(d);
        double best = -1.0;
        for (int sw : {1, 2, 3, 4, 6, 8, 12, 16}) {
            if (sw > 1 && sw * 8 > nkT) break;
            for (int sr : {1, 2, 3, 4, 6, 8, 12, 16}) {
                if (sr > 1 && sr * 8 > nkT) break;
                if ((int64_t)tiles * sw + (int64_t)rank_tiles * sr > max_gemm_blocks(d)) continue;
                // partial traffic: S writes, S reads and one result write per stored product
                const double fp = (double)rank_folded_pieces(d, sr), up = sr > 1 ? sr : 0;
                const double rank_traffic = 4.0 * ((fp > 0 ? 2.0 * fp + 1 : 0) * rp.folded +
                                                   (up > 0 ? 2.0 * up + 1 : 0) * rp.unfolded);
                std::vector<std::pair<int, double>> wgs{{tiles * sw, (double)cdiv(nkT, sw)}};
                for (const auto& e : rank) wgs.push_back({e.first * sr, cdiv(nkT, sr) / (e.second ? 2.0 : 1.0)});
                const double t = launch_makespan(wgs) +
                                 (sw > 1 ? (2.0 * sw + 1) * (double)MN * 4 / kPartialBytesPerUs : 0.0) +
                                 rank_traffic / kPartialBytesPerUs;
                if (best < 0 || t < best) {
                    best = t;
                    w.split = sw;
                    w.rank = sr;
                }
            }
        }
    }
    w.bytes = w.split > 1 ? align_up((size_t)w.split * MN * 4) : 0;
    if (r > 0) {
        const RankParts rp = rank_parts(d);
        const int64_t el = rank_folded_pieces(d, w.rank) * rp.folded + (w.rank > 1 ? w.rank * rp.unfolded : 0);
        w.rank_bytes = el > 0 ? align_up((size_t)el * 4) : 0;
    }
    return w;
}

// The plan depends only on the shape, and the search costs 10-20 us, paid by
// the workspace query, the forward's size check and the backward: the last
// eight plans are kept per thread.
WgradPlan plan_wgrad(const noble_linear_desc* d) {
    struct Entry {
        int64_t T, d_in, d_out, r;
        int32_t dtype, groups, mix;
        WgradPlan w;
    };
    thread_local Entry cache[8];
    thread_local int used = 0, next = 0;
    const int32_t G = ngroups(d), mix = (int32_t)n_mix(d);
    for (int i = 0; i < used; ++i) {
        const Entry& e = cache[i];
        if (e.T == d->T && e.d_in == d->d_in && e.d_out == d->d_out && e.r == d->r && e.dtype == d->dtype &&
            e.groups == G && e.mix == mix)
            return e.w;
    }
    const WgradPlan w = plan_wgrad_uncached(d);
    cache[next] = Entry{d->T, d->d_in, d->d_out, d->r, d->dtype, G, mix, w};
    next = (next + 1) % 8;
    used = std::min(used + 1, 8);
    return w;
}

size_t wgrad_need(const noble_linear_desc* d) {
    const WgradPlan w = plan_wgrad(d);
    return w.bytes + w.rank_bytes;
}

// Every GEMM launch of the call, unsplit, within max_gemm_blocks (the
// planner's splits stay within it too).  Only layers far beyond a GPU's
// memory come near: at the largest T the forward reaches it at d_out > 256.
noble_status check_grids(const noble_linear_desc* d) {
    const int64_t tile = gemm_tile_of(d), T = d->T, din = d->d_in, dout = d->d_out, r = d->r;
    const int64_t G = ngroups(d), dog = group_dout(d), R = rank_total(d);
    auto tiles = [tile](int64_t m, int64_t n) { return ((m + tile - 1) / tile) * ((n + tile - 1) / tile); };
    const int64_t fwd = G * tiles(T, dog), dx = tiles(T, din);
    const int64_t hl = hilo(d);
    const int64_t wgrad =
        tiles(din, dout) + (r > 0 ? tiles(din, hl * R) + G * (tiles(r, dog) + n_mix(d) * tiles(hl * r, hl * r)) : 0);
    // (an npair launch is chosen only when it has fewer weighted waves: at
    // most about twice the blocks of a launch of a few waves)
    return std::max({fwd, dx, wgrad}) <= max_gemm_blocks(d) ? NOBLE_OK : NOBLE_ERR_BAD_SHAPE;
}

// `plain`: the r = 0 forward, launched under its own kernel symbol so that
// profiles can tell it from the K-extended forward.
template <typename E, bool AK, bool BKM>
noble_status launch_gemm(const Batch& bt, hipStream_t st, bool plain = false) {
    if (bt.blocks == 0) return NOBLE_OK;
    if constexpr (sizeof(E) == 2) {
        if (AK && !BKM && plain)
            return launch(gemm_bf16_kernel<AK, BKM, false, 1>, dim3(bt.blocks), dim3(kDmaThreads), st, bt.b);
        return launch(gemm_bf16_kernel<AK, BKM, !AK && !BKM, 0>, dim3(bt.blocks), dim3(kDmaThreads), st, bt.b);
    } else {
        return launch(gemm_kernel<E, gemm_tile<E>(), gemm_tile<E>(), AK, BKM, !AK && !BKM>, dim3(bt.blocks),
                      dim3(kThreads), st, bt.b);
    }
}

// float32 path: chain kernels with their own rank projection, one launch per
// group (the arguments already point at the group's operands and columns).
noble_status launch_chain(bool fwd, int RP, int act, const ChainArgs& a, int T, hipStream_t st) {
    const dim3 grid = flat_grid(cdiv(T, kChainRows)), block(kThreads);
    return with_act(act, [&]<Act F, int L>() -> noble_status {
#define NOBLE_CHAIN(RPV)                                                                       \
    if (RP == RPV)                                                                             \
        return fwd ? launch(fwd_chain_kernel<float, RPV, F, L>, grid, block, st, a)            \
                   : launch(bwd_chain_kernel<float, RPV, F, L>, grid, block, st, a);
        NOBLE_CHAIN(32)
        NOBLE_CHAIN(64)
        NOBLE_CHAIN(128)
#undef NOBLE_CHAIN
        return NOBLE_ERR_BAD_SHAPE;
    });
}

// bf16 path, step 1: split-K rank projection into the float32 partials
// P [S][T][R], one job per (group, 128-rank block).  Forward: A = x, B =
// W_down's column block (MN-major, row stride R).  Backward: A = the group's
// column block of dy, B = the group's rows of W_up [R, d_out / G] (K-major).
noble_status launch_proj(bool fwd, const noble_linear_desc* d, const void* A, const void* B, float* P, int S,
                         hipStream_t st, const ZeroList* zero = nullptr) {
    const int64_t T = d->T, din = d->d_in, dout = d->d_out, r = d->r, R = rank_total(d), dog = group_dout(d);
    const int G = ngroups(d), NB = rank_blocks(d);
    ProjArgs a{};
    if (zero) a.z = *zero;
    a.J = 0;
    for (int g = 0; g < G; ++g)
        for (int b = 0; b < NB; ++b) {
            ProjJob& j = a.job[a.J++];
            const int64_t c0 = g * r + (int64_t)b * kSkN, n = std::min<int64_t>(kSkN, r - (int64_t)b * kSkN);
            if (fwd) {
                j.A = operand1(seg(A, din, din), T);
                j.B = operand1(seg(static_cast<const uint16_t*>(B) + c0, R, din), n);
            } else {
                j.A = operand1(seg(static_cast<const uint16_t*>(A) + g * dog, dout, dog), T);
                j.B = operand1(seg(static_cast<const uint16_t*>(B) + c0 * dog, dog, dog), n);
            }
            j.c0 = (int)c0;
        }
    a.P = P;
    a.ldp = (int)R;
    a.pstride = T * R;
    a.T = (int)T;
    a.nk = cdiv(fwd ? din : dog, 64);
    a.S = S;
    const dim3 grid = flat_grid((int64_t)cdiv(T, kPjRows) * S * a.J), block(kPjThreads);
    return fwd ? launch(proj_kernel<false>, grid, block, st, a) : launch(proj_kernel<true>, grid, block, st, a);
}

// bf16 path, step 2: the branch nonlinearity (forward or backward) from the
// summed partials, one workgroup per (32 tokens, group).
noble_status launch_branch(bool fwd, const noble_linear_desc* d, const ChainArgs& c, const float* P, int S,
                           hipStream_t st, float* copies = nullptr) {
    BranchArgs a{};
    a.copies = copies;
    a.P = P;
    a.pstride = d->T * rank_total(d);
    a.S = S;
    a.M = reinterpret_cast<const uint16_t*>(c.M);
    a.M2 = reinterpret_cast<const uint16_t*>(c.M2);
    a.w1 = c.w1;
    a.p1 = c.p1;
    a.w2 = c.w2;
    a.p2 = c.p2;
    a.w3 = c.w3;
    a.p3 = c.p3;
    a.H = c.H;
    a.C1s = reinterpret_cast<uint16_t*>(c.C1s);
    a.C2s = reinterpret_cast<uint16_t*>(c.C2s);
    a.dH2s = reinterpret_cast<uint16_t*>(c.dH2s);
    a.dHs = reinterpret_cast<uint16_t*>(c.dHs);
    a.C2ms = reinterpret_cast<uint16_t*>(c.C2ms);
    a.dH3s = reinterpret_cast<uint16_t*>(c.dH3s);
    a.dw1 = c.dw1;
    a.dp1 = c.dp1;
    a.dw2 = c.dw2;
    a.dp2 = c.dp2;
    a.dw3 = c.dw3;
    a.dp3 = c.dp3;
    a.T = (int)d->T;
    a.r = (int)d->r;
    a.G = ngroups(d);
    a.R = (int)rank_total(d);
    const int NT = rank_blocks(d);
    const dim3 grid = flat_grid((int64_t)cdiv(d->T, kSkRows) * a.G), block(kThreads * NT);
    return with_act(d->activation, [&]<Act F, int L>() -> noble_status {
        if (NT == 1)
            return fwd ? launch(branch_fwd_kernel<F, L, 1>, grid, block, st, a)
                       : launch(branch_bwd_kernel<F, L, 1>, grid, block, st, a);
        if constexpr (L != 3)   // the 3-layer form is validated to r <= 128 (NT = 1)
            return fwd ? launch(branch_fwd_kernel<F, L, 2>, grid, block, st, a)
                       : launch(branch_bwd_kernel<F, L, 2>, grid, block, st, a);
        return NOBLE_ERR_BAD_SHAPE;
    });
}

// K chunk of the large products (128 bytes of a row: 64 bf16 or 32 f32).
template <typename E>
constexpr int gemm_bk() {
    return Elt<E>::BK;
}

// Padded rank of the float32 chain kernels: a multiple of the K chunk,
// instantiated for 32, 64 and 128.
template <typename E>
int chain_rp(int64_t r) {
    if (r <= 32) return 32;
    return r <= 64 ? 64 : 128;
}

// Per-group view of the branch arguments for the float32 chain kernels: the
// group's operands, vectors and columns of the [T, R] arrays.
ChainArgs group_chain(const ChainArgs& a, const noble_linear_desc* d, int g, size_t es) {
    const int64_t r = d->r, c0 = g * r;
    ChainArgs c = a;
    auto off = [&](char* p, int64_t elems, size_t e) { return p ? p + elems * (int64_t)e : p; };
    auto offf = [&](auto* p, int64_t elems) { return p ? p + elems : p; };
    c.M = a.M ? a.M + g * r * r * (int64_t)es : a.M;
    c.M2 = a.M2 ? a.M2 + g * r * r * (int64_t)es : a.M2;
    c.w1 = offf(a.w1, c0);
    c.p1 = offf(a.p1, c0);
    c.w2 = offf(a.w2, c0);
    c.p2 = offf(a.p2, c0);
    c.w3 = offf(a.w3, c0);
    c.p3 = offf(a.p3, c0);
    c.H = offf(a.H, c0);
    c.C1s = off(a.C1s, c0, es);
    c.C2s = off(a.C2s, c0, es);
    c.dH2s = off(a.dH2s, c0, es);
    c.dHs = off(a.dHs, c0, es);
    c.C2ms = off(a.C2ms, c0, es);
    c.dH3s = off(a.dH3s, c0, es);
    c.dw1 = offf(a.dw1, c0);
    c.dp1 = offf(a.dp1, c0);
    c.dw2 = offf(a.dw2, c0);
    c.dp2 = offf(a.dp2, c0);
    c.dw3 = offf(a.dw3, c0);
    c.dp3 = offf(a.dp3, c0);
    return c;
}

// The mixing parameters: M [G][r][r] with omega2, phi2 [R]; the 3-layer form
// stores both mixing matrices as M [2][G][r][r] and the second and third
// frequency / phase vectors as omega2, phi2 [2][R].
void set_mixing(ChainArgs& a, const noble_linear_desc* d, const void* M, const float* w2, const float* p2) {
    a.M = static_cast<const char*>(M);
    a.w2 = w2;
    a.p2 = p2;
    if (three_layers(d)) {
        const int64_t R = rank_total(d);
        a.M2 = a.M + (int64_t)ngroups(d) * d->r * d->r * elt_size(d);
        a.w3 = w2 + R;
        a.p3 = p2 + R;
    }
}

template <typename E>
noble_status fwd_impl(const noble_linear_desc* d, const void* x, const void* W, const float* b, const void* Wd,
                      const float* w1, const float* p1, const void* M, const float* w2, const float* p2,
                      const void* Wu, void* y, void* reserve, void* scratch, hipStream_t st) {
    constexpr int BK = Elt<E>::BK;
    constexpr size_t ES = sizeof(E);
    const int64_t T = d->T, din = d->d_in, dout = d->d_out, r = d->r;
    const int64_t R = rank_total(d), dog = group_dout(d);
    const int G = ngroups(d);
    char* C2s = static_cast<char*>(scratch);
    if (r > 0) {
        ChainArgs a{};
        set_mixing(a, d, M, w2, p2);
        a.w1 = w1;
        a.p1 = p1;
        a.H = static_cast<float*>(reserve);
        a.C2s = C2s;
        a.T = (int)T;
        a.r = (int)r;
        a.ldr = (int)R;
        a.nk = cdiv(din, BK);
        if constexpr (sizeof(E) == 2) {
            float* P = reinterpret_cast<float*>(static_cast<char*>(scratch) + scratch_region(d));
            const int S = proj_split(T, din, proj_jobs(d));
            NOBLE_TRY(launch_proj(true, d, x, Wd, P, S, st));
            NOBLE_TRY(launch_branch(true, d, a, P, S, st));
        } else {
            for (int g = 0; g < G; ++g) {
                ChainArgs c = group_chain(a, d, g, ES);
                c.A = operand1(seg(x, din, din), T);
                c.B = operand1(seg(static_cast<const E*>(Wd) + g * r, R, din), r);
                NOBLE_TRY(launch_chain(true, chain_rp<E>(r), d->activation, c, (int)T, st));
            }
        }
    }
    // y[:, g] = [x | C2_g] [W_g ; W_up_g] + b_g, one problem per group (the
    // rank-r up-projection is a K-extension of the main product)
    constexpr int GBK = gemm_bk<E>();
    const int nk1 = cdiv(din, GBK);
    const int nk = nk1 + (r > 0 ? cdiv(r, GBK) : 0);
    Batch bt;
    bt.tile = gemm_tile<E>();
    if (sizeof(E) == 2)
        bt.npair = npair_pays((int64_t)G * cdiv(T, 256) * cdiv(dog, 256), (int64_t)G * cdiv(T, 256) * cdiv(dog, 128));
    for (int g = 0; g < G; ++g) {
        const E* Wg = static_cast<const E*>(W) + g * dog;
        const char* C2g = C2s + g * r * (int64_t)ES;
        const E* Wug = r > 0 ? static_cast<const E*>(Wu) + g * r * dog : nullptr;
        bt.add(operand2(seg(x, din, din), seg(C2g, R, r), nk1, T), operand2(seg(Wg, dout, din), seg(Wug, dog, r), nk1, dog),
               (int)T, (int)dog, nk, static_cast<E*>(y) + g * dog, dout, sizeof(E) == 4, b ? b + g * dog : nullptr,
               nullptr, 1);
    }
    return launch_gemm<E, true, false>(bt, st, r == 0 && G == 1);
}

template <typename E>
noble_status bwd_impl(const noble_linear_desc* d, const void* dy, const void* x, const void* W, const void* Wd,
                      const float* w1, const float* p1, const void* M, const float* w2, const float* p2,
                      const void* Wu, const void* reserve, void* dx, float* dW, float* db, float* dWd, float* dM,
                      float* dWu, float* dw1, float* dp1, float* dw2, float* dp2, void* scratch, hipStream_t st) {
    constexpr int BK = Elt<E>::BK;
    constexpr size_t ES = sizeof(E);
    const int64_t T = d->T, din = d->d_in, dout = d->d_out, r = d->r;
    const int64_t R = rank_total(d), dog = group_dout(d);
    const int G = ngroups(d);
    const bool two = act_two_layers(d->activation), three = three_layers(d);
    const int64_t nm = n_mix(d);   // mixing matrices per group
    const int64_t hl = hilo(d);    // C1, dH2, dH as high + low bf16 pairs on the bf16 path
    const size_t regw = scratch_region_w(d);
    char* base = static_cast<char*>(scratch);
    char* C2s = base;
    char* C1s = base + fwd_scratch_need(d);
    char* dH2s = C1s + regw;
    char* dHs = dH2s + regw;
    char* C2ms = three ? dHs + regw : nullptr;   // 3-layer form: the middle C2 and dH3
    char* dH3s = three ? C2ms + regw : nullptr;

    // dW, dW_down, dW_up and dM are overwritten by their products (or by
    // the sums of their split-K partials); db and the dw / dp vectors are
    // accumulated atomically and start from zero.  T = 0 zeroes every
    // gradient; so does a one-application activation for the unused dM, dw2
    // and dp2 (when given).  The 3-layer form's dM is [2][G][r][r] and its
    // dw2, dp2 are [2][R].
    constexpr int GBK = gemm_bk<E>();
    const int nkT = cdiv(T, GBK);
    const WgradPlan wp = plan_wgrad(d);
    char* after_rank = r > 0 ? C1s + bwd_regions(d) * regw : base;
    float* copies = copies_need(d) ? reinterpret_cast<float*>(after_rank) : nullptr;
    float* wpart = reinterpret_cast<float*>(after_rank + copies_need(d));
    float* rpart = reinterpret_cast<float*>(reinterpret_cast<char*>(wpart) + wp.bytes);

    ZeroList z{};
    auto zero = [&](float* p, int64_t n) {
        if (p && n > 0) {
            z.ptr[z.count] = p;
            z.n[z.count] = n;
            ++z.count;
        }
    };
    if (T == 0) zero(dW, din * dout);
    zero(db, dout);
    if (r > 0) {
        if (T == 0) {
            zero(dWd, din * R);
            zero(dWu, R * dog);
        }
        if (T == 0 || !two) zero(dM, nm * G * r * r);
        if (copies && T > 0) {
            // the reduction of the copies overwrites dw1, dp1 (and dw2, dp2)
            zero(copies, (int64_t)nvec(d) * kChainCopies * R);
            if (!two) {
                zero(dw2, R);
                zero(dp2, R);
            }
        } else {
            zero(dw1, R);
            zero(dp1, R);
            zero(dw2, nm * R);
            zero(dp2, nm * R);
        }
    }
    // On the bf16 path with a branch, the projection kernel does the zeroing.
    const bool zero_in_proj = sizeof(E) == 2 && r > 0 && T > 0;
    if (z.count > 0 && !zero_in_proj) {
        NOBLE_TRY(launch(zero_kernel, dim3(512), dim3(256), st, z));
    }
    if (T == 0) return NOBLE_OK;

    if (r > 0) {
        ChainArgs a{};
        set_mixing(a, d, M, w2, p2);
        a.w1 = w1;
        a.p1 = p1;
        a.H = static_cast<float*>(const_cast<void*>(reserve));
        a.C1s = C1s;
        a.C2s = C2s;
        a.dH2s = dH2s;
        a.dHs = dHs;
        a.C2ms = C2ms;
        a.dH3s = dH3s;
        a.dw1 = dw1;
        a.dp1 = dp1;
        a.dw2 = dw2;
        a.dp2 = dp2;
        if (three) {
            a.dw3 = dw2 + R;
            a.dp3 = dp2 + R;
        }
        a.T = (int)T;
        a.r = (int)r;
        a.ldr = (int)R;
        a.nk = cdiv(dog, BK);
        if constexpr (sizeof(E) == 2) {
            float* P = reinterpret_cast<float*>(base + scratch_region(d));
            const int S = proj_split(T, dog, proj_jobs(d));
            NOBLE_TRY(launch_proj(false, d, dy, Wu, P, S, st, &z));
            NOBLE_TRY(launch_branch(false, d, a, P, S, st, copies));
        } else {
            for (int g = 0; g < G; ++g) {
                ChainArgs c = group_chain(a, d, g, ES);
                // dC2_g = dy_g W_up_g^T: A = the group's columns of dy, B(k = j, n = q) = W_up_g[q][j]
                c.A = operand1(seg(static_cast<const E*>(dy) + g * dog, dout, dog), T);
                c.B = operand1(seg(static_cast<const E*>(Wu) + g * r * dog, dog, dog), r);
                NOBLE_TRY(launch_chain(false, chain_rp<E>(r), d->activation, c, (int)T, st));
            }
        }
    }

    // dx = [dy | dH] [W^T ; W_down^T]   (B(k, n) stored [n][k]: K-major); on
    // the bf16 path the K-extension reads dH's high part (row stride 2 R)
    {
        const int nk1 = cdiv(dout, GBK);
        const int nk = nk1 + (r > 0 ? cdiv(R, GBK) : 0);
        Batch bt;
        bt.tile = gemm_tile<E>();
        if (sizeof(E) == 2) bt.npair = npair_pays((int64_t)cdiv(T, 256) * cdiv(din, 256), (int64_t)cdiv(T, 256) * cdiv(din, 128));
        bt.add(operand2(seg(dy, dout, dout), seg(dHs, hl * R, R), nk1, T), operand2(seg(W, dout, dout), seg(Wd, R, R), nk1, din),
               (int)T, (int)din, nk, dx, din, sizeof(E) == 4, nullptr, nullptr, 1);
        NOBLE_TRY((launch_gemm<E, true, true>(bt, st)));
    }

    // Weight gradients, reduced over tokens (K = T), A and B both MN-major, in
    // one grouped launch: the rank-r gradients (dW_down, and dW_up, dM per
    // group) fill the CUs that dW leaves idle.  A split product stores its
    // partials, and one reduction pass sums them, with the copies of the
    // frequency / phase gradients.
    {
        ReduceList red{};
        static_assert(kChainCopies <= kMaxReduceSlices, "copies exceed the reduction's slices");
        static_assert(kMaxZero >= kMaxProblems + 6, "the reduction list holds every product and six copies");
        auto reduce = [&](const float* part, float* out, int64_t n, int S, int fw = 0, int fold = 0) {
            red.part[red.count] = part;
            red.out[red.count] = out;
            red.n[red.count] = n;
            red.S[red.count] = S;
            red.fw[red.count] = fw;
            red.fold[red.count] = fold;
            ++red.count;
        };
        Batch bt;
        bt.tile = gemm_tile<E>();
        const Operand xT = operand1(seg(x, din, T), din);
        const Operand dyN = operand1(seg(dy, dout, T), dout);
        bt.add(xT, dyN, (int)din, (int)dout, nkT, dW, dout, true, nullptr, db, wp.split,
               wp.split > 1 ? wpart : nullptr);
        if (wp.split > 1) reduce(wpart, dW, din * dout, wp.split);
        if (r > 0) {
            const int rs = wp.rank;
            float* rp = rpart;
            // One rank product [m, n]: a split product stores its pieces in the
            // next partial slots, as does (for any split) a product over high +
            // low operand pairs, whose output [m, n] the reduction folds into
            // `out` ([m / 2, n] or [m, n / 2] per the fold bits; F = its width).
            auto rank = [&](const Operand& A, const Operand& B, int64_t m, int64_t n, float* out, int fold, int64_t F) {
                const bool parts = fold != 0 || rs > 1;
                bt.add(A, B, (int)m, (int)n, nkT, out, n, true, nullptr, nullptr, rs, parts ? rp : nullptr);
                if (parts) {
                    const int64_t outn = m * n / ((fold & 1 ? 2 : 1) * (fold & 2 ? 2 : 1));
                    reduce(rp, out, outn, rs, fold ? (int)F : 0, fold);
                    rp += (int64_t)rs * m * n;
                }
            };
            // dW_down = x^T dH: on the bf16 path over [dH_hi | dH_lo] (N = 2 R)
            rank(xT, operand1(seg(dHs, hl * R, T), hl * R), din, hl * R, dWd, hl == 2 ? 1 : 0, R);
            for (int g = 0; g < G; ++g) {
                const int64_t c0 = g * r;
                const Operand C2T = operand1(seg(C2s + c0 * (int64_t)ES, R, T), r);
                const Operand dyg = operand1(seg(static_cast<const E*>(dy) + g * dog, dout, T), dog);
                rank(C2T, dyg, r, dog, dWu + c0 * dog, 0, 0);
                if (two) {
                    // dM_g = C1_g^T dH2_g: on the bf16 path over the group's
                    // [hi | lo] column pairs of C1 and dH2 (2r x 2r, both folded)
                    const Operand C1T = operand1(seg(C1s + hl * c0 * (int64_t)ES, hl * R, T), hl * r);
                    const Operand dH2N = operand1(seg(dH2s + hl * c0 * (int64_t)ES, hl * R, T), hl * r);
                    rank(C1T, dH2N, hl * r, hl * r, dM + g * r * r, hl == 2 ? 3 : 0, r);
                }
                if (three) {
                    // dM'_g = C2_g^T dH3_g (the middle layer's output and the
                    // third layer's pre-mixing gradient), stored after dM
                    const Operand C2mT = operand1(seg(C2ms + hl * c0 * (int64_t)ES, hl * R, T), hl * r);
                    const Operand dH3N = operand1(seg(dH3s + hl * c0 * (int64_t)ES, hl * R, T), hl * r);
                    rank(C2mT, dH3N, hl * r, hl * r, dM + (G + g) * r * r, hl == 2 ? 3 : 0, r);
                }
            }
        }
        hipEvent_t ev0 = t_wgrad_ev0, ev1 = t_wgrad_ev1;
        if (t_wgrad_wgs) *t_wgrad_wgs = bt.blocks;
        t_wgrad_ev0 = t_wgrad_ev1 = nullptr;
        t_wgrad_wgs = nullptr;
        if (ev0 && hipEventRecord(ev0, st) != hipSuccess) return NOBLE_ERR_HIP;
        NOBLE_TRY((launch_gemm<E, false, false>(bt, st)));
        if (ev1 && hipEventRecord(ev1, st) != hipSuccess) return NOBLE_ERR_HIP;
        if (copies) {
            const int64_t arr = (int64_t)kChainCopies * R;
            reduce(copies, dw1, R, kChainCopies);
            reduce(copies + arr, dp1, R, kChainCopies);
            if (two) {
                reduce(copies + 2 * arr, dw2, R, kChainCopies);
                reduce(copies + 3 * arr, dp2, R, kChainCopies);
            }
            if (three) {
                reduce(copies + 4 * arr, dw2 + R, R, kChainCopies);
                reduce(copies + 5 * arr, dp2 + R, R, kChainCopies);
            }
        }
        if (red.count > 0) {
            // up to 1024 blocks of 256 threads per array, four floats per thread
            red.first[0] = 0;
            for (int a = 0; a < red.count; ++a)
                red.first[a + 1] = red.first[a] + (int)std::min<int64_t>(1024, std::max<int64_t>(1, cdiv(red.n[a], 4 * 256)));
            NOBLE_TRY(launch(reduce_kernel, dim3(red.first[red.count]), dim3(256), st, red));
        }
    }
    return NOBLE_OK;
}

}  // namespace

extern "C" {

int noble_abi_version(void) { return NOBLE_ABI_VERSION; }

const char* noble_status_string(int status) {
    switch (status) {
        case NOBLE_OK: return "NOBLE_OK";
        case NOBLE_ERR_NULL_ARG: return "NOBLE_ERR_NULL_ARG: a required pointer is NULL";
        case NOBLE_ERR_BAD_SHAPE: return "NOBLE_ERR_BAD_SHAPE: dimension outside the supported ranges";
        case NOBLE_ERR_BAD_DTYPE: return "NOBLE_ERR_BAD_DTYPE: dtype is not NOBLE_BF16 or NOBLE_F32";
        case NOBLE_ERR_MISALIGNED: return "NOBLE_ERR_MISALIGNED: a pointer is not 16-byte aligned";
        case NOBLE_ERR_WORKSPACE_TOO_SMALL: return "NOBLE_ERR_WORKSPACE_TOO_SMALL: scratch buffer too small";
        case NOBLE_ERR_UNSUPPORTED_DEVICE: return "NOBLE_ERR_UNSUPPORTED_DEVICE: current device is not gfx950";
        case NOBLE_ERR_HIP: return "NOBLE_ERR_HIP: a HIP runtime call or kernel launch failed";
        case NOBLE_ERR_BAD_ACTIVATION: return "NOBLE_ERR_BAD_ACTIVATION: activation is not a noble_activation";
        default: return "NOBLE_ERR_UNKNOWN: not a noble_status value";
    }
}

noble_status noble_linear_workspace_size(const noble_linear_desc* desc, size_t* reserve_bytes,
                                         size_t* scratch_bytes) {
    NOBLE_TRY(check_desc(desc));
    NOBLE_TRY(check_grids(desc));
    if (reserve_bytes) *reserve_bytes = reserve_need(desc);
    if (scratch_bytes) *scratch_bytes = scratch_need(desc);
    return NOBLE_OK;
}

noble_status noble_linear_fwd_scratch_size(const noble_linear_desc* desc, size_t* scratch_bytes) {
    NOBLE_TRY(check_desc(desc));
    NOBLE_TRY(check_grids(desc));
    if (scratch_bytes) *scratch_bytes = fwd_scratch_need(desc);
    return NOBLE_OK;
}

}  // extern "C"

namespace {

// Argument checks of the forward; `scratch_bytes` < 0: the scratch is the
// static array (not checked here).
noble_status fwd_check(const noble_linear_desc* desc, const void* x, const void* W, const float* b,
                       const void* W_down, const float* omega1, const float* phi1, const void* M,
                       const float* omega2, const float* phi2, const void* W_up, const void* y,
                       const void* reserve, const void* scratch, int64_t scratch_bytes) {
    NOBLE_TRY(check_desc(desc));
    NOBLE_TRY(check_grids(desc));
    const bool rows = desc->T > 0, br = desc->r > 0;
    NOBLE_TRY(need(x, rows));
    NOBLE_TRY(need(W, true));
    NOBLE_TRY(optional(b));
    NOBLE_TRY(need(y, rows));
    if (br) {
        const bool l2 = act_two_layers(desc->activation);
        NOBLE_TRY(need(W_down, true));
        NOBLE_TRY(need(omega1, true));
        NOBLE_TRY(need(phi1, true));
        NOBLE_TRY(l2 ? need(M, true) : optional(M));
        NOBLE_TRY(l2 ? need(omega2, true) : optional(omega2));
        NOBLE_TRY(l2 ? need(phi2, true) : optional(phi2));
        NOBLE_TRY(need(W_up, true));
        NOBLE_TRY(optional(reserve));   // NULL: inference-only forward
        if (scratch_bytes >= 0) {
            NOBLE_TRY(need(scratch, rows));
            if ((size_t)scratch_bytes < fwd_scratch_need(desc)) return NOBLE_ERR_WORKSPACE_TOO_SMALL;
        } else if (fwd_scratch_need(desc) > kStaticScratchBytes) {
            return NOBLE_ERR_WORKSPACE_TOO_SMALL;
        }
    }
    return NOBLE_OK;
}

}  // namespace

extern "C" {

noble_status noble_linear_fwd(const noble_linear_desc* desc, const void* x, const void* W, const float* b,
                              const void* W_down, const float* omega1, const float* phi1, const void* M,
                              const float* omega2, const float* phi2, const void* W_up, void* y, void* reserve,
                              void* scratch, size_t scratch_bytes, void* stream) {
    NOBLE_TRY(fwd_check(desc, x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, scratch,
                        (int64_t)std::min<size_t>(scratch_bytes, (size_t)INT64_MAX)));
    if (desc->T == 0) return NOBLE_OK;
    NOBLE_TRY(check_device());
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (desc->dtype == NOBLE_BF16)
        return fwd_impl<uint16_t>(desc, x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, scratch, st);
    return fwd_impl<float>(desc, x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, scratch, st);
}

noble_status noble_linear_fwd_static(const noble_linear_desc* desc, const void* x, const void* W, const float* b,
                                     const void* W_down, const float* omega1, const float* phi1, const void* M,
                                     const float* omega2, const float* phi2, const void* W_up, void* y,
                                     void* reserve, void* stream) {
    NOBLE_TRY(fwd_check(desc, x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, nullptr, -1));
    if (desc->T == 0) return NOBLE_OK;
    int dev = 0;
    NOBLE_TRY(check_device(&dev));
    void* scratch = nullptr;
    if (desc->r > 0) NOBLE_TRY(static_scratch(dev, &scratch));
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (desc->dtype == NOBLE_BF16)
        return fwd_impl<uint16_t>(desc, x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, scratch, st);
    return fwd_impl<float>(desc, x, W, b, W_down, omega1, phi1, M, omega2, phi2, W_up, y, reserve, scratch, st);
}

noble_status noble_linear_bwd(const noble_linear_desc* desc, const void* dy, const void* x, const void* W,
                              const void* W_down, const float* omega1, const float* phi1, const void* M,
                              const float* omega2, const float* phi2, const void* W_up, const void* reserve, void* dx,
                              float* dW, float* db, float* dW_down, float* dM, float* dW_up, float* domega1,
                              float* dphi1, float* domega2, float* dphi2, void* scratch, size_t scratch_bytes,
                              void* stream) {
    NOBLE_TRY(check_desc(desc));
    NOBLE_TRY(check_grids(desc));
    const bool rows = desc->T > 0, br = desc->r > 0;
    NOBLE_TRY(need(dy, rows));
    NOBLE_TRY(need(x, rows));
    NOBLE_TRY(need(W, true));
    NOBLE_TRY(need(dx, rows));
    NOBLE_TRY(need(dW, true));
    NOBLE_TRY(optional(db));
    if (br) {
        const bool l2 = act_two_layers(desc->activation);
        NOBLE_TRY(need(W_down, true));
        NOBLE_TRY(need(omega1, true));
        NOBLE_TRY(need(phi1, true));
        NOBLE_TRY(l2 ? need(M, true) : optional(M));
        NOBLE_TRY(l2 ? need(omega2, true) : optional(omega2));
        NOBLE_TRY(l2 ? need(phi2, true) : optional(phi2));
        NOBLE_TRY(need(W_up, true));
        NOBLE_TRY(need(reserve, rows));
        NOBLE_TRY(need(dW_down, true));
        NOBLE_TRY(l2 ? need(dM, true) : optional(dM));
        NOBLE_TRY(need(dW_up, true));
        NOBLE_TRY(need(domega1, true));
        NOBLE_TRY(need(dphi1, true));
        NOBLE_TRY(l2 ? need(domega2, true) : optional(domega2));
        NOBLE_TRY(l2 ? need(dphi2, true) : optional(dphi2));
    }
    if (scratch_need(desc) > 0) {
        NOBLE_TRY(need(scratch, rows));
        if (rows && scratch_bytes < scratch_need(desc)) return NOBLE_ERR_WORKSPACE_TOO_SMALL;
    }
    NOBLE_TRY(check_device());
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (desc->dtype == NOBLE_BF16)
        return bwd_impl<uint16_t>(desc, dy, x, W, W_down, omega1, phi1, M, omega2, phi2, W_up, reserve, dx, dW, db,
                                  dW_down, dM, dW_up, domega1, dphi1, domega2, dphi2, scratch, st);
    return bwd_impl<float>(desc, dy, x, W, W_down, omega1, phi1, M, omega2, phi2, W_up, reserve, dx, dW, db, dW_down,
                           dM, dW_up, domega1, dphi1, domega2, dphi2, scratch, st);
}

noble_status noble_profile_next_wgrad(void* start_event, void* stop_event, int64_t* workgroups) {
    t_wgrad_ev0 = static_cast<hipEvent_t>(start_event);
    t_wgrad_ev1 = static_cast<hipEvent_t>(stop_event);
    t_wgrad_wgs = workgroups;
    return NOBLE_OK;
}

void noble_recipe_defaults(noble_recipe* r) {
    if (!r) return;
    r->alpha = 0.01;
    r->w_scale = 0.5;
    r->omega_min = 0.8;
    r->omega_max = 1.2;
    r->phi_std = 0.1;
    r->gamma = 0.3;
    r->gamma_M = 0.45;
    r->omega_lr = 3.0;
    r->phi_lr = 5.0;
}

noble_status noble_lr_multipliers(const noble_linear_desc* desc, const noble_recipe* recipe, noble_lr_mults* out) {
    if (!recipe || !out) return NOBLE_ERR_NULL_ARG;
    NOBLE_TRY(check_desc(desc));
    *out = noble_lr_mults{1.0, 1.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    if (desc->r == 0) return NOBLE_OK;
    // Sec. 3.3 Eqs. 3-4: the ratio of the smaller layer width to the rank,
    // raised to 2 gamma (W_up) and gamma_M (M); for a grouped layer the width
    // of one group (each group is its own d_in -> d_out / G layer)
    const double ratio = (double)std::min(desc->d_in, group_dout(desc)) / (double)desc->r;
    out->W_down = 1.0;
    out->W_up = std::pow(ratio, 2.0 * recipe->gamma);
    out->M = std::pow(ratio, recipe->gamma_M);
    out->omega = recipe->omega_lr;
    out->phi = recipe->phi_lr;
    return NOBLE_OK;
}

noble_status noble_init_params(const noble_linear_desc* desc, const noble_recipe* recipe, uint64_t seed, void* W,
                               float* b, void* W_down, float* omega1, float* phi1, void* M, float* omega2,
                               float* phi2, void* W_up, void* stream) {
    if (!recipe) return NOBLE_ERR_NULL_ARG;
    NOBLE_TRY(check_desc(desc));
    const bool bf = desc->dtype == NOBLE_BF16;
    const int64_t din = desc->d_in, dout = desc->d_out, r = desc->r;
    const int64_t R = rank_total(desc), G = ngroups(desc), dog = group_dout(desc);
    InitList L{};
    L.k0 = (uint32_t)seed;
    L.k1 = (uint32_t)(seed >> 32);
    auto add = [&](void* p, int64_t n, int kind, double a, double bb, bool storage, int id) -> noble_status {
        if (!p || n == 0) return NOBLE_OK;
        const uintptr_t align = storage && bf ? 2 : 4;
        if (reinterpret_cast<uintptr_t>(p) % align) return NOBLE_ERR_MISALIGNED;
        InitTensor& t = L.t[L.count++];
        t.ptr = p;
        t.n = n;
        t.kind = kind;
        t.a = a;
        t.b = bb;
        t.bf16 = storage && bf ? 1 : 0;
        t.tensor_id = id;
        return NOBLE_OK;
    };
    NOBLE_TRY(add(W, din * dout, 0, recipe->w_scale / std::sqrt((double)din), 0.0, true, 0));
    NOBLE_TRY(add(b, dout, 2, 0.0, 0.0, false, 8));
    if (r > 0) {
        const double dbound = 1.0 / std::sqrt((double)din);
        const double mbound = std::sqrt(3.0 / (double)r);   // Xavier uniform, fan_in = fan_out = r
        NOBLE_TRY(add(W_down, din * R, 1, -dbound, dbound, true, 1));
        NOBLE_TRY(add(omega1, R, 1, recipe->omega_min, recipe->omega_max, false, 2));
        NOBLE_TRY(add(phi1, R, 0, recipe->phi_std, 0.0, false, 3));
        // the 3-layer form: M [2][G][r][r], omega2 and phi2 [2][R]
        const int64_t nm = n_mix(desc);
        NOBLE_TRY(add(M, nm * G * r * r, 1, -mbound, mbound, true, 4));
        NOBLE_TRY(add(omega2, nm * R, 1, recipe->omega_min, recipe->omega_max, false, 5));
        NOBLE_TRY(add(phi2, nm * R, 0, recipe->phi_std, 0.0, false, 6));
        NOBLE_TRY(add(W_up, R * dog, 0, recipe->alpha / std::sqrt((double)r), 0.0, true, 7));
    }
    if (L.count == 0) return NOBLE_OK;
    NOBLE_TRY(check_device());
    return launch(init_kernel, dim3(1024), dim3(256), static_cast<hipStream_t>(stream), L);
}

}  // extern "C"
