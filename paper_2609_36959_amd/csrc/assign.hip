// Communication-aware task assignment (Section 3.3, Algorithm 1), one lane
// per token.
//
// Step 1 (select execution nodes): the token's experts without a replica on
// the source node form U_t, each with its remote-node mask (N-1 bits, bit i
// = the i-th node other than the source node). The masks are packed into
// SWAR words, one 8- or 16-bit lane per slot, and a candidate cover b is
// tested for all slots at once: it is feasible iff no lane of
// (packed & broadcast(b)) | fill is zero, where fill makes the lanes of
// slots outside U_t non-zero. Candidates are tried in the layout's
// (popcount, value) order and the first feasible one is the cover Algorithm 1
// keeps. Each expert of U_t then draws one of the cover's nodes holding it.
// Step 2 (select execution ranks): every task draws one rank of its node
// holding the expert. Draws hash the pair index with SplitMix64.
#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kAssignThreads = 256;

struct AssignArgs {
    const int32_t* topk;
    const int32_t* src;
    int64_t T;
    int64_t tok_per_src;
    int K, E, N, g, G, ncand, mode;
    uint64_t key;
    const uint32_t* node_mask;
    const uint32_t* rank_mask;
    const int32_t* owner;
    const uint16_t* cand;
    int32_t* out;
    uint16_t* remote;
};

__device__ __forceinline__ uint32_t draw(uint64_t key, int64_t p, uint32_t stream, uint32_t cnt) {
    if (cnt <= 1) return 0;
    const uint64_t h = splitmix64(key ^ (((uint64_t)p << 1) | stream));
    return (uint32_t)(((h >> 32) * (uint64_t)cnt) >> 32);
}

// position of the k-th (0-based) set bit of v
__device__ __forceinline__ int kth_bit(uint32_t v, uint32_t k) {
    for (uint32_t i = 0; i < k; ++i) v &= v - 1u;
    return __builtin_ctz(v);
}

template <int LB>  // SWAR lane width in bits: 8 (N <= 9) or 16 (N <= 16)
struct Swar {
    static constexpr int kLanes = 64 / LB;
    static constexpr int kWords = (kMaxK + kLanes - 1) / kLanes;
    static constexpr uint64_t kOnes = LB == 8 ? 0x0101010101010101ull : 0x0001000100010001ull;
    static constexpr uint64_t kHigh = kOnes << (LB - 1);
    static constexpr uint64_t kLaneMask = (1ull << LB) - 1ull;
    __device__ static bool has_zero_lane(uint64_t v) { return ((v - kOnes) & ~v & kHigh) != 0; }
};

template <int LB>
__global__ __launch_bounds__(kAssignThreads) void assign_kernel(AssignArgs a) {
    using SW = Swar<LB>;
    const int64_t t = (int64_t)blockIdx.x * kAssignThreads + threadIdx.x;
    if (t >= a.T) return;
    const int K = a.K;
    const int64_t p0 = t * K;
    const int s = a.src ? a.src[t] : (int)(t / a.tok_per_src);
    if (s < 0 || s >= a.G) {
        for (int j = 0; j < K; ++j) a.out[p0 + j] = -1;
        if (a.remote) a.remote[t] = 0;
        return;
    }
    const int home = s / a.g;
    const uint32_t home_bit = 1u << home;
    const uint32_t low = home_bit - 1u;

    int e[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        e[j] = -1;
        if (j < K) {
            const int v = a.topk[p0 + j];
            e[j] = (v >= 0 && v < a.E) ? v : -1;
        }
    }

    if (a.mode == 1) {  // owner-only baseline
        uint32_t nodes = 0;
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) {
            if (j < K) {
                int r = -1;
                if (e[j] >= 0) {
                    r = a.owner[e[j]];
                    const int n = r / a.g;
                    if (n != home) nodes |= 1u << n;
                }
                a.out[p0 + j] = r;
            }
        }
        if (a.remote) a.remote[t] = (uint16_t)nodes;
        return;
    }

    // Step 1: remote masks of U_t, packed one lane per slot.
    // packed lane j = m_j for experts of U_t, 0 otherwise; fill lane j is
    // non-zero exactly for the other slots, so (packed & b) | fill has a
    // zero lane iff some expert of U_t has no node in b.
    uint32_t m[kMaxK];
    uint64_t packed[SW::kWords], fill[SW::kWords];
#pragma unroll
    for (int w = 0; w < SW::kWords; ++w) {
        packed[w] = 0;
        fill[w] = SW::kOnes;
    }
    bool any_remote = false;
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        m[j] = 0;
        if (j < K && e[j] >= 0) {
            const uint32_t nm = a.node_mask[e[j]];
            if (!(nm & home_bit)) {
                m[j] = (nm & low) | ((nm >> (home + 1)) << home);
                const int w = j / SW::kLanes, sh = (j % SW::kLanes) * LB;
                packed[w] |= (uint64_t)m[j] << sh;
                fill[w] &= ~(SW::kLaneMask << sh);
                any_remote = true;
            }
        }
    }
    uint32_t bstar = 0;
    if (any_remote) {
        // The all-remote cover is feasible whenever every expert has a
        // replica, so the scan always stops; the bound guards bad layouts.
        bstar = (uint32_t)a.ncand - 1u;
        for (int i = 0; i < a.ncand; ++i) {
            const uint32_t b = a.cand[i];
            const uint64_t bb = (uint64_t)b * SW::kOnes;
            bool ok = true;
#pragma unroll
            for (int w = 0; w < SW::kWords; ++w)
                ok = ok && !SW::has_zero_lane((packed[w] & bb) | fill[w]);
            if (ok) {
                bstar = b;
                break;
            }
        }
    }

    // Node of each task, then its rank (Step 2).
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        if (j < K) {
            const int64_t p = p0 + j;
            int r = -1;
            if (e[j] >= 0) {
                int n = home;
                const uint32_t cand = bstar & m[j];  // empty only on invalid layouts
                if (m[j] && cand) {
                    const int bit = kth_bit(cand, draw(a.key, p, 0, __builtin_popcount(cand)));
                    n = bit + (bit >= home ? 1 : 0);
                }
                const uint32_t R = a.rank_mask[(int64_t)e[j] * a.N + n];
                if ((!m[j] || cand) && R)
                    r = n * a.g + kth_bit(R, draw(a.key, p, 1, __builtin_popcount(R)));
            }
            a.out[p] = r;
        }
    }
    if (a.remote) a.remote[t] = (uint16_t)((bstar & low) | ((bstar >> home) << (home + 1)));
}

}  // namespace

cobalt_status launch_assign(const DeviceLayout& L, const int32_t* topk, const int32_t* src,
                            int64_t T, int K, uint64_t key, int mode, int32_t* out,
                            uint16_t* remote, hipStream_t s) {
    AssignArgs a;
    a.topk = topk;
    a.src = src;
    a.T = T;
    a.tok_per_src = src ? 1 : T / L.G;
    a.K = K;
    a.E = L.E;
    a.N = L.N;
    a.g = L.g;
    a.G = L.G;
    a.ncand = L.ncand;
    a.mode = mode;
    a.key = key;
    a.node_mask = L.node_mask;
    a.rank_mask = L.rank_mask;
    a.owner = L.owner;
    a.cand = L.cand;
    a.out = out;
    a.remote = remote;
    const unsigned blocks = (unsigned)((T + kAssignThreads - 1) / kAssignThreads);
    if (L.N <= 9)
        hipLaunchKernelGGL(assign_kernel<8>, dim3(blocks), dim3(kAssignThreads), 0, s, a);
    else
        hipLaunchKernelGGL(assign_kernel<16>, dim3(blocks), dim3(kAssignThreads), 0, s, a);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
