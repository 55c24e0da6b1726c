// Communication-aware task assignment (Section 3.3, Algorithm 1), one lane
// per token.
//
// Step 1 (select execution nodes): the token's experts without a replica on
// the source node form U_t, each with its remote-node mask m (N-1 bits, bit
// i = the i-th node other than the source node). Algorithm 1 keeps the first
// feasible cover in order of (node count, mask value). The search here
// reaches the same cover without a table:
//  - F, the union of the masks with a single node, is contained in every
//    feasible cover. If F meets every mask of U_t, no other cover has as few
//    nodes, so F is the answer.
//  - Otherwise the answer is F | S, where S is the first subset, by (size,
//    value), of A = (union of the masks F misses) that meets each of those
//    masks (nodes outside A can only be dropped). Subsets of A of size c are
//    enumerated in increasing value with Gosper's next-combination step on
//    c-bit patterns deposited onto the bits of A; since F and S are disjoint
//    this is the order of F | S. The masks F misses are packed into SWAR
//    words, one 8- or 16-bit lane per slot, so each subset is tested for all
//    slots at once: it meets every mask iff no lane of
//    (packed & broadcast(S)) | fill is zero.
// Each expert of U_t then draws one of the cover's nodes holding it.
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
    int K, E, N, g, G, mode;
    uint64_t key;
    const uint32_t* node_mask;
    const uint32_t* rank_mask;
    const int32_t* owner;
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

// Writes a token's K ranks: two 16-byte stores for K = 8 (KV), one 4-byte
// store per slot otherwise.
template <bool KV>
__device__ __forceinline__ void store_ranks(int32_t* out, int K, const int (&r)[kMaxK]) {
    if constexpr (KV) {
        int4* o = reinterpret_cast<int4*>(out);
        o[0] = make_int4(r[0], r[1], r[2], r[3]);
        o[1] = make_int4(r[4], r[5], r[6], r[7]);
    } else {
#pragma unroll
        for (int j = 0; j < kMaxK; ++j)
            if (j < K) out[j] = r[j];
    }
}

// KV: K = 8 with 16-byte aligned topk and out, read and written with two
// 16-byte accesses per token.
template <int LB, bool KV>
__global__ __launch_bounds__(kAssignThreads) void assign_kernel(AssignArgs a) {
    using SW = Swar<LB>;
    const int64_t t = (int64_t)blockIdx.x * kAssignThreads + threadIdx.x;
    if (t >= a.T) return;
    const int K = KV ? 8 : a.K;
    const int64_t p0 = t * K;
    const int s = a.src ? a.src[t] : (int)(t / a.tok_per_src);
    int rr[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) rr[j] = -1;
    if (s < 0 || s >= a.G) {
        store_ranks<KV>(a.out + p0, K, rr);
        if (a.remote) a.remote[t] = 0;
        return;
    }
    const int home = s / a.g;
    const uint32_t home_bit = 1u << home;
    const uint32_t low = home_bit - 1u;

    int e[kMaxK];
    if constexpr (KV) {
        const int4* q = reinterpret_cast<const int4*>(a.topk + p0);
        const int4 v0 = q[0], v1 = q[1];
        e[0] = v0.x; e[1] = v0.y; e[2] = v0.z; e[3] = v0.w;
        e[4] = v1.x; e[5] = v1.y; e[6] = v1.z; e[7] = v1.w;
    }
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        if constexpr (!KV) e[j] = j < K ? a.topk[p0 + j] : -1;
        if (j >= K) e[j] = -1;
        e[j] = (e[j] >= 0 && e[j] < a.E) ? e[j] : -1;
    }

    if (a.mode == 1) {  // owner-only baseline
        uint32_t nodes = 0;
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) {
            if (j < K && e[j] >= 0) {
                rr[j] = a.owner[e[j]];
                const int n = rr[j] / a.g;
                if (n != home) nodes |= 1u << n;
            }
        }
        store_ranks<KV>(a.out + p0, K, rr);
        if (a.remote) a.remote[t] = (uint16_t)nodes;
        return;
    }

    // Step 1: remote masks of U_t and the nodes every cover needs.
    uint32_t m[kMaxK];
    uint32_t forced = 0;
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        m[j] = 0;
        if (j < K && e[j] >= 0) {
            const uint32_t nm = a.node_mask[e[j]];
            if (!(nm & home_bit)) {
                m[j] = (nm & low) | ((nm >> (home + 1)) << home);
                if ((m[j] & (m[j] - 1u)) == 0) forced |= m[j];
            }
        }
    }
    // Masks the forced nodes miss, packed one lane per slot; fill lane j is
    // non-zero exactly for the other slots.
    uint64_t packed[SW::kWords], fill[SW::kWords];
#pragma unroll
    for (int w = 0; w < SW::kWords; ++w) {
        packed[w] = 0;
        fill[w] = SW::kOnes;
    }
    uint32_t spare = 0;  // A: nodes that can still help
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        if (m[j] && !(m[j] & forced)) {
            const int w = j / SW::kLanes, sh = (j % SW::kLanes) * LB;
            packed[w] |= (uint64_t)m[j] << sh;
            fill[w] &= ~(SW::kLaneMask << sh);
            spare |= m[j];
        }
    }
    uint32_t bstar = forced;
    if (spare) {
        const int na = __builtin_popcount(spare);
        uint32_t extra = spare;  // the whole of A always meets every mask
        bool found = false;
        for (int c = 1; c <= na && !found; ++c) {
            for (uint32_t pat = (1u << c) - 1u; pat < (1u << na);) {
                // deposit the bits of pat onto the set bits of A, in order
                uint32_t sub = 0, rest = spare, pp = pat;
                while (pp) {
                    const uint32_t low_bit = rest & (0u - rest);
                    if (pp & 1u) sub |= low_bit;
                    rest ^= low_bit;
                    pp >>= 1;
                }
                const uint64_t bb = (uint64_t)sub * SW::kOnes;
                bool ok = true;
#pragma unroll
                for (int w = 0; w < SW::kWords; ++w)
                    ok = ok && !SW::has_zero_lane((packed[w] & bb) | fill[w]);
                if (ok) {
                    extra = sub;
                    found = true;
                    break;
                }
                // Gosper's hack: next larger pattern with the same popcount
                const uint32_t u = pat & (0u - pat);
                const uint32_t v = pat + u;
                pat = v + (((v ^ pat) >> __builtin_ctz(u)) >> 2);
            }
        }
        bstar |= extra;
    }

    // Node of each task, then its rank (Step 2).
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        if (j < K && e[j] >= 0) {
            const int64_t p = p0 + j;
            int n = home;
            const uint32_t cand = bstar & m[j];  // empty only on invalid layouts
            if (m[j] && cand) {
                const int bit = kth_bit(cand, draw(a.key, p, 0, __builtin_popcount(cand)));
                n = bit + (bit >= home ? 1 : 0);
            }
            const uint32_t R = a.rank_mask[(int64_t)e[j] * a.N + n];
            if ((!m[j] || cand) && R)
                rr[j] = n * a.g + kth_bit(R, draw(a.key, p, 1, __builtin_popcount(R)));
        }
    }
    store_ranks<KV>(a.out + p0, K, rr);
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
    a.mode = mode;
    a.key = key;
    a.node_mask = L.node_mask;
    a.rank_mask = L.rank_mask;
    a.owner = L.owner;
    a.out = out;
    a.remote = remote;
    const unsigned blocks = (unsigned)((T + kAssignThreads - 1) / kAssignThreads);
    const bool kv = K == 8 && ((uintptr_t)topk & 15u) == 0 && ((uintptr_t)out & 15u) == 0;
    auto launch = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kAssignThreads), 0, s, a);
    };
    if (L.N <= 9)
        kv ? launch(assign_kernel<8, true>) : launch(assign_kernel<8, false>);
    else
        kv ? launch(assign_kernel<16, true>) : launch(assign_kernel<16, false>);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
