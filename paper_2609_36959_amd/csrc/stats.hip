// Co-activation statistics (Section 3.2, Stage 1): per-pair co-selection
// counts c_ij and per-expert task counts w_e, as raw uint32 increments.
//
// The unordered pairs i < j form a triangle of E(E-1)/2 bins. It is split
// into nb row bands, nb a power of two, with the rows interleaved: band b
// holds the rows i = b, b + nb, b + 2nb, ... Interleaving gives every band
// nearly the same number of bins and, since popular experts are spread over
// the ids, a similar share of the increments. In band b, local row r (i =
// r*nb + b) starts at
//     off_b(r) = r (E - 1 - b) - nb r (r - 1) / 2
// and bin (i, j) is off_b(r) + j - i - 1.
//
// Two kernels:
//   count   grid = chunks x bands. A workgroup takes a contiguous chunk of
//           tokens and keeps its band's bins, and the counts of the experts
//           e = b (mod nb), in LDS. Each thread loads a token's ids (16-byte
//           loads for K = 8), sorts them in registers, and for every sorted
//           slot a whose expert is in the band adds one to the bins (e[a],
//           e[b]) of the later slots, with LDS atomics. The band's bins and
//           counts are then written to the chunk's slot of the workspace.
//           Bands split the LDS atomics of a chunk over more CUs without
//           more partial histograms to reduce: the partials total chunks x
//           triangle either way.
//   reduce  lanes per band bin sum that bin over the chunks (each lane a
//           stride of chunks, then shuffles); the first lane adds the total
//           to coact[i][j] and coact[j][i]. Another range of lanes does the
//           same for expert_count. Every output element has exactly one
//           writer, so the result does not depend on scheduling.
//
// Small calls (one band, at most kDirectUpdates bin updates over all
// chunks) skip the reduce: each count workgroup adds its nonzero bins
// straight into coact and expert_count with integer atomics, whose sums do
// not depend on their order. That saves the second launch, most of the time
// of such a call.
#include <algorithm>
#include <climits>
#include <cmath>
#include <mutex>
#include <set>
#include <utility>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kCountThreads = 1024;
constexpr int kReduceThreads = 256;
constexpr int kReduceLanes = 8;  // lanes per bin in the reduce kernel
constexpr int kMaxLgBands = 12;
constexpr int64_t kTokensPerChunk = 2048;
constexpr int64_t kMaxChunks = 64;
constexpr int kParBands = 4;            // bands for parallelism on large calls
constexpr int64_t kParPairs = 1 << 18;  // T*K from which bands are used for parallelism
constexpr int64_t kDirectUpdates = 65536;

struct Plan {
    int nchunks;
    int lgb;                // log2 of the number of bands
    int64_t tok_per_chunk;
    int64_t words;          // E(E-1)/2
    int64_t band_stride;    // bins of the largest band (band 0)
    size_t lds_bytes;
    size_t part_bytes;      // partial pair histograms
    size_t count_bytes;     // partial expert counts
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Rows of band b: i = r*nb + b < E - 1.
__host__ __device__ inline int32_t band_rows(int32_t E, int32_t nb, int32_t b) {
    return b < E - 1 ? (E - 1 - b + nb - 1) / nb : 0;
}
// Start of local row r of band b.
__host__ __device__ inline int32_t band_off(int32_t E, int32_t nb, int32_t b, int32_t r) {
    return r * (E - 1 - b) - nb * (r * (r - 1) / 2);
}
__host__ __device__ inline int32_t band_words(int32_t E, int32_t nb, int32_t b) {
    return band_off(E, nb, b, band_rows(E, nb, b));
}

bool make_plan(int64_t T, int64_t K, int E, int lds_bytes, Plan* p) {
    p->words = (int64_t)E * (E - 1) / 2;
    p->nchunks = (int)std::min<int64_t>(kMaxChunks, std::max<int64_t>(1, T / kTokensPerChunk));
    p->tok_per_chunk = std::max<int64_t>(1, (T + p->nchunks - 1) / p->nchunks);
    // fewest bands whose largest band (band 0) and counts fit the LDS
    int lgb = 0;
    auto fits = [&](int l) {
        const int nb = 1 << l;
        const int64_t need = (int64_t)band_words(E, nb, 0) + (E + nb - 1) / nb;
        return need * 4 <= lds_bytes;
    };
    while (lgb <= kMaxLgBands && !fits(lgb)) ++lgb;
    if (lgb > kMaxLgBands) return false;
    // large calls: more bands, for more workgroups (at most one row per band)
    if (T * K >= kParPairs)
        while ((1 << lgb) < kParBands && (1 << (lgb + 1)) <= std::max(E - 1, 1)) ++lgb;
    p->lgb = lgb;
    const int nb = 1 << lgb;
    p->band_stride = std::max<int64_t>(band_words(E, nb, 0), 1);
    p->lds_bytes = (size_t)(p->band_stride + (E + nb - 1) / nb) * 4;
    p->part_bytes = align256((size_t)p->nchunks * nb * p->band_stride * 4);
    p->count_bytes = align256((size_t)p->nchunks * E * 4);
    return true;
}

// Row i of triangle bin w (one band): the largest i with i-th row start <= w.
__device__ __forceinline__ int32_t tri_row(int32_t w, int32_t E) {
    const int32_t words = E * (E - 1) / 2;
    const int32_t r = words - 1 - w;  // index counted back from the last bin
    int32_t q = (int32_t)((sqrtf(8.0f * (float)r + 1.0f) - 1.0f) * 0.5f);
    while ((q + 1) * (q + 2) / 2 <= r) ++q;
    while (q > 0 && q * (q + 1) / 2 > r) --q;
    return E - 2 - q;
}

__device__ __forceinline__ void cswap(int& a, int& b) {
    const int lo = min(a, b), hi = max(a, b);
    a = lo;
    b = hi;
}

// Sorts e[0..KM) ascending: Batcher's odd-even merge sort network for 8
// (19 comparators), odd-even transposition otherwise.
template <int KM>
__device__ __forceinline__ void sort_ids(int (&e)[KM]) {
    if constexpr (KM == 8) {
        cswap(e[0], e[1]); cswap(e[2], e[3]); cswap(e[4], e[5]); cswap(e[6], e[7]);
        cswap(e[0], e[2]); cswap(e[1], e[3]); cswap(e[4], e[6]); cswap(e[5], e[7]);
        cswap(e[1], e[2]); cswap(e[5], e[6]);
        cswap(e[0], e[4]); cswap(e[1], e[5]); cswap(e[2], e[6]); cswap(e[3], e[7]);
        cswap(e[2], e[4]); cswap(e[3], e[5]);
        cswap(e[1], e[2]); cswap(e[3], e[4]); cswap(e[5], e[6]);
    } else {
#pragma unroll
        for (int r = 0; r < KM; ++r) {
#pragma unroll
            for (int a = r & 1; a + 1 < KM; a += 2) cswap(e[a], e[a + 1]);
        }
    }
}

// KC = compile-time K (0: any K up to 16, read at run time); kVec: K = 8
// and a 16-byte aligned topk, read with two 16-byte loads per token. Ids
// outside [0, E) sort last as INT_MAX and count nowhere.
template <int KC, bool kVec>
__global__ __launch_bounds__(kCountThreads) void coact_count_kernel(
    const int32_t* __restrict__ topk, int64_t T, int Kr, int E, int lgb, int nchunks,
    int64_t tok_per_chunk, int64_t band_stride, uint32_t* __restrict__ part,
    uint32_t* __restrict__ cpart, bool direct, uint32_t* __restrict__ coact,
    uint32_t* __restrict__ count) {
    constexpr int KM = KC ? KC : kMaxK;
    const int K = KC ? KC : Kr;
    extern __shared__ uint32_t lds[];
    const int nb = 1 << lgb;
    const int chunk = blockIdx.x % nchunks;
    const int band = blockIdx.x / nchunks;
    const int32_t nbins = band_words(E, nb, band);
    const int32_t ncnt = band < E ? (E - band + nb - 1) / nb : 0;
    const int32_t row_len0 = E - 1 - band;  // length of local row 0
    uint32_t* hist = lds;
    uint32_t* cnt = lds + nbins;

    for (int32_t w = threadIdx.x; w < nbins + ncnt; w += kCountThreads) lds[w] = 0;
    __syncthreads();

    const int64_t t0 = (int64_t)chunk * tok_per_chunk;
    const int64_t t1 = min(T, t0 + tok_per_chunk);
    for (int64_t t = t0 + threadIdx.x; t < t1; t += kCountThreads) {
        int e[KM];
        if constexpr (kVec) {
            const int4* p = reinterpret_cast<const int4*>(topk + t * 8);
            const int4 v0 = p[0], v1 = p[1];
            e[0] = v0.x; e[1] = v0.y; e[2] = v0.z; e[3] = v0.w;
            e[4] = v1.x; e[5] = v1.y; e[6] = v1.z; e[7] = v1.w;
        } else {
#pragma unroll
            for (int a = 0; a < KM; ++a) e[a] = a < K ? topk[t * K + a] : INT_MAX;
        }
#pragma unroll
        for (int a = 0; a < KM; ++a)
            if (e[a] < 0 || e[a] >= E) e[a] = INT_MAX;
#pragma unroll
        for (int a = 0; a < KM; ++a)
            if (e[a] != INT_MAX && (e[a] & (nb - 1)) == band) atomicAdd(&cnt[e[a] >> lgb], 1u);
        sort_ids<KM>(e);
#pragma unroll
        for (int a = 0; a < KM; ++a) {
            const int i = e[a];
            if (i == INT_MAX || (i & (nb - 1)) != band) continue;
            const int32_t r = i >> lgb;
            const int32_t base = r * row_len0 - nb * (r * (r - 1) / 2) - i - 1;
#pragma unroll
            for (int b = a + 1; b < KM; ++b) {
                const int j = e[b];
                if (j != INT_MAX && j != i) atomicAdd(&hist[base + j], 1u);
            }
        }
    }
    __syncthreads();

    if (direct) {  // one band: the chunk's bins go straight to the outputs
        for (int32_t bin = threadIdx.x; bin < nbins; bin += kCountThreads) {
            const uint32_t v = hist[bin];
            if (v == 0) continue;
            const int32_t i = tri_row(bin, E);
            const int32_t j = bin - band_off(E, 1, 0, i) + i + 1;
            atomicAdd(&coact[(int64_t)i * E + j], v);
            atomicAdd(&coact[(int64_t)j * E + i], v);
        }
        if (count)
            for (int e = threadIdx.x; e < ncnt; e += kCountThreads)
                if (cnt[e]) atomicAdd(&count[e], cnt[e]);
        return;
    }
    uint32_t* out = part + ((int64_t)band * nchunks + chunk) * band_stride;
    for (int32_t bin = threadIdx.x; bin < nbins; bin += kCountThreads) out[bin] = hist[bin];
    uint32_t* cout = cpart + (int64_t)chunk * E;
    for (int32_t k = threadIdx.x; k < ncnt; k += kCountThreads) cout[k * nb + band] = cnt[k];
}

// kReduceLanes lanes per bin: lane k sums chunks k, k + kReduceLanes, ...;
// the lanes then combine with shuffles and the first writes the totals.
// Items [0, nb * band_stride) are the band bins, then E expert counts.
__global__ __launch_bounds__(kReduceThreads) void coact_reduce_kernel(
    const uint32_t* __restrict__ part, const uint32_t* __restrict__ cpart, int E, int lgb,
    int nchunks, int64_t band_stride, bool do_count, uint32_t* __restrict__ coact,
    uint32_t* __restrict__ count) {
    const int nb = 1 << lgb;
    const int64_t nbins = (int64_t)nb * band_stride;
    const int64_t gid = (int64_t)blockIdx.x * kReduceThreads + threadIdx.x;
    const int64_t g = gid / kReduceLanes;
    const int k = (int)(gid % kReduceLanes);
    uint32_t sum = 0;
    int32_t i = 0, j = 0;
    bool bin_item = false;
    if (g < nbins) {
        const int band = (int)(g / band_stride);
        const int32_t w = (int32_t)(g % band_stride);
        if (w < band_words(E, nb, band)) {
            bin_item = true;
            // local row: the last r with band_off(r) <= w
            int32_t lo = 0, hi = band_rows(E, nb, band) - 1;
            while (lo < hi) {
                const int32_t mid = (lo + hi + 1) / 2;
                if (band_off(E, nb, band, mid) <= w) lo = mid; else hi = mid - 1;
            }
            i = lo * nb + band;
            j = w - band_off(E, nb, band, lo) + i + 1;
            const uint32_t* src = part + (int64_t)band * nchunks * band_stride + w;
#pragma unroll 8
            for (int c = k; c < nchunks; c += kReduceLanes) sum += src[(int64_t)c * band_stride];
        }
    } else if (do_count && g < nbins + E) {
        const int e = (int)(g - nbins);
#pragma unroll 8
        for (int c = k; c < nchunks; c += kReduceLanes) sum += cpart[(int64_t)c * E + e];
    }
#pragma unroll
    for (int o = 1; o < kReduceLanes; o <<= 1) sum += __shfl_xor(sum, o, kReduceLanes);
    if (k != 0 || sum == 0) return;
    if (bin_item) {
        coact[(int64_t)i * E + j] += sum;
        coact[(int64_t)j * E + i] += sum;
    } else if (do_count && g >= nbins && g < nbins + E) {
        count[g - nbins] += sum;
    }
}

}  // namespace

size_t coact_workspace_bytes(int64_t T, int K, int E, int lds_bytes) {
    Plan p;
    if (!make_plan(T, K, E, lds_bytes, &p)) return 0;
    return p.part_bytes + p.count_bytes;
}

cobalt_status launch_coact_stats(const int32_t* topk, int64_t T, int K, int E, uint32_t* coact,
                                 uint32_t* count, void* ws, size_t ws_bytes, hipStream_t s) {
    DeviceInfo di;
    if (cobalt_status st = device_info(&di)) return st;
    Plan p;
    if (!make_plan(T, K, E, di.lds_bytes, &p)) return COBALT_EUNSUPPORTED;
    if (ws_bytes < p.part_bytes + p.count_bytes) return COBALT_EINVAL;
    const int nb = 1 << p.lgb;
    const bool direct = nb == 1 && p.nchunks * (p.words + E) <= kDirectUpdates;
    uint32_t* part = (uint32_t*)ws;
    uint32_t* cpart = (uint32_t*)((char*)ws + p.part_bytes);
    // The LDS limit of each kernel variant is raised to the device maximum
    // once per device (host-side only, so the calls stay capturable).
    auto launch = [&](auto kernel, int variant) -> cobalt_status {
        static std::mutex mu;
        static std::set<std::pair<int, int>> raised;
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess) return COBALT_EHIP;
        {
            std::lock_guard<std::mutex> lock(mu);
            if (!raised.count({variant, dev})) {
                if (hipFuncSetAttribute((const void*)kernel,
                                        hipFuncAttributeMaxDynamicSharedMemorySize,
                                        di.lds_bytes) != hipSuccess)
                    return COBALT_EHIP;
                raised.insert({variant, dev});
            }
        }
        hipLaunchKernelGGL(kernel, dim3((unsigned)(p.nchunks * nb)), dim3(kCountThreads),
                           p.lds_bytes, s, topk, T, K, E, p.lgb, p.nchunks, p.tok_per_chunk,
                           p.band_stride, part, cpart, direct, coact, count);
        return COBALT_OK;
    };
    cobalt_status st;
    if (K == 8 && ((uintptr_t)topk & 15u) == 0)
        st = launch(coact_count_kernel<8, true>, 0);
    else if (K == 8)
        st = launch(coact_count_kernel<8, false>, 1);
    else
        st = launch(coact_count_kernel<0, false>, 2);
    if (st != COBALT_OK) return st;
    COBALT_LAUNCH_CHECK();
    if (direct) return COBALT_OK;
    const int64_t items = ((int64_t)nb * p.band_stride + (count ? E : 0)) * kReduceLanes;
    hipLaunchKernelGGL(coact_reduce_kernel,
                       dim3((unsigned)((items + kReduceThreads - 1) / kReduceThreads)),
                       dim3(kReduceThreads), 0, s, part, cpart, E, p.lgb, p.nchunks,
                       p.band_stride, count != nullptr, coact, count);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
