// Co-activation statistics (Section 3.2, Stage 1): per-pair co-selection
// counts c_ij and per-expert task counts w_e, as raw uint32 increments.
//
// Two kernels:
//   count   each workgroup takes a contiguous chunk of tokens and counts, in
//           LDS, every unordered pair i < j of each token (the upper
//           triangle of the pair matrix, row-major) and every selection, with
//           LDS atomics; then writes its LDS histogram to its slot of the
//           workspace with plain stores. A token's ids are sorted in
//           registers first, so the bin of pair (a, b) is the row base of
//           e[a] plus e[b]. Each pair of each token is looked at
//           exactly once; the bins are 32-bit, or two 16-bit bins per word
//           when the triangle only fits that way (a chunk then holds at most
//           65535 tokens, so a bin cannot overflow).
//           When even 16-bit bins do not fit (E above ~400), the triangle is
//           split in row bands and the grid is (chunks x bands): each band
//           re-reads the chunk and keeps the pairs whose smaller expert falls
//           in its rows.
//   reduce  eight lanes per triangle bin sum that bin over all chunks
//           (each lane every eighth chunk, then shuffles) and the first adds
//           the total to coact[i][j] and coact[j][i]; another range of lanes
//           does the same for expert_count. Every output element has exactly
//           one writer, so no atomics are needed and the result does not
//           depend on scheduling.
// The workspace holds the partial histograms; its size comes from
// cobalt_coact_stats_workspace_bytes.
//
// Small calls (one band, at most kDirectUpdates bin updates over all
// chunks) skip the reduce: each count workgroup adds its nonzero bins
// straight into coact and expert_count with integer atomics, whose sums do
// not depend on their order. That saves the second launch, most of the time
// of such a call; beyond the limit, contention on the atomics would cost
// more than the reduce.
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
constexpr int kMaxBands = 1024;
constexpr int64_t kTokensPerChunk = 2048;
constexpr int64_t kMaxChunks = 64;
constexpr int64_t kDirectUpdates = 65536;

struct Bands {
    int n;
    uint16_t row[kMaxBands + 1];  // band b covers rows [row[b], row[b+1])
};

struct Plan {
    int nchunks;
    int nbands;
    bool half;              // two 16-bit bins per LDS word
    int64_t tok_per_chunk;
    int64_t words;          // E(E-1)/2
    int64_t band_stride;    // 32-bit words of one band's partial histogram
    size_t lds_bytes;
    size_t part_bytes;      // partial pair histograms
    size_t count_bytes;     // partial expert counts
};

// Start of row i in the triangle minus (i + 1), so that bin(i, j) = row_base(i) + j.
// i < 4096 and 2E - i - 1 < 8192 fit the 24-bit multiplier.
__device__ __forceinline__ int32_t row_base(int32_t i, int32_t E) {
    return (int32_t)(__umul24((uint32_t)i, (uint32_t)(2 * E - i - 1)) >> 1) - i - 1;
}

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Band rows for a per-band word budget (greedy, whole rows).
bool make_bands(int E, int64_t budget, Bands* b, int64_t* max_words) {
    b->n = 0;
    b->row[0] = 0;
    *max_words = 0;
    int i = 0;
    while (i < E - 1) {
        int64_t w = 0;
        int j = i;
        while (j < E - 1 && w + (E - 1 - j) <= budget) {
            w += E - 1 - j;
            ++j;
        }
        if (j == i || b->n == kMaxBands) return false;
        b->row[++b->n] = (uint16_t)j;
        *max_words = std::max(*max_words, w);
        i = j;
    }
    return true;
}

bool make_plan(int64_t T, int E, int lds_bytes, Plan* p, Bands* bands) {
    p->words = (int64_t)E * (E - 1) / 2;
    p->nchunks = (int)std::min<int64_t>(kMaxChunks, std::max<int64_t>(1, T / kTokensPerChunk));
    p->tok_per_chunk = std::max<int64_t>(1, (T + p->nchunks - 1) / p->nchunks);
    const int64_t lds_words = lds_bytes / 4 - E - 16;
    p->half = false;
    if (p->words <= lds_words) {
        p->nbands = 1;
        bands->n = 1;
        bands->row[0] = 0;
        bands->row[1] = (uint16_t)std::max(E - 1, 1);
        p->band_stride = std::max<int64_t>(p->words, 1);
    } else if ((p->words + 1) / 2 <= lds_words && p->tok_per_chunk <= 65535) {
        p->half = true;
        p->nbands = 1;
        bands->n = 1;
        bands->row[0] = 0;
        bands->row[1] = (uint16_t)(E - 1);
        p->band_stride = p->words;
    } else {
        int64_t mw = 0;
        if (!make_bands(E, lds_words, bands, &mw)) return false;
        p->nbands = bands->n;
        p->band_stride = mw;
    }
    const int64_t lds_hist = p->half ? (p->band_stride + 1) / 2 : p->band_stride;
    p->lds_bytes = (size_t)(lds_hist + E) * 4;
    p->part_bytes = align256((size_t)p->nchunks * p->nbands * p->band_stride * 4);
    p->count_bytes = align256((size_t)p->nchunks * E * 4);
    return true;
}

// Row i of triangle bin w: the largest i with row_base(i) + i + 1 <= w.
__device__ __forceinline__ int32_t tri_row(int32_t w, int32_t E) {
    const int32_t words = E * (E - 1) / 2;
    const int32_t r = words - 1 - w;  // index counted back from the last bin
    int32_t q = (int32_t)((sqrtf(8.0f * (float)r + 1.0f) - 1.0f) * 0.5f);
    while ((q + 1) * (q + 2) / 2 <= r) ++q;
    while (q > 0 && q * (q + 1) / 2 > r) --q;
    return E - 2 - q;
}

// KC = compile-time K (0: any K up to 16, read at run time). The ids of a
// token are sorted first (invalid ids sort last as INT_MAX), so each pair
// (a < b) has i = e[a] <= j = e[b] and costs one add on the row base of e[a].
template <bool kHalf, int KC>
__global__ __launch_bounds__(kCountThreads) void coact_count_kernel(
    const int32_t* __restrict__ topk, int64_t T, int Kr, int E, Bands bands, int nchunks,
    int64_t tok_per_chunk, int64_t band_stride, uint32_t* __restrict__ part,
    uint32_t* __restrict__ cpart, bool direct, uint32_t* __restrict__ coact,
    uint32_t* __restrict__ count) {
    constexpr int KM = KC ? KC : kMaxK;
    const int K = KC ? KC : Kr;
    extern __shared__ uint32_t lds[];
    const int chunk = blockIdx.x % nchunks;
    const int band = blockIdx.x / nchunks;
    const int row_lo = bands.row[band], row_hi = bands.row[band + 1];
    const int32_t words = E * (E - 1) / 2;
    const int32_t first = E > 1 ? row_base(row_lo, E) + row_lo + 1 : 0;
    const int32_t last = (row_hi >= E - 1) ? words : row_base(row_hi, E) + row_hi + 1;
    const int32_t nbins = last - first;
    const int32_t hist_words = kHalf ? (nbins + 1) / 2 : nbins;
    uint32_t* hist = lds;
    uint32_t* cnt = lds + hist_words;
    const bool do_count = band == 0;

    for (int32_t w = threadIdx.x; w < hist_words; w += kCountThreads) hist[w] = 0;
    for (int e = threadIdx.x; e < E; e += kCountThreads) cnt[e] = 0;
    __syncthreads();

    const int64_t t0 = (int64_t)chunk * tok_per_chunk;
    const int64_t t1 = min(T, t0 + tok_per_chunk);
    for (int64_t t = t0 + threadIdx.x; t < t1; t += kCountThreads) {
        int e[KM];
#pragma unroll
        for (int a = 0; a < KM; ++a) {
            int v = INT_MAX;
            if (a < K) {
                v = topk[t * K + a];
                if (v < 0 || v >= E) v = INT_MAX;
            }
            e[a] = v;
        }
        if (do_count) {
#pragma unroll
            for (int a = 0; a < KM; ++a)
                if (e[a] != INT_MAX) atomicAdd(&cnt[e[a]], 1u);
        }
        // odd-even transposition sort of the K ids
#pragma unroll
        for (int r = 0; r < KM; ++r) {
#pragma unroll
            for (int a = r & 1; a + 1 < KM; a += 2) {
                const int lo = min(e[a], e[a + 1]), hi = max(e[a], e[a + 1]);
                e[a] = lo;
                e[a + 1] = hi;
            }
        }
#pragma unroll
        for (int a = 0; a < KM; ++a) {
            const int i = e[a];
            if (i == INT_MAX || i < row_lo || i >= row_hi) continue;
            const int32_t rb = row_base(i, E) - first;
#pragma unroll
            for (int b = a + 1; b < KM; ++b) {
                const int j = e[b];
                if (j != INT_MAX && j != i) {
                    const int32_t bin = rb + j;
                    if (kHalf)
                        atomicAdd(&hist[bin >> 1], 1u << (16 * (bin & 1)));
                    else
                        atomicAdd(&hist[bin], 1u);
                }
            }
        }
    }
    __syncthreads();

    if (direct) {  // one band: the chunk's bins go straight to the outputs
        for (int32_t bin = threadIdx.x; bin < nbins; bin += kCountThreads) {
            const uint32_t v = kHalf ? (hist[bin >> 1] >> (16 * (bin & 1))) & 0xffffu : hist[bin];
            if (v == 0) continue;
            const int32_t i = tri_row(bin, E);
            const int32_t j = bin - (row_base(i, E) + i + 1) + i + 1;
            atomicAdd(&coact[(int64_t)i * E + j], v);
            atomicAdd(&coact[(int64_t)j * E + i], v);
        }
        if (count)
            for (int e = threadIdx.x; e < E; e += kCountThreads)
                if (cnt[e]) atomicAdd(&count[e], cnt[e]);
        return;
    }
    uint32_t* out = part + (int64_t)blockIdx.x * band_stride;
    for (int32_t bin = threadIdx.x; bin < nbins; bin += kCountThreads)
        out[bin] = kHalf ? (hist[bin >> 1] >> (16 * (bin & 1))) & 0xffffu : hist[bin];
    if (do_count) {
        uint32_t* cout = cpart + (int64_t)chunk * E;
        for (int e = threadIdx.x; e < E; e += kCountThreads) cout[e] = cnt[e];
    }
}

// kReduceLanes lanes per bin: lane k sums chunks k, k + kReduceLanes, ...;
// the lanes then combine with shuffles and the first writes the totals.
__global__ __launch_bounds__(kReduceThreads) void coact_reduce_kernel(
    const uint32_t* __restrict__ part, const uint32_t* __restrict__ cpart, int E, Bands bands,
    int nchunks, int64_t band_stride, bool do_count, uint32_t* __restrict__ coact,
    uint32_t* __restrict__ count) {
    const int32_t words = E * (E - 1) / 2;
    const int64_t gid = (int64_t)blockIdx.x * kReduceThreads + threadIdx.x;
    const int64_t g = gid / kReduceLanes;
    const int k = (int)(gid % kReduceLanes);
    uint32_t sum = 0;
    int32_t i = 0, j = 0;
    if (g < words) {
        i = tri_row((int32_t)g, E);
        j = (int32_t)g - (row_base(i, E) + i + 1) + i + 1;
        int lo = 0, hi = bands.n - 1;  // band holding row i
        while (lo < hi) {
            const int mid = (lo + hi + 1) / 2;
            if (bands.row[mid] <= i) lo = mid; else hi = mid - 1;
        }
        const int64_t off = g - (row_base(bands.row[lo], E) + bands.row[lo] + 1);
        const uint32_t* src = part + (int64_t)lo * nchunks * band_stride + off;
#pragma unroll 8
        for (int c = k; c < nchunks; c += kReduceLanes) sum += src[(int64_t)c * band_stride];
    } else if (do_count && g < words + E) {
        const int e = (int)(g - words);
#pragma unroll 8
        for (int c = k; c < nchunks; c += kReduceLanes) sum += cpart[(int64_t)c * E + e];
    }
#pragma unroll
    for (int o = 1; o < kReduceLanes; o <<= 1) sum += __shfl_xor(sum, o, kReduceLanes);
    if (k != 0 || sum == 0) return;
    if (g < words) {
        coact[(int64_t)i * E + j] += sum;
        coact[(int64_t)j * E + i] += sum;
    } else if (do_count && g < words + E) {
        count[g - words] += sum;
    }
}

}  // namespace

size_t coact_workspace_bytes(int64_t T, int E, int lds_bytes) {
    Plan p;
    Bands b;
    if (!make_plan(T, E, lds_bytes, &p, &b)) return 0;
    return p.part_bytes + p.count_bytes;
}

cobalt_status launch_coact_stats(const int32_t* topk, int64_t T, int K, int E, uint32_t* coact,
                                 uint32_t* count, void* ws, size_t ws_bytes, hipStream_t s) {
    DeviceInfo di;
    if (cobalt_status st = device_info(&di)) return st;
    Plan p;
    Bands bands;
    if (!make_plan(T, E, di.lds_bytes, &p, &bands)) return COBALT_EUNSUPPORTED;
    if (ws_bytes < p.part_bytes + p.count_bytes) return COBALT_EINVAL;
    const bool direct = p.nbands == 1 && p.nchunks * (p.words + E) <= kDirectUpdates;
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
        hipLaunchKernelGGL(kernel, dim3((unsigned)(p.nchunks * p.nbands)), dim3(kCountThreads),
                           p.lds_bytes, s, topk, T, K, E, bands, p.nchunks, p.tok_per_chunk,
                           p.band_stride, part, cpart, direct, coact, count);
        return COBALT_OK;
    };
    cobalt_status st;
    if (K == 8)
        st = p.half ? launch(coact_count_kernel<true, 8>, 0) : launch(coact_count_kernel<false, 8>, 1);
    else
        st = p.half ? launch(coact_count_kernel<true, 0>, 2) : launch(coact_count_kernel<false, 0>, 3);
    if (st != COBALT_OK) return st;
    COBALT_LAUNCH_CHECK();
    if (direct) return COBALT_OK;
    const int64_t items = (p.words + (count ? E : 0)) * kReduceLanes;
    hipLaunchKernelGGL(coact_reduce_kernel,
                       dim3((unsigned)((items + kReduceThreads - 1) / kReduceThreads)),
                       dim3(kReduceThreads), 0, s, part, cpart, E, bands, p.nchunks,
                       p.band_stride, count != nullptr, coact, count);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
