// Co-activation statistics (Section 3.2, Stage 1): per-pair co-selection
// counts c_ij and per-expert task counts w_e, as raw uint32 increments.
//
// Each workgroup keeps a private histogram of the unordered pairs i < j in
// LDS (the upper triangle, row-major), restricted to a band of rows so that
// the band fits the workgroup's LDS; blockIdx.y selects the band and
// blockIdx.x a contiguous chunk of tokens. Tokens' pairs are added with LDS
// atomics; at the end the non-zero bins are added to coact[i][j] and
// coact[j][i] with global atomics (the matrix is symmetric by definition).
// The expert counts use a second small LDS histogram in band 0.
#include <algorithm>
#include <vector>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kStatsThreads = 512;
constexpr int kMaxBands = 256;

struct Bands {
    int n;
    int row[kMaxBands + 1];  // band b covers rows [row[b], row[b+1])
};

__host__ __device__ inline uint32_t tri_index(uint32_t i, uint32_t j, uint32_t E) {
    // position of (i, j), i < j, in the row-major upper triangle
    return i * (2u * E - i - 1u) / 2u + (j - i - 1u);
}

__global__ __launch_bounds__(kStatsThreads) void coact_kernel(
    const int32_t* __restrict__ topk, int64_t T, int K, int E, Bands bands,
    int64_t tok_per_blk, uint32_t* __restrict__ coact, uint32_t* __restrict__ count) {
    extern __shared__ uint32_t lds[];
    const int band = blockIdx.y;
    const int row_lo = bands.row[band], row_hi = bands.row[band + 1];
    const uint32_t first = tri_index(row_lo, row_lo + 1, E);
    const uint32_t last = (row_hi >= E - 1) ? (uint32_t)E * (E - 1) / 2 : tri_index(row_hi, row_hi + 1, E);
    const uint32_t nwords = last - first;
    uint32_t* hist = lds;
    uint32_t* cnt = lds + nwords;
    const bool do_count = count != nullptr && band == 0;

    for (uint32_t w = threadIdx.x; w < nwords; w += kStatsThreads) hist[w] = 0;
    if (do_count)
        for (int e = threadIdx.x; e < E; e += kStatsThreads) cnt[e] = 0;
    __syncthreads();

    const int64_t t0 = (int64_t)blockIdx.x * tok_per_blk;
    const int64_t t1 = min(T, t0 + tok_per_blk);
    for (int64_t t = t0 + threadIdx.x; t < t1; t += kStatsThreads) {
        int e[kMaxK];
#pragma unroll
        for (int a = 0; a < kMaxK; ++a) {
            e[a] = -1;
            if (a < K) {
                const int v = topk[t * K + a];
                e[a] = (v >= 0 && v < E) ? v : -1;
            }
        }
        if (do_count) {
#pragma unroll
            for (int a = 0; a < kMaxK; ++a)
                if (a < K && e[a] >= 0) atomicAdd(&cnt[e[a]], 1u);
        }
#pragma unroll
        for (int a = 0; a < kMaxK; ++a) {
#pragma unroll
            for (int b = a + 1; b < kMaxK; ++b) {
                if (b < K && e[a] >= 0 && e[b] >= 0 && e[a] != e[b]) {
                    const int i = min(e[a], e[b]), j = max(e[a], e[b]);
                    if (i >= row_lo && i < row_hi) atomicAdd(&hist[tri_index(i, j, E) - first], 1u);
                }
            }
        }
    }
    __syncthreads();

    for (int i = row_lo; i < row_hi; ++i) {
        const uint32_t rb = tri_index(i, i + 1, E) - first;
        for (int j = i + 1 + threadIdx.x; j < E; j += kStatsThreads) {
            const uint32_t v = hist[rb + (j - i - 1)];
            if (v) {
                atomicAdd(&coact[(int64_t)i * E + j], v);
                atomicAdd(&coact[(int64_t)j * E + i], v);
            }
        }
    }
    if (do_count)
        for (int e = threadIdx.x; e < E; e += kStatsThreads) {
            const uint32_t v = cnt[e];
            if (v) atomicAdd(&count[e], v);
        }
}

}  // namespace

cobalt_status launch_coact_stats(const int32_t* topk, int64_t T, int K, int E, uint32_t* coact,
                                 uint32_t* count, hipStream_t s) {
    DeviceInfo di;
    if (cobalt_status st = device_info(&di)) return st;
    const size_t budget_words = (size_t)di.lds_bytes / 4 - (size_t)E;
    Bands bands{};
    bands.n = 0;
    bands.row[0] = 0;
    if (E == 1) {
        bands.n = 1;
        bands.row[1] = 1;
    }
    size_t max_words = 0;
    for (int i = 0; i < E - 1;) {
        size_t words = 0;
        int j = i;
        while (j < E - 1 && words + (size_t)(E - 1 - j) <= budget_words) {
            words += (size_t)(E - 1 - j);
            ++j;
        }
        if (j == i) return COBALT_EUNSUPPORTED;  // a single row exceeds LDS
        if (bands.n == kMaxBands) return COBALT_EUNSUPPORTED;
        bands.row[++bands.n] = j;
        max_words = std::max(max_words, words);
        i = j;
    }
    // Tokens per workgroup: enough pair increments to amortise clearing and
    // flushing the band, but at least one workgroup per CU overall.
    const int64_t pairs_per_tok = std::max<int64_t>(1, (int64_t)K * (K - 1) / 2);
    const int64_t want = std::max<int64_t>(1, (int64_t)max_words / pairs_per_tok);
    int64_t chunks = std::max<int64_t>(1, T / std::max<int64_t>(want, 1));
    chunks = std::max<int64_t>(chunks, (di.cus + bands.n - 1) / bands.n);
    chunks = std::min<int64_t>(chunks, (T + 63) / 64);
    chunks = std::max<int64_t>(chunks, 1);
    const int64_t tok_per_blk = (T + chunks - 1) / chunks;
    chunks = (T + tok_per_blk - 1) / tok_per_blk;
    const size_t lds = (max_words + (size_t)E) * sizeof(uint32_t);
    if (lds > 64 * 1024 &&
        hipFuncSetAttribute((const void*)coact_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds) != hipSuccess)
        return COBALT_EHIP;
    dim3 grid((unsigned)chunks, (unsigned)bands.n);
    hipLaunchKernelGGL(coact_kernel, grid, dim3(kStatsThreads), lds, s, topk, T, K, E, bands,
                       tok_per_blk, coact, count);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
