// Per-replica workload (Section 3.1, the workload model: w_er is the number
// of tasks of expert e executed by its replica on rank r; Section 3.2,
// Stage 2 tracks it per replica for the intra-node rebalancing).
//
// load[e][r] += #{pairs p : topk_idx[p] = e and assigned_rank[p] = r}.
// Same two-kernel scheme as the co-activation statistics: each workgroup
// counts a contiguous chunk of pairs into an LDS histogram of a band of
// expert rows (all of them when E*G fits), writes it to the workspace with
// plain stores, and a reduce kernel with eight lanes per bin sums the chunks
// and adds the total into load with a single writer per element.
#include <algorithm>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kLoadThreads = 1024;
constexpr int kReduceThreads = 256;
constexpr int kReduceLanes = 8;
constexpr int64_t kPairsPerChunk = 16384;
constexpr int64_t kMaxChunks = 64;
constexpr int64_t kBandWords = 16384;  // 64 KiB of LDS

struct LoadPlan {
    int nchunks, nbands, band_rows;
    int64_t pairs_per_chunk;
    int64_t stride;  // words of one (chunk, band) partial
    size_t bytes;
};

LoadPlan make_plan(int64_t T, int K, int E, int G) {
    LoadPlan p;
    const int64_t pairs = T * K;
    p.nchunks = (int)std::min<int64_t>(kMaxChunks, std::max<int64_t>(1, pairs / kPairsPerChunk));
    p.pairs_per_chunk = std::max<int64_t>(1, (pairs + p.nchunks - 1) / p.nchunks);
    p.band_rows = (int)std::max<int64_t>(1, std::min<int64_t>(E, kBandWords / G));
    p.nbands = (E + p.band_rows - 1) / p.band_rows;
    p.stride = (int64_t)p.band_rows * G;
    p.bytes = ((size_t)p.nchunks * p.nbands * p.stride * 4 + 255) & ~size_t(255);
    return p;
}

__global__ __launch_bounds__(kLoadThreads) void load_count_kernel(
    const int32_t* __restrict__ topk, const int32_t* __restrict__ assigned, int64_t TK, int E,
    int G, int nchunks, int band_rows, int64_t pairs_per_chunk, int64_t stride,
    uint32_t* __restrict__ part) {
    __shared__ uint32_t hist[kBandWords];
    const int chunk = blockIdx.x % nchunks;
    const int band = blockIdx.x / nchunks;
    const int e_lo = band * band_rows;
    const int e_hi = min(E, e_lo + band_rows);
    const int nbins = (e_hi - e_lo) * G;
    for (int b = threadIdx.x; b < nbins; b += kLoadThreads) hist[b] = 0;
    __syncthreads();
    const int64_t p0 = (int64_t)chunk * pairs_per_chunk;
    const int64_t p1 = min(TK, p0 + pairs_per_chunk);
    for (int64_t p = p0 + threadIdx.x; p < p1; p += kLoadThreads) {
        const int e = topk[p];
        const int r = assigned[p];
        if (e >= e_lo && e < e_hi && r >= 0 && r < G) atomicAdd(&hist[(e - e_lo) * G + r], 1u);
    }
    __syncthreads();
    uint32_t* out = part + (int64_t)blockIdx.x * stride;
    for (int b = threadIdx.x; b < nbins; b += kLoadThreads) out[b] = hist[b];
}

__global__ __launch_bounds__(kReduceThreads) void load_reduce_kernel(
    const uint32_t* __restrict__ part, int E, int G, int nchunks, int band_rows, int64_t stride,
    uint32_t* __restrict__ load) {
    const int64_t gid = (int64_t)blockIdx.x * kReduceThreads + threadIdx.x;
    const int64_t bin = gid / kReduceLanes;
    const int k = (int)(gid % kReduceLanes);
    const int64_t nbins = (int64_t)E * G;
    uint32_t sum = 0;
    if (bin < nbins) {
        const int e = (int)(bin / G);
        const int band = e / band_rows;
        const uint32_t* src = part + (int64_t)band * nchunks * stride + (bin - (int64_t)band * band_rows * G);
#pragma unroll 8
        for (int c = k; c < nchunks; c += kReduceLanes) sum += src[(int64_t)c * stride];
    }
#pragma unroll
    for (int o = 1; o < kReduceLanes; o <<= 1) sum += __shfl_xor(sum, o, kReduceLanes);
    if (k == 0 && bin < nbins && sum) load[bin] += sum;
}

}  // namespace

size_t replica_load_workspace_bytes(int64_t T, int K, int E, int G) {
    return std::max<size_t>(make_plan(T, K, E, G).bytes, 256);
}

cobalt_status launch_replica_load(const int32_t* topk, const int32_t* assigned, int64_t T, int K,
                                  int E, int G, uint32_t* load, void* ws, size_t ws_bytes,
                                  hipStream_t s) {
    const LoadPlan p = make_plan(T, K, E, G);
    if (ws_bytes < p.bytes) return COBALT_EINVAL;
    uint32_t* part = (uint32_t*)ws;
    hipLaunchKernelGGL(load_count_kernel, dim3((unsigned)(p.nchunks * p.nbands)),
                       dim3(kLoadThreads), 0, s, topk, assigned, T * K, E, G, p.nchunks,
                       p.band_rows, p.pairs_per_chunk, p.stride, part);
    COBALT_LAUNCH_CHECK();
    const int64_t items = (int64_t)E * G * kReduceLanes;
    hipLaunchKernelGGL(load_reduce_kernel,
                       dim3((unsigned)((items + kReduceThreads - 1) / kReduceThreads)),
                       dim3(kReduceThreads), 0, s, part, E, G, p.nchunks, p.band_rows, p.stride,
                       load);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
