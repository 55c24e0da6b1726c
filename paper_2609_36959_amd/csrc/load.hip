// Per-replica workload (Section 3.1, the workload model: w_er is the number
// of tasks of expert e executed by its replica on rank r; Section 3.2,
// Stage 2 tracks it per replica for the intra-node rebalancing).
//
// load[e][r] += #{pairs p : topk_idx[p] = e and assigned_rank[p] = r}.
// Same two-kernel scheme as the co-activation statistics:
//   count   grid = chunks x bands. A workgroup takes a contiguous chunk of
//           pairs and keeps the bins of a band of expert rows in LDS (all
//           rows when E*G fits and the grid is large enough without bands).
//           Pairs come four at a time with 16-byte loads of topk_idx and
//           assigned_rank where both are aligned. The band's bins are then
//           written out as uint16 where a chunk's pair count fits, else as
//           uint32.
//   reduce  sixteen lanes per group of eight bins sum the chunks (one
//           16-byte load of eight uint16 bins per chunk), add pairwise
//           across lanes k and k + 8, exchange halves in three shuffle
//           rounds, and lane k < 8 adds the total of bin k into load: one
//           writer per element.
#include <algorithm>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kLoadThreads = 1024;
constexpr int kReduceThreads = 256;
constexpr int kReduceLanes = 16;
constexpr int64_t kPairsPerChunk = 16384;
constexpr int64_t kMaxChunks = 64;
constexpr int64_t kBandWords = 16384;  // 64 KiB of LDS
constexpr int kMinGroups = 256;        // workgroups from which bands are not split further

struct LoadPlan {
    int nchunks, nbands, band_rows;
    bool u16;                // partial bins stored as uint16
    int64_t pairs_per_chunk; // a multiple of 4
    int64_t stride;          // bins of one (chunk, band) partial, a multiple of 8
    size_t bytes;
};

LoadPlan make_plan(int64_t T, int K, int E, int G) {
    LoadPlan p;
    const int64_t pairs = T * K;
    p.nchunks = (int)std::min<int64_t>(kMaxChunks, std::max<int64_t>(1, pairs / kPairsPerChunk));
    p.pairs_per_chunk = std::max<int64_t>(4, ((pairs + p.nchunks - 1) / p.nchunks + 3) & ~3);
    p.band_rows = (int)std::max<int64_t>(1, std::min<int64_t>(E, kBandWords / G));
    // more bands (fewer rows each) until the grid fills the chip
    while (p.nchunks * ((E + p.band_rows - 1) / p.band_rows) < kMinGroups && p.band_rows > 1)
        p.band_rows = (p.band_rows + 1) / 2;
    p.nbands = (E + p.band_rows - 1) / p.band_rows;
    p.u16 = p.pairs_per_chunk <= 65535;
    p.stride = ((int64_t)p.band_rows * G + 7) & ~int64_t(7);
    p.bytes = ((size_t)p.nchunks * p.nbands * p.stride * (p.u16 ? 2 : 4) + 255) & ~size_t(255);
    return p;
}

// kVec: four pairs per 16-byte load of each input (both 16-byte aligned and
// every chunk a multiple of four pairs, the last one included).
template <bool kVec, bool U16>
__global__ __launch_bounds__(kLoadThreads) void load_count_kernel(
    const int32_t* __restrict__ topk, const int32_t* __restrict__ assigned, int64_t TK, int E,
    int G, int nchunks, int band_rows, int64_t pairs_per_chunk, int64_t stride,
    void* __restrict__ part) {
    __shared__ __align__(16) uint32_t hist[kBandWords];
    const int chunk = blockIdx.x % nchunks;
    const int band = blockIdx.x / nchunks;
    const int e_lo = band * band_rows;
    const int e_hi = min(E, e_lo + band_rows);
    for (int b = threadIdx.x; b < stride; b += kLoadThreads) hist[b] = 0;
    __syncthreads();
    const int64_t p0 = (int64_t)chunk * pairs_per_chunk;
    const int64_t p1 = min(TK, p0 + pairs_per_chunk);
    auto add = [&](int e, int r) {
        if (e >= e_lo && e < e_hi && r >= 0 && r < G) atomicAdd(&hist[(e - e_lo) * G + r], 1u);
    };
    if constexpr (kVec) {
        const int4* t4 = reinterpret_cast<const int4*>(topk);
        const int4* a4 = reinterpret_cast<const int4*>(assigned);
        for (int64_t q = p0 / 4 + threadIdx.x; q < p1 / 4; q += kLoadThreads) {
            const int4 e = t4[q], r = a4[q];
            add(e.x, r.x);
            add(e.y, r.y);
            add(e.z, r.z);
            add(e.w, r.w);
        }
    } else {
        for (int64_t p = p0 + threadIdx.x; p < p1; p += kLoadThreads) add(topk[p], assigned[p]);
    }
    __syncthreads();
    // bins past the band's rows are zero (cleared above, never counted)
    const int64_t at = (int64_t)blockIdx.x * stride;
    for (int g = threadIdx.x; g < stride / 8; g += kLoadThreads) {
        const u32x4 lo = *reinterpret_cast<const u32x4*>(hist + g * 8);
        const u32x4 hi = *reinterpret_cast<const u32x4*>(hist + g * 8 + 4);
        if constexpr (U16) {
            const u32x4 packed = {lo.x | (lo.y << 16), lo.z | (lo.w << 16), hi.x | (hi.y << 16),
                                  hi.z | (hi.w << 16)};
            *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(part) + at + g * 8) = packed;
        } else {
            u32x4* out = reinterpret_cast<u32x4*>(static_cast<uint32_t*>(part) + at + g * 8);
            out[0] = lo;
            out[1] = hi;
        }
    }
}

template <bool U16>
__global__ __launch_bounds__(kReduceThreads) void load_reduce_kernel(
    const void* __restrict__ part, int E, int G, int nchunks, int band_rows, int64_t stride,
    uint32_t* __restrict__ load) {
    const int64_t groups = stride / 8;
    const int64_t gid = (int64_t)blockIdx.x * kReduceThreads + threadIdx.x;
    const int64_t item = gid / kReduceLanes;
    const int k = (int)(gid % kReduceLanes);
    const int band = (int)(item / groups);
    if (band >= (E + band_rows - 1) / band_rows) return;  // whole groups of lanes
    const int64_t w0 = (item % groups) * 8;
    const int64_t band_bins = (int64_t)(min(E, (band + 1) * band_rows) - band * band_rows) * G;
    const int64_t w = w0 + (k & 7);
    const int64_t bin = (int64_t)band * band_rows * G + w;
    const bool real = k < 8 && w < band_bins;
    const uint32_t prev = real ? load[bin] : 0u;
    uint32_t s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const int64_t base = (int64_t)band * nchunks * stride + w0;
    if constexpr (U16) {
        const uint16_t* src = static_cast<const uint16_t*>(part) + base;
#pragma unroll 4
        for (int c = k; c < nchunks; c += kReduceLanes) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(src + (int64_t)c * stride);
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                s[2 * h] += v[h] & 0xffffu;
                s[2 * h + 1] += v[h] >> 16;
            }
        }
    } else {
        const uint32_t* src = static_cast<const uint32_t*>(part) + base;
#pragma unroll 4
        for (int c = k; c < nchunks; c += kReduceLanes) {
            const u32x4* q = reinterpret_cast<const u32x4*>(src + (int64_t)c * stride);
            const u32x4 lo = q[0], hi = q[1];
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                s[h] += lo[h];
                s[4 + h] += hi[h];
            }
        }
    }
    // lanes k, k ^ 8 add; then each round halves the bins a lane holds
#pragma unroll
    for (int o = 8; o < kReduceLanes; o <<= 1)
#pragma unroll
        for (int m = 0; m < 8; ++m) s[m] += __shfl_xor(s[m], o, kReduceLanes);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const bool up = k & 4;
        const uint32_t keep = up ? s[4 + m] : s[m], give = up ? s[m] : s[4 + m];
        s[m] = keep + __shfl_xor(give, 4, kReduceLanes);
    }
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const bool up = k & 2;
        const uint32_t keep = up ? s[2 + m] : s[m], give = up ? s[m] : s[2 + m];
        s[m] = keep + __shfl_xor(give, 2, kReduceLanes);
    }
    {
        const bool up = k & 1;
        const uint32_t keep = up ? s[1] : s[0], give = up ? s[0] : s[1];
        s[0] = keep + __shfl_xor(give, 1, kReduceLanes);
    }
    if (real && s[0]) load[bin] = prev + s[0];
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
    const int64_t TK = T * K;
    const bool vec = TK % 4 == 0 && ((uintptr_t)topk & 15u) == 0 && ((uintptr_t)assigned & 15u) == 0;
    auto count = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3((unsigned)(p.nchunks * p.nbands)), dim3(kLoadThreads), 0, s,
                           topk, assigned, TK, E, G, p.nchunks, p.band_rows, p.pairs_per_chunk,
                           p.stride, ws);
    };
    if (p.u16)
        vec ? count(load_count_kernel<true, true>) : count(load_count_kernel<false, true>);
    else
        vec ? count(load_count_kernel<true, false>) : count(load_count_kernel<false, false>);
    COBALT_LAUNCH_CHECK();
    const int64_t items = (int64_t)p.nbands * (p.stride / 8) * kReduceLanes;
    const dim3 grid((unsigned)((items + kReduceThreads - 1) / kReduceThreads));
    if (p.u16)
        hipLaunchKernelGGL(load_reduce_kernel<true>, grid, dim3(kReduceThreads), 0, s, ws, E, G,
                           p.nchunks, p.band_rows, p.stride, load);
    else
        hipLaunchKernelGGL(load_reduce_kernel<false>, grid, dim3(kReduceThreads), 0, s, ws, E, G,
                           p.nchunks, p.band_rows, p.stride, load);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
