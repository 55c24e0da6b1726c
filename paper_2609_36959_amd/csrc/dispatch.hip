// Dispatch layout and pack: one packed row per (token, expert) pair, grouped
// in buckets (source rank, destination rank) in row-major order, stable in
// the pair index p = t*K + j.
//
// With source ranks non-decreasing in t, the pairs before p that share p's
// destination r and have a smaller source are exactly the column prefix
// sum_{s' < s} counts[s'][r]. The packed row of p is therefore
//     pos[p] = offsets[s][r] - colprefix[s][r] + prefix_r(p),
// where prefix_r(p) counts the pairs before p with destination r regardless
// of source: a G-way stable partition, computed here with a single-pass
// decoupled look-back scan over tiles of pairs.
//
// Kernels, in stream order:
//   init   clears send_counts and the look-back state in the workspace
//   count  send_counts[s][r] (LDS window over the block's sources, global
//          atomics to flush)
//   scan   one workgroup: send_offsets and base[s][r] = offsets - colprefix
//          (counts staged in LDS when G <= 128)
//   rank   per tile: wave multi-split ranks (ballots over the bits of r),
//          per-wave running counts in LDS, aggregates published, look-back
//          over predecessor tiles per destination, then pos
//   copy   each wave reads a 1-2 KiB slice of one token row of x once
//          into registers and stores it to the token's K packed rows
#include <algorithm>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kInitThreads = 256;
constexpr int kCountThreads = 256;
constexpr int kCountWin = 8192;  // LDS bins: (source - first source) * G + destination
constexpr int kScanThreads = 1024;
constexpr int kScanLds = 16384;  // G*G entries staged in LDS (G <= 128)
constexpr int kRankWaves = 4;
constexpr int kRankChunks = 8;
constexpr int kRankThreads = kRankWaves * 64;
constexpr int64_t kTile = (int64_t)kRankWaves * 64 * kRankChunks;  // pairs per tile
constexpr uint64_t kFlagAgg = 1ull << 62;
constexpr uint64_t kFlagInc = 2ull << 62;
constexpr uint64_t kFlagMask = 3ull << 62;
constexpr int kCopyWaves = 4;

struct Workspace {
    uint32_t* ctrl;    // [0] = next tile id
    int32_t* base;     // [G*G]
    uint64_t* status;  // [ntiles][G] look-back words: flag | count
    int64_t ntiles;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

Workspace carve(void* ws, int64_t T, int K, int G) {
    Workspace w;
    char* p = (char*)ws;
    w.ntiles = (T * K + kTile - 1) / kTile;
    w.ctrl = (uint32_t*)p;
    p += 256;
    w.base = (int32_t*)p;
    p += align256(sizeof(int32_t) * (size_t)G * G);
    w.status = (uint64_t*)p;
    return w;
}

__device__ __forceinline__ int src_of(const int32_t* src, int64_t t, int64_t tok_per_src) {
    return src ? src[t] : (int)(t / tok_per_src);
}

__global__ __launch_bounds__(kInitThreads) void init_kernel(int32_t* counts, int64_t ncounts,
                                                            uint32_t* ctrl, uint64_t* status,
                                                            int64_t nstatus) {
    const int64_t i0 = (int64_t)blockIdx.x * kInitThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kInitThreads;
    for (int64_t i = i0; i < ncounts; i += stride) counts[i] = 0;
    for (int64_t i = i0; i < nstatus; i += stride) status[i] = 0;
    if (i0 < 64) ctrl[i0] = 0;
}

__global__ __launch_bounds__(kCountThreads) void count_kernel(
    const int32_t* __restrict__ assigned, const int32_t* __restrict__ src, int64_t T, int K, int G,
    int64_t tok_per_src, int64_t tok_per_blk, int32_t* __restrict__ counts) {
    __shared__ uint32_t h[kCountWin];
    const int64_t t0 = (int64_t)blockIdx.x * tok_per_blk;
    const int64_t t1 = min(T, t0 + tok_per_blk);
    if (t0 >= t1) return;
    const int s_lo = src_of(src, t0, tok_per_src);
    const int s_hi = src_of(src, t1 - 1, tok_per_src);
    const bool win = s_lo >= 0 && s_hi < G && s_hi >= s_lo && (s_hi - s_lo + 1) * G <= kCountWin;
    const int nwin = win ? (s_hi - s_lo + 1) * G : 0;
    for (int i = threadIdx.x; i < nwin; i += kCountThreads) h[i] = 0;
    __syncthreads();
    const int64_t p1 = t1 * K;
    for (int64_t p = t0 * K + threadIdx.x; p < p1; p += kCountThreads) {
        const int r = assigned[p];
        const int s = src_of(src, p / K, tok_per_src);
        if (r < 0 || r >= G || s < 0 || s >= G) continue;
        if (win && s >= s_lo && s <= s_hi)
            atomicAdd(&h[(s - s_lo) * G + r], 1u);
        else
            atomicAdd(&counts[(int64_t)s * G + r], 1);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nwin; i += kCountThreads) {
        const uint32_t v = h[i];
        if (v) atomicAdd(&counts[(int64_t)s_lo * G + i], (int32_t)v);
    }
}

// Exclusive scan of one value per thread across the workgroup.
__device__ int64_t block_exclusive_scan(int64_t v, int64_t* total) {
    __shared__ int64_t wsum[kScanThreads / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    if (wave == 0) {
        int64_t w = lane < kScanThreads / 64 ? wsum[lane] : 0;
#pragma unroll
        for (int o = 1; o < kScanThreads / 64; o <<= 1) {
            const int64_t y = __shfl_up(w, o, 64);
            if (lane >= o) w += y;
        }
        if (lane < kScanThreads / 64) wsum[lane] = w;  // inclusive over waves
    }
    __syncthreads();
    const int64_t before = (wave > 0 ? wsum[wave - 1] : 0) + x - v;
    *total = wsum[kScanThreads / 64 - 1];
    return before;
}

// With G*G <= kScanLds the counts and offsets are staged in LDS, so the
// sequential column pass reads LDS instead of global memory.
template <bool kLds>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(const int32_t* __restrict__ counts,
                                                            int G, int64_t* __restrict__ offsets,
                                                            int32_t* __restrict__ base) {
    __shared__ int32_t c_lds[kLds ? kScanLds : 1];
    __shared__ int32_t o_lds[kLds ? kScanLds : 1];
    const int64_t n = (int64_t)G * G;
    if (kLds) {
        for (int64_t b = threadIdx.x; b < n; b += kScanThreads) c_lds[b] = counts[b];
        __syncthreads();
    }
    auto cnt = [&](int64_t b) -> int64_t { return kLds ? c_lds[b] : counts[b]; };
    const int64_t seg = (n + kScanThreads - 1) / kScanThreads;
    const int64_t lo = min(n, (int64_t)threadIdx.x * seg), hi = min(n, lo + seg);
    int64_t local = 0;
    for (int64_t b = lo; b < hi; ++b) local += cnt(b);
    int64_t total = 0;
    int64_t run = block_exclusive_scan(local, &total);
    for (int64_t b = lo; b < hi; ++b) {
        offsets[b] = run;
        if (kLds) o_lds[b] = (int32_t)run;
        run += cnt(b);
    }
    if (threadIdx.x == 0) offsets[n] = total;
    __syncthreads();
    for (int r = threadIdx.x; r < G; r += kScanThreads) {
        int64_t col = 0;
        for (int s = 0; s < G; ++s) {
            const int64_t b = (int64_t)s * G + r;
            base[b] = (int32_t)((kLds ? (int64_t)o_lds[b] : offsets[b]) - col);
            col += cnt(b);
        }
    }
}

__device__ __forceinline__ uint64_t ld_status(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_status(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kRankThreads) void rank_kernel(
    const int32_t* __restrict__ assigned, const int32_t* __restrict__ src, int K, int G,
    int64_t tok_per_src, int64_t TK, int64_t ntiles, uint32_t* __restrict__ ctrl,
    const int32_t* __restrict__ base, uint64_t* __restrict__ status, int32_t* __restrict__ pos) {
    __shared__ uint32_t wcnt[kRankWaves][kMaxG];  // running counts, then wave bases
    __shared__ uint32_t tile_agg[kMaxG];
    __shared__ uint32_t tile_excl[kMaxG];
    __shared__ int tile_sh;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

    // Tiles are numbered in the order workgroups start, so a tile only ever
    // waits for tiles whose workgroups are already running.
    if (threadIdx.x == 0) tile_sh = (int)atomicAdd(ctrl, 1u);
    for (int i = threadIdx.x; i < kRankWaves * G; i += kRankThreads) wcnt[i / G][i % G] = 0;
    __syncthreads();
    const int64_t tile = tile_sh;
    if (tile >= ntiles) return;

    const uint64_t lt_mask = (1ull << lane) - 1ull;
    int rank_bits = 0;
    while ((1 << rank_bits) < G) ++rank_bits;
    const int64_t p_wave = tile * kTile + (int64_t)wave * 64 * kRankChunks;
    int lr[kRankChunks], rr[kRankChunks], ss[kRankChunks];
#pragma unroll
    for (int c = 0; c < kRankChunks; ++c) {
        const int64_t p = p_wave + c * 64 + lane;
        int r = -1, s = -1;
        if (p < TK) {
            r = assigned[p];
            s = src_of(src, p / K, tok_per_src);
        }
        const bool valid = r >= 0 && r < G && s >= 0 && s < G;
        // lanes holding the same destination, by agreement on every bit
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < rank_bits; ++b) {
            const bool bit = valid && ((r >> b) & 1);
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        int prior = 0;
        if (valid) prior = (int)wcnt[wave][r];
        if (valid && (peers & lt_mask) == 0) wcnt[wave][r] = prior + __popcll(peers);
        lr[c] = prior + __popcll(peers & lt_mask);
        rr[c] = valid ? r : -1;
        ss[c] = s;
    }
    __syncthreads();
    for (int r = threadIdx.x; r < G; r += kRankThreads) {
        uint32_t run = 0;
#pragma unroll
        for (int w = 0; w < kRankWaves; ++w) {
            const uint32_t v = wcnt[w][r];
            wcnt[w][r] = run;
            run += v;
        }
        tile_agg[r] = run;
    }
    // Publish this tile's aggregates, then look back for the exclusive
    // prefix of each destination.
    for (int r = threadIdx.x; r < G; r += kRankThreads) {
        const uint32_t agg = tile_agg[r];
        uint64_t* mine = status + tile * G + r;
        uint32_t excl = 0;
        if (tile == 0) {
            st_status(mine, kFlagInc | agg);
        } else {
            st_status(mine, kFlagAgg | agg);
            int64_t q = tile - 1;
            for (;;) {
                const uint64_t v = ld_status(status + q * G + r);
                const uint64_t f = v & kFlagMask;
                if (f == 0) {
                    __builtin_amdgcn_s_sleep(1);
                    continue;
                }
                excl += (uint32_t)v;
                if (f == kFlagInc) break;
                --q;
            }
            st_status(mine, kFlagInc | (uint64_t)(excl + agg));
        }
        tile_excl[r] = excl;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < kRankChunks; ++c) {
        const int64_t p = p_wave + c * 64 + lane;
        if (p >= TK) continue;
        const int r = rr[c];
        int out = -1;
        if (r >= 0)
            out = base[(int64_t)ss[c] * G + r] + (int)tile_excl[r] + (int)wcnt[wave][r] + lr[c];
        pos[p] = out;
    }
}

// Row copy. Each wave takes one (token, column group): it loads CG 16-byte
// chunks per lane of x[t] (64*CG chunks, a contiguous 1-2 KiB slice of the
// row) once, then stores them to the K packed rows of the token. Small
// per-wave state keeps many waves in flight; plain stores sustain a higher
// write rate than non-temporal ones on this access pattern.
// KC = compile-time K (0: any K up to 16); with KC the scalar loads of the
// token's pos entries are issued together.
template <int CG, int KC>
__global__ __launch_bounds__(kCopyWaves * 64) void copy_kernel(
    const u32x4* __restrict__ x, const int32_t* __restrict__ pos, int64_t T, int Kr, int64_t nch,
    int64_t TK, u32x4* __restrict__ packed) {
    constexpr int KM = KC ? KC : kMaxK;
    const int K = KC ? KC : Kr;
    const int64_t groups = (nch + 64 * CG - 1) / (64 * CG);
    // wave-uniform item index, so pos comes in through scalar loads
    const int64_t item = (int64_t)blockIdx.x * kCopyWaves +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (item >= T * groups) return;
    const int64_t t = item / groups;
    const int64_t c0 = (item - t * groups) * 64 * CG + (threadIdx.x & 63);
    int p[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) p[j] = j < K ? pos[t * K + j] : -1;
    const u32x4* row = x + t * nch;
    u32x4 v[CG];
#pragma unroll
    for (int i = 0; i < CG; ++i)
        if (c0 + 64 * i < nch) v[i] = __builtin_nontemporal_load(row + c0 + 64 * i);
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        if (p[j] < 0 || p[j] >= TK) continue;
        u32x4* dst = packed + (int64_t)p[j] * nch;
#pragma unroll
        for (int i = 0; i < CG; ++i)
            if (c0 + 64 * i < nch) dst[c0 + 64 * i] = v[i];
    }
}

}  // namespace

size_t dispatch_workspace_bytes(int64_t T, int K, int G) {
    const int64_t ntiles = (T * K + kTile - 1) / kTile;
    return 256 + align256(sizeof(int32_t) * (size_t)G * G) +
           align256(sizeof(uint64_t) * (size_t)std::max<int64_t>(ntiles, 1) * G);
}

cobalt_status launch_dispatch(const int32_t* assigned, const int32_t* src, int64_t T, int K,
                              int G, const void* x, int64_t d, int32_t* counts, int64_t* offsets,
                              int32_t* pos, void* packed, void* ws, hipStream_t s) {
    DeviceInfo di;
    if (cobalt_status st = device_info(&di)) return st;
    const Workspace w = carve(ws, T, K, G);
    const int64_t TK = T * K;
    const int64_t tok_per_src = src ? 1 : std::max<int64_t>(1, T / G);
    const int64_t nstatus = w.ntiles * G;

    const int64_t init_work = std::max<int64_t>((int64_t)G * G, nstatus);
    const unsigned init_blocks =
        (unsigned)std::min<int64_t>(std::max<int64_t>(1, (init_work + kInitThreads - 1) / kInitThreads),
                                    4 * di.cus);
    hipLaunchKernelGGL(init_kernel, dim3(init_blocks), dim3(kInitThreads), 0, s, counts,
                       (int64_t)G * G, w.ctrl, w.status, nstatus);
    COBALT_LAUNCH_CHECK();
    if (T > 0) {
        const int64_t tok_per_blk =
            std::max<int64_t>(64, (T + 2 * di.cus - 1) / (2 * di.cus));
        const unsigned cblocks = (unsigned)((T + tok_per_blk - 1) / tok_per_blk);
        hipLaunchKernelGGL(count_kernel, dim3(cblocks), dim3(kCountThreads), 0, s, assigned, src,
                           T, K, G, tok_per_src, tok_per_blk, counts);
        COBALT_LAUNCH_CHECK();
    }
    if ((int64_t)G * G <= kScanLds)
        hipLaunchKernelGGL(scan_kernel<true>, dim3(1), dim3(kScanThreads), 0, s, counts, G,
                           offsets, w.base);
    else
        hipLaunchKernelGGL(scan_kernel<false>, dim3(1), dim3(kScanThreads), 0, s, counts, G,
                           offsets, w.base);
    COBALT_LAUNCH_CHECK();
    if (T == 0) return COBALT_OK;
    hipLaunchKernelGGL(rank_kernel, dim3((unsigned)w.ntiles), dim3(kRankThreads), 0, s, assigned,
                       src, K, G, tok_per_src, TK, w.ntiles, w.ctrl, w.base, w.status, pos);
    COBALT_LAUNCH_CHECK();
    if (!x) return COBALT_OK;

    const int64_t nch = d / 8;
    const u32x4* xv = (const u32x4*)x;
    u32x4* pv = (u32x4*)packed;
    auto launch = [&](auto kernel, int64_t cg) {
        const int64_t items = T * ((nch + 64 * cg - 1) / (64 * cg));
        hipLaunchKernelGGL(kernel, dim3((unsigned)((items + kCopyWaves - 1) / kCopyWaves)),
                           dim3(kCopyWaves * 64), 0, s, xv, pos, T, K, nch, TK, pv);
    };
    if (nch >= 128)
        K == 8 ? launch(copy_kernel<2, 8>, 2) : launch(copy_kernel<2, 0>, 2);
    else
        K == 8 ? launch(copy_kernel<1, 8>, 1) : launch(copy_kernel<1, 0>, 1);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
