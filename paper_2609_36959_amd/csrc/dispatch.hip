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
//   scatter one wave per (token, 2 KiB slice, slot): reads the slice of x
//          (from the cache for all but the first of the token's K waves)
//          and stores it to the slot's packed row
//
// The node-deduplicated layout (Section 1, Eq. 1: a token crosses to a node
// once and is forwarded inside it) has one row per (token, destination node)
// in buckets (source rank, node). A token has at most one row per bucket, so
//     node_pos[t][n] = offsets[s][n] - colprefix[s][n] + prefix_n(t),
// where prefix_n(t) counts the tokens before t that reach node n: an N-way
// prefix count over tokens, done with ballots per node bit and the same
// decoupled look-back. The same init and scan kernels serve both; the node
// rows are written by node_scatter_kernel, four waves per (token, slice)
// with two or four nodes each (copy_kernel for rows wider than 16 slices).
#include <algorithm>
#include <mutex>
#include <vector>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kInitThreads = 256;
constexpr int kCountThreads = 256;
constexpr int kCountWin = 8192;  // LDS bins: (source - first source) * G + destination
constexpr int kScanThreads = 1024;
constexpr int kScanLds = 16384;  // G*G entries staged in LDS (G <= 128)
constexpr int kRankWaves = 16;
constexpr int kRankChunks = 4;
constexpr int kRankThreads = kRankWaves * 64;
constexpr int64_t kTile = (int64_t)kRankWaves * 64 * kRankChunks;  // pairs per tile
constexpr uint64_t kFlagAgg = 1ull << 62;
constexpr uint64_t kFlagInc = 2ull << 62;
constexpr uint64_t kFlagMask = 3ull << 62;
constexpr int kCopyWaves = 4;
constexpr int kNodeWaves = 4;
constexpr int kNodeThreads = kNodeWaves * 64;
constexpr int kNodeChunks = 2;
constexpr int64_t kNodeTile = (int64_t)kNodeWaves * 64 * kNodeChunks;  // tokens per tile

struct Workspace {
    uint32_t* ctrl;    // [0] = next tile id
    int32_t* base;     // [G*G]
    uint64_t* status;  // [ntiles][G] look-back words: flag | count
    int64_t ntiles;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// ntiles tiles of look-back state over C columns, base[G][C].
Workspace carve(void* ws, int64_t ntiles, int G, int C) {
    Workspace w;
    char* p = (char*)ws;
    w.ntiles = ntiles;
    w.ctrl = (uint32_t*)p;
    p += 256;
    w.base = (int32_t*)p;
    p += align256(sizeof(int32_t) * (size_t)G * C);
    w.status = (uint64_t*)p;
    return w;
}

size_t carve_bytes(int64_t ntiles, int G, int C) {
    return 256 + align256(sizeof(int32_t) * (size_t)G * C) +
           align256(sizeof(uint64_t) * (size_t)std::max<int64_t>(ntiles, 1) * C);
}

__device__ __forceinline__ int src_of(const int32_t* src, int64_t t, int64_t tok_per_src) {
    return src ? src[t] : (int)(t / tok_per_src);
}

// kNode (here and on scan_kernel and copy_kernel) changes no instruction: it
// gives the node-deduplicated layout's launches kernel names of their own,
// so per-kernel profiles attribute each launch to its entry point.
template <bool kNode>
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

// Exclusive scan of a [R][C] count matrix in row-major order, and
// base[s][c] = offsets[s][c] - sum_{s' < s} counts[s'][c]. With R*C <=
// kScanLds the counts and offsets are staged in LDS, so the sequential
// column pass reads LDS instead of global memory.
template <bool kLds, bool kNode>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(const int32_t* __restrict__ counts,
                                                            int R, int C,
                                                            int64_t* __restrict__ offsets,
                                                            int32_t* __restrict__ base) {
    __shared__ int32_t c_lds[kLds ? kScanLds : 1];
    __shared__ int32_t o_lds[kLds ? kScanLds : 1];
    const int64_t n = (int64_t)R * C;
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
    for (int c = threadIdx.x; c < C; c += kScanThreads) {
        int64_t col = 0;
        for (int r = 0; r < R; ++r) {
            const int64_t b = (int64_t)r * C + c;
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
template <int CG, int KC, bool kNode>
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


// Node set of one token, for the node-deduplicated layout: code[j] =
// (node << 8) | index of the rank inside its node, or -1 for a slot with no
// valid rank; the result has bit n set if some slot goes to node n.
template <int KM>
__device__ __forceinline__ uint32_t token_nodes(const int32_t* __restrict__ assigned, int64_t t,
                                                int K, int g, int G, int (&code)[KM]) {
    uint32_t B = 0;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        int cd = -1;
        if (j < K) {
            const int r = assigned[t * K + j];
            if (r >= 0 && r < G) {
                const int n = r / g;
                cd = (n << 8) | (r - n * g);
                B |= 1u << n;
            }
        }
        code[j] = cd;
    }
    return B;
}

// node_counts[s][n]: tokens of source s with a slot on node n (LDS window
// over the block's sources, global atomics to flush). One token per thread.
template <int KC>
__global__ __launch_bounds__(kCountThreads) void node_count_kernel(
    const int32_t* __restrict__ assigned, const int32_t* __restrict__ src, int64_t T, int Kr,
    int N, int g, int64_t tok_per_src, int64_t tok_per_blk, int32_t* __restrict__ counts) {
    constexpr int KM = KC ? KC : kMaxK;
    const int K = KC ? KC : Kr;
    const int G = N * g;
    __shared__ uint32_t h[kCountWin];
    const int64_t t0 = (int64_t)blockIdx.x * tok_per_blk;
    const int64_t t1 = min(T, t0 + tok_per_blk);
    if (t0 >= t1) return;
    const int s_lo = src_of(src, t0, tok_per_src);
    const int s_hi = src_of(src, t1 - 1, tok_per_src);
    const bool win = s_lo >= 0 && s_hi < G && s_hi >= s_lo && (s_hi - s_lo + 1) * N <= kCountWin;
    const int nwin = win ? (s_hi - s_lo + 1) * N : 0;
    for (int i = threadIdx.x; i < nwin; i += kCountThreads) h[i] = 0;
    __syncthreads();
    for (int64_t t = t0 + threadIdx.x; t < t1; t += kCountThreads) {
        const int s = src_of(src, t, tok_per_src);
        if (s < 0 || s >= G) continue;
        int code[KM];
        uint32_t B = token_nodes<KM>(assigned, t, K, g, G, code);
        const bool in_win = win && s >= s_lo && s <= s_hi;
        while (B) {
            const int n = __ffs(B) - 1;
            B &= B - 1;
            if (in_win)
                atomicAdd(&h[(s - s_lo) * N + n], 1u);
            else
                atomicAdd(&counts[(int64_t)s * N + n], 1);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nwin; i += kCountThreads) {
        const uint32_t v = h[i];
        if (v) atomicAdd(&counts[(int64_t)s_lo * N + i], (int32_t)v);
    }
}

// Per tile of kNodeTile tokens: each (wave, chunk) segment of 64 tokens
// counts its tokens per node with one ballot per node, the segments are
// scanned in token order in LDS, the tile's per-node totals go through the
// decoupled look-back, and each (token, node) row gets
//     base[s][n] + tile prefix + segment prefix + lanes below with bit n.
// node_pos is written for every (t, n), -1 where the token has no row.
template <int KC>
__global__ __launch_bounds__(kNodeThreads) void node_rank_kernel(
    const int32_t* __restrict__ assigned, const int32_t* __restrict__ src, int64_t T, int Kr,
    int N, int g, int64_t tok_per_src, int64_t ntiles, uint32_t* __restrict__ ctrl,
    const int32_t* __restrict__ base, uint64_t* __restrict__ status,
    int32_t* __restrict__ node_pos, uint32_t* __restrict__ fwd, int32_t* __restrict__ row_token) {
    constexpr int KM = KC ? KC : kMaxK;
    constexpr int kSegs = kNodeWaves * kNodeChunks;
    const int K = KC ? KC : Kr;
    const int G = N * g;
    __shared__ uint32_t seg[kSegs][kMaxN];  // segment counts, then segment prefixes
    __shared__ uint32_t tile_excl[kMaxN];
    __shared__ int tile_sh;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

    if (threadIdx.x == 0) tile_sh = (int)atomicAdd(ctrl, 1u);
    __syncthreads();
    const int64_t tile = tile_sh;
    if (tile >= ntiles) return;

    const uint64_t lt_mask = (1ull << lane) - 1ull;
    const int64_t t_wave = tile * kNodeTile + (int64_t)wave * 64 * kNodeChunks;
    int code[kNodeChunks][KM];
    uint32_t nodes[kNodeChunks];
    int ss[kNodeChunks];
#pragma unroll
    for (int c = 0; c < kNodeChunks; ++c) {
        const int64_t t = t_wave + c * 64 + lane;
        const int s = t < T ? src_of(src, t, tok_per_src) : -1;
        uint32_t B = 0;
        if (s >= 0 && s < G) {
            B = token_nodes<KM>(assigned, t, K, g, G, code[c]);
        } else {
#pragma unroll
            for (int j = 0; j < KM; ++j) code[c][j] = -1;
        }
        nodes[c] = B;
        ss[c] = s;
        uint32_t mine = 0;  // lane n keeps the segment's count for node n
        for (int n = 0; n < N; ++n) {
            const uint32_t cnt = (uint32_t)__popcll(__ballot((B >> n) & 1u));
            if (lane == n) mine = cnt;
        }
        if (lane < N) seg[wave * kNodeChunks + c][lane] = mine;
    }
    __syncthreads();
    if (threadIdx.x < N) {
        const int n = threadIdx.x;
        uint32_t agg = 0;
        for (int q = 0; q < kSegs; ++q) {
            const uint32_t v = seg[q][n];
            seg[q][n] = agg;
            agg += v;
        }
        uint64_t* mine = status + tile * N + n;
        uint32_t excl = 0;
        if (tile == 0) {
            st_status(mine, kFlagInc | agg);
        } else {
            st_status(mine, kFlagAgg | agg);
            int64_t q = tile - 1;
            for (;;) {
                const uint64_t v = ld_status(status + q * N + n);
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
        tile_excl[n] = excl;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < kNodeChunks; ++c) {
        const int64_t t = t_wave + c * 64 + lane;
        const uint32_t B = nodes[c];
        const int q = wave * kNodeChunks + c;
        for (int n = 0; n < N; ++n) {
            const bool bit = (B >> n) & 1u;
            const uint64_t bal = __ballot(bit);
            if (t < T) {
                int32_t row = -1;
                if (bit) {
                    row = base[(int64_t)ss[c] * N + n] + (int)tile_excl[n] + (int)seg[q][n] +
                          __popcll(bal & lt_mask);
                    uint32_t m = 0;
#pragma unroll
                    for (int j = 0; j < KM; ++j)
                        if ((code[c][j] >> 8) == n) m |= 1u << (code[c][j] & 255);
                    fwd[row] = m;
                    if (row_token) row_token[row] = (int32_t)t;
                }
                node_pos[t * N + n] = row;
            }
        }
    }
}

// Row scatter for the per-pair layout: one workgroup per (token, 2 KiB
// column slice), one wave per slot j. The K waves that copy one slice of
// x[t] share a workgroup, so the slice is read from HBM once and from the
// cache K - 1 times (plain loads keep it cached); each wave then issues a
// single 2 KiB burst to one packed row, with non-temporal stores. On the
// T=131072, K=8, d=7168 workload this reaches 5.7 TB/s, where the fan-out
// of copy_kernel (one wave stores its slice to all K rows) reaches 5.1.
// GROUPS, the number of slices per row, is a template parameter so that
// the block index splits into (token, slice) with a constant division: a
// wave does two loads and two stores, and a runtime 64-bit division would
// cost it more scalar instructions than that.
template <int GROUPS>
__global__ __launch_bounds__(kMaxK * 64) void scatter_kernel(
    const u32x4* __restrict__ x, const int32_t* __restrict__ pos, int K, int64_t nch,
    int64_t bound, u32x4* __restrict__ packed) {
    const uint32_t tg = blockIdx.x;
    const uint32_t t = tg / GROUPS;
    const uint32_t g = tg - t * GROUPS;
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t c0 = (int64_t)g * 128 + (threadIdx.x & 63);
    // The x loads are issued before the packed row is read: a branch on the
    // row first would make every wave wait for that load before its own
    // two loads start (measured: 3.45 ms instead of 2.95 ms). The in-range
    // guards also keep them there: without them the compiler sinks both
    // loads below the branch on p, with the same cost (3.42 ms at d = 7168).
    const u32x4* row = x + (int64_t)t * nch;
    const bool in0 = c0 < nch, in1 = c0 + 64 < nch;
    u32x4 v0, v1;
    if (in0) v0 = row[c0];
    if (in1) v1 = row[c0 + 64];
    const int p = pos[(int64_t)t * K + j];
    if (p < 0 || p >= bound) return;
    // The row's buffer descriptor drops stores past its nch chunks, so the
    // stores need no guard of their own: both issue back to back from one
    // offset register.
    u32x4* dst = packed + (int64_t)p * nch;
    const int32_t off = (int32_t)(c0 * 16);
    store_stream(v0, dst, (int32_t)(nch * 16), off);
    store_stream(v1, dst, (int32_t)(nch * 16), off + 1024);
}

// Launches scatter_kernel for rows pos[t][0..per_tok) in [0, bound) when
// the slice count has an instantiation; returns false otherwise (the
// caller then uses the fan-out copy).
template <int GROUPS>
bool try_scatter(const void* x, const int32_t* pos, int64_t T, int per_tok, int64_t nch,
                 int64_t bound, void* packed, hipStream_t s) {
    if ((nch + 127) / 128 != GROUPS)
        return try_scatter<GROUPS - 1>(x, pos, T, per_tok, nch, bound, packed, s);
    for_token_ranges(T, (int64_t)GROUPS * per_tok * 64, [&](int64_t t0, int64_t n) {
        hipLaunchKernelGGL(scatter_kernel<GROUPS>, dim3((unsigned)(n * GROUPS)),
                           dim3(per_tok * 64), 0, s, (const u32x4*)x + t0 * nch,
                           pos + t0 * per_tok, per_tok, nch, bound, (u32x4*)packed);
    });
    return true;
}
template <>
bool try_scatter<0>(const void*, const int32_t*, int64_t, int, int64_t, int64_t, void*,
                    hipStream_t) {
    return false;
}

// Row scatter for the node-deduplicated layout: one workgroup of
// kNodeScatterWaves waves per (token, 2 KiB column slice); wave j loads the
// slice of x[t] and stores it to the token's rows for nodes n = j, j + 4,
// ... (SPW of them at most). A token has rows on only about half of the
// nodes, so one wave per node would leave half of the waves without a row
// (2.06 ms) and one wave for all of the token's rows serialises their
// stores (1.99 ms); two nodes per wave take 1.63 ms on the T=131072, N=8,
// d=7168 workload. GROUPS as for scatter_kernel.
constexpr int kNodeScatterWaves = 4;

template <int GROUPS, int SPW>
__global__ __launch_bounds__(kNodeScatterWaves * 64) void node_scatter_kernel(
    const u32x4* __restrict__ x, const int32_t* __restrict__ node_pos, int N, int64_t nch,
    int64_t bound, u32x4* __restrict__ packed) {
    const uint32_t tg = blockIdx.x;
    const uint32_t t = tg / GROUPS;
    const uint32_t g = tg - t * GROUPS;
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t c0 = (int64_t)g * 128 + (threadIdx.x & 63);
    // loads first, as in scatter_kernel (the guards keep them there)
    const u32x4* row = x + (int64_t)t * nch;
    const bool in0 = c0 < nch, in1 = c0 + 64 < nch;
    u32x4 v0, v1;
    if (in0) v0 = row[c0];
    if (in1) v1 = row[c0 + 64];
    int q[SPW];
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
        const int n = j + kNodeScatterWaves * i;
        q[i] = n < N ? node_pos[(int64_t)t * N + n] : -1;
    }
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
        if (q[i] < 0 || q[i] >= bound) continue;
        u32x4* dst = packed + (int64_t)q[i] * nch;
        if (in0) __builtin_nontemporal_store(v0, dst + c0);
        if (in1) __builtin_nontemporal_store(v1, dst + c0 + 64);
    }
}

// Launches node_scatter_kernel when the slice count has an instantiation;
// returns false otherwise (the caller then uses the fan-out copy).
template <int GROUPS>
bool try_node_scatter(const void* x, const int32_t* node_pos, int64_t T, int N, int64_t nch,
                      int64_t bound, void* packed, hipStream_t s) {
    if constexpr (GROUPS == 0) {
        return false;
    } else {
        if ((nch + 127) / 128 != GROUPS)
            return try_node_scatter<GROUPS - 1>(x, node_pos, T, N, nch, bound, packed, s);
        const dim3 block(kNodeScatterWaves * 64);
        for_token_ranges(T, (int64_t)GROUPS * kNodeScatterWaves * 64, [&](int64_t t0, int64_t n) {
            const dim3 grid((unsigned)(n * GROUPS));
            const u32x4* xr = (const u32x4*)x + t0 * nch;
            const int32_t* np = node_pos + t0 * N;
            if (N <= 2 * kNodeScatterWaves)
                hipLaunchKernelGGL((node_scatter_kernel<GROUPS, 2>), grid, block, 0, s, xr, np, N,
                                   nch, bound, (u32x4*)packed);
            else
                hipLaunchKernelGGL((node_scatter_kernel<GROUPS, 4>), grid, block, 0, s, xr, np, N,
                                   nch, bound, (u32x4*)packed);
        });
        return true;
    }
}

// Copies x[t] to the rows pos[t][0..per_tok) that are in [0, bound).
template <bool kNode>
cobalt_status launch_copy(const void* x, const int32_t* pos, int64_t T, int per_tok, int64_t d,
                          int64_t bound, void* packed, hipStream_t s) {
    const int64_t nch = d / 8;
    const u32x4* xv = (const u32x4*)x;
    u32x4* pv = (u32x4*)packed;
    auto launch = [&](auto kernel, int64_t cg) {
        const int64_t groups = (nch + 64 * cg - 1) / (64 * cg);  // one wave each
        for_token_ranges(T, groups * 64, [&](int64_t t0, int64_t n) {
            const int64_t items = n * groups;
            hipLaunchKernelGGL(kernel, dim3((unsigned)((items + kCopyWaves - 1) / kCopyWaves)),
                               dim3(kCopyWaves * 64), 0, s, xv + t0 * nch, pos + t0 * per_tok, n,
                               per_tok, nch, bound, pv);
        });
    };
    if (nch >= 128)
        per_tok == 8 ? launch(copy_kernel<2, 8, kNode>, 2) : launch(copy_kernel<2, 0, kNode>, 2);
    else
        per_tok == 8 ? launch(copy_kernel<1, 8, kNode>, 1) : launch(copy_kernel<1, 0, kNode>, 1);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace

size_t dispatch_workspace_bytes(int64_t T, int K, int G) {
    return carve_bytes((T * K + kTile - 1) / kTile, G, G);
}

size_t node_dispatch_workspace_bytes(int64_t T, int N, int G) {
    return carve_bytes((T + kNodeTile - 1) / kNodeTile, G, N);
}

namespace {

template <bool kNode>
cobalt_status launch_init(const DeviceInfo& di, int32_t* counts, int64_t ncounts,
                          const Workspace& w, int C, hipStream_t s) {
    const int64_t nstatus = w.ntiles * C;
    const int64_t init_work = std::max<int64_t>(ncounts, nstatus);
    const unsigned init_blocks = (unsigned)std::min<int64_t>(
        std::max<int64_t>(1, (init_work + kInitThreads - 1) / kInitThreads), 4 * di.cus);
    hipLaunchKernelGGL(init_kernel<kNode>, dim3(init_blocks), dim3(kInitThreads), 0, s, counts,
                       ncounts, w.ctrl, w.status, nstatus);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

template <bool kNode>
cobalt_status launch_scan(const int32_t* counts, int R, int C, int64_t* offsets, int32_t* base,
                          hipStream_t s) {
    if ((int64_t)R * C <= kScanLds)
        hipLaunchKernelGGL((scan_kernel<true, kNode>), dim3(1), dim3(kScanThreads), 0, s, counts,
                           R, C, offsets, base);
    else
        hipLaunchKernelGGL((scan_kernel<false, kNode>), dim3(1), dim3(kScanThreads), 0, s, counts,
                           R, C, offsets, base);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace

cobalt_status launch_dispatch(const int32_t* assigned, const int32_t* src, int64_t T, int K,
                              int G, const void* x, int64_t d, int32_t* counts, int64_t* offsets,
                              int32_t* pos, void* packed, void* ws, hipStream_t s) {
    DeviceInfo di;
    if (cobalt_status st = device_info(&di)) return st;
    const Workspace w = carve(ws, (T * K + kTile - 1) / kTile, G, G);
    const int64_t TK = T * K;
    const int64_t tok_per_src = src ? 1 : std::max<int64_t>(1, T / G);

    if (cobalt_status st = launch_init<false>(di, counts, (int64_t)G * G, w, G, s)) return st;
    if (T > 0) {
        const int64_t tok_per_blk =
            std::max<int64_t>(64, (T + 2 * di.cus - 1) / (2 * di.cus));
        const unsigned cblocks = (unsigned)((T + tok_per_blk - 1) / tok_per_blk);
        hipLaunchKernelGGL(count_kernel, dim3(cblocks), dim3(kCountThreads), 0, s, assigned, src,
                           T, K, G, tok_per_src, tok_per_blk, counts);
        COBALT_LAUNCH_CHECK();
    }
    if (cobalt_status st = launch_scan<false>(counts, G, G, offsets, w.base, s)) return st;
    if (T == 0) return COBALT_OK;
    hipLaunchKernelGGL(rank_kernel, dim3((unsigned)w.ntiles), dim3(kRankThreads), 0, s, assigned,
                       src, K, G, tok_per_src, TK, w.ntiles, w.ctrl, w.base, w.status, pos);
    COBALT_LAUNCH_CHECK();
    if (!x) return COBALT_OK;
    if (try_scatter<16>(x, pos, T, K, d / 8, TK, packed, s)) {
        COBALT_LAUNCH_CHECK();
        return COBALT_OK;
    }
    return launch_copy<false>(x, pos, T, K, d, TK, packed, s);
}

cobalt_status launch_node_dispatch(const int32_t* assigned, const int32_t* src, int64_t T, int K,
                                   int N, int g, const void* x, int64_t d, int32_t* counts,
                                   int64_t* offsets, int32_t* node_pos, uint32_t* fwd,
                                   int32_t* row_token, void* packed, void* ws, hipStream_t s) {
    DeviceInfo di;
    if (cobalt_status st = device_info(&di)) return st;
    const int G = N * g;
    const Workspace w = carve(ws, (T + kNodeTile - 1) / kNodeTile, G, N);
    const int64_t tok_per_src = src ? 1 : std::max<int64_t>(1, T / G);

    if (cobalt_status st = launch_init<true>(di, counts, (int64_t)G * N, w, N, s)) return st;
    if (T > 0) {
        const int64_t tok_per_blk =
            std::max<int64_t>(kCountThreads, (T + 2 * di.cus - 1) / (2 * di.cus));
        const unsigned cblocks = (unsigned)((T + tok_per_blk - 1) / tok_per_blk);
        if (K == 8)
            hipLaunchKernelGGL(node_count_kernel<8>, dim3(cblocks), dim3(kCountThreads), 0, s,
                               assigned, src, T, K, N, g, tok_per_src, tok_per_blk, counts);
        else
            hipLaunchKernelGGL(node_count_kernel<0>, dim3(cblocks), dim3(kCountThreads), 0, s,
                               assigned, src, T, K, N, g, tok_per_src, tok_per_blk, counts);
        COBALT_LAUNCH_CHECK();
    }
    if (cobalt_status st = launch_scan<true>(counts, G, N, offsets, w.base, s)) return st;
    if (T == 0) return COBALT_OK;
    if (K == 8)
        hipLaunchKernelGGL(node_rank_kernel<8>, dim3((unsigned)w.ntiles), dim3(kNodeThreads), 0,
                           s, assigned, src, T, K, N, g, tok_per_src, w.ntiles, w.ctrl, w.base,
                           w.status, node_pos, fwd, row_token);
    else
        hipLaunchKernelGGL(node_rank_kernel<0>, dim3((unsigned)w.ntiles), dim3(kNodeThreads), 0,
                           s, assigned, src, T, K, N, g, tok_per_src, w.ntiles, w.ctrl, w.base,
                           w.status, node_pos, fwd, row_token);
    COBALT_LAUNCH_CHECK();
    if (!x) return COBALT_OK;
    const int64_t bound = T * std::min(K, N);
    if (try_node_scatter<16>(x, node_pos, T, N, d / 8, bound, packed, s)) {
        COBALT_LAUNCH_CHECK();
        return COBALT_OK;
    }
    return launch_copy<true>(x, node_pos, T, N, d, bound, packed, s);
}

// Scratch of cobalt_dispatch_pack_noalloc: the dispatch workspace as a fixed
// array in the library's device memory. Each GPU the library runs on holds
// its own copy, from when the code object is loaded there until the process
// ends. In host code the array's name denotes a host-side stand-in, not a
// device address: the device address is looked up once per device and only
// that address is handed to kernels. The init kernel clears the look-back
// state and the tile counter at the start of every call, and the scan
// writes every base entry before the rank kernel reads it, so what a
// previous call left in the array does not matter.
static __device__ __align__(256) uint8_t scratch[COBALT_DISPATCH_NOALLOC_SCRATCH_BYTES];

cobalt_status dispatch_noalloc_scratch(void** out) {
    static std::mutex mu;
    static std::vector<void*> addr;  // per device
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return COBALT_EHIP;
    std::lock_guard<std::mutex> lock(mu);
    if ((int)addr.size() <= dev) addr.resize(dev + 1, nullptr);
    if (!addr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return COBALT_EHIP;
        addr[dev] = p;
    }
    *out = addr[dev];
    return COBALT_OK;
}

}  // namespace cobalt
