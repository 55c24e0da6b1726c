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
//           e[b]) of the later slots, with LDS atomics. The band's bins are
//           then written to the chunk's slot of the workspace, as uint16
//           where no bin of a chunk can pass 65535, else as uint32.
//   reduce  sixteen lanes per group of eight band bins sum the group over
//           the chunks (lane k takes chunks k, k + 16, ..., one 16-byte load
//           of eight uint16 bins each), add pairwise across lanes k and
//           k + 8, then exchange halves in three shuffle rounds so that lane
//           k < 8 ends with the total of bin k, which it adds to coact[i][j]
//           and coact[j][i]. Other lanes do the same for expert_count. Every
//           output element has exactly one writer, so the result does not
//           depend on scheduling.
//
// Checks. Ids outside [0, E) count nowhere. A token that repeats an id adds
// the product of the multiplicities to a pair, and m (m - 1) to the
// diagonal entry of an id it holds m times: the diagonal is kept per band in
// LDS beside the counts and added to coact with one atomic per nonzero entry
// (top-k selections never repeat an id, so this costs nothing on real
// routing). When every token a wave holds has K distinct ids in range (the
// normal case, found with one ballot), the wave adds its pairs without
// per-pair tests.
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
constexpr int kReduceLanes = 16;  // lanes per group of eight bins (and per count)
constexpr int kMaxLgBands = 12;
constexpr int64_t kTokensPerChunk = 1024;
constexpr int64_t kMaxChunks = 128;
constexpr int64_t kMaxChunks16 = 128;  // more chunks allowed to keep uint16 partials
constexpr int kParBands = 2;            // bands for parallelism on large calls
constexpr int64_t kParPairs = 1 << 18;  // T*K from which bands are used for parallelism
constexpr int64_t kDirectUpdates = 65536;

struct Plan {
    int nchunks;
    int lgb;                // log2 of the number of bands
    bool u16;               // partial bins stored as uint16
    int64_t tok_per_chunk;
    int64_t words;          // E(E-1)/2
    int64_t band_stride;    // bins of the largest band (band 0), rounded up to 8
    int32_t cnt_off;        // LDS word of the band's expert counts (then its diagonal)
    size_t lds_bytes;
    size_t part_bytes;      // partial pair histograms
    size_t count_bytes;     // partial expert counts
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }
int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

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

// LDS words of band 0 (the largest) and of its expert counts (or diagonal)
// with nb bands, rounded up for 16-byte accesses.
int64_t hist_words(int E, int nb) { return round_up(std::max(band_words(E, nb, 0), 1), 8); }
int64_t cnt_words(int E, int nb) { return round_up((E + nb - 1) / nb, 4); }

bool make_plan(int64_t T, int64_t K, int E, int lds_bytes, Plan* p) {
    p->words = (int64_t)E * (E - 1) / 2;
    p->nchunks = (int)std::min<int64_t>(kMaxChunks, std::max<int64_t>(1, T / kTokensPerChunk));
    p->tok_per_chunk = std::max<int64_t>(1, (T + p->nchunks - 1) / p->nchunks);
    // A token adds at most floor(K/2) * ceil(K/2) to one bin (two experts,
    // each repeated), so a chunk's bins fit in uint16 when its tokens times
    // that product stay within 65535. More chunks are used to get there when
    // at most kMaxChunks16 suffice.
    const int64_t maxpair = (K / 2) * ((K + 1) / 2);
    p->u16 = p->tok_per_chunk * maxpair <= 65535;
    if (!p->u16) {
        const int64_t n16 = (T * maxpair + 65534) / 65535;
        if (n16 <= kMaxChunks16) {
            p->nchunks = (int)n16;
            p->tok_per_chunk = (T + n16 - 1) / n16;
            p->u16 = p->tok_per_chunk * maxpair <= 65535;
        }
    }
    const int64_t lds_words = lds_bytes / 4;
    auto fits = [&](int l) { return hist_words(E, 1 << l) + 2 * cnt_words(E, 1 << l) <= lds_words; };
    // fewest bands whose largest band and counts fit the LDS
    int lgb = 0;
    while (lgb <= kMaxLgBands && !fits(lgb)) ++lgb;
    if (lgb > kMaxLgBands) return false;
    // large calls: more bands, for more workgroups (at most one row per band)
    if (T * K >= kParPairs)
        while ((1 << lgb) < kParBands && (1 << (lgb + 1)) <= std::max(E - 1, 1)) ++lgb;
    p->lgb = lgb;
    const int nb = 1 << lgb;
    p->band_stride = hist_words(E, nb);
    p->cnt_off = (int32_t)p->band_stride;
    p->lds_bytes = (size_t)(p->band_stride + 2 * cnt_words(E, nb)) * 4;
    p->part_bytes = align256((size_t)p->nchunks * nb * p->band_stride * (p->u16 ? 2 : 4));
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

// Local row of bin w of band b: the last r with off_b(r) <= w.
__device__ __forceinline__ int32_t band_row_of(int32_t E, int32_t nb, int32_t b, int32_t w) {
    int32_t lo = 0, hi = band_rows(E, nb, b) - 1;
    while (lo < hi) {
        const int32_t mid = (lo + hi + 1) / 2;
        if (band_off(E, nb, b, mid) <= w) lo = mid; else hi = mid - 1;
    }
    return lo;
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

// Loads token t's ids into e (INT_MAX past K).
template <int KC, bool kVec, int KM>
__device__ __forceinline__ void load_ids(const int32_t* __restrict__ topk, int64_t t, int K,
                                         int (&e)[KM]) {
    if constexpr (kVec) {
        const int4* p = reinterpret_cast<const int4*>(topk + t * 8);
        const int4 v0 = p[0], v1 = p[1];
        e[0] = v0.x; e[1] = v0.y; e[2] = v0.z; e[3] = v0.w;
        e[4] = v1.x; e[5] = v1.y; e[6] = v1.z; e[7] = v1.w;
    } else {
#pragma unroll
        for (int a = 0; a < KM; ++a) e[a] = a < K ? topk[t * K + a] : INT_MAX;
    }
}

// One token of the count kernel: its counts, pairs and repeats in band `band`.
template <int KC, int KM>
__device__ __forceinline__ void count_token(int (&e)[KM], int E, int lgb, int band,
                                            int32_t row_len0, uint32_t* hist, uint32_t* cnt,
                                            uint32_t* diag) {
    const int nb = 1 << lgb;
#pragma unroll
    for (int a = 0; a < KM; ++a)
        if ((uint32_t)e[a] >= (uint32_t)E) e[a] = INT_MAX;
#pragma unroll
    for (int a = 0; a < KM; ++a)
        if (e[a] != INT_MAX && (e[a] & (nb - 1)) == band) atomicAdd(&cnt[e[a] >> lgb], 1u);
    sort_ids<KM>(e);
    bool fast = false;
    if constexpr (KC == 8) {
        // K distinct ids in range: strictly increasing, the last not INT_MAX
        bool ok = e[KM - 1] != INT_MAX;
#pragma unroll
        for (int a = 0; a + 1 < KM; ++a) ok = ok && e[a] < e[a + 1];
        fast = __builtin_amdgcn_ballot_w64(!ok) == 0;  // one value for the wave
    }
    if (fast) {
#pragma unroll
        for (int a = 0; a + 1 < KM; ++a) {
            const int i = e[a];
            if ((i & (nb - 1)) != band) continue;
            const int32_t r = i >> lgb;
            const int32_t base = r * row_len0 - nb * (r * (r - 1) / 2) - i - 1;
#pragma unroll
            for (int b = a + 1; b < KM; ++b) atomicAdd(&hist[base + e[b]], 1u);
        }
    } else {
#pragma unroll
        for (int a = 0; a < KM; ++a) {
            const int i = e[a];
            if (i == INT_MAX || (i & (nb - 1)) != band) continue;
            const int32_t r = i >> lgb;
            const int32_t base = r * row_len0 - nb * (r * (r - 1) / 2) - i - 1;
            int m = 1;  // copies of i from slot a on (they follow a, sorted)
#pragma unroll
            for (int b = a + 1; b < KM; ++b) {
                const int j = e[b];
                if (j == i)
                    ++m;
                else if (j != INT_MAX)
                    atomicAdd(&hist[base + j], 1u);
            }
            const bool first = a == 0 || e[a > 0 ? a - 1 : 0] != i;
            if (first && m > 1) atomicAdd(&diag[i >> lgb], (uint32_t)(m * (m - 1)));
        }
    }
}

// KC = compile-time K (0: any K up to 16, read at run time); kVec: K = 8
// and a 16-byte aligned topk, read with two 16-byte loads per token. Ids
// outside [0, E) sort last as INT_MAX and count nowhere. U16: partial bins
// written as uint16. A thread takes two tokens per iteration and issues
// both loads before either is counted.
template <int KC, bool kVec, bool U16>
__global__ __launch_bounds__(kCountThreads) void coact_count_kernel(
    const int32_t* __restrict__ topk, int64_t T, int Kr, int E, int lgb, int nchunks,
    int64_t tok_per_chunk, int64_t band_stride, int cnt_off, void* __restrict__ part,
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
    uint32_t* cnt = lds + cnt_off;
    uint32_t* diag = cnt + (((E + nb - 1) / nb + 3) & ~3);

    // band_stride and the count words are multiples of 4 words
    const int32_t lds_words = (int32_t)(diag - lds) + ((ncnt + 3) & ~3);
    for (int32_t w = threadIdx.x * 4; w < lds_words; w += kCountThreads * 4)
        *reinterpret_cast<u32x4*>(lds + w) = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();

    const int64_t t0 = (int64_t)chunk * tok_per_chunk;
    const int64_t t1 = min(T, t0 + tok_per_chunk);
    for (int64_t t = t0 + threadIdx.x; t < t1; t += 2 * kCountThreads) {
        const int64_t u = t + kCountThreads;
        int e[KM], f[KM];
        load_ids<KC, kVec>(topk, t, K, e);
        if (u < t1) load_ids<KC, kVec>(topk, u, K, f);
        count_token<KC>(e, E, lgb, band, row_len0, hist, cnt, diag);
        if (u < t1) count_token<KC>(f, E, lgb, band, row_len0, hist, cnt, diag);
    }
    __syncthreads();

    // Write-out: thread g takes bins [8g, 8g + 8).
    const int32_t groups = (int32_t)(band_stride / 8);
    for (int32_t g = threadIdx.x; g < groups; g += kCountThreads) {
        const u32x4 lo = *reinterpret_cast<const u32x4*>(lds + g * 8);
        const u32x4 hi = *reinterpret_cast<const u32x4*>(lds + g * 8 + 4);
        if (direct) {  // one band: the chunk's bins go straight to the outputs
            const uint32_t v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int32_t bin = g * 8 + k;
                if (v[k] == 0 || bin >= nbins) continue;
                const int32_t i = tri_row(bin, E);
                const int32_t j = bin - band_off(E, 1, 0, i) + i + 1;
                atomicAdd(&coact[(int64_t)i * E + j], v[k]);
                atomicAdd(&coact[(int64_t)j * E + i], v[k]);
            }
            continue;
        }
        const int64_t at = ((int64_t)band * nchunks + chunk) * band_stride + g * 8;
        if constexpr (U16) {
            const u32x4 packed = {lo.x | (lo.y << 16), lo.z | (lo.w << 16), hi.x | (hi.y << 16),
                                  hi.z | (hi.w << 16)};
            *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(part) + at) = packed;
        } else {
            u32x4* out = reinterpret_cast<u32x4*>(static_cast<uint32_t*>(part) + at);
            out[0] = lo;
            out[1] = hi;
        }
    }
    for (int32_t k = threadIdx.x; k < ncnt; k += kCountThreads) {
        const uint32_t v = cnt[k];
        if (direct) {
            if (count && v) atomicAdd(&count[k], v);
        } else {
            cpart[(int64_t)chunk * E + k * nb + band] = v;
        }
        const int64_t ex = (int64_t)k * nb + band;
        if (diag[k]) atomicAdd(&coact[ex * E + ex], diag[k]);
    }
}

// Items [0, nb * band_stride / 8) are groups of eight band bins, then E
// expert counts; kReduceLanes lanes per item, lane k summing chunks k,
// k + kReduceLanes, ...
template <bool U16>
__global__ __launch_bounds__(kReduceThreads) void coact_reduce_kernel(
    const void* __restrict__ part, const uint32_t* __restrict__ cpart, int E, int lgb,
    int nchunks, int64_t band_stride, bool do_count, uint32_t* __restrict__ coact,
    uint32_t* __restrict__ count) {
    static_assert(kReduceLanes >= 8 && kReduceLanes <= 64 && (kReduceLanes & (kReduceLanes - 1)) == 0,
                  "a power of two of at least eight lanes");
    const int nb = 1 << lgb;
    const int64_t groups_per_band = band_stride / 8;
    const int64_t ngroups = (int64_t)nb * groups_per_band;
    const int64_t gid = (int64_t)blockIdx.x * kReduceThreads + threadIdx.x;
    const int64_t item = gid / kReduceLanes;
    const int k = (int)(gid % kReduceLanes);
    if (item < ngroups) {
        const int band = (int)(item / groups_per_band);
        const int32_t w0 = (int32_t)(item % groups_per_band) * 8;
        // The bin of lane k < 8 and its two outputs, read before the
        // partials so that both loads are in flight together; lanes from 8 on
        // help with the sums only.
        const int32_t w = w0 + (k & 7);
        const bool real = k < 8 && w < band_words(E, nb, band);
        int64_t ij = 0, ji = 0;
        uint32_t cij = 0, cji = 0;
        if (real) {
            const int32_t r = band_row_of(E, nb, band, w);
            const int32_t i = r * nb + band;
            const int32_t j = w - band_off(E, nb, band, r) + i + 1;
            ij = (int64_t)i * E + j;
            ji = (int64_t)j * E + i;
            cij = coact[ij];
            cji = coact[ji];
        }
        uint32_t s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const int64_t base = (int64_t)band * nchunks * band_stride + w0;
        if constexpr (U16) {
            const uint16_t* src = static_cast<const uint16_t*>(part) + base;
#pragma unroll 8
            for (int c = k; c < nchunks; c += kReduceLanes) {
                const u32x4 v = *reinterpret_cast<const u32x4*>(src + (int64_t)c * band_stride);
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
                const u32x4* q = reinterpret_cast<const u32x4*>(src + (int64_t)c * band_stride);
                const u32x4 lo = q[0], hi = q[1];
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    s[h] += lo[h];
                    s[4 + h] += hi[h];
                }
            }
        }
        // Lanes k, k ^ 8, k ^ 16, ... add their sums, then three rounds each
        // halve the bins a lane holds: the lane keeps the half its bit
        // selects and adds the partner's sums of that half. Lane k ends with
        // the total of bin w0 + k % 8.
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
        const uint32_t sum = s[0];
        if (sum == 0 || !real) return;
        coact[ij] = cij + sum;
        coact[ji] = cji + sum;
    } else if (do_count && item < ngroups + E) {
        const int e = (int)(item - ngroups);
        uint32_t sum = 0;
#pragma unroll 8
        for (int c = k; c < nchunks; c += kReduceLanes) sum += cpart[(int64_t)c * E + e];
#pragma unroll
        for (int o = 1; o < kReduceLanes; o <<= 1) sum += __shfl_xor(sum, o, kReduceLanes);
        if (k == 0 && sum != 0) count[e] += sum;
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
    void* part = ws;
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
                           p.band_stride, p.cnt_off, part, cpart, direct, coact, count);
        return COBALT_OK;
    };
    const bool vec = K == 8 && ((uintptr_t)topk & 15u) == 0;
    cobalt_status st;
    if (p.u16)
        st = vec      ? launch(coact_count_kernel<8, true, true>, 0)
             : K == 8 ? launch(coact_count_kernel<8, false, true>, 1)
                      : launch(coact_count_kernel<0, false, true>, 2);
    else
        st = vec      ? launch(coact_count_kernel<8, true, false>, 3)
             : K == 8 ? launch(coact_count_kernel<8, false, false>, 4)
                      : launch(coact_count_kernel<0, false, false>, 5);
    if (st != COBALT_OK) return st;
    COBALT_LAUNCH_CHECK();
    if (direct) return COBALT_OK;
    const int64_t items = (int64_t)nb * (p.band_stride / 8) + (count ? E : 0);
    const dim3 grid((unsigned)((items * kReduceLanes + kReduceThreads - 1) / kReduceThreads));
    if (p.u16)
        hipLaunchKernelGGL(coact_reduce_kernel<true>, grid, dim3(kReduceThreads), 0, s, part,
                           cpart, E, p.lgb, p.nchunks, p.band_stride, count != nullptr, coact,
                           count);
    else
        hipLaunchKernelGGL(coact_reduce_kernel<false>, grid, dim3(kReduceThreads), 0, s, part,
                           cpart, E, p.lgb, p.nchunks, p.band_stride, count != nullptr, coact,
                           count);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
