// C entry points: argument checks, the layout handle, and dispatch to the
// kernel launchers.
#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "internal.hpp"

using namespace cobalt;

struct cobalt_layout_s {
    DeviceLayout d;
};

extern "C" const char* cobalt_status_string(cobalt_status s) {
    switch (s) {
        case COBALT_OK: return "ok";
        case COBALT_EINVAL: return "invalid argument";
        case COBALT_EUNSUPPORTED: return "unsupported size";
        case COBALT_ENOMEM: return "device allocation failed";
        case COBALT_EHIP: return "HIP runtime error";
        case COBALT_EDATA: return "input data violates the layout or routing model";
    }
    return "unknown status";
}

namespace cobalt {

cobalt_status device_info(DeviceInfo* out) {
    static std::mutex mu;
    static std::vector<DeviceInfo> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return COBALT_EHIP;
    std::lock_guard<std::mutex> lock(mu);
    if ((int)cache.size() <= dev) cache.resize(dev + 1, DeviceInfo{0, 0});
    if (cache[dev].cus == 0) {
        int cus = 0, lds = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return COBALT_EHIP;
        if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
            hipSuccess)
            return COBALT_EHIP;
        cache[dev] = DeviceInfo{cus, lds};
    }
    *out = cache[dev];
    return COBALT_OK;
}

}  // namespace cobalt

static void free_layout(DeviceLayout& d) {
    (void)hipFree(d.node_mask);
    (void)hipFree(d.rank_mask);
    (void)hipFree(d.owner);
    d.node_mask = nullptr;
    d.rank_mask = nullptr;
    d.owner = nullptr;
}

extern "C" cobalt_status cobalt_layout_create(int32_t N, int32_t gpn, int32_t E, int32_t S,
                                              const int32_t* slot, const int32_t* owner_in,
                                              cobalt_layout_t* out) {
    if (!out || !slot) return COBALT_EINVAL;
    *out = nullptr;
    if (N < 1 || N > kMaxN || gpn < 1 || gpn > kMaxGpn || E < 1 || E > kMaxE || S < 1)
        return COBALT_EINVAL;
    const int32_t G = N * gpn;
    if (G > kMaxG) return COBALT_EUNSUPPORTED;

    std::vector<uint32_t> node_mask(E, 0u), rank_mask((size_t)E * N, 0u);
    std::vector<int32_t> owner(E, -1);
    for (int32_t r = 0; r < G; ++r) {
        const int32_t n = r / gpn, i = r % gpn;
        for (int32_t k = 0; k < S; ++k) {
            const int32_t e = slot[(size_t)r * S + k];
            if (e == -1) continue;
            if (e < 0 || e >= E) return COBALT_EDATA;
            uint32_t& rm = rank_mask[(size_t)e * N + n];
            if (rm & (1u << i)) return COBALT_EDATA;  // expert twice on one rank
            rm |= 1u << i;
            node_mask[e] |= 1u << n;
            if (owner[e] < 0) owner[e] = r;
        }
    }
    for (int32_t e = 0; e < E; ++e) {
        if (!node_mask[e]) return COBALT_EDATA;  // uncovered expert
        if (owner_in) {
            const int32_t o = owner_in[e];
            if (o < 0 || o >= G) return COBALT_EDATA;
            if (!(rank_mask[(size_t)e * N + o / gpn] & (1u << (o % gpn)))) return COBALT_EDATA;
            owner[e] = o;
        }
    }
    auto* L = new (std::nothrow) cobalt_layout_s();
    if (!L) return COBALT_ENOMEM;
    DeviceLayout& d = L->d;
    if (hipGetDevice(&d.device) != hipSuccess) {
        delete L;
        return COBALT_EHIP;
    }
    d.N = N;
    d.g = gpn;
    d.G = G;
    d.E = E;
    d.S = S;
    if (hipMalloc(&d.node_mask, sizeof(uint32_t) * E) != hipSuccess ||
        hipMalloc(&d.rank_mask, sizeof(uint32_t) * E * N) != hipSuccess ||
        hipMalloc(&d.owner, sizeof(int32_t) * E) != hipSuccess) {
        free_layout(d);
        delete L;
        return COBALT_ENOMEM;
    }
    if (hipMemcpy(d.node_mask, node_mask.data(), sizeof(uint32_t) * E, hipMemcpyHostToDevice) !=
            hipSuccess ||
        hipMemcpy(d.rank_mask, rank_mask.data(), sizeof(uint32_t) * E * N,
                  hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(d.owner, owner.data(), sizeof(int32_t) * E, hipMemcpyHostToDevice) !=
            hipSuccess) {
        free_layout(d);
        delete L;
        return COBALT_EHIP;
    }
    *out = L;
    return COBALT_OK;
}

extern "C" cobalt_status cobalt_layout_destroy(cobalt_layout_t L) {
    if (!L) return COBALT_EINVAL;
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return COBALT_EHIP;
    if (cur != L->d.device && hipSetDevice(L->d.device) != hipSuccess) return COBALT_EHIP;
    free_layout(L->d);
    if (cur != L->d.device) (void)hipSetDevice(cur);
    delete L;
    return COBALT_OK;
}

static cobalt_status check_device(const cobalt_layout_s* L) {
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return COBALT_EHIP;
    return cur == L->d.device ? COBALT_OK : COBALT_EINVAL;
}

extern "C" cobalt_status cobalt_layout_tables(cobalt_layout_t L, uint32_t* node_mask,
                                              uint32_t* rank_mask, int32_t* owner) {
    if (!L) return COBALT_EINVAL;
    if (cobalt_status st = check_device(L)) return st;
    const DeviceLayout& d = L->d;
    if (node_mask && hipMemcpy(node_mask, d.node_mask, sizeof(uint32_t) * d.E,
                               hipMemcpyDeviceToHost) != hipSuccess)
        return COBALT_EHIP;
    if (rank_mask && hipMemcpy(rank_mask, d.rank_mask, sizeof(uint32_t) * d.E * d.N,
                               hipMemcpyDeviceToHost) != hipSuccess)
        return COBALT_EHIP;
    if (owner &&
        hipMemcpy(owner, d.owner, sizeof(int32_t) * d.E, hipMemcpyDeviceToHost) != hipSuccess)
        return COBALT_EHIP;
    return COBALT_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

namespace cobalt {
int64_t max_launch_items() {
    const char* v = std::getenv("COBALT_MAX_LAUNCH_ITEMS");
    if (!v || !*v) return kMaxLaunchItems;
    char* end = nullptr;
    const long long n = std::strtoll(v, &end, 10);
    if (*end != '\0' || n < 64) return kMaxLaunchItems;
    return n < kMaxLaunchItems ? (int64_t)n : kMaxLaunchItems;
}
}  // namespace cobalt


extern "C" size_t cobalt_coact_stats_workspace_bytes(int64_t T, int32_t K, int32_t E) {
    if (T < 0 || K < 1 || K > kMaxK || E < 1 || E > kMaxE) return 0;
    // the larger of the plans for 64 KiB and 160 KiB of LDS per workgroup
    return std::max<size_t>(std::max<size_t>(coact_workspace_bytes(T, K, E, 64 * 1024),
                                             coact_workspace_bytes(T, K, E, 160 * 1024)),
                            256);
}

extern "C" cobalt_status cobalt_coact_stats(const int32_t* topk, int64_t T, int32_t K, int32_t E,
                                            uint32_t* coact, uint32_t* count, void* ws,
                                            size_t ws_bytes, void* stream) {
    if (T < 0 || K < 1 || K > kMaxK || E < 1 || E > kMaxE || !coact || !ws) return COBALT_EINVAL;
    if (K > E) return COBALT_EINVAL;  // a token's K experts are distinct
    if (T > 0 && !topk) return COBALT_EINVAL;
    if (((uintptr_t)ws & 255u) != 0) return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    if (ws_bytes < cobalt_coact_stats_workspace_bytes(T, K, E)) return COBALT_EINVAL;
    if (T == 0) return COBALT_OK;
    return launch_coact_stats(topk, T, K, E, coact, count, ws, ws_bytes, (hipStream_t)stream);
}

extern "C" cobalt_status cobalt_assign(cobalt_layout_t L, const int32_t* topk,
                                       const int32_t* src, int64_t T, int32_t K, uint64_t seed,
                                       uint64_t step, int32_t mode, int32_t* out,
                                       uint16_t* remote, void* stream) {
    if (!L || T < 0 || K < 1 || K > kMaxK || (mode != 0 && mode != 1)) return COBALT_EINVAL;
    if (K > L->d.E) return COBALT_EINVAL;  // a token's K experts are distinct
    if (T > 0 && (!topk || !out)) return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    if (!src && T % L->d.G != 0) return COBALT_EINVAL;
    if (cobalt_status st = check_device(L)) return st;
    if (T == 0) return COBALT_OK;
    const uint64_t key = splitmix64(splitmix64(seed) ^ step);
    return launch_assign(L->d, topk, src, T, K, key, mode, out, remote, (hipStream_t)stream);
}

extern "C" size_t cobalt_dispatch_workspace_bytes(int64_t T, int32_t K, int32_t G) {
    if (T < 0 || K < 1 || K > kMaxK || G < 1 || G > kMaxG) return 0;
    return dispatch_workspace_bytes(T, K, G);
}

// Host checks shared by both dispatch entry points (all but the workspace).
static cobalt_status check_dispatch(const int32_t* assigned, const int32_t* src, int64_t T,
                                    int32_t K, int32_t G, const void* x, int64_t d,
                                    const int32_t* counts, const int64_t* offsets,
                                    const int32_t* pos, const void* packed) {
    if (T < 0 || K < 1 || K > kMaxK || G < 1 || G > kMaxG) return COBALT_EINVAL;
    if (!counts || !offsets) return COBALT_EINVAL;
    if (T > 0 && (!assigned || !pos)) return COBALT_EINVAL;
    if ((x == nullptr) != (packed == nullptr)) return COBALT_EINVAL;
    if (x && (d < 8 || d % 8 != 0 || !aligned16(x) || !aligned16(packed))) return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    if (!src && T % G != 0) return COBALT_EINVAL;
    return COBALT_OK;
}

extern "C" cobalt_status cobalt_dispatch_pack(const int32_t* assigned, const int32_t* src,
                                              int64_t T, int32_t K, int32_t G, const void* x,
                                              int64_t d, int32_t* counts, int64_t* offsets,
                                              int32_t* pos, void* packed, void* ws,
                                              size_t ws_bytes, void* stream) {
    if (cobalt_status st = check_dispatch(assigned, src, T, K, G, x, d, counts, offsets, pos,
                                          packed))
        return st;
    if (!ws || ((uintptr_t)ws & 255u) != 0) return COBALT_EINVAL;
    if (ws_bytes < dispatch_workspace_bytes(T, K, G)) return COBALT_EINVAL;
    return launch_dispatch(assigned, src, T, K, G, x, x ? d : 0, counts, offsets, pos, packed, ws,
                           (hipStream_t)stream);
}

extern "C" cobalt_status cobalt_dispatch_pack_noalloc(const int32_t* assigned,
                                                      const int32_t* src, int64_t T, int32_t K,
                                                      int32_t G, const void* x, int64_t d,
                                                      int32_t* counts, int64_t* offsets,
                                                      int32_t* pos, void* packed, void* stream) {
    if (cobalt_status st = check_dispatch(assigned, src, T, K, G, x, d, counts, offsets, pos,
                                          packed))
        return st;
    if (dispatch_workspace_bytes(T, K, G) > COBALT_DISPATCH_NOALLOC_SCRATCH_BYTES)
        return COBALT_EUNSUPPORTED;
    void* ws = nullptr;
    if (cobalt_status st = dispatch_noalloc_scratch(&ws)) return st;
    return launch_dispatch(assigned, src, T, K, G, x, x ? d : 0, counts, offsets, pos, packed, ws,
                           (hipStream_t)stream);
}

extern "C" size_t cobalt_node_dispatch_workspace_bytes(int64_t T, int32_t N, int32_t gpn) {
    if (T < 0 || N < 1 || N > kMaxN || gpn < 1 || gpn > kMaxGpn || N * gpn > kMaxG) return 0;
    return node_dispatch_workspace_bytes(T, N, N * gpn);
}

extern "C" cobalt_status cobalt_node_dispatch_pack(const int32_t* assigned, const int32_t* src,
                                                   int64_t T, int32_t K, int32_t N, int32_t gpn,
                                                   const void* x, int64_t d, int32_t* counts,
                                                   int64_t* offsets, int32_t* node_pos,
                                                   uint32_t* fwd, int32_t* row_token,
                                                   void* packed, void* ws, size_t ws_bytes,
                                                   void* stream) {
    if (T < 0 || K < 1 || K > kMaxK || N < 1 || N > kMaxN || gpn < 1 || gpn > kMaxGpn)
        return COBALT_EINVAL;
    const int32_t G = N * gpn;
    if (G > kMaxG) return COBALT_EUNSUPPORTED;
    if (!counts || !offsets || !ws) return COBALT_EINVAL;
    if (T > 0 && (!assigned || !node_pos || !fwd)) return COBALT_EINVAL;
    if ((x == nullptr) != (packed == nullptr)) return COBALT_EINVAL;
    if (x && (d < 8 || d % 8 != 0 || !aligned16(x) || !aligned16(packed))) return COBALT_EINVAL;
    if (((uintptr_t)ws & 255u) != 0) return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    if (!src && T % G != 0) return COBALT_EINVAL;
    if (ws_bytes < node_dispatch_workspace_bytes(T, N, G)) return COBALT_EINVAL;
    return launch_node_dispatch(assigned, src, T, K, N, gpn, x, x ? d : 0, counts, offsets,
                                node_pos, fwd, row_token, packed, ws, (hipStream_t)stream);
}

namespace {
bool ema_args_ok(float decay, int32_t flags) {
    return decay >= 0.0f && decay <= 1.0f && (flags & ~(COBALT_EMA_INIT | COBALT_EMA_CLEAR)) == 0;
}
}  // namespace

extern "C" cobalt_status cobalt_coact_ema(uint32_t* coact, uint32_t* count, int32_t E,
                                          float decay, int32_t flags, float* ema_coact,
                                          float* ema_count, float* ochiai, void* stream) {
    if (E < 1 || E > kMaxE || !coact || !count || !ema_args_ok(decay, flags))
        return COBALT_EINVAL;
    return launch_coact_ema(coact, count, E, decay, flags & COBALT_EMA_INIT,
                            flags & COBALT_EMA_CLEAR, ema_coact, ema_count, ochiai,
                            (hipStream_t)stream);
}

extern "C" cobalt_status cobalt_count_ema(uint32_t* counts, int64_t n, float decay,
                                          int32_t flags, float* ema, void* stream) {
    if (n < 0 || !ema_args_ok(decay, flags)) return COBALT_EINVAL;
    if (n > 0 && !counts) return COBALT_EINVAL;
    return launch_count_ema(counts, n, decay, flags & COBALT_EMA_INIT, flags & COBALT_EMA_CLEAR,
                            ema, (hipStream_t)stream);
}

extern "C" cobalt_status cobalt_combine(const void* eo, const int32_t* pos, const float* gates,
                                        int64_t T, int32_t K, int64_t d, void* y, float* y32,
                                        void* stream) {
    if (T < 0 || K < 1 || K > kMaxK || d < 8 || d % 8 != 0) return COBALT_EINVAL;
    if (T > 0 && (!eo || !pos || !gates || !y)) return COBALT_EINVAL;
    if (T > 0 && (!aligned16(eo) || !aligned16(y) || (y32 && !aligned16(y32))))
        return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    if (T == 0) return COBALT_OK;
    return launch_combine(eo, pos, gates, T, K, d, y, y32, (hipStream_t)stream);
}

extern "C" cobalt_status cobalt_node_combine(const void* eo, const int32_t* pos,
                                             const int32_t* assigned, const float* gates,
                                             const int32_t* node_pos, int64_t T, int32_t K,
                                             int32_t N, int32_t gpn, int64_t d, void* partial,
                                             void* y, void* stream) {
    if (T < 0 || K < 1 || K > kMaxK || N < 1 || N > kMaxN || gpn < 1 || gpn > kMaxGpn || d < 8 ||
        d % 8 != 0)
        return COBALT_EINVAL;  // N * gpn <= kMaxN * kMaxGpn = kMaxG
    if (T > 0 && (!eo || !pos || !assigned || !gates || !node_pos || !partial || !y))
        return COBALT_EINVAL;
    if (T > 0 && (!aligned16(eo) || !aligned16(partial) || !aligned16(y))) return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    if (T == 0) return COBALT_OK;
    return launch_node_combine(eo, pos, assigned, gates, node_pos, T, K, N, gpn, d, partial, y,
                               (hipStream_t)stream);
}

extern "C" size_t cobalt_replica_load_workspace_bytes(int64_t T, int32_t K, int32_t E,
                                                     int32_t G) {
    if (T < 0 || K < 1 || K > kMaxK || E < 1 || E > kMaxE || G < 1 || G > kMaxG) return 0;
    return replica_load_workspace_bytes(T, K, E, G);
}

extern "C" cobalt_status cobalt_replica_load(const int32_t* topk, const int32_t* assigned,
                                             int64_t T, int32_t K, int32_t E, int32_t G,
                                             uint32_t* load, void* ws, size_t ws_bytes,
                                             void* stream) {
    if (T < 0 || K < 1 || K > kMaxK || E < 1 || E > kMaxE || G < 1 || G > kMaxG) return COBALT_EINVAL;
    if (!load || !ws || (T > 0 && (!topk || !assigned))) return COBALT_EINVAL;
    if (((uintptr_t)ws & 255u) != 0) return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    if (ws_bytes < replica_load_workspace_bytes(T, K, E, G)) return COBALT_EINVAL;
    if (T == 0) return COBALT_OK;
    return launch_replica_load(topk, assigned, T, K, E, G, load, ws, ws_bytes, (hipStream_t)stream);
}

extern "C" cobalt_status cobalt_validate_routing(const int32_t* topk, const int32_t* src,
                                                 int64_t T, int32_t K, int32_t E, int32_t G,
                                                 uint32_t* host_flags, void* stream) {
    if (T < 0 || K < 1 || K > kMaxK || E < 1 || G < 1 || G > kMaxG) return COBALT_EINVAL;
    if (T > 0 && !topk) return COBALT_EINVAL;
    if (T * K >= (int64_t(1) << 31)) return COBALT_EUNSUPPORTED;
    uint32_t flags = 0;
    if (T > 0) {
        uint32_t* dflags = nullptr;
        if (hipMalloc(&dflags, sizeof(uint32_t)) != hipSuccess) return COBALT_ENOMEM;
        hipStream_t s = (hipStream_t)stream;
        cobalt_status st = launch_validate(topk, src, T, K, E, G, dflags, s);
        if (st == COBALT_OK &&
            (hipMemcpyAsync(&flags, dflags, sizeof(uint32_t), hipMemcpyDeviceToHost, s) !=
                 hipSuccess ||
             hipStreamSynchronize(s) != hipSuccess))
            st = COBALT_EHIP;
        (void)hipFree(dflags);
        if (st != COBALT_OK) return st;
    }
    if (host_flags) *host_flags = flags;
    return flags ? COBALT_EDATA : COBALT_OK;
}
