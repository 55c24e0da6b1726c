// Internal declarations of the HIP routing library (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "cobalt.h"

namespace cobalt {

constexpr int kMaxN = 16;
constexpr int kMaxGpn = 32;
constexpr int kMaxG = 512;
static_assert(kMaxN * kMaxGpn <= kMaxG, "N and gpus_per_node in range bound G");
constexpr int kMaxK = 16;
constexpr int kMaxE = 4096;

// 16-byte vector: eight bf16 values, the unit of every row copy.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Streaming row store: a 16-byte raw buffer store with the non-temporal
// (nt) cache bit, through a buffer descriptor of `bytes` bytes at `base`.
// The hardware drops stores outside the descriptor, so a row's stores need
// no guard branches of their own and issue back to back from one offset
// register (with a branch per store the compiler can make the second wait
// for the first). The descriptor's third dword is the gfx9 raw-buffer
// format word.
__device__ __forceinline__ void store_stream(const u32x4& v, void* base, int32_t bytes,
                                             int32_t offset) {
    constexpr int kNt = 2;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(base, (short)0, bytes, 0x00020000);
    __builtin_amdgcn_raw_buffer_store_b128(v, rs, offset, 0, kNt);
}

struct DeviceLayout {
    int device;
    int32_t N, g, G, E, S;
    uint32_t* node_mask;       // [E]
    uint32_t* rank_mask;       // [E][N]
    int32_t* owner;            // [E]
};

// A dispatch packet holds the grid size in work-items as a 32-bit value,
// and a larger grid is cut short without an error. Kernels that take one
// workgroup (or wave) per token slice are therefore launched over ranges of
// tokens of at most max_launch_items() work-items each, with their
// per-token arrays offset to the range; the rows they address through pos
// or node_pos stay absolute.
constexpr int64_t kMaxLaunchItems = int64_t(1) << 31;

// kMaxLaunchItems, or a smaller limit from the environment variable
// COBALT_MAX_LAUNCH_ITEMS (read at every launch, at least 64), so that
// tests can split ordinary sizes into many ranges.
int64_t max_launch_items();

// Calls launch(t0, n) for consecutive token ranges [t0, t0 + n) covering
// [0, T), each of at most max_launch_items() / items_per_token tokens (at
// least one).
template <typename F>
void for_token_ranges(int64_t T, int64_t items_per_token, F&& launch) {
    const int64_t per = items_per_token > 0 ? items_per_token : 1;
    const int64_t lim = max_launch_items();
    const int64_t step = lim / per > 0 ? lim / per : 1;
    for (int64_t t0 = 0; t0 < T; t0 += step) launch(t0, T - t0 < step ? T - t0 : step);
}

#define COBALT_LAUNCH_CHECK()                                        \
    do {                                                             \
        if (hipGetLastError() != hipSuccess) return COBALT_EHIP;     \
    } while (0)

// Per-device properties used to size launches.
struct DeviceInfo {
    int cus;
    int lds_bytes;  // usable LDS per workgroup
};
cobalt_status device_info(DeviceInfo* out);

// Launchers (argument checks are done by the C entry points).
size_t coact_workspace_bytes(int64_t T, int K, int E, int lds_bytes);
cobalt_status launch_coact_stats(const int32_t* topk, int64_t T, int K, int E, uint32_t* coact,
                                 uint32_t* count, void* ws, size_t ws_bytes, hipStream_t s);
cobalt_status launch_assign(const DeviceLayout& L, const int32_t* topk, const int32_t* src,
                            int64_t T, int K, uint64_t key, int mode, int32_t* out,
                            uint16_t* remote, hipStream_t s);
size_t dispatch_workspace_bytes(int64_t T, int K, int G);
cobalt_status launch_dispatch(const int32_t* assigned, const int32_t* src, int64_t T, int K,
                              int G, const void* x, int64_t d, int32_t* counts,
                              int64_t* offsets, int32_t* pos, void* packed, void* ws,
                              hipStream_t s);
// Device address of the fixed dispatch scratch on the current device
// (COBALT_DISPATCH_NOALLOC_SCRATCH_BYTES bytes, 256-byte aligned); looked up
// on the first call on each device, allocates nothing.
cobalt_status dispatch_noalloc_scratch(void** out);
size_t node_dispatch_workspace_bytes(int64_t T, int N, int G);
cobalt_status launch_node_dispatch(const int32_t* assigned, const int32_t* src, int64_t T, int K,
                                   int N, int g, const void* x, int64_t d, int32_t* counts,
                                   int64_t* offsets, int32_t* node_pos, uint32_t* fwd,
                                   int32_t* row_token, void* packed, void* ws, hipStream_t s);
cobalt_status launch_combine(const void* eo, const int32_t* pos, const float* gates, int64_t T,
                             int K, int64_t d, void* y, float* y32, hipStream_t s);
cobalt_status launch_node_combine(const void* eo, const int32_t* pos, const int32_t* assigned,
                                  const float* gates, const int32_t* node_pos, int64_t T, int K,
                                  int N, int gpn, int64_t d, void* partial, void* y,
                                  hipStream_t s);
size_t replica_load_workspace_bytes(int64_t T, int K, int E, int G);
cobalt_status launch_replica_load(const int32_t* topk, const int32_t* assigned, int64_t T, int K,
                                  int E, int G, uint32_t* load, void* ws, size_t ws_bytes,
                                  hipStream_t s);
cobalt_status launch_count_ema(uint32_t* counts, int64_t n, float decay, bool init, bool clear,
                               float* ema, hipStream_t s);
cobalt_status launch_coact_ema(uint32_t* coact, uint32_t* count, int E, float decay, bool init,
                               bool clear, float* ema_coact, float* ema_count, float* ochiai,
                               hipStream_t s);
cobalt_status launch_validate(const int32_t* topk, const int32_t* src, int64_t T, int K, int E,
                              int G, uint32_t* dflags, hipStream_t s);

// SplitMix64 (Steele, Lea & Flood 2014): output of the generator for state z.
__host__ __device__ inline uint64_t splitmix64(uint64_t z) {
    z += 0x9e3779b97f4a7c15ull;
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

}  // namespace cobalt
