// Reference kernels that measure what this GPU's HBM sustains for the access
// shapes of the routing path, timed by the benchmark beside the library's
// calls. They are measurement instruments, not part of the routing library
// or its C ABI; each does the memory traffic it names and computes a small
// checkable result so that no access can be optimised away.
//
//   ceil_read         streams a buffer once (16 B non-temporal load per
//                     thread, one pass wide, no grid-stride loop) and writes
//                     the XOR of each workgroup's words
//   ceil_fill         writes a buffer once (16 B non-temporal store per
//                     thread, one pass wide)
//   ceil_copy         copies a buffer once (16 B load and store per thread)
//   ceil_pack_store   the pack's stores without its loads: one workgroup per
//                     (token, 2 KiB slice), one wave per slot, each wave
//                     writing one 2 KiB burst to its packed row with
//                     non-temporal stores; the data is a pattern of (token,
//                     slot, chunk)
//   ceil_gather_read  the combine's loads without its fold or stores: one
//                     workgroup per (token, 2 KiB slice), one wave per slot,
//                     each wave loading one 2 KiB burst of its packed row with
//                     non-temporal loads; each workgroup writes the XOR of
//                     what it read
//
// All sizes are checked on the host; a bad argument returns 1, a launch
// error 2.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kMaxK = 16;
constexpr int64_t kMaxItems = int64_t(1) << 31;  // work-items of one dispatch

__device__ uint32_t block_xor(uint32_t v) {
    __shared__ uint32_t part[16];
    for (int o = 32; o > 0; o >>= 1) v ^= __shfl_xor(v, o, 64);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) part[wave] = v;
    __syncthreads();
    uint32_t r = 0;
    if (threadIdx.x == 0)
        for (int w = 0; w < (int)(blockDim.x >> 6); ++w) r ^= part[w];
    return r;
}

__global__ __launch_bounds__(kThreads) void read_kernel(const u32x4* __restrict__ buf, int64_t n,
                                                        uint32_t* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    uint32_t v = 0;
    if (i < n) {
        const u32x4 a = __builtin_nontemporal_load(buf + i);
        v = a.x ^ a.y ^ a.z ^ a.w;
    }
    v = block_xor(v);
    if (threadIdx.x == 0) out[blockIdx.x] = v;
}

__global__ __launch_bounds__(kThreads) void fill_kernel(u32x4* __restrict__ buf, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) {
        const uint32_t k = (uint32_t)i;
        const u32x4 v = {k, k ^ 0x9e3779b9u, ~k, k * 3u};
        __builtin_nontemporal_store(v, buf + i);
    }
}

__global__ __launch_bounds__(kThreads) void copy_kernel(const u32x4* __restrict__ src,
                                                        u32x4* __restrict__ dst, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

template <int GROUPS>
__global__ __launch_bounds__(kMaxK * 64) void pack_store_kernel(const int32_t* __restrict__ pos,
                                                                int K, int64_t nch, int64_t TK,
                                                                u32x4* __restrict__ packed) {
    const uint32_t tg = blockIdx.x;
    const uint32_t t = tg / GROUPS;
    const uint32_t g = tg - t * GROUPS;
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t c0 = (int64_t)g * 128 + (threadIdx.x & 63);
    const int p = pos[(int64_t)t * K + j];
    if (p < 0 || p >= TK) return;
    u32x4* dst = packed + (int64_t)p * nch;
    const u32x4 v0 = {t, (uint32_t)j, (uint32_t)c0, 0x5a5a5a5au};
    const u32x4 v1 = {t, (uint32_t)j, (uint32_t)(c0 + 64), 0x5a5a5a5au};
    if (c0 < nch) __builtin_nontemporal_store(v0, dst + c0);
    if (c0 + 64 < nch) __builtin_nontemporal_store(v1, dst + c0 + 64);
}

template <int GROUPS>
__global__ __launch_bounds__(kMaxK * 64) void gather_read_kernel(
    const u32x4* __restrict__ rows, const int32_t* __restrict__ pos, int K, int64_t nch,
    int64_t TK, uint32_t* __restrict__ out) {
    const uint32_t tg = blockIdx.x;
    const uint32_t t = tg / GROUPS;
    const uint32_t g = tg - t * GROUPS;
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t c0 = (int64_t)g * 128 + (threadIdx.x & 63);
    const int p = pos[(int64_t)t * K + j];
    uint32_t v = 0;
    if (p >= 0 && p < TK) {
        const u32x4* src = rows + (int64_t)p * nch;
        if (c0 < nch) {
            const u32x4 a = __builtin_nontemporal_load(src + c0);
            v ^= a.x ^ a.y ^ a.z ^ a.w;
        }
        if (c0 + 64 < nch) {
            const u32x4 a = __builtin_nontemporal_load(src + c0 + 64);
            v ^= a.x ^ a.y ^ a.z ^ a.w;
        }
    }
    v = block_xor(v);
    if (threadIdx.x == 0) out[blockIdx.x] = v;
}

int launched() { return hipGetLastError() == hipSuccess ? 0 : 2; }

}  // namespace

extern "C" {

// Blocks written by ceil_read and ceil_fill etc. for a buffer of `bytes`.
int64_t ceil_stream_blocks(int64_t bytes) {
    return (bytes / 16 + kThreads - 1) / kThreads;
}

int ceil_read(const void* buf, int64_t bytes, uint32_t* out, void* stream) {
    if (!buf || !out || bytes <= 0 || bytes % 16 != 0 || bytes / 16 >= kMaxItems) return 1;
    const int64_t n = bytes / 16;
    hipLaunchKernelGGL(read_kernel, dim3((unsigned)ceil_stream_blocks(bytes)), dim3(kThreads), 0,
                       (hipStream_t)stream, (const u32x4*)buf, n, out);
    return launched();
}

int ceil_fill(void* buf, int64_t bytes, void* stream) {
    if (!buf || bytes <= 0 || bytes % 16 != 0 || bytes / 16 >= kMaxItems) return 1;
    const int64_t n = bytes / 16;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)ceil_stream_blocks(bytes)), dim3(kThreads), 0,
                       (hipStream_t)stream, (u32x4*)buf, n);
    return launched();
}

int ceil_copy(const void* src, void* dst, int64_t bytes, void* stream) {
    if (!src || !dst || bytes <= 0 || bytes % 16 != 0 || bytes / 16 >= kMaxItems) return 1;
    const int64_t n = bytes / 16;
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)ceil_stream_blocks(bytes)), dim3(kThreads), 0,
                       (hipStream_t)stream, (const u32x4*)src, (u32x4*)dst, n);
    return launched();
}

#define CEIL_GROUP_CASES(X) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) \
    X(13) X(14) X(15) X(16)

// pos [T][K]: packed row of each pair (rows outside [0, T*K) are skipped);
// packed [T*K][d] bf16. d % 8 == 0, d <= 16384, 1 <= K <= 16.
int ceil_pack_store(const int32_t* pos, int64_t T, int K, int64_t d, void* packed, void* stream) {
    if (!pos || !packed || T <= 0 || K < 1 || K > kMaxK || d < 8 || d % 8 != 0 || d > 16384)
        return 1;
    const int64_t nch = d / 8, groups = (nch + 127) / 128, TK = T * K;
    if (T * groups * K * 64 >= kMaxItems || TK >= kMaxItems) return 1;
    const dim3 grid((unsigned)(T * groups)), block(K * 64);
    hipStream_t s = (hipStream_t)stream;
    switch (groups) {
#define CASE(G) case G: hipLaunchKernelGGL(pack_store_kernel<G>, grid, block, 0, s, pos, K, nch, TK, (u32x4*)packed); break;
        CEIL_GROUP_CASES(CASE)
#undef CASE
        default: return 1;
    }
    return launched();
}

// rows [T*K][d] bf16 in the packed layout, pos as above; out [T * ceil(d /
// 1024)] receives each workgroup's XOR.
int ceil_gather_read(const void* rows, const int32_t* pos, int64_t T, int K, int64_t d,
                     uint32_t* out, void* stream) {
    if (!rows || !pos || !out || T <= 0 || K < 1 || K > kMaxK || d < 8 || d % 8 != 0 ||
        d > 16384)
        return 1;
    const int64_t nch = d / 8, groups = (nch + 127) / 128, TK = T * K;
    if (T * groups * K * 64 >= kMaxItems || TK >= kMaxItems) return 1;
    const dim3 grid((unsigned)(T * groups)), block(K * 64);
    hipStream_t s = (hipStream_t)stream;
    switch (groups) {
#define CASE(G) case G: hipLaunchKernelGGL(gather_read_kernel<G>, grid, block, 0, s, (const u32x4*)rows, pos, K, nch, TK, out); break;
        CEIL_GROUP_CASES(CASE)
#undef CASE
        default: return 1;
    }
    return launched();
}

}  // extern "C"
