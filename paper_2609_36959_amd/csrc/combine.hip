// Combine and weighted sum (Fig. 1, last stage). Each wave takes one
// (token, 1 KiB column slice): every lane loads its 16-byte chunk of the K
// expert rows (rows pos[t][j] of the packed expert outputs) together, folds
// them into eight fp32 accumulators with one fused multiply-add per slot in
// slot order, and stores the round-to-nearest-even bf16 result (and the fp32
// sums when asked). A wave issues all its loads before its single store, so
// no load waits behind a store; loads and stores are non-temporal (every
// byte is touched once).
#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kCombineWaves = 16;

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// KC = compile-time K (0: any K up to 16, read at run time); with KC the
// scalar loads of pos and gates are issued back to back before the rows.
template <bool kF32, int KC>
__global__ __launch_bounds__(kCombineWaves * 64) void combine_kernel(
    const u32x4* __restrict__ eo, const int32_t* __restrict__ pos, const float* __restrict__ gates,
    int64_t T, int Kr, int64_t nch, int64_t TK, u32x4* __restrict__ y, float* __restrict__ y32) {
    constexpr int KM = KC ? KC : kMaxK;
    const int K = KC ? KC : Kr;
    const int64_t groups = (nch + 63) / 64;
    // wave-uniform item index, so pos and gates come in through scalar loads
    const int64_t item = (int64_t)blockIdx.x * kCombineWaves +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (item >= T * groups) return;
    const int64_t t = item / groups;
    const int64_t c = (item - t * groups) * 64 + (threadIdx.x & 63);
    int p[KM];
    float g[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        p[j] = -1;
        g[j] = 0.f;
        if (j < K) {
            p[j] = pos[t * K + j];
            g[j] = gates[t * K + j];
        }
    }
    u32x4 v[KM];
    bool ok[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        ok[j] = p[j] >= 0 && p[j] < TK && c < nch;
        if (ok[j]) v[j] = __builtin_nontemporal_load(eo + (int64_t)p[j] * nch + c);
    }
    if (c >= nch) return;
    float acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.f;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        if (!ok[j]) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float lo = __uint_as_float(v[j][q] << 16);
            const float hi = __uint_as_float(v[j][q] & 0xffff0000u);
            acc[2 * q] = __builtin_fmaf(g[j], lo, acc[2 * q]);
            acc[2 * q + 1] = __builtin_fmaf(g[j], hi, acc[2 * q + 1]);
        }
    }
    u32x4 out;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        out[q] = f32_to_bf16_rne(acc[2 * q]) | (f32_to_bf16_rne(acc[2 * q + 1]) << 16);
    __builtin_nontemporal_store(out, y + t * nch + c);
    if (kF32) {
        float4* o = (float4*)(y32 + (t * nch + c) * 8);
        o[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        o[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    }
}

}  // namespace

cobalt_status launch_combine(const void* eo, const int32_t* pos, const float* gates, int64_t T,
                             int K, int64_t d, void* y, float* y32, hipStream_t s) {
    const int64_t nch = d / 8;
    const int64_t items = T * ((nch + 63) / 64);
    const dim3 grid((unsigned)((items + kCombineWaves - 1) / kCombineWaves));
    auto launch = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, grid, dim3(kCombineWaves * 64), 0, s, (const u32x4*)eo, pos,
                           gates, T, K, nch, T * K, (u32x4*)y, y32);
    };
    if (K == 8)
        y32 ? launch(combine_kernel<true, 8>) : launch(combine_kernel<false, 8>);
    else
        y32 ? launch(combine_kernel<true, 0>) : launch(combine_kernel<false, 0>);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

// ---------------------------------------------------------------- validation

namespace {

__global__ void zero_flag_kernel(uint32_t* f) { *f = 0; }

__global__ __launch_bounds__(256) void validate_kernel(const int32_t* __restrict__ topk,
                                                       const int32_t* __restrict__ src, int64_t T,
                                                       int K, int E, int G, uint32_t* flags) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= T) return;
    uint32_t f = 0;
    for (int j = 0; j < K; ++j) {
        const int e = topk[t * K + j];
        if (e < 0 || e >= E) f |= 1u;
        for (int i = 0; i < j; ++i)
            if (topk[t * K + i] == e) f |= 2u;
    }
    if (src) {
        const int s = src[t];
        if (s < 0 || s >= G) f |= 4u;
        if (t > 0 && src[t - 1] > s) f |= 8u;
    }
    if (f) atomicOr(flags, f);
}

}  // namespace

cobalt_status launch_validate(const int32_t* topk, const int32_t* src, int64_t T, int K, int E,
                              int G, uint32_t* dflags, hipStream_t s) {
    hipLaunchKernelGGL(zero_flag_kernel, dim3(1), dim3(1), 0, s, dflags);
    COBALT_LAUNCH_CHECK();
    hipLaunchKernelGGL(validate_kernel, dim3((unsigned)((T + 255) / 256)), dim3(256), 0, s, topk,
                       src, T, K, E, G, dflags);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

}  // namespace cobalt
