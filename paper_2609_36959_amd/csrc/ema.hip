// Planner statistics on the device (Section 3.2): exponential moving
// averages of the step's counts, and the Ochiai similarity of expert pairs
// (Section 1, the footnote on Fig. 3).
//
// One EMA update of m with the step's count x, in fp32:
//     init:      m = x
//     otherwise: m = fma(decay, m, (1 - decay) * x),
// with x the count rounded to fp32 and 1 - decay rounded once. Ochiai from
// co-activation counts c and expert counts n:
//     O_ij = c_ij / sqrt(n_i * n_j),   O_ii = 1 for an active expert,
// 0 where the pair shares no token or an expert is inactive; every
// operation is one correctly rounded fp32 operation (hipcc's default
// division and square root), with no contraction.
//
// coact_ema_kernel makes one pass over the E x E counts: it reads c_ij and
// the two expert counts, writes O_ij and the EMA of c_ij, and clears c_ij.
// The expert counts are updated and cleared by count_ema_kernel, launched
// after it in stream order, so no thread reads a count another has cleared.
#include <cmath>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kEmaThreads = 256;

__device__ __forceinline__ float ema_step(float m, uint32_t x, float decay, float gain,
                                          bool init) {
#pragma clang fp contract(off)
    const float xf = (float)x;
    return init ? xf : __builtin_fmaf(decay, m, gain * xf);
}

__global__ __launch_bounds__(kEmaThreads) void coact_ema_kernel(
    uint32_t* __restrict__ coact, const uint32_t* __restrict__ count, int E, float decay,
    float gain, int init, int clear, float* __restrict__ ema, float* __restrict__ ochiai) {
#pragma clang fp contract(off)
    const int64_t idx = (int64_t)blockIdx.x * kEmaThreads + threadIdx.x;
    if (idx >= (int64_t)E * E) return;
    const int i = (int)(idx / E);
    const int j = (int)(idx - (int64_t)i * E);
    const uint32_t c = coact[idx];
    if (ochiai) {
        const uint32_t ni = count[i], nj = count[j];
        const uint32_t common = i == j ? ni : c;
        float o = 0.f;
        if (common != 0 && ni != 0 && nj != 0) o = (float)common / sqrtf((float)ni * (float)nj);
        ochiai[idx] = o;
    }
    if (ema) ema[idx] = ema_step(ema[idx], c, decay, gain, init != 0);
    if (clear) coact[idx] = 0;
}

__global__ __launch_bounds__(kEmaThreads) void count_ema_kernel(uint32_t* __restrict__ counts,
                                                                int64_t n, float decay,
                                                                float gain, int init, int clear,
                                                                float* __restrict__ ema) {
    const int64_t i = (int64_t)blockIdx.x * kEmaThreads + threadIdx.x;
    if (i >= n) return;
    const uint32_t x = counts[i];
    if (ema) ema[i] = ema_step(ema[i], x, decay, gain, init != 0);
    if (clear) counts[i] = 0;
}

unsigned blocks_for(int64_t n) { return (unsigned)((n + kEmaThreads - 1) / kEmaThreads); }

}  // namespace

cobalt_status launch_count_ema(uint32_t* counts, int64_t n, float decay, bool init, bool clear,
                               float* ema, hipStream_t s) {
    if (n == 0 || (!ema && !clear)) return COBALT_OK;
    const float gain = 1.0f - decay;
    hipLaunchKernelGGL(count_ema_kernel, dim3(blocks_for(n)), dim3(kEmaThreads), 0, s, counts, n,
                       decay, gain, (int)init, (int)clear, ema);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

cobalt_status launch_coact_ema(uint32_t* coact, uint32_t* count, int E, float decay, bool init,
                               bool clear, float* ema_coact, float* ema_count, float* ochiai,
                               hipStream_t s) {
    const float gain = 1.0f - decay;
    if (ema_coact || ochiai || clear) {
        hipLaunchKernelGGL(coact_ema_kernel, dim3(blocks_for((int64_t)E * E)), dim3(kEmaThreads),
                           0, s, coact, count, E, decay, gain, (int)init, (int)clear, ema_coact,
                           ochiai);
        COBALT_LAUNCH_CHECK();
    }
    return launch_count_ema(count, E, decay, init, clear, ema_count, s);
}

}  // namespace cobalt
