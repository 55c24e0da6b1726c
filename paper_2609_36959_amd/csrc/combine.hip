// Combine and weighted sum (Fig. 1, last stage):
//   y[t][c] = bf16_rne( sum_j gates[t][j] * expert_out[pos[t][j]][c] ),
// accumulated in fp32 from 0 with one fused multiply-add per slot in slot
// order; slots whose row is outside [0, T*K) are skipped.
//
// fold_kernel: one workgroup per (token, 2 KiB column slice), one wave per
// slot j (at least two waves). Wave j loads its row's slice (non-temporal,
// two 16-byte chunks per lane) into LDS; after a barrier two waves fold the
// K slices in slot order, one 16-byte chunk (eight bf16 values) per thread,
// and store the slice of y. Each wave has a single row to fetch, so many
// independent row loads are in flight; on the T=131072, K=8, d=7168
// workload this runs at 6.5-6.6 TB/s, against 5.6 TB/s for combine_kernel.
// Four folding waves storing 8 bytes per thread took 3 % longer, and one
// wave folding two chunks per lane holds the stage longer still.
//
// combine_kernel (other shapes): each wave takes one (token, 1 KiB slice)
// and loads the chunks of all K rows itself, issuing every load before its
// single store so that no load waits behind a store.
//
// The node-level combine (the reverse of the node-deduplicated dispatch)
// follows: node_fold_kernel sums each node's slots into a bf16 partial row,
// node_sum_kernel sums a token's partial rows in node order.
#include <algorithm>

#include "internal.hpp"

namespace cobalt {
namespace {

constexpr int kCombineWaves = 16;
constexpr int kFoldWaves = 2;  // waves that fold or sum a staged slice (128 chunks, one per thread)
constexpr int kNodeWaves = 4;  // least waves of node_fold_kernel; waves of node_sum_kernel

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Rounds a and b to bf16, nearest even, and packs them with a in the low
// half: one v_cvt_pk_bf16_f32. In the floating-point mode of these kernels
// (IEEE, fp32 denormals kept) it gives the bits of the IEEE-754 rule written
// out (a quiet NaN keeps its sign and the top bits of its payload) on every
// one of the 2^32 inputs, and costs one instruction where the bit rule
// costs about ten for the pair.
__device__ __forceinline__ uint32_t pack_bf16_rne(float a, float b) {
    const f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
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
        out[q] = pack_bf16_rne(acc[2 * q], acc[2 * q + 1]);
    __builtin_nontemporal_store(out, y + t * nch + c);
    if (kF32) {
        float4* o = (float4*)(y32 + (t * nch + c) * 8);
        o[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        o[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    }
}

// GROUPS = slices of 128 chunks per row, a template parameter so that the
// block index splits into (token, slice) with a constant division.
template <bool kF32, int GROUPS>
__global__ __launch_bounds__(kMaxK * 64) void fold_kernel(
    const u32x4* __restrict__ eo, const int32_t* __restrict__ pos, const float* __restrict__ gates,
    int K, int64_t nch, int64_t TK, u32x4* __restrict__ y, float* __restrict__ y32) {
    // K slices of 128 chunks (K * 2 KiB, sized at launch): a small stage
    // lets further workgroups start on a CU once the loading waves of a
    // workgroup have exited, which the wave count alone would not limit
    extern __shared__ u32x4 stage[];
    __shared__ float gate[kMaxK];
    __shared__ int valid[kMaxK];
    const uint32_t tg = blockIdx.x;
    const uint32_t t = tg / GROUPS;
    const uint32_t g = tg - t * GROUPS;
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int64_t c0 = (int64_t)g * 128 + lane;
    const bool in0 = c0 < nch, in1 = c0 + 64 < nch;
    if (j < K) {
        const int p = pos[(int64_t)t * K + j];
        const bool ok = p >= 0 && p < TK;
        // both loads are issued before either LDS write: a write right after
        // its own load would make the second load wait for the first
        const u32x4* row = eo + (int64_t)(ok ? p : 0) * nch;
        u32x4 v0, v1;
        if (ok && in0) v0 = __builtin_nontemporal_load(row + c0);
        if (ok && in1) v1 = __builtin_nontemporal_load(row + c0 + 64);
        if (ok && in0) stage[j * 128 + lane] = v0;
        if (ok && in1) stage[j * 128 + lane + 64] = v1;
        const float gj = gates[(int64_t)t * K + j];
        if (lane == 0) {
            valid[j] = ok;
            gate[j] = gj;
        }
    }
    __syncthreads();
    // kFoldWaves waves fold: thread i takes chunk i of the slice (eight bf16
    // values), summing the K slots in slot order, and stores 16 bytes of y
    if (j >= kFoldWaves) return;
    const int i = threadIdx.x;
    const int64_t c = (int64_t)g * 128 + i;
    if (c >= nch) return;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < K; ++k) {
        if (!valid[k]) continue;
        const float gk = gate[k];
        const u32x4 v = stage[k * 128 + i];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            acc[2 * q] = __builtin_fmaf(gk, __uint_as_float(v[q] << 16), acc[2 * q]);
            acc[2 * q + 1] = __builtin_fmaf(gk, __uint_as_float(v[q] & 0xffff0000u), acc[2 * q + 1]);
        }
    }
    u32x4 out;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        out[q] = pack_bf16_rne(acc[2 * q], acc[2 * q + 1]);
    __builtin_nontemporal_store(out, y + (int64_t)t * nch + c);
    if (kF32) {
        float4* o = (float4*)(y32 + ((int64_t)t * nch + c) * 8);
        o[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        o[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    }
}

template <bool kF32, int GROUPS>
bool try_fold(const void* eo, const int32_t* pos, const float* gates, int64_t T, int K,
              int64_t nch, void* y, float* y32, hipStream_t s) {
    if constexpr (GROUPS == 0) {
        return false;  // wider rows: combine_kernel
    } else {
        if ((nch + 127) / 128 != GROUPS)
            return try_fold<kF32, GROUPS - 1>(eo, pos, gates, T, K, nch, y, y32, s);
        const int threads = std::max(K, kFoldWaves) * 64;
        for_token_ranges(T, (int64_t)GROUPS * threads, [&](int64_t t0, int64_t n) {
            hipLaunchKernelGGL((fold_kernel<kF32, GROUPS>), dim3((unsigned)(n * GROUPS)),
                               dim3(threads), (size_t)K * 128 * sizeof(u32x4), s,
                               (const u32x4*)eo, pos + t0 * K, gates + t0 * K, K, nch, T * K,
                               (u32x4*)y + t0 * nch, y32 ? y32 + t0 * nch * 8 : nullptr);
        });
        return true;
    }
}

// Node side of the node-level combine: one workgroup per (token, 2 KiB
// column slice), one wave per slot j (at least four waves). Wave j loads its
// row's slice like fold_kernel and records its gate and its rank's node;
// after a barrier each wave folds whole node rows: for each node the token
// reaches, the slots on that node in slot order, stored as the bf16 partial
// in the token's row for that node. GROUPS as for fold_kernel.
template <int GROUPS>
__global__ __launch_bounds__(kMaxK * 64) void node_fold_kernel(
    const u32x4* __restrict__ eo, const int32_t* __restrict__ pos,
    const int32_t* __restrict__ assigned, const float* __restrict__ gates,
    const int32_t* __restrict__ node_pos, int K, int N, int gpn, int64_t nch, int64_t TK,
    int64_t node_rows, int groups_rt, u32x4* __restrict__ partial) {
    extern __shared__ u32x4 stage[];
    __shared__ float gate[kMaxK];
    __shared__ int slot_node[kMaxK];  // node of slot j's rank, -1 for a skipped slot
    __shared__ int nrow[kMaxN];       // row of (t, n) in partial, -1 if none
    const uint32_t groups = GROUPS ? GROUPS : (uint32_t)groups_rt;
    const uint32_t tg = blockIdx.x;
    const uint32_t t = tg / groups;
    const uint32_t g = tg - t * groups;
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int64_t c0 = (int64_t)g * 128 + lane;
    const bool in0 = c0 < nch, in1 = c0 + 64 < nch;
    if (j < K) {
        const int p = pos[(int64_t)t * K + j];
        const int r = assigned[(int64_t)t * K + j];
        const bool ok = p >= 0 && p < TK && r >= 0 && r < N * gpn;
        const u32x4* row = eo + (int64_t)(ok ? p : 0) * nch;
        u32x4 v0, v1;
        if (ok && in0) v0 = __builtin_nontemporal_load(row + c0);
        if (ok && in1) v1 = __builtin_nontemporal_load(row + c0 + 64);
        if (ok && in0) stage[j * 128 + lane] = v0;
        if (ok && in1) stage[j * 128 + lane + 64] = v1;
        const float gj = gates[(int64_t)t * K + j];
        if (lane == 0) {
            gate[j] = gj;
            slot_node[j] = ok ? r / gpn : -1;
        }
    }
    if (j == 0 && lane < N) {
        const int q = node_pos[(int64_t)t * N + lane];
        nrow[lane] = q >= 0 && q < node_rows ? q : -1;
    }
    __syncthreads();
    // Wave w folds the rows of nodes w, w + waves, ...: for each, it sums the
    // node's slots in slot order over its two chunks per lane and stores the
    // row's 2 KiB slice itself (splitting a row over four waves, eight bytes
    // per lane, took 3 % longer).
    const int waves = blockDim.x >> 6;
    for (int n = j; n < N; n += waves) {
        const int q = nrow[n];
        if (q < 0) continue;
        float acc[2][8];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
        for (int k = 0; k < K; ++k) {
            if (slot_node[k] != n) continue;
            const float gk = gate[k];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const u32x4 v = stage[k * 128 + lane + 64 * h];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[h][2 * e] = __builtin_fmaf(gk, __uint_as_float(v[e] << 16), acc[h][2 * e]);
                    acc[h][2 * e + 1] =
                        __builtin_fmaf(gk, __uint_as_float(v[e] & 0xffff0000u), acc[h][2 * e + 1]);
                }
            }
        }
        u32x4* dst = partial + (int64_t)q * nch;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if (!(h == 0 ? in0 : in1)) continue;
            u32x4 out;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                out[e] = pack_bf16_rne(acc[h][2 * e], acc[h][2 * e + 1]);
            __builtin_nontemporal_store(out, dst + c0 + 64 * h);
        }
    }
}

template <int GROUPS>
void launch_node_fold(const void* eo, const int32_t* pos, const int32_t* assigned,
                      const float* gates, const int32_t* node_pos, int64_t T, int K, int N,
                      int gpn, int64_t nch, int64_t node_rows, void* partial, hipStream_t s) {
    const int64_t groups = (nch + 127) / 128;
    if constexpr (GROUPS > 0) {
        if (groups != GROUPS)
            return launch_node_fold<GROUPS - 1>(eo, pos, assigned, gates, node_pos, T, K, N, gpn,
                                                nch, node_rows, partial, s);
    }
    const int threads = std::max(K, kNodeWaves) * 64;
    for_token_ranges(T, groups * threads, [&](int64_t t0, int64_t n) {
        hipLaunchKernelGGL(node_fold_kernel<GROUPS>, dim3((unsigned)(n * groups)), dim3(threads),
                           (size_t)K * 128 * sizeof(u32x4), s, (const u32x4*)eo, pos + t0 * K,
                           assigned + t0 * K, gates + t0 * K, node_pos + t0 * N, K, N, gpn, nch,
                           T * K, node_rows, (int)groups, (u32x4*)partial);
    });
}

// Source side of the node-level combine: one workgroup of four waves per
// (token, 2 KiB column slice). Wave j loads the node rows n = j, j + 4, ...
// (SPW of them at most) that node_pos names for the token; after a barrier
// two waves sum the staged rows in increasing n, one 16-byte chunk per
// thread, and store the slice of y (four waves at 8 bytes per thread were
// no faster). A token reaches only about
// half of the nodes, so one loading wave per node would leave half the
// waves idle at the barrier (1.91 ms against 1.65 ms on the T=131072, N=8,
// d=7168 workload).
// GROUPS as for node_fold_kernel.
template <int GROUPS, int SPW>
__global__ __launch_bounds__(kNodeWaves * 64) void node_sum_kernel(
    const u32x4* __restrict__ partial, const int32_t* __restrict__ node_pos, int N, int64_t nch,
    int64_t node_rows, int groups_rt, u32x4* __restrict__ y) {
    extern __shared__ u32x4 stage[];
    __shared__ int valid[kMaxN];
    const uint32_t groups = GROUPS ? GROUPS : (uint32_t)groups_rt;
    const uint32_t tg = blockIdx.x;
    const uint32_t t = tg / groups;
    const uint32_t g = tg - t * groups;
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int64_t c0 = (int64_t)g * 128 + lane;
    // Lanes past the end of a ragged last slice load chunk 0 instead and
    // stage values that no thread sums: with no lane-dependent branch around
    // the loads, every row load is issued before the first wait (guarded
    // loads here each waited for the one before).
    const int64_t c0a = c0 < nch ? c0 : 0, c0b = c0 + 64 < nch ? c0 + 64 : 0;
    u32x4 v[SPW][2];
    bool ok[SPW];
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
        const int n = j + kNodeWaves * i;
        const int q = n < N ? node_pos[(int64_t)t * N + n] : -1;
        ok[i] = q >= 0 && q < node_rows;
        if (ok[i]) {
            const u32x4* row = partial + (int64_t)q * nch;
            v[i][0] = __builtin_nontemporal_load(row + c0a);
            v[i][1] = __builtin_nontemporal_load(row + c0b);
        }
    }
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
        const int n = j + kNodeWaves * i;
        if (n < N) {
            if (ok[i]) {
                stage[n * 128 + lane] = v[i][0];
                stage[n * 128 + lane + 64] = v[i][1];
            }
            if (lane == 0) valid[n] = ok[i];
        }
    }
    __syncthreads();
    // kFoldWaves waves sum: thread i takes chunk i of the slice
    if (j >= kFoldWaves) return;
    const int i = threadIdx.x;
    const int64_t c = (int64_t)g * 128 + i;
    if (c >= nch) return;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int n = 0; n < N; ++n) {
        if (!valid[n]) continue;
        const u32x4 a = stage[n * 128 + i];
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            acc[2 * h] += __uint_as_float(a[h] << 16);
            acc[2 * h + 1] += __uint_as_float(a[h] & 0xffff0000u);
        }
    }
    u32x4 out;
#pragma unroll
    for (int h = 0; h < 4; ++h)
        out[h] = pack_bf16_rne(acc[2 * h], acc[2 * h + 1]);
    __builtin_nontemporal_store(out, y + (int64_t)t * nch + c);
}

template <int GROUPS>
void launch_node_sum(const void* partial, const int32_t* node_pos, int64_t T, int N, int64_t nch,
                     int64_t node_rows, void* y, hipStream_t s) {
    const int64_t groups = (nch + 127) / 128;
    if constexpr (GROUPS > 0) {
        if (groups != GROUPS)
            return launch_node_sum<GROUPS - 1>(partial, node_pos, T, N, nch, node_rows, y, s);
    }
    const dim3 block(kNodeWaves * 64);
    const size_t lds = (size_t)N * 128 * sizeof(u32x4);
    for_token_ranges(T, groups * kNodeWaves * 64, [&](int64_t t0, int64_t n) {
        const dim3 grid((unsigned)(n * groups));
        if (N <= 2 * kNodeWaves)
            hipLaunchKernelGGL((node_sum_kernel<GROUPS, 2>), grid, block, lds, s,
                               (const u32x4*)partial, node_pos + t0 * N, N, nch, node_rows,
                               (int)groups, (u32x4*)y + t0 * nch);
        else
            hipLaunchKernelGGL((node_sum_kernel<GROUPS, 4>), grid, block, lds, s,
                               (const u32x4*)partial, node_pos + t0 * N, N, nch, node_rows,
                               (int)groups, (u32x4*)y + t0 * nch);
    });
}

}  // namespace

cobalt_status launch_combine(const void* eo, const int32_t* pos, const float* gates, int64_t T,
                             int K, int64_t d, void* y, float* y32, hipStream_t s) {
    const int64_t nch = d / 8;
    if (y32 ? try_fold<true, 16>(eo, pos, gates, T, K, nch, y, y32, s)
            : try_fold<false, 16>(eo, pos, gates, T, K, nch, y, y32, s)) {
        COBALT_LAUNCH_CHECK();
        return COBALT_OK;
    }
    const int64_t g64 = (nch + 63) / 64;  // one wave per (token, 1 KiB slice)
    auto launch = [&](auto kernel) {
        for_token_ranges(T, g64 * 64, [&](int64_t t0, int64_t n) {
            const int64_t items = n * g64;
            hipLaunchKernelGGL(kernel, dim3((unsigned)((items + kCombineWaves - 1) / kCombineWaves)),
                               dim3(kCombineWaves * 64), 0, s, (const u32x4*)eo, pos + t0 * K,
                               gates + t0 * K, n, K, nch, T * K, (u32x4*)y + t0 * nch,
                               y32 ? y32 + t0 * nch * 8 : nullptr);
        });
    };
    if (K == 8)
        y32 ? launch(combine_kernel<true, 8>) : launch(combine_kernel<false, 8>);
    else
        y32 ? launch(combine_kernel<true, 0>) : launch(combine_kernel<false, 0>);
    COBALT_LAUNCH_CHECK();
    return COBALT_OK;
}

cobalt_status launch_node_combine(const void* eo, const int32_t* pos, const int32_t* assigned,
                                  const float* gates, const int32_t* node_pos, int64_t T, int K,
                                  int N, int gpn, int64_t d, void* partial, void* y,
                                  hipStream_t s) {
    const int64_t nch = d / 8;
    const int64_t node_rows = T * std::min(K, N);
    launch_node_fold<16>(eo, pos, assigned, gates, node_pos, T, K, N, gpn, nch, node_rows,
                         partial, s);
    COBALT_LAUNCH_CHECK();
    // source side: y[t] = sum over n of partial[node_pos[t][n]], n increasing
    launch_node_sum<16>(partial, node_pos, T, N, nch, node_rows, y, s);
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
