// Merge of key-split partial results, shared by the attention and MLA
// decode entry points (internal to libtileattn).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace tileattn_detail {

typedef uint32_t cu32x2 __attribute__((ext_vector_type(2)));
typedef float cf32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 cbf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t combine_pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(cf32x2{lo, hi}, cbf16x2));
}

// Merge the partial results of the key splits of every row:
//   LSE = log sum_s exp(LSE_s),  O = sum_s exp(LSE_s - LSE) O_s,
// where (O_s, LSE_s) is the softmax result over the keys of split s alone
// (LSE_s = -inf, O_s = 0 for a split without a visible key).  D/4 threads
// per row, 4 consecutive elements each.  Up to UNROLL splits are read with
// all their loads issued before the first is used (the merge is bound by
// the latency of these loads, not by their bytes); more splits take further
// rounds of UNROLL.  The arithmetic is the same, in the same order, either way.
template <int D, bool OBF16>
__global__ __launch_bounds__(256) void combine_kernel(const float *Op, const float *Lp, void *O,
                                                      float *LSE, int n_rows, int n_split,
                                                      size_t o_split, size_t l_split)
{
    constexpr int TPR = D / 4;
    constexpr int RPB = 256 / TPR;
    constexpr int UNROLL = 8;
    const int t = threadIdx.x % TPR;
    const int row = blockIdx.x * RPB + threadIdx.x / TPR;
    if (row >= n_rows)
        return;
    float m = -INFINITY;
    for (int s0 = 0; s0 < n_split; s0 += UNROLL) {
        float ls[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
            ls[u] = s0 + u < n_split ? Lp[(s0 + u) * l_split + row] : -INFINITY;
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
            m = fmaxf(m, ls[u]);
    }
    float4 acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    for (int s0 = 0; s0 < n_split; s0 += UNROLL) {
        float ls[UNROLL];
        float4 o[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const bool in = s0 + u < n_split;
            ls[u] = in ? Lp[(s0 + u) * l_split + row] : -INFINITY;
            o[u] = in ? *(const float4 *)(Op + (s0 + u) * o_split + (size_t)row * D + 4 * t)
                      : float4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            if (s0 + u < n_split) {
                const float w = ls[u] == -INFINITY ? 0.f : expf(ls[u] - m);
                acc.x += w * o[u].x;
                acc.y += w * o[u].y;
                acc.z += w * o[u].z;
                acc.w += w * o[u].w;
                wsum += w;
            }
        }
    }
    const float inv = 1.f / wsum;
    const float x0 = acc.x * inv, x1 = acc.y * inv, x2 = acc.z * inv, x3 = acc.w * inv;
    if (OBF16) {
        const cu32x2 v = {combine_pack_bf16(x0, x1), combine_pack_bf16(x2, x3)};
        *(cu32x2 *)((uint16_t *)O + (size_t)row * D + 4 * t) = v;
    } else {
        *(float4 *)((float *)O + (size_t)row * D + 4 * t) = float4{x0, x1, x2, x3};
    }
    if (t == 0)
        LSE[row] = m + logf(wsum);
}

template <int D, bool OBF16>
hipError_t launch_combine(const float *Op, const float *Lp, void *O, float *LSE, int n_rows,
                          int n_split, size_t o_split, size_t l_split, hipStream_t stream)
{
    constexpr int RPB = 256 / (D / 4);
    hipLaunchKernelGGL((combine_kernel<D, OBF16>), dim3((n_rows + RPB - 1) / RPB), dim3(256), 0,
                       stream, Op, Lp, O, LSE, n_rows, n_split, o_split, l_split);
    return hipGetLastError();
}

}  // namespace tileattn_detail
