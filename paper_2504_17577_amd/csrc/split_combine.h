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
// per row, 4 consecutive elements each.
template <int D, bool OBF16>
__global__ __launch_bounds__(256) void combine_kernel(const float *Op, const float *Lp, void *O,
                                                      float *LSE, int n_rows, int n_split,
                                                      size_t o_split, size_t l_split)
{
    constexpr int TPR = D / 4;
    constexpr int RPB = 256 / TPR;
    const int t = threadIdx.x % TPR;
    const int row = blockIdx.x * RPB + threadIdx.x / TPR;
    if (row >= n_rows)
        return;
    float m = -INFINITY;
    for (int s = 0; s < n_split; ++s)
        m = fmaxf(m, Lp[s * l_split + row]);
    float4 acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    for (int s = 0; s < n_split; ++s) {
        const float ls = Lp[s * l_split + row];
        const float w = ls == -INFINITY ? 0.f : expf(ls - m);
        const float4 o = *(const float4 *)(Op + s * o_split + (size_t)row * D + 4 * t);
        acc.x += w * o.x;
        acc.y += w * o.y;
        acc.z += w * o.z;
        acc.w += w * o.w;
        wsum += w;
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
