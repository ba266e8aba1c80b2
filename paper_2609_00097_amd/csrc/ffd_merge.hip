// Log-sum-exp merge of split partials (the flash-decoding reduction, Sec. 2): for each (sequence,
// query head), M* = max_s m_s, l* = sum_s e^{m_s - M*} l_s, out = sum_s e^{m_s - M*} acc_s / l*,
// lse = M* + ln l*. Splits that kept nothing carry m = -inf and are skipped; a head with no split
// gets out = 0 and lse = -inf.
//
// Partial rows of head bh = b * Hq + h: without a table, rows bh * S + s for s < S (the dense path's
// fixed splits); with a table (the FFD path), rows (first + i) * G + bh % G for i < count, where
// (first, count) = table[bh / G] describes the refinement workgroups given to that KV group.
//
// Mapping: one workgroup per (sequence, query head); thread (d4, r) folds the splits s = r (mod 8)
// of dims 4*d4..4*d4+3 into an online (max, sum, acc) with 8 float4 loads in flight, then the
// 8 threads of a d4 combine with shuffles.
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

constexpr int kMergeLanes = 8;     // threads per 4-dim group

__device__ __forceinline__ void lse_fold(float& M, float& l, float4& acc, float m2, float l2, float4 a2) {
    const float mn = fmaxf(M, m2);
    if (mn == -INFINITY) return;
    const float c1 = __expf(M - mn), c2 = __expf(m2 - mn);
    l = l * c1 + l2 * c2;
    acc.x = acc.x * c1 + a2.x * c2;
    acc.y = acc.y * c1 + a2.y * c2;
    acc.z = acc.z * c1 + a2.z * c2;
    acc.w = acc.w * c1 + a2.w * c2;
    M = mn;
}

}  // namespace

__global__ __launch_bounds__(kThreads) void lse_merge_kernel(const float* __restrict__ part_m,
                                                             const float* __restrict__ part_l,
                                                             const float* __restrict__ part_acc, int S,
                                                             const int2* __restrict__ table, int G,
                                                             uint16_t* __restrict__ out, float* __restrict__ lse) {
    size_t row0 = (size_t)blockIdx.x * S, stride = 1;      // blockIdx.x = b * Hq + h
    if (table) {
        const int2 fc = table[blockIdx.x / G];
        row0 = (size_t)fc.x * G + blockIdx.x % G;
        stride = (size_t)G;
        S = fc.y;
    }
    const int d4 = threadIdx.x / kMergeLanes, r = threadIdx.x % kMergeLanes;
    float M = -INFINITY, l = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    constexpr int U = 8;
    for (int s0 = r; s0 < S; s0 += U * kMergeLanes) {
        float ms[U], ls[U];
        float4 as[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = s0 + u * kMergeLanes;
            ms[u] = -INFINITY;
            ls[u] = 0.f;
            as[u] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (s < S) {
                const size_t row = row0 + (size_t)s * stride;
                ms[u] = part_m[row];
                ls[u] = part_l[row];
                as[u] = *reinterpret_cast<const float4*>(part_acc + row * kD + 4 * d4);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) lse_fold(M, l, acc, ms[u], ls[u], as[u]);
    }
#pragma unroll
    for (int o = 1; o < kMergeLanes; o <<= 1) {
        const float M2 = __shfl_xor(M, o), l2 = __shfl_xor(l, o);
        const float4 a2 = make_float4(__shfl_xor(acc.x, o), __shfl_xor(acc.y, o), __shfl_xor(acc.z, o),
                                      __shfl_xor(acc.w, o));
        lse_fold(M, l, acc, M2, l2, a2);
    }
    if (r == 0) {
        const bool any = M != -INFINITY;
        const float inv = any ? 1.f / l : 0.f;
        uint2 packed;
        packed.x = (uint32_t)f32_to_bf16(acc.x * inv) | ((uint32_t)f32_to_bf16(acc.y * inv) << 16);
        packed.y = (uint32_t)f32_to_bf16(acc.z * inv) | ((uint32_t)f32_to_bf16(acc.w * inv) << 16);
        *reinterpret_cast<uint2*>(out + (size_t)blockIdx.x * kD + 4 * d4) = packed;
        if (lse && d4 == 0) lse[blockIdx.x] = any ? M + logf(l) : -INFINITY;
    }
}

}  // namespace ffd
