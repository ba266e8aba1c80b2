// Device-side helpers shared by the FFD and dense decode kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ffd {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kD = 128;        // head dimension
constexpr int kBlock = 64;     // KV block (tokens)
constexpr int kWaves = 4;      // waves per workgroup
constexpr int kThreads = 256;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bf16 bits, round to nearest even (inf/nan preserved)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Reductions over the 16 lanes of one MFMA row group (lanes 16g..16g+15).
__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, __shfl_xor(x, 1));
    x = fmaxf(x, __shfl_xor(x, 2));
    x = fmaxf(x, __shfl_xor(x, 4));
    x = fmaxf(x, __shfl_xor(x, 8));
    return x;
}
__device__ __forceinline__ float row16_sum(float x) {
    x += __shfl_xor(x, 1);
    x += __shfl_xor(x, 2);
    x += __shfl_xor(x, 4);
    x += __shfl_xor(x, 8);
    return x;
}
__device__ __forceinline__ float wave_max(float x) {
    for (int o = 1; o < 64; o <<= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}
__device__ __forceinline__ int wave_sum_i(int x) {
    for (int o = 1; o < 64; o <<= 1) x += __shfl_xor(x, o);
    return x;
}

// Orders this wave's LDS writes before its later LDS reads (one wave's LDS ops execute in order;
// this keeps the compiler from moving them across).
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Online-softmax state for the PV product of one wave, G_T = 4 * NT heads.
// Lane (g, n) = (lane >> 4, lane & 15) accumulates tokens t = g (mod 4) of every block, dims
// 8n..8n+7, for all heads. acc[h][e] is the unnormalised sum of p * v.
template <int NT>
struct PvAcc {
    float acc[4 * NT][8];
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int h = 0; h < 4 * NT; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    }
};

// Per-wave LDS scratch for one block: probabilities p[token][head] and per-head rescale factors.
template <int NT>
struct WaveP {
    float p[kBlock][4 * NT];
    float corr[4 * NT];
};

// acc[h] = acc[h] * corr[h] + sum over this lane's tokens of p[t][h] * V[t][8n..8n+7].
// vblk points at V row 0 of the block (bf16 [64][128]); tokens at or after `valid` have p = 0 and
// are skipped.
template <int NT>
__device__ __forceinline__ void pv_update(PvAcc<NT>& pv, const WaveP<NT>& wp, const uint16_t* vblk,
                                          int g, int n, int valid) {
#pragma unroll
    for (int h = 0; h < 4 * NT; ++h) {
        const float c = wp.corr[h];
#pragma unroll
        for (int e = 0; e < 8; ++e) pv.acc[h][e] *= c;
    }
    const uint4* vp = reinterpret_cast<const uint4*>(vblk) + n;   // 16 uint4 per 128-dim row
    uint4 vv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int t = 4 * i + g;
        vv[i] = t < valid ? vp[t * 16] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int t = 4 * i + g;
        float v[8];
        v[0] = bf16_lo(vv[i].x); v[1] = bf16_hi(vv[i].x);
        v[2] = bf16_lo(vv[i].y); v[3] = bf16_hi(vv[i].y);
        v[4] = bf16_lo(vv[i].z); v[5] = bf16_hi(vv[i].z);
        v[6] = bf16_lo(vv[i].w); v[7] = bf16_hi(vv[i].w);
#pragma unroll
        for (int h = 0; h < 4 * NT; ++h) {
            const float p = wp.p[t][h];
#pragma unroll
            for (int e = 0; e < 8; ++e) pv.acc[h][e] = fmaf(p, v[e], pv.acc[h][e]);
        }
    }
}

// Workgroup epilogue: combine the four waves' (m, l, acc) and write this split's partial state.
// m_w[h], l_w[h] are row-uniform per head (lane n == 0 of row g holds head 4t + g); pv holds
// per-lane partial sums over tokens t = g (mod 4).
template <int NT>
struct EpilogueLds {
    float m[kWaves][4 * NT];
    float l[kWaves][4 * NT];
    float acc[kWaves][4 * NT][kD];
};

template <int NT>
__device__ __forceinline__ void write_partials(EpilogueLds<NT>& E, PvAcc<NT>& pv,
                                               const float (&m_run)[NT], const float (&l_part)[NT],
                                               int wave, int lane, int G, int hq0, int Hq, int S,
                                               int b, int s, float* part_m, float* part_l,
                                               float* part_acc) {
    const int g = lane >> 4, n = lane & 15;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const float l = row16_sum(l_part[t]);
        if (n == 0) {
            E.m[wave][4 * t + g] = m_run[t];
            E.l[wave][4 * t + g] = l;
        }
    }
#pragma unroll
    for (int h = 0; h < 4 * NT; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float x = pv.acc[h][e];
            x += __shfl_xor(x, 16);
            x += __shfl_xor(x, 32);
            pv.acc[h][e] = x;
        }
    if (g == 0) {
#pragma unroll
        for (int h = 0; h < 4 * NT; ++h)
#pragma unroll
            for (int e = 0; e < 8; ++e) E.acc[wave][h][8 * n + e] = pv.acc[h][e];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * kD; idx += kThreads) {
        const int h = idx >> 7, d = idx & (kD - 1);
        float mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, E.m[w][h]);
        float l = 0.f, a = 0.f;
        if (mx != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                const float mw = E.m[w][h];
                if (mw != -INFINITY) {
                    const float sc = __expf(mw - mx);
                    l = fmaf(sc, E.l[w][h], l);
                    a = fmaf(sc, E.acc[w][h][d], a);
                }
            }
        }
        const size_t row = ((size_t)b * Hq + hq0 + h) * S + s;
        part_acc[row * kD + d] = a;
        if (d == 0) {
            part_m[row] = mx;
            part_l[row] = l;
        }
    }
}

}  // namespace ffd
