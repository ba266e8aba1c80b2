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

// Reductions over the 16 lanes of one MFMA row group (lanes 16g..16g+15), every lane receiving
// the result: DPP quad permutes (xor 1, xor 2) then row rotations by 4 and 8.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppRor4 = 0x124;    // row_ror:4
constexpr int kDppRor8 = 0x128;    // row_ror:8

__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dpp_f<kDppXor1>(x));
    x = fmaxf(x, dpp_f<kDppXor2>(x));
    x = fmaxf(x, dpp_f<kDppRor4>(x));
    x = fmaxf(x, dpp_f<kDppRor8>(x));
    return x;
}
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp_f<kDppXor1>(x);
    x += dpp_f<kDppXor2>(x);
    x += dpp_f<kDppRor4>(x);
    x += dpp_f<kDppRor8>(x);
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

// Wave-wide reductions through DPP within each 16-lane row and four readlanes across the rows
// (cheaper than a chain of LDS permutes; the same results, max and integer sums being exact).
__device__ __forceinline__ float wave_max_dpp(float x) {
    x = fmaxf(x, dpp_f<kDppXor1>(x));
    x = fmaxf(x, dpp_f<kDppXor2>(x));
    x = fmaxf(x, dpp_f<kDppRor4>(x));
    x = fmaxf(x, dpp_f<kDppRor8>(x));
    const int v = __float_as_int(x);
    return fmaxf(fmaxf(__int_as_float(__builtin_amdgcn_readlane(v, 0)), __int_as_float(__builtin_amdgcn_readlane(v, 16))),
                 fmaxf(__int_as_float(__builtin_amdgcn_readlane(v, 32)), __int_as_float(__builtin_amdgcn_readlane(v, 48))));
}
__device__ __forceinline__ int wave_sum_dpp(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, kDppXor1, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, kDppXor2, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, kDppRor4, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, kDppRor8, 0xf, 0xf, false);
    return __builtin_amdgcn_readlane(x, 0) + __builtin_amdgcn_readlane(x, 16) +
           __builtin_amdgcn_readlane(x, 32) + __builtin_amdgcn_readlane(x, 48);
}

// Inclusive prefix sum over the 64 lanes of a wave (lane order).
__device__ __forceinline__ int wave_inclusive_scan(int x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    return x;
}

// Orders this wave's LDS writes before its later LDS reads (one wave's LDS ops execute in order;
// this keeps the compiler from moving them across).
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Exclusive prefix sum over the workgroup (thread order) of x; *total receives the sum. One
// barrier: consecutive calls must alternate between the two halves of wsum[2][kWaves] (a wave
// reaching call k + 2 has passed call k + 1's barrier, so every wave has read call k's half).
template <int NW = kWaves>
__device__ __forceinline__ int wg_exclusive_scan(int x, int* wsum, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int incl = x;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const int s = wsum[w];
        before += w < wave ? s : 0;
        tot += s;
    }
    *total = tot;
    return before + incl - x;
}

// Work decomposition of the attention kernels: wave w owns tokens [16 (w mod 4), 16 (w mod 4) + 16)
// (one MFMA tile) of the 64-token blocks it handles. The dense kernel's 4-wave workgroups take every
// block of their run; the FFD kernels' 8-wave workgroups give waves w and w + 4 alternate kept
// blocks. Each wave keeps its own online-softmax state over its tiles, and the workgroup's states
// are merged in the epilogue.

// PV accumulators of one wave for 4 * NT heads: lane l holds dims 2l and 2l + 1 of every head;
// acc[h][e] is the unnormalised sum of p * v.
template <int NT>
struct PvAcc {
    float acc[4 * NT][2];
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int h = 0; h < 4 * NT; ++h) acc[h][0] = acc[h][1] = 0.f;
    }
};

// Per-wave LDS scratch for one tile: probabilities p[token][head] and per-head rescale factors.
template <int NT>
struct __attribute__((aligned(16))) TileP {
    float p[16][4 * NT];
    float corr[4 * NT];
};

// This lane's dword (dims 2l, 2l + 1) of the 16 value rows of a tile.
struct VTile {
    uint32_t v[16];
};

// Rows row0 .. row0 + 15 of v_bh (bf16 [rows][128]), each clamped to last_row: rows past the end
// of the sequence read the last valid row, a finite value whose probability is zero, so no select
// is needed and the loads stay unconditional (the compiler can count them).
__device__ __forceinline__ VTile load_vtile(const uint16_t* v_bh, int row0, int last_row, int lane) {
    const uint32_t* vp = reinterpret_cast<const uint32_t*>(v_bh) + lane;
    VTile r;
#pragma unroll
    for (int t = 0; t < 16; ++t) r.v[t] = vp[(size_t)min(row0 + t, last_row) * 64];
    return r;
}

// acc[h] = acc[h] * corr[h] + sum_t p[t][h] * v[t]. Tokens go in groups of four with a scheduling
// barrier between groups, so the compiler does not hoist all sixteen probability reads at once
// (which would cost ~64 registers).
template <int NT>
__device__ __forceinline__ void pv_tile(PvAcc<NT>& pv, const TileP<NT>& tp, const VTile& vt) {
#pragma unroll
    for (int h = 0; h < 4 * NT; ++h) {
        const float c = tp.corr[h];
        pv.acc[h][0] *= c;
        pv.acc[h][1] *= c;
    }
#pragma unroll
    for (int t0 = 0; t0 < 16; t0 += 4) {
#pragma unroll
        for (int t = t0; t < t0 + 4; ++t) {
            const float v0 = bf16_lo(vt.v[t]), v1 = bf16_hi(vt.v[t]);
#pragma unroll
            for (int q4 = 0; q4 < NT; ++q4) {
                const float4 p = *reinterpret_cast<const float4*>(&tp.p[t][4 * q4]);
                pv.acc[4 * q4 + 0][0] = fmaf(p.x, v0, pv.acc[4 * q4 + 0][0]);
                pv.acc[4 * q4 + 0][1] = fmaf(p.x, v1, pv.acc[4 * q4 + 0][1]);
                pv.acc[4 * q4 + 1][0] = fmaf(p.y, v0, pv.acc[4 * q4 + 1][0]);
                pv.acc[4 * q4 + 1][1] = fmaf(p.y, v1, pv.acc[4 * q4 + 1][1]);
                pv.acc[4 * q4 + 2][0] = fmaf(p.z, v0, pv.acc[4 * q4 + 2][0]);
                pv.acc[4 * q4 + 2][1] = fmaf(p.z, v1, pv.acc[4 * q4 + 2][1]);
                pv.acc[4 * q4 + 3][0] = fmaf(p.w, v0, pv.acc[4 * q4 + 3][0]);
                pv.acc[4 * q4 + 3][1] = fmaf(p.w, v1, pv.acc[4 * q4 + 3][1]);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Online-softmax update of one tile for the heads of this lane (head 4t + g, token n): keeps the
// running max m_run and per-lane partial sum l_part, and writes p and the rescale factor to LDS.
// Heads with use[t] false contribute p = 0 and keep their state.
template <int NT>
__device__ __forceinline__ void softmax_tile(const float (&z)[NT], const bool (&use)[NT], float (&m_run)[NT],
                                             float (&l_part)[NT], TileP<NT>& tp, int g, int n) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float corr = 1.f, p = 0.f;
        if (use[t]) {
            const float mn = fmaxf(m_run[t], row16_max(z[t]));
            if (mn != -INFINITY) {                   // a tile wholly past the end changes nothing
                corr = __expf(m_run[t] - mn);
                p = z[t] == -INFINITY ? 0.f : __expf(z[t] - mn);
                l_part[t] = fmaf(l_part[t], corr, p);
                m_run[t] = mn;
            }
        }
        tp.p[n][4 * t + g] = p;
        if (n == 0) tp.corr[4 * t + g] = corr;
    }
}

// Workgroup epilogue: combine the NW waves' (m, l, acc) and write one partial state per head.
// Head h (0 <= h < G) of the group goes to partial row row0 + h * head_stride. With out != null the
// workgroup holds the head's only partial state, so it writes the normalised bf16 output row
// out + h * kD and lse[h] (when lse != null) instead, as lse_merge_kernel would from that one row:
// out = acc / l, lse = m + ln l; no kept token gives out = 0 and lse = -inf.
template <int NT, int NW = kWaves>
struct EpilogueLds {
    float m[NW][4 * NT];
    float l[NW][4 * NT];
    float acc[NW][4 * NT][kD];
};

template <int NT, int NW = kWaves>
__device__ __forceinline__ void write_partials(EpilogueLds<NT, NW>& E, const PvAcc<NT>& pv,
                                               const float (&m_run)[NT], const float (&l_part)[NT],
                                               int wave, int lane, int G, size_t row0, size_t head_stride,
                                               float* part_m, float* part_l, float* part_acc,
                                               uint16_t* out = nullptr, float* lse = nullptr) {
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
        *reinterpret_cast<float2*>(&E.acc[wave][h][2 * lane]) = make_float2(pv.acc[h][0], pv.acc[h][1]);
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * kD; idx += 64 * NW) {
        const int h = idx >> 7, d = idx & (kD - 1);
        float mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < NW; ++w) mx = fmaxf(mx, E.m[w][h]);
        float l = 0.f, a = 0.f;
        if (mx != -INFINITY) {
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                const float mw = E.m[w][h];
                if (mw != -INFINITY) {
                    const float sc = __expf(mw - mx);
                    l = fmaf(sc, E.l[w][h], l);
                    a = fmaf(sc, E.acc[w][h][d], a);
                }
            }
        }
        if (out) {
            const bool any = mx != -INFINITY;
            out[(size_t)h * kD + d] = f32_to_bf16(a * (any ? 1.f / l : 0.f));
            if (lse && d == 0) lse[h] = any ? mx + logf(l) : -INFINITY;
            continue;
        }
        const size_t row = row0 + (size_t)h * head_stride;
        part_acc[row * kD + d] = a;
        if (d == 0) {
            part_m[row] = mx;
            part_l[row] = l;
        }
    }
}

// Log-sum-exp merge of `count` partial rows row0 + i * stride (i < count) of one head into its bf16
// output row and lse (Sec. 2, flash-decoding): M* = max m_i, l* = sum e^{m_i - M*} l_i,
// out = sum e^{m_i - M*} acc_i / l*, lse = M* + ln l*. Rows with m = -inf are skipped (their l and
// acc may hold anything); no row gives out = 0, lse = -inf. Run by all 256 threads of a workgroup: thread (d4, r) folds rows
// i = r (mod 8) of dims 4*d4 .. 4*d4 + 3, U rows at a time with the next U rows' loads already in
// flight (a head can have hundreds of partials), then the 8 threads of a d4 combine with shuffles.
constexpr int kMergeLanes = 8;

__device__ __forceinline__ void lse_fold(float& M, float& l, float4& acc, float m2, float l2, float4 a2) {
    if (m2 == -INFINITY) return;               // an empty row: its l and acc are not read
    const float mn = fmaxf(M, m2);
    const float c1 = __expf(M - mn), c2 = __expf(m2 - mn);
    l = l * c1 + l2 * c2;
    acc.x = acc.x * c1 + a2.x * c2;
    acc.y = acc.y * c1 + a2.y * c2;
    acc.z = acc.z * c1 + a2.z * c2;
    acc.w = acc.w * c1 + a2.w * c2;
    M = mn;
}

template <int U>
struct MergeBatch {
    float m[U], l[U];
    float4 a[U];
};

// Rows s0 + u * kMergeLanes (u < U) of the head, or empty rows (m = -inf) past count. The row
// index is clamped so the loads are unconditional.
template <int U>
__device__ __forceinline__ void load_merge_batch(MergeBatch<U>& bt, const float* __restrict__ part_m,
                                                 const float* __restrict__ part_l,
                                                 const float* __restrict__ part_acc, size_t row0,
                                                 size_t stride, int count, int s0, int d4) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int s = s0 + u * kMergeLanes;
        const size_t row = row0 + (size_t)min(s, count - 1) * stride;
        bt.m[u] = part_m[row];
        bt.l[u] = part_l[row];
        bt.a[u] = *reinterpret_cast<const float4*>(part_acc + row * kD + 4 * d4);
        if (s >= count) bt.m[u] = -INFINITY;
    }
}

__device__ __forceinline__ void merge_partial_rows(const float* __restrict__ part_m,
                                                   const float* __restrict__ part_l,
                                                   const float* __restrict__ part_acc, size_t row0,
                                                   size_t stride, int count, uint16_t* __restrict__ out_row,
                                                   float* __restrict__ lse_out) {
    const int d4 = threadIdx.x / kMergeLanes, r = threadIdx.x % kMergeLanes;
    float M = -INFINITY, l = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    constexpr int U = 8;
    constexpr int kStep = U * kMergeLanes;
    if (count > 0) {
        MergeBatch<U> cur, nxt;
        load_merge_batch<U>(cur, part_m, part_l, part_acc, row0, stride, count, r, d4);
        for (int s0 = r; s0 < count; s0 += kStep) {
            load_merge_batch<U>(nxt, part_m, part_l, part_acc, row0, stride, count, s0 + kStep, d4);
#pragma unroll
            for (int u = 0; u < U; ++u) lse_fold(M, l, acc, cur.m[u], cur.l[u], cur.a[u]);
            cur = nxt;
        }
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
        *reinterpret_cast<uint2*>(out_row + 4 * d4) = packed;
        if (lse_out && d4 == 0) *lse_out = any ? M + logf(l) : -INFINITY;
    }
}

}  // namespace ffd
