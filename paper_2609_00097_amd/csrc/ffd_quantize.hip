// Key quantization for gfx950 (Sec. 3.1; App. A): each bf16 key vector of 128 dims becomes 2-bit
// codes on the scale s = M/1.5 (M = max |k_i|, nearest level of {-1.5,-0.5,0.5,1.5}, ties to the
// upper level), the absmax M, and an int8 residual r = rint(381 k / M) - 254 c + 381.
//
// Exactness: 3k, 2M and 381k are exact in fp32 for bf16 k and M, so the code decisions are exact
// comparisons; 381k / M is one correctly rounded fp32 division, which cannot move a value across a
// half-integer (381k has at most 17 significant bits and M at most 8, so a non-tie sits at least
// 2^-18 relatively away from the nearest half-integer, far above fp32 rounding), so rintf gives
// the exact round-half-even result.
//
// Mapping: 16 lanes per token, each lane owns 8 consecutive dims (one 16-byte load); the absmax is
// a 16-lane max reduction. Writes go straight into the storage layouts documented in ffd.h.
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

// One token's quantization by 16 lanes: lane j16 holds dims 8*j16 .. 8*j16 + 7 as one 16-byte
// chunk of bf16 (raw). All 16 lanes must be active. Returns the token's absmax M in every lane;
// word = the 16 codes of the lane pair's 16-dim group (identical in both lanes of the pair), rlo/rhi =
// the lane's 8 int8 residuals.
struct QuantToken {
    float m;
    uint32_t word, rlo, rhi;
};

__device__ __forceinline__ QuantToken quantize_token(uint4 raw, int j16) {
    float x[8];
    x[0] = bf16_lo(raw.x); x[1] = bf16_hi(raw.x);
    x[2] = bf16_lo(raw.y); x[3] = bf16_hi(raw.y);
    x[4] = bf16_lo(raw.z); x[5] = bf16_hi(raw.z);
    x[6] = bf16_lo(raw.w); x[7] = bf16_hi(raw.w);
    float m = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(x[e]));
    m = fmaxf(m, __shfl_xor(m, 1));
    m = fmaxf(m, __shfl_xor(m, 2));
    m = fmaxf(m, __shfl_xor(m, 4));
    m = fmaxf(m, __shfl_xor(m, 8));

    const float two_m = 2.f * m;
    uint32_t word = 0, rlo = 0, rhi = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float xv = x[e];
        const float x3 = 3.f * xv;
        int c = x3 >= two_m ? 3 : (xv >= 0.f ? 2 : (x3 >= -two_m ? 1 : 0));
        int r = 0;
        if (m == 0.f) {
            c = 2;
        } else {
            r = (int)rintf((381.f * xv) / m) - 254 * c + 381;
        }
        const int e16 = 8 * (j16 & 1) + e;              // position inside the 16-dim group
        word |= (uint32_t)c << (8 * (e16 & 3) + 2 * (e16 >> 2));
        const uint32_t rb = (uint32_t)(r & 0xff);
        if (e < 4) rlo |= rb << (8 * e); else rhi |= rb << (8 * (e - 4));
    }
    word |= __shfl_xor(word, 1);                        // the pair of lanes covering 16 dims
    return QuantToken{m, word, rlo, rhi};
}

// Store token t of (b, kvh) = row bh into the codes / absmax / residual layouts (lane j16's share).
__device__ __forceinline__ void store_token(const QuantToken& qt, int j16, size_t bh, int t, int Lcap,
                                            uint32_t* codes, uint16_t* absmax, int8_t* resid) {
    const int n16 = t & 15;
    if ((j16 & 1) == 0) {
        const int w = j16 >> 1;                         // 16-dim group 0..7
        const int cc = w >> 2, g = w & 3;
        codes[((bh * (size_t)(Lcap / 64) + (t >> 6)) * 64 + n16 + 16 * g) * 8 + 2 * ((t >> 4) & 3) + cc] = qt.word;
    }
    {
        const int cc = j16 >> 3, g = (j16 & 7) >> 1, e0 = 8 * (j16 & 1);
        int8_t* dst = resid + (((bh * (size_t)(Lcap / 16) + (t >> 4)) * 2 + cc) * 64 + n16 + 16 * g) * 16 + e0;
        *reinterpret_cast<uint2*>(dst) = make_uint2(qt.rlo, qt.rhi);
    }
    if (j16 == 0)
        absmax[bh * (size_t)Lcap + (size_t)(t >> 6) * 64 + n16 * 4 + ((t >> 4) & 3)] =
            (uint16_t)(__float_as_uint(qt.m) >> 16);
}

}  // namespace

__global__ __launch_bounds__(kThreads) void quantize_keys_kernel(QuantArgs a) {
    const int tid = threadIdx.x, j16 = tid & 15;
    const int t = a.t_begin + blockIdx.x * 16 + (tid >> 4);
    const int kvh = blockIdx.y, b = blockIdx.z;
    const size_t bh = (size_t)b * a.Hkv + kvh;
    const bool live = t < a.t_end;

    uint4 raw = make_uint4(0, 0, 0, 0);
    if (live) raw = *reinterpret_cast<const uint4*>(a.k + (bh * a.Lcap + t) * kD + 8 * j16);
    const QuantToken qt = quantize_token(raw, j16);
    if (!live) return;
    store_token(qt, j16, bh, t, a.Lcap, a.codes, a.absmax, a.resid);
}

// Decode-step append: workgroup b writes the new token of every KV head of sequence b at position
// L = seq_lens[b] (bf16 K/V rows when the caches are given, and its quantized key), then sets
// seq_lens[b] = L + 1. 16 lanes per KV head; a sequence already at capacity is left unchanged.
__global__ __launch_bounds__(kThreads) void append_kv_kernel(AppendArgs a) {
    const int tid = threadIdx.x, j16 = tid & 15;
    const int b = blockIdx.x;
    const int L = a.seq_lens[b];
    const bool room = L >= 0 && L < a.Lcap;
    for (int kvh = tid >> 4; kvh < a.Hkv; kvh += kThreads / 16) {
        const size_t bh = (size_t)b * a.Hkv + kvh;
        const uint4 kraw = *reinterpret_cast<const uint4*>(a.k_new + bh * kD + 8 * j16);
        const uint4 vraw = *reinterpret_cast<const uint4*>(a.v_new + bh * kD + 8 * j16);
        const QuantToken qt = quantize_token(kraw, j16);
        if (room) {
            const size_t row = (bh * a.Lcap + L) * kD + 8 * j16;
            if (a.k_cache) *reinterpret_cast<uint4*>(a.k_cache + row) = kraw;
            if (a.v_cache) *reinterpret_cast<uint4*>(a.v_cache + row) = vraw;
            store_token(qt, j16, bh, L, a.Lcap, a.codes, a.absmax, a.resid);
        }
    }
    __syncthreads();                    // every thread has read L before it moves
    if (tid == 0 && room) a.seq_lens[b] = L + 1;
}

}  // namespace ffd
