// Key quantization for gfx950 (Sec. 3.1; App. A; App. C depths): each bf16 key vector of 128 dims
// becomes b-bit codes on the scale s = M/Lv (M = max |k_i|, Lv = (2^b - 1)/2, nearest level c - Lv,
// ties to the upper level), the absmax M, and an int8 residual r = rint(254 Lv k / M) - 254 c + 254 Lv.
// b = 2 is App. A's codebook {-1.5, -0.5, 0.5, 1.5} with the residual rint(381 k / M) - 254 c + 381.
//
// Exactness:
//  * code: x/s = Lv k / M has the integers as bin edges, so c = floor((2^b - 1) k / (2M)) + 2^(b-1).
//    The quotient is taken as a product with the token's reciprocal 1/(2M) (off by at most one in
//    the floor); (2^b - 1) k and i * 2M are products of 8-bit significands, exact in fp32 while
//    2^-100 < M < 2^100 (no overflow, reciprocals normal), so exact comparisons then settle the
//    floor. For b = 2 this is App. A's rule as three exact comparisons of 3k with -2M, 0, 2M.
//  * residual: 254 Lv k is exact; q = 254 Lv k * (1/M) is within 2^-23 |q| of the true quotient, so
//    rint(q) is the exact round-half-even result whenever q lies further than 2^-21 |q| from every
//    half-integer. Otherwise (a tie or a near-tie), and for M outside (2^-100, 2^100), the element
//    is redone in fp64, where nothing overflows and a quotient that is not a tie lies at least
//    2^-24 Q from every half-integer (254 Lv < 2^15, k has 8 significant bits) while the division
//    moves it by at most 2^-53 Q.
//
// Mapping: 16 lanes per token, each lane owns 8 consecutive dims (one 16-byte load); the absmax is
// a 16-lane max reduction. Writes go straight into the storage layouts documented in ffd.h.
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

// One token's quantization by 16 lanes: lane j16 holds dims 8*j16 .. 8*j16 + 7 as one 16-byte
// chunk of bf16 (raw). The 16 lanes must be one aligned DPP row (lanes 16r .. 16r + 15), all active. Returns the token's absmax M in every lane, the
// lane's code words and its 8 int8 residuals (rlo/rhi). Code words: b = 2, the 16 codes of the lane
// pair's 16-dim group (identical in both lanes of the pair); b = 4, the lane's 8 codes; b = 8, its 8
// code bytes c - 128.
template <int BITS>
struct QuantToken {
    float m;
    uint32_t word[BITS == 8 ? 2 : 1];
    uint32_t rlo, rhi;
};

template <int BITS>
__device__ __forceinline__ QuantToken<BITS> quantize_token(uint4 raw, int j16) {
#pragma clang fp contract(off)          // the rounding arguments above assume no fused products
    constexpr int kLevels = 1 << BITS;
    constexpr double kTwoLv = kLevels - 1;                 // 2 Lv
    constexpr double kFull = 127.0 * (kLevels - 1);        // 254 Lv
    float x[8];
    x[0] = bf16_lo(raw.x); x[1] = bf16_hi(raw.x);
    x[2] = bf16_lo(raw.y); x[3] = bf16_hi(raw.y);
    x[4] = bf16_lo(raw.z); x[5] = bf16_hi(raw.z);
    x[6] = bf16_lo(raw.w); x[7] = bf16_hi(raw.w);
    float m = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(x[e]));
    m = row16_max(m);                      // the token's 16 lanes are one DPP row

    QuantToken<BITS> qt;
    qt.m = m;
    const bool fast = m < 0x1p100f && m > 0x1p-100f;
    const float two_m = 2.f * m, r_two_m = 1.f / two_m, r_m = 1.f / m;
#pragma unroll
    for (int w = 0; w < (BITS == 8 ? 2 : 1); ++w) qt.word[w] = 0;
    qt.rlo = qt.rhi = 0;
    // fp32 pass over the 8 elements; the rare ones it cannot settle are redone in fp64 below
    int cs[8], ns[8];
    uint32_t slow = fast || m == 0.f ? 0u : 0xffu;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        if constexpr (BITS == 2) {
            // the three bin edges 3k = -2M, 0, 2M, ties up (a branch-free count of edges passed)
            const float x3 = 3.f * x[e];
            cs[e] = (int)(x3 >= two_m) + (int)(x[e] >= 0.f) + (int)(x3 >= -two_m);
        } else {
            const float u = (float)kTwoLv * x[e];
            float i = floorf(u * r_two_m);
            i += (i + 1.f) * two_m <= u ? 1.f : 0.f;
            i -= i * two_m > u ? 1.f : 0.f;
            cs[e] = (int)i + kLevels / 2;
        }
        const float q = ((float)kFull * x[e]) * r_m;
        const bool near_tie = !(fabsf(q - floorf(q) - 0.5f) > fabsf(q) * 0x1p-21f);
        slow |= (uint32_t)(fast & near_tie) << e;
        ns[e] = (int)rintf(q);
    }
    if (slow) {
        const double md = m, two_md = 2.0 * md;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (slow & (1u << e)) {
                const double xv = x[e], u = kTwoLv * xv;
                double i = floor(u / two_md);
                if ((i + 1.0) * two_md <= u) i += 1.0;
                if (i * two_md > u) i -= 1.0;
                cs[e] = (int)i + kLevels / 2;
                ns[e] = (int)rint((kFull * xv) / md);
            }
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        int c = kLevels / 2, r = 0;                        // M = 0: level +0.5, residual 0
        if (m != 0.f) {
            c = min(max(cs[e], 0), kLevels - 1);
            r = ns[e] - 254 * c + (int)kFull;
        }
        if constexpr (BITS == 2) {
            const int e16 = 8 * (j16 & 1) + e;             // position inside the 16-dim group
            qt.word[0] |= (uint32_t)c << (8 * (e16 & 3) + 2 * (e16 >> 2));
        } else if constexpr (BITS == 4) {
            qt.word[0] |= (uint32_t)c << (8 * (e & 3) + 4 * (e >> 2));
        } else {
            qt.word[e >> 2] |= (uint32_t)((c - 128) & 0xff) << (8 * (e & 3));
        }
        const uint32_t rb = (uint32_t)(r & 0xff);
        if (e < 4) qt.rlo |= rb << (8 * e); else qt.rhi |= rb << (8 * (e - 4));
    }
    if constexpr (BITS == 2)                                           // the lane pair's 16 dims
        qt.word[0] |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)qt.word[0], kDppXor1, 0xf, 0xf, false);
    return qt;
}

// Store token t of (b, kvh) = row bh into the codes / absmax / residual layouts (lane j16's share).
// Codes: lane l = n16 + 16g of block t/64 holds the (t4, cc) group's b/2 words from (2 t4 + cc) b/2;
// its word w sits at [w / 4][l][w % 4] of the block's 4b x 64 words.
template <int BITS>
__device__ __forceinline__ void store_token(const QuantToken<BITS>& qt, int j16, size_t bh, int t, int Lcap,
                                            uint32_t* codes, uint16_t* absmax, int8_t* resid) {
    const int n16 = t & 15, t4 = (t >> 4) & 3;
    const int w16 = j16 >> 1;                              // 16-dim group 0..7
    const int cc = w16 >> 2, g = w16 & 3;
    const int w = (2 * t4 + cc) * (BITS / 2) + (BITS == 2 ? 0 : (BITS / 4) * (j16 & 1));   // first word
    uint32_t* dst = codes + (bh * (size_t)(Lcap / 64) + (t >> 6)) * (64 * 4 * BITS) + (w >> 2) * 256 +
                    (n16 + 16 * g) * 4 + (w & 3);
    if constexpr (BITS == 2) {
        if ((j16 & 1) == 0) dst[0] = qt.word[0];
    } else if constexpr (BITS == 4) {
        dst[0] = qt.word[0];
    } else {
        *reinterpret_cast<uint2*>(dst) = make_uint2(qt.word[0], qt.word[1]);   // words w, w + 1 (w even)
    }
    {
        const int rc = j16 >> 3, rg = (j16 & 7) >> 1, e0 = 8 * (j16 & 1);
        int8_t* dst = resid + (((bh * (size_t)(Lcap / 16) + (t >> 4)) * 2 + rc) * 64 + n16 + 16 * rg) * 16 + e0;
        *reinterpret_cast<uint2*>(dst) = make_uint2(qt.rlo, qt.rhi);
    }
    if (j16 == 0)
        absmax[bh * (size_t)Lcap + (size_t)(t >> 6) * 64 + n16 * 4 + t4] = (uint16_t)(__float_as_uint(qt.m) >> 16);
}

}  // namespace

// Workgroup x covers the 64-token block t0 = 64 * (t_begin / 64 + x) of one (b, kvh): 16 tokens per
// pass, the four loads issued first, so the block's code words, absmaxes and residual tiles are all
// written by this workgroup (whole cache lines); only tokens in [t_begin, t_end) are stored.
template <int BITS>
__global__ __launch_bounds__(kThreads) void quantize_keys_kernel(QuantArgs a) {
    const int tid = threadIdx.x, j16 = tid & 15;
    const int t0 = (a.t_begin & ~63) + blockIdx.x * 64 + (tid >> 4);
    const int kvh = blockIdx.y, b = blockIdx.z;
    const size_t bh = (size_t)b * a.Hkv + kvh;

    uint4 raw[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const int t = t0 + 16 * p;
        raw[p] = make_uint4(0, 0, 0, 0);
        if (t >= a.t_begin && t < a.t_end)
            raw[p] = *reinterpret_cast<const uint4*>(a.k + (bh * a.Lcap + t) * kD + 8 * j16);
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const int t = t0 + 16 * p;
        const QuantToken<BITS> qt = quantize_token<BITS>(raw[p], j16);
        if (t >= a.t_begin && t < a.t_end) store_token<BITS>(qt, j16, bh, t, a.Lcap, a.codes, a.absmax, a.resid);
    }
}

// Decode-step append: workgroup b writes the new token of every KV head of sequence b at position
// L = seq_lens[b] (bf16 K/V rows when the caches are given, and its quantized key), then sets
// seq_lens[b] = L + 1. 16 lanes per KV head; a sequence already at capacity is left unchanged.
template <int BITS>
__global__ __launch_bounds__(kThreads) void append_kv_kernel(AppendArgs a) {
    const int tid = threadIdx.x, j16 = tid & 15;
    const int b = blockIdx.x;
    const int L = a.seq_lens[b];
    const bool room = L >= 0 && L < a.Lcap;
    for (int kvh = tid >> 4; kvh < a.Hkv; kvh += kThreads / 16) {
        const size_t bh = (size_t)b * a.Hkv + kvh;
        const uint4 kraw = *reinterpret_cast<const uint4*>(a.k_new + bh * kD + 8 * j16);
        const uint4 vraw = *reinterpret_cast<const uint4*>(a.v_new + bh * kD + 8 * j16);
        const QuantToken<BITS> qt = quantize_token<BITS>(kraw, j16);
        if (room) {
            const size_t row = (bh * a.Lcap + L) * kD + 8 * j16;
            if (a.k_cache) *reinterpret_cast<uint4*>(a.k_cache + row) = kraw;
            if (a.v_cache) *reinterpret_cast<uint4*>(a.v_cache + row) = vraw;
            store_token<BITS>(qt, j16, bh, L, a.Lcap, a.codes, a.absmax, a.resid);
        }
    }
    __syncthreads();                    // every thread has read L before it moves
    if (tid == 0 && room) a.seq_lens[b] = L + 1;
}

template __global__ void quantize_keys_kernel<2>(QuantArgs);
template __global__ void quantize_keys_kernel<4>(QuantArgs);
template __global__ void quantize_keys_kernel<8>(QuantArgs);
template __global__ void append_kv_kernel<2>(AppendArgs);
template __global__ void append_kv_kernel<4>(AppendArgs);
template __global__ void append_kv_kernel<8>(AppendArgs);

}  // namespace ffd
