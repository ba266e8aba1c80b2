// FFD decode attention for gfx950: 2-bit scan + top-delta selection + refinement + online softmax.
//
// Method (Alg. 1; Eq. 1-4): for each query head h of a KV group,
//   s_hat[t] = alpha * q . k^quant_t                      (thumbnail scan)
//   m~       = max of s_hat over the first n_sink and last n_local tokens      (pseudo-max, Eq. 3)
//   keep j   iff max_{t in block j} s_hat[t] >= m~ - delta                       (top-delta, Eq. 1)
//   z[t]     = s_hat[t] + alpha * q . k^res_t   for t in kept blocks            (scan reuse, Eq. 4)
//   out      = softmax(z) . V over kept tokens, split along the sequence and merged by LSE.
//
// Mapping to the hardware. One workgroup (4 waves) serves one (sequence, KV head, split); each wave
// walks the split's blocks with stride 4. The group's queries stay in registers as the A operand of
// v_mfma_i32_16x16x64_i8: each query is held in fixed point Q = rint(q * 2^(22-E)) (|q| < 2^E),
// split into three signed 8-bit limbs, one MFMA row per (head, limb). The B operand is either the
// 2-bit codes expanded to bytes (two VALU ops per 4 codes) or the stored int8 residual, so both dot
// products are exact integer sums, combined and rounded once to fp32:
//   sum_d Q_d (2 c_d - 3) = T  (int32, exact),     s_hat = T * M_t * alpha 2^(E-23) / 1.5
//   sum_d Q_d r_d         = R  (three int32 limbs), z = s_hat + R * M_t * alpha 2^(E-22) / 381
// Output register i of lane (g, n) is row 4g + i, column n: head g's limbs for token n of a 16-token
// tile, so each 16-lane row group owns one head and block maxima are 16-lane reductions.
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

__device__ __forceinline__ int limb_of(int Q, int which) {
    const int l0 = ((Q + 128) & 255) - 128;
    const int q1 = (Q - l0) >> 8;
    const int l1 = ((q1 + 128) & 255) - 128;
    const int l2 = (q1 - l1) >> 8;
    return which == 0 ? l0 : (which == 1 ? l1 : l2);
}

__device__ __forceinline__ v4i expand_codes(uint32_t w) {
    v4i r;
    r.x = (int)(w & 0x03030303u);
    r.y = (int)((w >> 2) & 0x03030303u);
    r.z = (int)((w >> 4) & 0x03030303u);
    r.w = (int)((w >> 6) & 0x03030303u);
    return r;
}

template <int NT>
struct HeadConsts {
    v4i A[NT][2];      // MFMA A operand per head tile and 64-dim chunk
    int off[NT];       // 3 * sum_d Q_d of head 4t + g
    float kap[NT];     // alpha * 2^(E-23) / 1.5
    float kap2[NT];    // alpha * 2^(E-22) / 381
    bool live[NT];     // head 4t + g exists
};

// Thumbnail scores of block j for this lane's head(s) and tokens 64j + 16*T4 + n.
template <int NT>
__device__ __forceinline__ void scan_block(const uint32_t* __restrict__ codes_bh,
                                           const uint16_t* __restrict__ absmax_bh, int j, int lane,
                                           int L, const HeadConsts<NT>& hc, float (&sc)[NT][4],
                                           float (&Mf)[4]) {
    const int n = lane & 15;
    const uint4* cp = reinterpret_cast<const uint4*>(codes_bh) + (size_t)(2 * j) * 64 + lane;
    const uint4 w0 = cp[0];
    const uint4 w1 = cp[64];
    const uint2 mm = *reinterpret_cast<const uint2*>(absmax_bh + (size_t)j * 64 + n * 4);
    Mf[0] = bf16_lo(mm.x); Mf[1] = bf16_hi(mm.x);
    Mf[2] = bf16_lo(mm.y); Mf[3] = bf16_hi(mm.y);
    const uint32_t words[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4) {
        const v4i b0 = expand_codes(words[2 * T4 + 0]);
        const v4i b1 = expand_codes(words[2 * T4 + 1]);
        const int tok = 64 * j + 16 * T4 + n;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], b0, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], b1, acc, 0, 0, 0);
            const uint32_t s = (uint32_t)acc.x + ((uint32_t)acc.y << 8) + ((uint32_t)acc.z << 16);
            const int T = (int)(2u * s - (uint32_t)hc.off[t]);     // exact modulo 2^32, |T| < 2^31
            sc[t][T4] = tok < L ? (float)T * (Mf[T4] * hc.kap[t]) : -INFINITY;
        }
    }
}

// Refined logits of block j (scan term reused): z = s_hat + alpha * q . k^res.
template <int NT>
__device__ __forceinline__ void refine_block(const int8_t* __restrict__ resid_bh, int j, int lane,
                                             int L, const HeadConsts<NT>& hc,
                                             const float (&sc)[NT][4], const float (&Mf)[4],
                                             float (&z)[NT][4]) {
    const int n = lane & 15;
    const v4i* rp = reinterpret_cast<const v4i*>(resid_bh) + (size_t)(8 * j) * 64 + lane;
    v4i r[4][2];
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4)
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) r[T4][cc] = rp[(2 * T4 + cc) * 64];
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4) {
        const int tok = 64 * j + 16 * T4 + n;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], r[T4][0], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], r[T4][1], acc, 0, 0, 0);
            const float R = fmaf(65536.f, (float)acc.z, fmaf(256.f, (float)acc.y, (float)acc.x));
            z[t][T4] = tok < L ? fmaf(R, Mf[T4] * hc.kap2[t], sc[t][T4]) : -INFINITY;
        }
    }
}

template <int NT>
struct DecodeLds {
    float q[4 * NT][kD];
    int qq[4 * NT][kD];
    int off[4 * NT];
    float kap[4 * NT];
    float kap2[4 * NT];
    float pm[kWaves][4 * NT];
    WaveP<NT> wp[kWaves];
    EpilogueLds<NT> epi;
};

}  // namespace

template <int NT>
__global__ __launch_bounds__(kThreads) void ffd_decode_kernel(DecodeArgs a) {
    __shared__ DecodeLds<NT> sm;
    const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, n = lane & 15;
    const int G = a.G, hq0 = kvh * G;
    const size_t bh = (size_t)b * a.Hkv + kvh;
    const int L = min(max(a.seq_lens[b], 0), a.Lcap);
    const int nblk = (L + kBlock - 1) / kBlock;
    const int nblk_cap = a.Lcap / kBlock;
    const int bps = (nblk + a.S - 1) / a.S;
    const int jb = min(s * bps, nblk), je = min(jb + bps, nblk);

    const uint32_t* codes_bh = a.codes + bh * (size_t)(a.Lcap / 32) * 256;
    const uint16_t* absmax_bh = a.absmax + bh * (size_t)a.Lcap;
    const int8_t* resid_bh = a.resid + bh * (size_t)a.Lcap * kD;
    const uint16_t* v_bh = a.v + bh * (size_t)a.Lcap * kD;

    // Mask entries past the end of the sequence are zero (spread over the splits).
    if (a.mask) {
        for (int j = nblk + s * kThreads + tid; j < nblk_cap; j += a.S * kThreads)
            for (int h = 0; h < G; ++h) a.mask[((size_t)b * a.Hq + hq0 + h) * nblk_cap + j] = 0;
    }

    // ---- queries -> fixed point, per-head constants ----------------------------------------
    for (int i = tid; i < G * kD; i += kThreads)
        sm.q[i >> 7][i & (kD - 1)] = bf16_to_f32(a.q[((size_t)b * a.Hq + hq0) * kD + i]);
    __syncthreads();
    for (int h = wave; h < G; h += kWaves) {
        const float x0 = sm.q[h][lane], x1 = sm.q[h][lane + 64];
        const float mx = wave_max(fmaxf(fabsf(x0), fabsf(x1)));
        int E = 0;
        (void)frexpf(mx, &E);                       // mx < 2^E (mx == 0 -> E = 0)
        const int Q0 = (int)rintf(ldexpf(x0, 22 - E));
        const int Q1 = (int)rintf(ldexpf(x1, 22 - E));
        sm.qq[h][lane] = Q0;
        sm.qq[h][lane + 64] = Q1;
        const int sum = wave_sum_i(Q0 + Q1);
        if (lane == 0) {
            sm.off[h] = 3 * sum;
            sm.kap[h] = ldexpf(a.scale / 1.5f, E - 23);
            sm.kap2[h] = ldexpf(a.scale / 381.f, E - 22);
        }
    }
    __syncthreads();

    HeadConsts<NT> hc;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        // A operand: row m = n is (head 4t + n/4, limb n%4); bytes e are dims 64cc + 16g + e.
        const int hrow = 4 * t + (n >> 2), limb = n & 3;
        const bool rlive = hrow < G && limb < 3;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            int words[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                uint32_t w = 0;
#pragma unroll
                for (int bb = 0; bb < 4; ++bb) {
                    const int d = 64 * cc + 16 * g + 4 * k + bb;
                    const int v = rlive ? limb_of(sm.qq[hrow][d], limb) : 0;
                    w |= ((uint32_t)v & 0xffu) << (8 * bb);
                }
                words[k] = (int)w;
            }
            hc.A[t][cc] = v4i{words[0], words[1], words[2], words[3]};
        }
        const int hh = 4 * t + g;      // this lane's output head
        hc.live[t] = hh < G;
        hc.off[t] = hc.live[t] ? sm.off[hh] : 0;
        hc.kap[t] = hc.live[t] ? sm.kap[hh] : 0.f;
        hc.kap2[t] = hc.live[t] ? sm.kap2[hh] : 0.f;
    }

    // ---- pseudo-max over sink and local windows (Eq. 3) ----------------------------------
    const int sink_end = min(a.n_sink, L);
    const int loc_beg = max(0, L - a.n_local);
    const int sink_blk_end = (sink_end + kBlock - 1) / kBlock;
    const int loc_blk_beg = max(loc_beg / kBlock, sink_blk_end);
    const int npm = sink_blk_end + max(nblk - loc_blk_beg, 0);
    float pm[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) pm[t] = -INFINITY;
    for (int idx = wave; idx < npm; idx += kWaves) {
        const int j = idx < sink_blk_end ? idx : loc_blk_beg + (idx - sink_blk_end);
        float sc[NT][4], Mf[4];
        scan_block<NT>(codes_bh, absmax_bh, j, lane, L, hc, sc, Mf);
#pragma unroll
        for (int T4 = 0; T4 < 4; ++T4) {
            const int tok = 64 * j + 16 * T4 + n;
            const bool in_win = tok < L && (tok < sink_end || tok >= loc_beg);
#pragma unroll
            for (int t = 0; t < NT; ++t) pm[t] = fmaxf(pm[t], in_win ? sc[t][T4] : -INFINITY);
        }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        pm[t] = row16_max(pm[t]);
        if (n == 0) sm.pm[wave][4 * t + g] = pm[t];
    }
    __syncthreads();
    float thr[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float m = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) m = fmaxf(m, sm.pm[w][4 * t + g]);
        thr[t] = m - a.delta;                      // -inf when both windows are empty
    }

    // ---- main loop: scan, decide, refine + attend kept blocks ---------------------------
    PvAcc<NT> pv;
    pv.zero();
    float m_run[NT], l_part[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { m_run[t] = -INFINITY; l_part[t] = 0.f; }
    WaveP<NT>& wp = sm.wp[wave];

    for (int j = jb + wave; j < je; j += kWaves) {
        float sc[NT][4], Mf[4];
        scan_block<NT>(codes_bh, absmax_bh, j, lane, L, hc, sc, Mf);
        bool keep[NT], any = false;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float sig = row16_max(fmaxf(fmaxf(sc[t][0], sc[t][1]), fmaxf(sc[t][2], sc[t][3])));
            keep[t] = hc.live[t] && sig >= thr[t];
            any |= keep[t];
            if (a.mask && n == 0 && hc.live[t])
                a.mask[((size_t)b * a.Hq + hq0 + 4 * t + g) * nblk_cap + j] = keep[t] ? 1 : 0;
        }
        if (__ballot(any) == 0) continue;          // no head of the group keeps the block

        float z[NT][4];
        refine_block<NT>(resid_bh, j, lane, L, hc, sc, Mf, z);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            float corr = 1.f, p[4] = {0.f, 0.f, 0.f, 0.f};
            if (keep[t]) {
                const float mb = row16_max(fmaxf(fmaxf(z[t][0], z[t][1]), fmaxf(z[t][2], z[t][3])));
                const float mn = fmaxf(m_run[t], mb);
                corr = __expf(m_run[t] - mn);
                float ls = 0.f;
#pragma unroll
                for (int T4 = 0; T4 < 4; ++T4) {
                    p[T4] = z[t][T4] == -INFINITY ? 0.f : __expf(z[t][T4] - mn);
                    ls += p[T4];
                }
                l_part[t] = fmaf(l_part[t], corr, ls);
                m_run[t] = mn;
            }
#pragma unroll
            for (int T4 = 0; T4 < 4; ++T4) wp.p[16 * T4 + n][4 * t + g] = p[T4];
            if (n == 0) wp.corr[4 * t + g] = corr;
        }
        wave_lds_fence();
        pv_update<NT>(pv, wp, v_bh + (size_t)j * kBlock * kD, g, n, L - 64 * j);
        wave_lds_fence();
    }

    write_partials<NT>(sm.epi, pv, m_run, l_part, wave, lane, G, hq0, a.Hq, a.S, b, s, a.part_m,
                       a.part_l, a.part_acc);
}

template __global__ void ffd_decode_kernel<1>(DecodeArgs);
template __global__ void ffd_decode_kernel<2>(DecodeArgs);

}  // namespace ffd
