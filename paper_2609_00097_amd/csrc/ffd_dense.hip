// Dense flash-decode attention for gfx950 (the exact comparator): softmax(alpha q K^T) V over all
// tokens of each sequence, split along the sequence and merged by log-sum-exp.
//
// Mapping. One workgroup (4 waves) serves one (sequence, KV head, split); waves take the split's
// 64-token blocks with stride 4. QK^T runs on v_mfma_f32_16x16x32_bf16 with the queries as the A
// operand (head h of a 4-head tile on row 4h, other rows zero) and 16 tokens per tile as B: lane
// (g, n) loads token n's dims 32g..32g+31 (64 contiguous bytes), so its output register 0 is head
// g's score for token n. PV runs on the VALU in fp32 (see pv_update).
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

template <int NT>
struct DenseLds {
    WaveP<NT> wp[kWaves];
    EpilogueLds<NT> epi;
};

}  // namespace

template <int NT>
__global__ __launch_bounds__(kThreads) void dense_decode_kernel(DenseArgs a) {
    __shared__ DenseLds<NT> sm;
    const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, n = lane & 15;
    const int G = a.G, hq0 = kvh * G;
    const size_t bh = (size_t)b * a.Hkv + kvh;
    const int L = min(max(a.seq_lens[b], 0), a.Lcap);
    const int nblk = (L + kBlock - 1) / kBlock;
    const int bps = (nblk + a.S - 1) / a.S;
    const int jb = min(s * bps, nblk), je = min(jb + bps, nblk);
    const uint16_t* k_bh = a.k + bh * (size_t)a.Lcap * kD;
    const uint16_t* v_bh = a.v + bh * (size_t)a.Lcap * kD;

    // A operand: lane (m = n, g), k-step ks holds q[head][32g + 8ks .. +8] on rows m = 4h.
    v8bf Aq[NT][4];
    bool live[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int hrow = 4 * t + (n >> 2);
        const bool rl = (n & 3) == 0 && hrow < G;
        const uint4* qp = reinterpret_cast<const uint4*>(a.q + ((size_t)b * a.Hq + hq0 + hrow) * kD + 32 * g);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const uint4 w = rl ? qp[ks] : make_uint4(0, 0, 0, 0);
            Aq[t][ks] = __builtin_bit_cast(v8bf, w);
        }
        live[t] = 4 * t + g < G;
    }

    PvAcc<NT> pv;
    pv.zero();
    float m_run[NT], l_part[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { m_run[t] = -INFINITY; l_part[t] = 0.f; }
    WaveP<NT>& wp = sm.wp[wave];

    for (int j = jb + wave; j < je; j += kWaves) {
        float z[NT][4];
#pragma unroll
        for (int T4 = 0; T4 < 4; ++T4) {
            const int tok = 64 * j + 16 * T4 + n;
            const uint4* kp = reinterpret_cast<const uint4*>(k_bh + (size_t)tok * kD + 32 * g);
            uint4 kk[4];
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) kk[ks] = tok < L ? kp[ks] : make_uint4(0, 0, 0, 0);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Aq[t][ks], __builtin_bit_cast(v8bf, kk[ks]),
                                                                  acc, 0, 0, 0);
                z[t][T4] = tok < L ? acc.x * a.scale : -INFINITY;
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            float corr = 1.f, p[4] = {0.f, 0.f, 0.f, 0.f};
            if (live[t]) {
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

template __global__ void dense_decode_kernel<1>(DenseArgs);
template __global__ void dense_decode_kernel<2>(DenseArgs);

// Log-sum-exp merge of the split partials (flash-decoding reduction): one workgroup per (b, h),
// one thread per output dim.
__global__ __launch_bounds__(kD) void lse_merge_kernel(const float* part_m, const float* part_l,
                                                       const float* part_acc, int S, uint16_t* out,
                                                       float* lse) {
    const size_t bh = blockIdx.x;
    const int d = threadIdx.x;
    const float* pm = part_m + bh * S;
    const float* pl = part_l + bh * S;
    const float* pa = part_acc + bh * (size_t)S * kD + d;
    float mx = -INFINITY;
    for (int s = 0; s < S; ++s) mx = fmaxf(mx, pm[s]);
    float l = 0.f, o = 0.f;
    if (mx != -INFINITY) {
        for (int s = 0; s < S; ++s) {
            const float ms = pm[s];
            if (ms != -INFINITY) {
                const float w = __expf(ms - mx);
                l = fmaf(w, pl[s], l);
                o = fmaf(w, pa[(size_t)s * kD], o);
            }
        }
    }
    out[bh * kD + d] = f32_to_bf16(mx != -INFINITY ? o / l : 0.f);
    if (lse && d == 0) lse[bh] = mx != -INFINITY ? mx + logf(l) : -INFINITY;
}

}  // namespace ffd
