// FFD decode attention for gfx950: 2-bit scan + top-delta selection + refinement + online softmax.
//
// Method (Alg. 1; Eq. 1-4): for each query head h of a KV group,
//   s_hat[t] = alpha * q . k^quant_t                      (thumbnail scan)
//   m~       = max of s_hat over the first n_sink and last n_local tokens      (pseudo-max, Eq. 3)
//   keep j   iff max_{t in block j} s_hat[t] >= m~ - delta                       (top-delta, Eq. 1)
//   z[t]     = s_hat[t] + alpha * q . k^res_t   for t in kept blocks            (scan reuse, Eq. 4)
//   out      = softmax(z) . V over kept tokens, split along the sequence and merged by LSE.
//
// Mapping to the hardware. A workgroup (4 waves) serves one (sequence, KV head, split); wave w
// owns the 16-token tile w of every 64-token block. The group's queries stay in registers as the A
// operand of v_mfma_i32_16x16x64_i8: each query is held in fixed point Q = rint(q * 2^(22-E))
// (|q| < 2^E), split into three signed 8-bit limbs, one MFMA row per (head, limb). The B operand is
// either the tile's 2-bit codes expanded to bytes (two VALU ops per 4 codes) or the stored int8
// residual, so both dot products are exact integer sums, combined and rounded once to fp32:
//   sum_d Q_d (2 c_d - 3) = T  (int32, exact),     s_hat = T * M_t * alpha 2^(E-23) / 1.5
//   sum_d Q_d r_d         = R  (three int32 limbs), z = s_hat + R * M_t * alpha 2^(E-22) / 381
// Output register i of lane (g, n) is row 4g + i, column n: head g's limbs for token n, so each
// 16-lane row group owns one head and a tile's maximum is a 16-lane DPP reduction.
//
// Schedule. Wave w of a workgroup owns blocks w, w+4, w+8, ... of the split and keeps its own
// online-softmax state; there is no barrier after the pseudo-max. Each wave streams its blocks'
// codes and absmaxes through a ring of kRing register slots, refilling a slot as soon as it is
// scored, so kRing blocks stay in flight. It takes the keep decision for each block itself and
// parks a kept block's scan scores in its own small LDS queue; after each round of kRing blocks it
// fetches each queued block's int8 residual and values tile by tile (two 16-token tiles in flight),
// refines the parked scan scores (Eq. 4) and updates its softmax and PV state, while the ring's
// scan loads keep streaming.
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

constexpr int kRing = 4;    // scan loads in flight per wave (blocks)
constexpr int kPMW = 2;     // pseudo-max window blocks per wave per pass

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

// One lane's share of a block's thumbnail: 32 B of codes (both 64-dim halves of its token in each
// of the four tiles) and the absmax of its four tokens.
struct BlockScan {
    uint4 w0, w1;
    uint2 mm;
};

__device__ __forceinline__ BlockScan load_block_scan(const uint32_t* __restrict__ codes_bh,
                                                     const uint16_t* __restrict__ absmax_bh, int j,
                                                     int lane) {
    const uint4* cp = reinterpret_cast<const uint4*>(codes_bh) + ((size_t)j * 64 + lane) * 2;
    BlockScan r;
    r.w0 = cp[0];
    r.w1 = cp[1];
    r.mm = *reinterpret_cast<const uint2*>(absmax_bh + (size_t)j * 64 + (lane & 15) * 4);
    return r;
}

// Thumbnail scores of block j for this lane's head(s) and tokens 64j + 16*T4 + n.
template <int NT>
__device__ __forceinline__ void block_scores(const BlockScan& ld, int j, int lane, int L,
                                             const HeadConsts<NT>& hc, float (&sc)[NT][4],
                                             float (&M)[4]) {
    const int n = lane & 15;
    M[0] = bf16_lo(ld.mm.x); M[1] = bf16_hi(ld.mm.x);
    M[2] = bf16_lo(ld.mm.y); M[3] = bf16_hi(ld.mm.y);
    const uint32_t words[8] = {ld.w0.x, ld.w0.y, ld.w0.z, ld.w0.w, ld.w1.x, ld.w1.y, ld.w1.z, ld.w1.w};
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4) {
        const v4i b0 = expand_codes(words[2 * T4 + 0]);
        const v4i b1 = expand_codes(words[2 * T4 + 1]);
        const bool valid = 64 * j + 16 * T4 + n < L;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], b0, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], b1, acc, 0, 0, 0);
            const uint32_t s = (uint32_t)acc.x + ((uint32_t)acc.y << 8) + ((uint32_t)acc.z << 16);
            const int T = (int)(2u * s - (uint32_t)hc.off[t]);     // exact modulo 2^32, |T| < 2^31
            sc[t][T4] = valid ? (float)T * (M[T4] * hc.kap[t]) : -INFINITY;
        }
    }
}

// A kept block parked by one wave: its scan scores per (tile, head-tile, lane), absmaxes, index and
// per-head keep bits (bit 4t + g).
template <int NT>
struct Parked {
    float sc[4][NT][64];
    float M[4][16];
    int j;
    uint32_t keep;
};

// One wave's fetch for one 16-token tile of a kept block: int8 residual and its lane's value dwords.
struct TileGather {
    v4i r0, r1;
    VTile vt;
};

__device__ __forceinline__ TileGather load_tile_gather(const int8_t* __restrict__ resid_bh,
                                                       const uint16_t* __restrict__ v_bh, int tile,
                                                       int lane, int L) {
    TileGather r;
    const v4i* rp = reinterpret_cast<const v4i*>(resid_bh) + (size_t)tile * 128 + lane;
    r.r0 = rp[0];
    r.r1 = rp[64];
    r.vt = load_vtile(v_bh, 16 * tile, max(L, 1) - 1, lane);
    return r;
}

template <int NT>
struct DecodeLds {
    alignas(16) int8_t limbs[4][4 * NT][kD];     // [limb][head][dim]; limb 3 is zero
    int off[4 * NT];
    float kap[4 * NT];
    float kap2[4 * NT];
    float pm[kWaves][4 * NT];
    Parked<NT> park[kWaves][kRing];
    TileP<NT> tp[kWaves];
    EpilogueLds<NT> epi;
};

}  // namespace

template <int NT>
__global__ __launch_bounds__(kThreads, 2) void ffd_decode_kernel(DecodeArgs a) {
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

    const uint32_t* codes_bh = a.codes + bh * (size_t)a.Lcap * 8;
    const uint16_t* absmax_bh = a.absmax + bh * (size_t)a.Lcap;
    const int8_t* resid_bh = a.resid + bh * (size_t)a.Lcap * kD;
    const uint16_t* v_bh = a.v + bh * (size_t)a.Lcap * kD;

    // Ring of this wave's scan loads: slot r holds block jb + 4*(i0 + r) + wave of round i0.
    // The first chunk and the first pseudo-max window blocks are requested before the setup.
    // Loads are issued unconditionally (out-of-range indices are clamped to valid data that is then
    // ignored): uniform control flow lets the compiler wait for exactly the load it needs instead of
    // draining every load in flight. Order: queries, pseudo-max window blocks, the first chunk.
    uint32_t qw[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
        qw[t] = reinterpret_cast<const uint32_t*>(a.q + ((size_t)b * a.Hq + hq0 + min(wave + 4 * t, G - 1)) * kD)[lane];
    const int jlast = max(nblk, 1) - 1;
    const int sink_end = min(a.n_sink, L);
    const int loc_beg = max(0, L - a.n_local);
    const int sink_blk_end = (sink_end + kBlock - 1) / kBlock;
    const int loc_blk_beg = max(loc_beg / kBlock, sink_blk_end);
    const int npm = sink_blk_end + max(nblk - loc_blk_beg, 0);
    auto pm_block = [&](int idx) { return idx < sink_blk_end ? idx : loc_blk_beg + (idx - sink_blk_end); };
    BlockScan win[kPMW];
#pragma unroll
    for (int i = 0; i < kPMW; ++i)
        win[i] = load_block_scan(codes_bh, absmax_bh, min(pm_block(min(kWaves * i + wave, max(npm, 1) - 1)), jlast), lane);
    BlockScan ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) ring[i] = load_block_scan(codes_bh, absmax_bh, min(jb + kWaves * i + wave, jlast), lane);


    // ---- queries -> fixed point limbs in LDS, per-head constants ------------------------------
    // Head h (wave h % 4): E with max|q| < 2^E, Q = rint(q 2^(22-E)) split into three signed bytes
    // stored as limbs[limb][h][d]; the fourth limb row and heads past G stay zero.
    for (int i = tid; i < 4 * 4 * NT * kD / 4; i += kThreads) reinterpret_cast<int*>(sm.limbs)[i] = 0;
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int h = wave + 4 * t;
        if (h >= G) continue;
        const float x0 = bf16_lo(qw[t]), x1 = bf16_hi(qw[t]);         // dims 2*lane, 2*lane + 1
        const float mx = wave_max(fmaxf(fabsf(x0), fabsf(x1)));
        int E = 0;
        (void)frexpf(mx, &E);                       // mx < 2^E (mx == 0 -> E = 0)
        const int Q0 = (int)rintf(ldexpf(x0, 22 - E));
        const int Q1 = (int)rintf(ldexpf(x1, 22 - E));
#pragma unroll
        for (int li = 0; li < 3; ++li) {
            const uint32_t pair = ((uint32_t)limb_of(Q0, li) & 0xffu) | (((uint32_t)limb_of(Q1, li) & 0xffu) << 8);
            reinterpret_cast<uint16_t*>(&sm.limbs[li][h][0])[lane] = (uint16_t)pair;
        }
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
        // A operand: row m = n is (head 4t + n/4, limb n%4); its 16 bytes are dims 64cc + 16g + e.
        const int hrow = 4 * t + (n >> 2), limb = n & 3;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc)
            hc.A[t][cc] = *reinterpret_cast<const v4i*>(&sm.limbs[limb][hrow][64 * cc + 16 * g]);
        const int hh = 4 * t + g;      // this lane's output head
        hc.live[t] = hh < G;
        hc.off[t] = hc.live[t] ? sm.off[hh] : 0;
        hc.kap[t] = hc.live[t] ? sm.kap[hh] : 0.f;
        hc.kap2[t] = hc.live[t] ? sm.kap2[hh] : 0.f;
    }

    // ---- pseudo-max over sink and local windows (Eq. 3) ----------------------------------
    float pm[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) pm[t] = -INFINITY;
    for (int base = 0; base < npm; base += kWaves * kPMW) {
        if (base > 0) {
#pragma unroll
            for (int i = 0; i < kPMW; ++i)
                win[i] = load_block_scan(codes_bh, absmax_bh, pm_block(min(base + kWaves * i + wave, npm - 1)), lane);
        }
#pragma unroll
        for (int i = 0; i < kPMW; ++i) {
            const int idx = base + kWaves * i + wave;
            const int j = pm_block(min(idx, npm - 1));
            float sc[NT][4], M[4];
            block_scores<NT>(win[i], j, lane, L, hc, sc, M);
#pragma unroll
            for (int T4 = 0; T4 < 4; ++T4) {
                const int tok = 64 * j + 16 * T4 + n;
                const bool in_win = idx < npm && tok < L && (tok < sink_end || tok >= loc_beg);
#pragma unroll
                for (int t = 0; t < NT; ++t) pm[t] = fmaxf(pm[t], in_win ? sc[t][T4] : -INFINITY);
            }
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

    // ---- main loop: scan, decide, and attend kept blocks, per wave ----------------------
    PvAcc<NT> pv;
    pv.zero();
    float m_run[NT], l_part[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { m_run[t] = -INFINITY; l_part[t] = 0.f; }
    TileP<NT>& tp = sm.tp[wave];

    // refine (Eq. 4) and attend one tile of a parked block from its fetched residual and values
    auto attend_tile = [&](const TileGather& tg, const Parked<NT>& pk, int T4) {
        float z[NT];
        bool keep[NT];
        const float Mt = pk.M[T4][n];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], tg.r0, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], tg.r1, acc, 0, 0, 0);
            const float R = fmaf(65536.f, (float)acc.z, fmaf(256.f, (float)acc.y, (float)acc.x));
            const float sct = pk.sc[T4][t][lane];
            z[t] = sct == -INFINITY ? -INFINITY : fmaf(R, Mt * hc.kap2[t], sct);
            keep[t] = (pk.keep >> (4 * t + g)) & 1u;
        }
        softmax_tile<NT>(z, keep, m_run, l_part, tp, g, n);
        wave_lds_fence();
        pv_tile<NT>(pv, tp, tg.vt);
        wave_lds_fence();
    };

    for (int i0 = 0; jb + kWaves * i0 + wave < je; i0 += kRing) {
        int parked = 0;                                       // wave-uniform
#pragma unroll
        for (int r = 0; r < kRing; ++r) {
            const int j = jb + kWaves * (i0 + r) + wave;      // wave-uniform
            if (j < je) {
                float sc[NT][4], M[4];
                block_scores<NT>(ring[r], j, lane, L, hc, sc, M);
                ring[r] = load_block_scan(codes_bh, absmax_bh, min(j + kWaves * kRing, jlast), lane);
                bool keep[NT], any = false;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const float sig = row16_max(fmaxf(fmaxf(sc[t][0], sc[t][1]), fmaxf(sc[t][2], sc[t][3])));
                    keep[t] = hc.live[t] && sig >= thr[t];
                    any |= keep[t];
                    if (a.mask && n == 0 && hc.live[t])
                        a.mask[((size_t)b * a.Hq + hq0 + 4 * t + g) * nblk_cap + j] = keep[t] ? 1 : 0;
                }
                if (__ballot(any) != 0) {                   // some head of the group keeps block j
                    uint32_t bits = 0;
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const uint64_t bl = __ballot(keep[t] && n == 0);
                        bits |= (uint32_t)(((bl >> 0) & 1u) | ((bl >> 15) & 2u) | ((bl >> 30) & 4u) |
                                           ((bl >> 45) & 8u)) << (4 * t);
                    }
                    Parked<NT>& pk = sm.park[wave][parked];
#pragma unroll
                    for (int T4 = 0; T4 < 4; ++T4) {
#pragma unroll
                        for (int t = 0; t < NT; ++t) pk.sc[T4][t][lane] = sc[t][T4];
                        if (g == 0) pk.M[T4][n] = M[T4];
                    }
                    if (lane == 0) {
                        pk.j = j;
                        pk.keep = bits;
                    }
                    ++parked;
                }
            }
        }
        if (parked == 0) continue;
        wave_lds_fence();
        // attend the parked blocks' tiles k = 4e + T4 in pairs, two tiles in flight; the pair loop
        // is not unrolled, so the tile code exists twice and the register budget stays bounded
        const int ntile = 4 * parked;
        auto tile_of = [&](int k) { return 4 * sm.park[wave][k >> 2].j + (k & 3); };
        TileGather g0 = load_tile_gather(resid_bh, v_bh, tile_of(0), lane, L);
        TileGather g1 = load_tile_gather(resid_bh, v_bh, tile_of(1), lane, L);
#pragma unroll 1
        for (int k = 0; k < ntile; k += 2) {
            attend_tile(g0, sm.park[wave][k >> 2], k & 3);
            g0 = load_tile_gather(resid_bh, v_bh, tile_of(min(k + 2, ntile - 1)), lane, L);
            attend_tile(g1, sm.park[wave][(k + 1) >> 2], (k + 1) & 3);
            g1 = load_tile_gather(resid_bh, v_bh, tile_of(min(k + 3, ntile - 1)), lane, L);
        }
    }

    write_partials<NT>(sm.epi, pv, m_run, l_part, wave, lane, G, hq0, a.Hq, a.S, b, s, a.part_m,
                       a.part_l, a.part_acc);

    // Mask entries past the end of the sequence are zero (spread over the splits).
    if (a.mask) {
        for (int j = nblk + s * kThreads + tid; j < nblk_cap; j += a.S * kThreads)
            for (int h = 0; h < G; ++h) a.mask[((size_t)b * a.Hq + hq0 + h) * nblk_cap + j] = 0;
    }
}

template __global__ void ffd_decode_kernel<1>(DecodeArgs);
template __global__ void ffd_decode_kernel<2>(DecodeArgs);

}  // namespace ffd
