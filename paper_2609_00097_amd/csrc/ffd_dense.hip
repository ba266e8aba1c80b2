// Dense flash-decode attention for gfx950 (the exact comparator): softmax(alpha q K^T) V over all
// tokens of each sequence, split along the sequence and merged by log-sum-exp.
//
// Mapping. A workgroup (4 waves) serves one run of blocks of a (sequence, KV head): in balanced
// mode (batches of up to kDenseBalanceMaxSeqs sequences) the runs have equal lengths across the
// whole ragged batch, the workgroups being given to the sequences in proportion to their blocks;
// otherwise each sequence is split into S equal runs. Wave w owns the 16-token tile w of every
// 64-token block and keeps its own online-softmax state. QK^T runs on
// v_mfma_f32_16x16x32_bf16 with the queries as the A operand (head h of a 4-head tile on row 4h,
// other rows zero) and the tile's keys as B: lane (g, n) loads token n's dims 32g..32g+31 (64
// contiguous bytes), so its output register 0 is head g's score for token n. PV runs on the VALU
// in fp32. The next block's key and value tiles are requested before the current one is used.
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

template <int NT>
struct DenseLds {
    TileP<NT> tp[kWaves];
    EpilogueLds<NT> epi;
};

struct KTile {
    uint4 k[4];
};

// Key row `tok`, clamped to last_row (a valid row): the score of a token past the end is masked to
// -inf by the caller. The loads are unconditional so the compiler can count them.
__device__ __forceinline__ KTile load_ktile(const uint16_t* k_bh, int tok, int last_row, int g) {
    KTile r;
    const uint4* kp = reinterpret_cast<const uint4*>(k_bh + (size_t)min(tok, last_row) * kD + 32 * g);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) r.k[ks] = kp[ks];
    return r;
}

}  // namespace

// Balanced mode: this workgroup's (sequence, KV head) and run of blocks, computed by every wave
// alone from the sequence lengths (lane l: sequences 4l .. 4l + 3). Returns false for a workgroup
// past the last one used.
__device__ __forceinline__ bool dense_balanced_share(const DenseArgs& a, int wg, int lane, int& b, int& kvh,
                                                     int& jb, int& je) {
    int nb[4], sum = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int bi = 4 * lane + k;
        const int L = bi < a.B ? min(max(a.seq_lens[bi], 0), a.Lcap) : 0;
        nb[k] = (L + kBlock - 1) / kBlock;
        sum += nb[k];
    }
    const int incl = wave_inclusive_scan(sum);
    const long long N = (long long)__builtin_amdgcn_readlane(incl, 63) * a.Hkv;
    const long long W = (long long)a.S * a.B * a.Hkv;
    const long long Weff = N > 0 ? min(W, N) : 1;
    int wb[4], span = 0;                            // workgroups per KV head of each sequence
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int bi = 4 * lane + k;
        wb[k] = bi < a.B ? (nb[k] > 0 ? (int)(((long long)nb[k] * Weff + N - 1) / N) : 1) : 0;
        span += wb[k] * a.Hkv;
    }
    const int sincl = wave_inclusive_scan(span);
    int q0 = sincl - span, hit = -1;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (hit < 0 && wg >= q0 && wg < q0 + wb[k] * a.Hkv) hit = k;
        if (hit < 0) q0 += wb[k] * a.Hkv;
    }
    const uint64_t hb = __ballot(hit >= 0);
    if (hb == 0) return false;                      // uniform: past the last sequence's workgroups
    const int src = __builtin_amdgcn_readfirstlane((int)__builtin_ctzll(hb));
    const int kk = __builtin_amdgcn_readlane(hit, src);
    int wsel = wb[0], nsel = nb[0];
#pragma unroll
    for (int k = 1; k < 4; ++k) if (kk == k) { wsel = wb[k]; nsel = nb[k]; }
    const int Wb = __builtin_amdgcn_readlane(wsel, src), n = __builtin_amdgcn_readlane(nsel, src);
    const int Qb = __builtin_amdgcn_readlane(q0, src);
    b = 4 * src + kk;
    kvh = (wg - Qb) / Wb;
    const int p = (wg - Qb) % Wb;
    jb = (int)((long long)p * n / Wb);
    je = (int)((long long)(p + 1) * n / Wb);
    if (p == 0 && lane == 0 && threadIdx.x == 0)
        a.table[(size_t)b * a.Hkv + kvh] = make_int2(Qb + kvh * Wb, Wb);
    return true;
}

template <int NT>
__global__ __launch_bounds__(kThreads, NT == 1 ? 4 : 2) void dense_decode_kernel(DenseArgs a) {
    __shared__ DenseLds<NT> sm;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, n = lane & 15;
    const bool balanced = a.table != nullptr;
    int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z, jb = 0, je = 0;
    if (balanced) {
        if (!dense_balanced_share(a, blockIdx.x, lane, b, kvh, jb, je)) return;
        b = __builtin_amdgcn_readfirstlane(b);
        kvh = __builtin_amdgcn_readfirstlane(kvh);
        jb = __builtin_amdgcn_readfirstlane(jb);
        je = __builtin_amdgcn_readfirstlane(je);
    }
    const int G = a.G, hq0 = kvh * G;
    const size_t bh = (size_t)b * a.Hkv + kvh;
    const int L = min(max(a.seq_lens[b], 0), a.Lcap);
    const int nblk = (L + kBlock - 1) / kBlock;
    if (!balanced) {
        const int bps = (nblk + a.S - 1) / a.S;
        jb = min(s * bps, nblk);
        je = min(jb + bps, nblk);
    }
    const uint16_t* k_bh = a.k + bh * (size_t)a.Lcap * kD;
    const uint16_t* v_bh = a.v + bh * (size_t)a.Lcap * kD;

    // First block's tiles before the setup. Rows are clamped to the last valid row, so look-ahead
    // past the split never leaves the sequence; the real index decides what is valid.
    const int last_row = max(L, 1) - 1;
    KTile kc = load_ktile(k_bh, 64 * jb + 16 * wave + n, last_row, g);
    VTile vc = load_vtile(v_bh, 64 * jb + 16 * wave, last_row, lane);

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
    TileP<NT>& tp = sm.tp[wave];

    for (int j = jb; j < je; ++j) {
        const int tok = 64 * j + 16 * wave + n;
        const KTile kn = load_ktile(k_bh, 64 * (j + 1) + 16 * wave + n, last_row, g);
        const VTile vn = load_vtile(v_bh, 64 * (j + 1) + 16 * wave, last_row, lane);
        float z[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Aq[t][ks], __builtin_bit_cast(v8bf, kc.k[ks]),
                                                              acc, 0, 0, 0);
            z[t] = tok < L ? acc.x * a.scale : -INFINITY;
        }
        softmax_tile<NT>(z, live, m_run, l_part, tp, g, n);
        wave_lds_fence();
        pv_tile<NT>(pv, tp, vc);
        wave_lds_fence();
        kc = kn;
        vc = vn;
    }

    if (balanced)
        write_partials<NT>(sm.epi, pv, m_run, l_part, wave, lane, G, (size_t)blockIdx.x * G, 1, a.part_m,
                           a.part_l, a.part_acc);
    else
        write_partials<NT>(sm.epi, pv, m_run, l_part, wave, lane, G, ((size_t)b * a.Hq + hq0) * a.S + s,
                           (size_t)a.S, a.part_m, a.part_l, a.part_acc);
}

template __global__ void dense_decode_kernel<1>(DenseArgs);
template __global__ void dense_decode_kernel<2>(DenseArgs);

}  // namespace ffd
