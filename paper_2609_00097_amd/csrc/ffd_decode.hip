// FFD decode attention for gfx950: b-bit thumbnail scan (b = 2, 4, 8; App. C) + top-delta
// selection, then refinement + online softmax over the kept blocks.
//
// Method (Alg. 1; Eq. 1-4): for each query head h of a KV group,
//   s_hat[t] = alpha * q . k^quant_t                      (thumbnail scan)
//   m~       = max of s_hat over the first n_sink and last n_local tokens      (pseudo-max, Eq. 3)
//   keep j   iff max_{t in block j} s_hat[t] >= m~ - delta                       (top-delta, Eq. 1)
//   z[t]     = s_hat[t] + alpha * q . k^res_t   for t in kept blocks            (scan reuse, Eq. 4)
//   out      = softmax(z) . V over kept tokens, split into partial states merged by LSE.
//
// Arithmetic. The group's queries are the A operand of v_mfma_i32_16x16x64_i8: each query is held in
// fixed point Q = rint(q * 2^(22-E)) (|q| < 2^E), split into three signed 8-bit limbs, one MFMA row
// per (head, limb). The B operand is either a 16-token tile's codes as bytes (2- and 4-bit codes
// expanded by two VALU ops per 4 codes, 8-bit codes stored as the signed bytes c - 128) or its stored
// int8 residual, so both dot products are exact integer sums, combined and rounded once to fp32:
//   sum_d Q_d (2 c_d - (2^b - 1)) = T  (exact: int32 for b = 2, int64 otherwise),
//                                   s_hat = T * M_t * alpha 2^(E-23) / Lv,   Lv = (2^b - 1) / 2
//   sum_d Q_d r_d                 = R  (three int32 limbs), z = s_hat + R * M_t * alpha 2^(E-22) / (254 Lv)
// Output register i of lane (g, n) is row 4g + i, column n: head g's limbs for token n, so each
// 16-lane row group owns one head and a tile's maximum is a 16-lane DPP reduction.
//
// Two ways to run a step, chosen by the host (FFD_KERNELS_*):
//  * ffd_decode_kernel, the fused kernel (short and mid contexts: at most 64 blocks per
//    workgroup): S1 workgroups per (sequence, KV head) each scan an interleaved share of the group's
//    blocks (j = s + S1 i), decide them, and refine and attend their own kept blocks; one partial
//    state per head (or, with S1 = 1, the outputs themselves).
//  * the split kernels, where the kept blocks are too many for their owners to refine in time:
//    - ffd_scan_kernel streams the codes and absmaxes of every block once (the dominant, perfectly
//      regular stream; one 8-wave workgroup per CU whose waves take blocks from an LDS counter),
//      keeps each block's per-head maximum score in LDS and, once its stream and the pseudo-max are
//      done, takes the keep decision per (head, block): the kept blocks, with their per-head keep
//      bits, form its workgroup's kept list (in block order) in the workspace, plus the list's
//      length;
//    - ffd_refine_kernel gives each (sequence, KV head) a number of workgroups proportional to its
//      kept blocks (every workgroup computes the same allocation from the scan's counts, so no
//      cross-workgroup synchronisation is needed); each 8-wave workgroup refines an equal share of
//      its group's kept blocks, wave w taking 16-token tile w % 4 of every other block, with
//      several tiles' residual and value loads in flight, and writes one partial (m, l, acc) per
//      head; lse_merge_kernel combines the partials of each head through a small per-group table.
// Both recompute the scan scores s_hat of each kept tile from its codes (Eq. 4's reuse term: the
// same integer MFMA and fp32 operations as the scan, so the same values; storing them would cost
// as many bytes, written then read).
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

#ifndef FFD_SCAN_RING
#define FFD_SCAN_RING 4
#endif
#ifndef FFD_REFINE_RING
#define FFD_REFINE_RING 2
#endif
constexpr int kRing2 = FFD_SCAN_RING;         // 2-bit scan loads in flight per wave (blocks)
constexpr int kRefineRing = FFD_REFINE_RING;  // refinement tiles in flight per wave
constexpr int kChunk = kFfdChunk;             // list entries staged per pass of the refinement kernel

__device__ __forceinline__ int limb_of(int Q, int which) {
    const int l0 = ((Q + 128) & 255) - 128;
    const int q1 = (Q - l0) >> 8;
    const int l1 = ((q1 + 128) & 255) - 128;
    const int l2 = (q1 - l1) >> 8;
    return which == 0 ? l0 : (which == 1 ? l1 : l2);
}

// The 16 codes of one (tile, 64-dim chunk) group of a lane, from its b/2 words, as the MFMA B
// operand: byte i of dword k is dim 4k + i of the lane's 16-dim slice.
template <int BITS>
__device__ __forceinline__ v4i expand_codes(const uint32_t* w) {
    v4i r;
    if constexpr (BITS == 2) {
        r.x = (int)(w[0] & 0x03030303u);
        r.y = (int)((w[0] >> 2) & 0x03030303u);
        r.z = (int)((w[0] >> 4) & 0x03030303u);
        r.w = (int)((w[0] >> 6) & 0x03030303u);
    } else if constexpr (BITS == 4) {
        r.x = (int)(w[0] & 0x0f0f0f0fu);
        r.y = (int)((w[0] >> 4) & 0x0f0f0f0fu);
        r.z = (int)(w[1] & 0x0f0f0f0fu);
        r.w = (int)((w[1] >> 4) & 0x0f0f0f0fu);
    } else {
        r.x = (int)w[0]; r.y = (int)w[1]; r.z = (int)w[2]; r.w = (int)w[3];
    }
    return r;
}

template <int NT>
struct HeadConsts {
    v4i A[NT][2];      // MFMA A operand per head tile and 64-dim chunk
    int sumq[NT];      // sum_d Q_d of head 4t + g
    float kap[NT];     // alpha * 2^(E-23) / Lv
    float kap2[NT];    // alpha * 2^(E-22) / (254 Lv)
    bool live[NT];     // head 4t + g exists
};

template <int NT>
struct QueryLds {
    alignas(16) int8_t limbs[4][4 * NT][kD];     // [limb][head][dim]; limb 3 is zero
    int sumq[4 * NT];
    float kap[4 * NT];
    float kap2[4 * NT];
};

// This lane's dword (dims 2*lane, 2*lane + 1) of the queries of heads wave + 4t of the group.
template <int NT>
__device__ __forceinline__ void load_query_words(const uint16_t* __restrict__ q, int b, int Hq, int hq0,
                                                 int G, int wave, int lane, uint32_t (&qw)[NT]) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
        qw[t] = reinterpret_cast<const uint32_t*>(q + ((size_t)b * Hq + hq0 + min(wave + 4 * t, G - 1)) * kD)[lane];
}

// Queries -> fixed-point limbs in LDS and this lane's per-head constants. Head h (wave h % 4): E with
// max|q| < 2^E, Q = rint(q 2^(22-E)) split into three signed bytes stored as limbs[limb][h][d]; the
// fourth limb row and heads past G stay zero. lv is the thumbnail's outer level Lv. Contains two
// workgroup barriers.
template <int NT>
__device__ __forceinline__ void build_query_consts(QueryLds<NT>& sm, const uint32_t (&qw)[NT], int G,
                                                   float scale, float lv, int tid, HeadConsts<NT>& hc) {
    const int wave = tid >> 6, lane = tid & 63, g = lane >> 4, n = lane & 15;
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
            sm.sumq[h] = sum;
            sm.kap[h] = ldexpf(scale / lv, E - 23);
            sm.kap2[h] = ldexpf(scale / (254.f * lv), E - 22);
        }
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        // A operand: row m = n is (head 4t + n/4, limb n%4); its 16 bytes are dims 64cc + 16g + e.
        const int hrow = 4 * t + (n >> 2), limb = n & 3;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc)
            hc.A[t][cc] = *reinterpret_cast<const v4i*>(&sm.limbs[limb][hrow][64 * cc + 16 * g]);
        const int hh = 4 * t + g;      // this lane's output head
        hc.live[t] = hh < G;
        hc.sumq[t] = hc.live[t] ? sm.sumq[hh] : 0;
        hc.kap[t] = hc.live[t] ? sm.kap[hh] : 0.f;
        hc.kap2[t] = hc.live[t] ? sm.kap2[hh] : 0.f;
    }
}

// The same constants built by one wave alone, with no workgroup barrier: the wave computes every
// head (qa[h]: this lane's dword of head h, any value for h >= G) and writes the whole limb table;
// every wave of a workgroup writes identical values, so each may read back what it wrote itself
// (one wave's LDS operations execute in order) without waiting for the others. Bit for bit the
// values of build_query_consts.
template <int NT>
__device__ __forceinline__ void build_query_consts_wave(QueryLds<NT>& sm, const uint32_t (&qa)[4 * NT], int G,
                                                        float scale, float lv, int lane, HeadConsts<NT>& hc) {
    const int g = lane >> 4, n = lane & 15;
#pragma unroll
    for (int h = 0; h < 4 * NT; ++h) {
        const bool live = h < G;
        const float x0 = live ? bf16_lo(qa[h]) : 0.f, x1 = live ? bf16_hi(qa[h]) : 0.f;
        const float mx = wave_max_dpp(fmaxf(fabsf(x0), fabsf(x1)));
        int E = 0;
        (void)frexpf(mx, &E);                       // mx < 2^E (mx == 0 -> E = 0)
        const int Q0 = (int)rintf(ldexpf(x0, 22 - E));
        const int Q1 = (int)rintf(ldexpf(x1, 22 - E));
#pragma unroll
        for (int li = 0; li < 3; ++li) {
            const uint32_t pair = ((uint32_t)limb_of(Q0, li) & 0xffu) | (((uint32_t)limb_of(Q1, li) & 0xffu) << 8);
            reinterpret_cast<uint16_t*>(&sm.limbs[li][h][0])[lane] = (uint16_t)pair;
        }
        reinterpret_cast<uint16_t*>(&sm.limbs[3][h][0])[lane] = 0;
        const int sum = wave_sum_dpp(Q0 + Q1);
        if (lane == 0) {
            sm.sumq[h] = sum;
            sm.kap[h] = ldexpf(scale / lv, E - 23);
            sm.kap2[h] = ldexpf(scale / (254.f * lv), E - 22);
        }
    }
    wave_lds_fence();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int hrow = 4 * t + (n >> 2), limb = n & 3;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc)
            hc.A[t][cc] = *reinterpret_cast<const v4i*>(&sm.limbs[limb][hrow][64 * cc + 16 * g]);
        const int hh = 4 * t + g;
        hc.live[t] = hh < G;
        hc.sumq[t] = hc.live[t] ? sm.sumq[hh] : 0;
        hc.kap[t] = hc.live[t] ? sm.kap[hh] : 0.f;
        hc.kap2[t] = hc.live[t] ? sm.kap2[hh] : 0.f;
    }
}

// One lane's share of a block's thumbnail: its 4b code words (both 64-dim halves of its token in
// each of the four tiles; w[i] = words 4i .. 4i + 3, each load 1 KiB contiguous over the wave) and
// the absmax of its four tokens.
template <int BITS>
struct BlockScan {
    uint4 w[BITS];
    uint2 mm;
};

template <int BITS>
__device__ __forceinline__ BlockScan<BITS> load_block_scan(const uint32_t* __restrict__ codes_bh,
                                                           const uint16_t* __restrict__ absmax_bh, int j,
                                                           int lane) {
    const uint4* cp = reinterpret_cast<const uint4*>(codes_bh) + (size_t)j * 64 * BITS + lane;
    BlockScan<BITS> r;
#pragma unroll
    for (int i = 0; i < BITS; ++i) r.w[i] = cp[64 * i];               // words 4i .. 4i + 3
    r.mm = *reinterpret_cast<const uint2*>(absmax_bh + (size_t)j * 64 + (lane & 15) * 4);
    return r;
}

// The same loads through buffer resources whose ranges end at a workgroup's last block: a block
// index at or past that end reads zeros without touching memory (the hardware range check of a raw
// buffer), so a wave may request blocks that turn out not to exist.
constexpr int kRawBufferWord3 = 0x00020000;    // gfx9 raw buffer: 32-bit data format, no swizzle
template <int BITS>
__device__ __forceinline__ BlockScan<BITS> load_block_scan_rsrc(__amdgpu_buffer_rsrc_t rc, __amdgpu_buffer_rsrc_t ra,
                                                                int j, int lane) {
    BlockScan<BITS> r;
    const uint32_t base = (uint32_t)j * (1024u * BITS) + (uint32_t)lane * 16u;
#pragma unroll
    for (int i = 0; i < BITS; ++i) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(rc, (int)(base + 1024u * i), 0, 0);
        r.w[i] = make_uint4(v[0], v[1], v[2], v[3]);
    }
    const auto m = __builtin_amdgcn_raw_buffer_load_b64(ra, (int)((uint32_t)j * 128u + (uint32_t)(lane & 15) * 8u), 0, 0);
    r.mm = make_uint2(m[0], m[1]);
    return r;
}

// Thumbnail scores of one 16-token tile for this lane's head(s) and token n: tw holds the lane's b
// words of the tile (64-dim chunk 0, then chunk 1), M the token's absmax; -inf for a token past L.
template <int NT, int BITS>
__device__ __forceinline__ void tile_scores(const uint32_t* tw, float M, bool valid, const HeadConsts<NT>& hc,
                                            float (&sc)[NT]) {
    const v4i b0 = expand_codes<BITS>(tw);
    const v4i b1 = expand_codes<BITS>(tw + BITS / 2);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        v4i acc = {0, 0, 0, 0};
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], b0, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], b1, acc, 0, 0, 0);
        float Tf;
        if constexpr (BITS == 2) {
            // |sum_d Q_d (2 c_d - 3)| <= 3 * 128 * 2^22 < 2^31: exact modulo 2^32
            const uint32_t s = (uint32_t)acc.x + ((uint32_t)acc.y << 8) + ((uint32_t)acc.z << 16);
            Tf = (float)(int)(2u * s - 3u * (uint32_t)hc.sumq[t]);
        } else {
            const long long s = (long long)acc.x + ((long long)acc.y << 8) + ((long long)acc.z << 16);
            // 8-bit codes are the bytes c - 128, and 2c - 255 = 2 (c - 128) + 1
            const long long T = BITS == 8 ? 2 * s + hc.sumq[t]
                                          : 2 * s - (long long)((1 << BITS) - 1) * hc.sumq[t];
            Tf = (float)T;
        }
        sc[t] = valid ? Tf * (M * hc.kap[t]) : -INFINITY;
    }
}

// Thumbnail scores of block j for this lane's head(s) and tokens 64j + 16*T4 + n; -inf past L.
// Lane words of tile T4 are words T4*b .. T4*b + b - 1 (the storage layout of ffd.h).
template <int NT, int BITS>
__device__ __forceinline__ void block_scores(const BlockScan<BITS>& ld, int j, int lane, int L,
                                             const HeadConsts<NT>& hc, float (&sc)[NT][4]) {
    const int n = lane & 15;
    const float M[4] = {bf16_lo(ld.mm.x), bf16_hi(ld.mm.x), bf16_lo(ld.mm.y), bf16_hi(ld.mm.y)};
    uint32_t words[4 * BITS];
#pragma unroll
    for (int i = 0; i < BITS; ++i) {
        words[4 * i] = ld.w[i].x; words[4 * i + 1] = ld.w[i].y;
        words[4 * i + 2] = ld.w[i].z; words[4 * i + 3] = ld.w[i].w;
    }
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4) {
        float st[NT];
        tile_scores<NT, BITS>(&words[T4 * BITS], M[T4], 64 * j + 16 * T4 + n < L, hc, st);
#pragma unroll
        for (int t = 0; t < NT; ++t) sc[t][T4] = st[t];
    }
}

template <int NT>
struct ScanLds {
    QueryLds<NT> qs;
    alignas(16) float pm[kScanWaves][4 * NT];             // each wave's window maxima per head
    alignas(16) float sig[kFfdMaxScanBlocks][4 * NT];     // block maxima of the thumbnail scores per head
    int nkept[kScanWaves];                    // kept blocks per wave
    int next;                                 // next block to hand out
};

// ---- refinement helpers ---------------------------------------------------------------------

// One wave's loads for one 16-token tile of a kept block: int8 residual, its lane's value dwords,
// the token's absmax and the lane's RBITS code words of the tile, from which the scan scores are
// recomputed.
template <int NT, int RBITS>
struct RefineTile {
    v4i r0, r1;
    VTile vt;
    uint32_t cw[RBITS];
    uint32_t m;       // absmax bf16 bits in the low half
};

// An address every lane holds alike, moved to scalar registers: a buffer resource built from it is
// then one scalar value (the compiler cannot always see that the block number and the wave index
// are uniform, and otherwise loops over the lanes' distinct resources).
template <typename T>
__device__ __forceinline__ void* uniform_ptr(const T* p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
}

// All five loads go through buffer resources based at the tile (the block number is wave-uniform):
// the per-lane offsets are 32-bit and shared, the per-row ones immediates, which saves the 64-bit
// address arithmetic of every row (about a tenth of the tile's instructions). The value resource
// ends at the sequence end, so value rows past it read zeros (their probability is zero).
template <int NT, int RBITS>
__device__ __forceinline__ RefineTile<NT, RBITS> load_refine_tile(const int8_t* __restrict__ resid_bh,
                                                                  const uint16_t* __restrict__ v_bh,
                                                                  const uint32_t* __restrict__ codes_bh,
                                                                  const uint16_t* __restrict__ absmax_bh,
                                                                  int j, int T4, int lane, int L) {
    RefineTile<NT, RBITS> r;
    const int tile = 4 * j + T4;
    const uint32_t lo16 = (uint32_t)lane * 16u;
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        uniform_ptr(resid_bh + (size_t)tile * 2048), (short)0, 2048, kRawBufferWord3);
    r.r0 = (v4i)__builtin_amdgcn_raw_buffer_load_b128(rr, (int)lo16, 0, 0);
    r.r1 = (v4i)__builtin_amdgcn_raw_buffer_load_b128(rr, (int)(lo16 + 1024u), 0, 0);
    const int vrows = __builtin_amdgcn_readfirstlane(min(max(L - 16 * tile, 0), 16));
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        uniform_ptr(v_bh + (size_t)tile * (16 * kD)), (short)0, vrows * (2 * kD), kRawBufferWord3);
#pragma unroll
    for (int t = 0; t < 16; ++t) r.vt.v[t] = __builtin_amdgcn_raw_buffer_load_b32(rv, lane * 4 + t * (2 * kD), 0, 0);
    // tile T4 is the lane's words T4*b .. T4*b + b - 1 of block j; word w at [w / 4][lane][w % 4]
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        uniform_ptr(codes_bh + (size_t)j * (256 * RBITS)), (short)0, 1024 * RBITS, kRawBufferWord3);
    if constexpr (RBITS == 2) {
        const auto w = __builtin_amdgcn_raw_buffer_load_b64(rc, (int)(lo16 + (T4 >> 1) * 1024u + (T4 & 1) * 8u), 0, 0);
        r.cw[0] = w[0]; r.cw[1] = w[1];
    } else {
#pragma unroll
        for (int i = 0; i < RBITS / 4; ++i) {
            const auto w = __builtin_amdgcn_raw_buffer_load_b128(rc, (int)(lo16 + (T4 * (RBITS / 4) + i) * 1024u), 0, 0);
            r.cw[4 * i] = w[0]; r.cw[4 * i + 1] = w[1]; r.cw[4 * i + 2] = w[2]; r.cw[4 * i + 3] = w[3];
        }
    }
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        uniform_ptr(absmax_bh + (size_t)j * 64), (short)0, 128, kRawBufferWord3);
    r.m = __builtin_amdgcn_raw_buffer_load_b16(ra, ((lane & 15) * 4 + T4) * 2, 0, 0);
    return r;
}

constexpr int kPairChunk = 4 * kThreads;     // KV groups allocated per pass (4 per thread)
constexpr int kCountCache = 4096;            // scan counts kept in LDS when they all fit

template <int NT>
struct RefineLds {
    QueryLds<NT> qs;
    int wsum[2][kRefineWaves];           // wg_exclusive_scan scratch, alternating halves
    int sel[4];                          // this workgroup's KV group: pair, first workgroup, workgroups, kept
    int pn[kPairChunk];                  // kept blocks per KV group of the current pass (large inputs)
    int cnt[kCountCache + 1];            // exclusive prefix of all scan counts, when they fit
    int pref[kFfdMaxScanSplits + 1];     // exclusive prefix of the group's per-split counts (large inputs)
    TileP<NT> tp[kRefineWaves];
    union {
        uint32_t list[kChunk];           // kept blocks of the share: j | keep bits << 24
        EpilogueLds<NT, kRefineWaves> epi;
    } u;
};

}  // namespace

// ================================================================================================
// Scan: b-bit thumbnail scan and pseudo-max, then the keep decisions; the kept list (or, for the
// top-k rule, every block's scores) to the workspace.
// Grid (S1, Hkv, B) of kScanWaves-wave workgroups; workgroup s1 scans blocks [s1 * bps, (s1 + 1) *
// bps) of one (sequence, KV head), bps = ceil(nblk / S1) <= kFfdMaxScanBlocks; its waves take the
// blocks one at a time from an LDS counter and keep kRing blocks in flight each.
// ================================================================================================
// Blocks in flight per wave, fewer for the wider thumbnails (whose blocks are 2x and 4x larger).
template <int BITS> constexpr int scan_ring() { return BITS == 2 ? kRing2 : 2; }

// Adds the residual term of Eq. 4 to the thumbnail scores sc of block j (the refined logits of its
// tokens, computed exactly as the refinement kernel computes them).
template <int NT>
__device__ __forceinline__ void add_residual_term(const int8_t* __restrict__ resid_bh, uint2 mm, int j,
                                                  int lane, const HeadConsts<NT>& hc, float (&sc)[NT][4]) {
    const float M[4] = {bf16_lo(mm.x), bf16_hi(mm.x), bf16_lo(mm.y), bf16_hi(mm.y)};
    v4i r[4][2];
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4) {
        const v4i* rp = reinterpret_cast<const v4i*>(resid_bh) + (size_t)(4 * j + T4) * 128 + lane;
        r[T4][0] = rp[0];
        r[T4][1] = rp[64];
    }
#pragma unroll
    for (int T4 = 0; T4 < 4; ++T4) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], r[T4][0], acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], r[T4][1], acc, 0, 0, 0);
            const float R = fmaf(65536.f, (float)acc.z, fmaf(256.f, (float)acc.y, (float)acc.x));
            const float sct = sc[t][T4];
            sc[t][T4] = sct == -INFINITY ? -INFINITY : fmaf(R, M[T4] * hc.kap2[t], sct);
        }
    }
}

// Workgroups per CU the registers must allow: two, so that a grid slightly larger than the CU count
// (S1 rounded up) runs in one wave of workgroups; the 8-bit blocks need more registers.
template <int BITS> constexpr int scan_occupancy() { return BITS == 8 ? 1 : 2; }

template <int NT, int BITS, int MODE>
__global__ __launch_bounds__(kScanThreads, scan_occupancy<BITS>()) void ffd_scan_kernel(ScanArgs a) {
    constexpr bool kTopK = MODE == kSelTopK;
    constexpr int kRing = scan_ring<BITS>();
    __shared__ ScanLds<NT> sm;
    const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, n = lane & 15;
    const int G = a.G, hq0 = kvh * G;
    const size_t bh = (size_t)b * a.Hkv + kvh;
    const int L = min(max(a.seq_lens[b], 0), a.Lcap);
    const int nblk = (L + kBlock - 1) / kBlock;
    const int nblk_cap = a.Lcap / kBlock;
    const int bps = (nblk + a.S1 - 1) / a.S1;
    const int jb = min(s * bps, nblk), je = min(jb + bps, nblk);
    if (jb >= je && (kTopK || !a.mask)) {       // nothing to scan (short sequence), nothing to clear
        if constexpr (!kTopK) {
            if (tid == 0) a.counts[bh * a.S1 + s] = 0;
            if (a.m_tilde && s == 0 && tid < G) a.m_tilde[(size_t)b * a.Hq + hq0 + tid] = -INFINITY;   // L = 0
        }
        return;
    }

    const uint32_t* codes_bh = a.codes + bh * (size_t)a.Lcap * (4 * BITS);
    const uint16_t* absmax_bh = a.absmax + bh * (size_t)a.Lcap;

    // The stream reads through buffer resources whose ranges end at block je, so a request for a
    // block >= je reads zeros without touching memory (the hardware range check of a raw buffer):
    // every load is issued unconditionally, and uniform control flow lets the compiler wait for
    // exactly the load it needs instead of draining every load in flight (which a conditional load
    // made it do). Offsets and sizes are unsigned 32-bit: at most 2^18 blocks of 8 KiB.
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(codes_bh), (short)0, (int)((uint32_t)je * (1024u * BITS)), kRawBufferWord3);
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(absmax_bh), (short)0, (int)((uint32_t)je * 128u), kRawBufferWord3);
    // Work distribution: wave w starts with blocks jb + kRing w + r (r < kRing), then takes the next
    // block from an LDS counter each time it scores one, so the waves of a CU finish together however
    // its memory requests are served (a CU serves its oldest waves first: with fixed shares, the
    // workgroups of one CU ended up to 12 us apart at 4 x 128K).
    int js[kRing];                                  // block held by each ring slot (>= je: none)
#pragma unroll
    for (int r = 0; r < kRing; ++r) js[r] = jb + kRing * wave + r;

    // Order of requests: queries, the window blocks of the first pseudo-max pass (clamped to valid
    // blocks), the first ring round. Each wave scores its window blocks on its own before its first
    // block (the refined logits: after the stream, with the window blocks' residual tiles) and only
    // writes their maxima to LDS; every keep decision waits for the end of the stream, where the
    // pseudo-max is known, so no wave waits on another before or during its stream (a
    // workgroup-wide window pass before the stream held every wave until the slowest one's window
    // blocks had arrived behind the whole chip's first round: 6 us at the median, 20 us at worst at
    // 4 x 128K). Until then a block costs G floats of LDS.
    uint32_t qw[NT];
    load_query_words<NT>(a.q, b, a.Hq, hq0, G, wave, lane, qw);
    const int jlast = max(nblk, 1) - 1;
    const int sink_end = min(a.n_sink, L);
    const int loc_beg = max(0, L - a.n_local);
    const int sink_blk_end = (sink_end + kBlock - 1) / kBlock;
    const int loc_blk_beg = max(loc_beg / kBlock, sink_blk_end);
    const int npm = sink_blk_end + max(nblk - loc_blk_beg, 0);
    auto pm_block = [&](int idx) { return idx < sink_blk_end ? idx : loc_blk_beg + (idx - sink_blk_end); };
    auto win_block = [&](int idx) { return min(pm_block(min(idx, max(npm, 1) - 1)), jlast); };
    constexpr bool kEarlyWindows = MODE == kSelThumbnailPM;
    BlockScan<BITS> win;                            // wave w's window block of the current pass
    auto load_window = [&](int base) { win = load_block_scan<BITS>(codes_bh, absmax_bh, win_block(base + wave), lane); };
    if constexpr (kEarlyWindows) load_window(0);
    BlockScan<BITS> ring[kRing];
#pragma unroll
    for (int i = 0; i < kRing; ++i) ring[i] = load_block_scan_rsrc<BITS>(rc, ra, min(js[i], je), lane);
    if (tid == 0) sm.next = jb + kScanWaves * kRing;   // visible after the barriers below
    if constexpr (MODE == kSelRefinedPM) load_window(0);

    HeadConsts<NT> hc;
    build_query_consts<NT>(sm.qs, qw, G, a.scale, thumb_top_level(BITS), tid, hc);

    // ---- scan (Alg. 1): block maxima sigma per head, and the pseudo-max's window maxima -------
    float pm[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) pm[t] = -INFINITY;
    auto window_max = [&](const float (&sc)[NT][4], int j) {     // over the window tokens of block j
#pragma unroll
        for (int T4 = 0; T4 < 4; ++T4) {
            const int tok = 64 * j + 16 * T4 + n;
            const bool in_win = tok < L && (tok < sink_end || tok >= loc_beg);
#pragma unroll
            for (int t = 0; t < NT; ++t) pm[t] = fmaxf(pm[t], in_win ? sc[t][T4] : -INFINITY);
        }
    };
    auto window_pass = [&](int base) {              // wave w: window block base + w
        const int idx = base + wave;
        if (idx >= npm) return;                     // wave-uniform
        const int j = pm_block(idx);
        float sc[NT][4];
        block_scores<NT, BITS>(win, j, lane, L, hc, sc);
        if constexpr (MODE == kSelRefinedPM)
            add_residual_term<NT>(a.resid + bh * (size_t)a.Lcap * kD, win.mm, j, lane, hc, sc);
        window_max(sc, j);
    };
    auto consume = [&](const BlockScan<BITS>& blk, int j) {
        float sc[NT][4];
        block_scores<NT, BITS>(blk, j, lane, L, hc, sc);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            // + 0 turns a -0 score (a zero key) into +0, so that equal scores compare equal
            const float sig = row16_max(fmaxf(fmaxf(sc[t][0], sc[t][1]), fmaxf(sc[t][2], sc[t][3]))) + 0.f;
            if constexpr (kTopK) {
                if (n == 0 && hc.live[t]) a.sigma[(bh * (size_t)nblk_cap + j) * G + 4 * t + g] = sig;
            } else {
                if (n == 0) sm.sig[j - jb][4 * t + g] = sig;
            }
        }
    };
    if constexpr (kEarlyWindows) window_pass(0);     // its block arrives ahead of the first round
    // Each slot in turn: take the next block number (its LDS round trip hides behind the scoring),
    // score the slot's block if it has one, refill the slot. The loop ends once a whole round has
    // taken no block below je: every slot then holds none, and its last loads read no memory.
    for (bool more = true; more;) {                 // wave-uniform
        more = false;
#pragma unroll
        for (int r = 0; r < kRing; ++r) {
            int jn = 0;
            if (lane == 0) jn = atomicAdd(&sm.next, 1);
            jn = __builtin_amdgcn_readfirstlane(jn);
            if (js[r] < je) consume(ring[r], js[r]);
            ring[r] = load_block_scan_rsrc<BITS>(rc, ra, min(jn, je), lane);
            js[r] = jn;
            more |= jn < je;
        }
    }

    if constexpr (kTopK) return;                // the top-k rule compares block scores with each other

    // ---- pseudo-max over the sink and local windows (Eq. 3): the first pass unless done during
    // the stream, further passes (wide windows) loaded now -------------------------------------
    if constexpr (!kEarlyWindows) window_pass(0);
    for (int base = kScanWaves; base < npm; base += kScanWaves) {
        load_window(base);
        window_pass(base);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        pm[t] = row16_max(pm[t]);
        if (n == 0) sm.pm[wave][4 * t + g] = pm[t];
    }
    __syncthreads();

    // ---- decide (Eq. 1) per (head, block): keep iff sigma >= m~ - delta; the workgroup's kept
    // list in block order, its length and the optional mask -----------------------------------
    float thr[4 * NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float4 m = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
#pragma unroll
        for (int w = 0; w < kScanWaves; ++w) {
            const float4 p = reinterpret_cast<const float4*>(sm.pm[w])[t];
            m.x = fmaxf(m.x, p.x); m.y = fmaxf(m.y, p.y); m.z = fmaxf(m.z, p.z); m.w = fmaxf(m.w, p.w);
        }
        thr[4 * t] = m.x - a.delta;                     // -inf when both windows are empty
        thr[4 * t + 1] = m.y - a.delta;
        thr[4 * t + 2] = m.z - a.delta;
        thr[4 * t + 3] = m.w - a.delta;
    }
    if (a.m_tilde && s == 0 && tid < G) {
        float m = -INFINITY;
#pragma unroll
        for (int w = 0; w < kScanWaves; ++w) m = fmaxf(m, sm.pm[w][tid]);
        a.m_tilde[(size_t)b * a.Hq + hq0 + tid] = m;
    }
    // lane i of wave w decides block jb + 64 w + i (bps <= kFfdMaxScanBlocks <= 64 kScanWaves)
    static_assert(kFfdMaxScanBlocks <= 64 * kScanWaves, "one decision per lane");
    uint32_t bits = 0;
    const int jl = jb + 64 * wave + lane;
    if (jl < je) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float4 sg = reinterpret_cast<const float4*>(sm.sig[jl - jb])[t];
            bits |= ((uint32_t)(sg.x >= thr[4 * t]) | (uint32_t)(sg.y >= thr[4 * t + 1]) << 1 |
                     (uint32_t)(sg.z >= thr[4 * t + 2]) << 2 | (uint32_t)(sg.w >= thr[4 * t + 3]) << 3) << (4 * t);
        }
        bits &= (1u << G) - 1u;                         // heads past G are never kept
        if (a.mask)
            for (int h = 0; h < G; ++h) a.mask[((size_t)b * a.Hq + hq0 + h) * nblk_cap + jl] = (bits >> h) & 1u;
    }
    const uint64_t kept = __ballot(bits != 0);
    const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(kept >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)kept, 0u));
    if (lane == 0) sm.nkept[wave] = __popcll(kept);
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kScanWaves; ++w) {
        const int c = sm.nkept[w];
        before += w < wave ? c : 0;
        total += c;
    }
    if (bits != 0) a.lists[bh * (size_t)nblk_cap + jb + before + below] = (uint32_t)jl | (bits << 24);
    if (tid == 0) a.counts[bh * a.S1 + s] = total;

    // Mask entries past the end of the sequence are zero (spread over the scan workgroups).
    if (a.mask) {
        for (int j = nblk + s * kScanThreads + tid; j < nblk_cap; j += a.S1 * kScanThreads)
            for (int h = 0; h < G; ++h) a.mask[((size_t)b * a.Hq + hq0 + h) * nblk_cap + j] = 0;
    }
}

// ================================================================================================
// Fused top-delta decode: one workgroup per (sequence, KV head, split s) of kScanWaves waves.
// Workgroup s owns the blocks j = s + S1 i (i < cnt) of its group, an interleaved share, so the kept
// blocks of a group (windows, planted clusters) spread evenly over its S1 workgroups. It
//  1. streams the thumbnail codes of its blocks (waves take block numbers i from an LDS counter,
//     kRing blocks in flight each) and keeps each block's per-head maximum score in LDS, while each
//     wave also scores its share of the pseudo-max window blocks (Alg. 1; Eq. 3);
//  2. decides per (head, block): keep iff sigma >= m~ - delta (Eq. 1), the kept blocks (with their
//     keep bits) forming a list in LDS, in block order;
//  3. refines and attends its own kept blocks (Eq. 4; online softmax and PV): wave w takes tile
//     w % 4 of the kept entries w / 4, w / 4 + 2, ..., with kRefineRing tiles in flight; the
//     thumbnail term of each kept tile is recomputed from its codes with the same integer MFMA and
//     fp32 operations as in step 1, so it equals the value the decision used;
//  4. combines the eight waves' states into one partial state per head (rows [B, Hq, S1]), or,
//     when it is the group's only workgroup (S1 == 1), writes the bf16 output and lse itself.
// No workgroup waits for another: each needs only its own blocks, the window blocks (re-read by
// every workgroup of the group, L2-resident) and the query.
// ================================================================================================
template <int NT>
struct FusedLds {
    QueryLds<NT> qs;
    alignas(16) float pm[kScanWaves][4 * NT];             // each wave's window maxima per head
    alignas(16) float sig[kFfdMaxScanBlocks][4 * NT];     // block maxima per head, by share index i
    uint32_t list[kFfdMaxScanBlocks];                     // kept blocks j | keep bits << 24
    int nkept[kScanWaves];
    int next;                                             // next share index to hand out
    TileP<NT> tp[kScanWaves];
    EpilogueLds<NT, kScanWaves> epi;
};

template <int NT, int BITS, int MODE>
__global__ __launch_bounds__(kScanThreads, 1) void ffd_decode_kernel(FusedArgs a) {
    static_assert(MODE == kSelThumbnailPM || MODE == kSelRefinedPM, "top-delta modes only");
    constexpr int kRing = scan_ring<BITS>();
    __shared__ FusedLds<NT> sm;
    const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, n = lane & 15;
    const int G = a.G, hq0 = kvh * G, S1 = a.S1;
    const size_t bh = (size_t)b * a.Hkv + kvh;
    const size_t hrow0 = (size_t)b * a.Hq + hq0;             // [B, Hq] row of the group's head 0
    const int L = min(max(a.seq_lens[b], 0), a.Lcap);
    const int nblk = (L + kBlock - 1) / kBlock;
    const int nblk_cap = a.Lcap / kBlock;
    const int cnt = nblk > s ? (nblk - 1 - s) / S1 + 1 : 0;  // blocks of this workgroup
    uint16_t* out_h = a.out ? a.out + hrow0 * kD : nullptr;
    float* lse_h = a.out && a.lse ? a.lse + hrow0 : nullptr;

    // Mask entries past the end of the sequence are zero (spread over the group's workgroups).
    if (a.mask) {
        for (int j = nblk + s * kScanThreads + tid; j < nblk_cap; j += S1 * kScanThreads)
            for (int h = 0; h < G; ++h) a.mask[(hrow0 + h) * nblk_cap + j] = 0;
    }
    if (cnt == 0) {                                 // uniform: nothing to scan
        if (out_h) {                                // an empty sequence: out = 0, lse = -inf
            for (int idx = tid; idx < G * kD; idx += kScanThreads) out_h[idx] = 0;
            if (lse_h && tid < G) lse_h[tid] = -INFINITY;
        } else if (tid < G) {
            a.part_m[(hrow0 + tid) * S1 + s] = -INFINITY;     // an empty partial state
        }
        if (a.m_tilde && s == 0 && tid < G) a.m_tilde[hrow0 + tid] = -INFINITY;   // L = 0
        return;
    }

    const uint32_t* codes_bh = a.codes + bh * (size_t)a.Lcap * (4 * BITS);
    const uint16_t* absmax_bh = a.absmax + bh * (size_t)a.Lcap;

    // The stream reads through buffer resources whose ranges end after this workgroup's last block
    // s + S1 (cnt - 1): a request for an index i >= cnt (block s + S1 i beyond it) reads zeros
    // without touching memory, so every load is issued unconditionally (uniform control flow keeps
    // the compiler's in-order vmcnt accounting exact). Offsets are unsigned 32-bit: at most 2^18 + S1
    // blocks of 8 KiB.
    const uint32_t jend = (uint32_t)(s + S1 * (cnt - 1)) + 1u;
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(codes_bh), (short)0, (int)(jend * (1024u * BITS)), kRawBufferWord3);
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(absmax_bh), (short)0, (int)(jend * 128u), kRawBufferWord3);
    auto block_of = [&](int i) { return s + S1 * min(i, cnt); };     // i >= cnt: past the range
    int is[kRing];                                  // share index held by each ring slot (>= cnt: none)
#pragma unroll
    for (int r = 0; r < kRing; ++r) is[r] = kRing * wave + r;

    // Requests: queries, the first window blocks, the first ring round.
    uint32_t qw[NT];
    load_query_words<NT>(a.q, b, a.Hq, hq0, G, wave, lane, qw);
    const int jlast = nblk - 1;
    const int sink_end = min(a.n_sink, L);
    const int loc_beg = max(0, L - a.n_local);
    const int sink_blk_end = (sink_end + kBlock - 1) / kBlock;
    const int loc_blk_beg = max(loc_beg / kBlock, sink_blk_end);
    const int npm = sink_blk_end + max(nblk - loc_blk_beg, 0);
    auto pm_block = [&](int idx) { return idx < sink_blk_end ? idx : loc_blk_beg + (idx - sink_blk_end); };
    auto win_block = [&](int idx) { return min(pm_block(min(idx, max(npm, 1) - 1)), jlast); };
    constexpr bool kEarlyWindows = MODE == kSelThumbnailPM;
    BlockScan<BITS> win;
    auto load_window = [&](int base) { win = load_block_scan<BITS>(codes_bh, absmax_bh, win_block(base + wave), lane); };
    if constexpr (kEarlyWindows) load_window(0);
    BlockScan<BITS> ring[kRing];
#pragma unroll
    for (int r = 0; r < kRing; ++r) ring[r] = load_block_scan_rsrc<BITS>(rc, ra, block_of(is[r]), lane);
    if (tid == 0) sm.next = kScanWaves * kRing;
    if constexpr (MODE == kSelRefinedPM) load_window(0);

    HeadConsts<NT> hc;
    build_query_consts<NT>(sm.qs, qw, G, a.scale, thumb_top_level(BITS), tid, hc);

    // ---- scan (Alg. 1): block maxima per head, and the window maxima of the pseudo-max ---------
    float pm[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) pm[t] = -INFINITY;
    auto window_pass = [&](int base) {
        const int idx = base + wave;
        if (idx >= npm) return;                     // wave-uniform
        const int j = pm_block(idx);
        float sc[NT][4];
        block_scores<NT, BITS>(win, j, lane, L, hc, sc);
        if constexpr (MODE == kSelRefinedPM)
            add_residual_term<NT>(a.resid + bh * (size_t)a.Lcap * kD, win.mm, j, lane, hc, sc);
#pragma unroll
        for (int T4 = 0; T4 < 4; ++T4) {
            const int tok = 64 * j + 16 * T4 + n;
            const bool in_win = tok < L && (tok < sink_end || tok >= loc_beg);
#pragma unroll
            for (int t = 0; t < NT; ++t) pm[t] = fmaxf(pm[t], in_win ? sc[t][T4] : -INFINITY);
        }
    };
    auto consume = [&](const BlockScan<BITS>& blk, int i) {
        float sc[NT][4];
        block_scores<NT, BITS>(blk, s + S1 * i, lane, L, hc, sc);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float sig = row16_max(fmaxf(fmaxf(sc[t][0], sc[t][1]), fmaxf(sc[t][2], sc[t][3])));
            if (n == 0) sm.sig[i][4 * t + g] = sig;
        }
    };
    if constexpr (kEarlyWindows) window_pass(0);
    for (bool more = true; more;) {                 // wave-uniform
        more = false;
#pragma unroll
        for (int r = 0; r < kRing; ++r) {
            int in = 0;
            if (lane == 0) in = atomicAdd(&sm.next, 1);
            in = __builtin_amdgcn_readfirstlane(in);
            if (is[r] < cnt) consume(ring[r], is[r]);
            ring[r] = load_block_scan_rsrc<BITS>(rc, ra, block_of(in), lane);
            is[r] = in;
            more |= in < cnt;
        }
    }
    if constexpr (!kEarlyWindows) window_pass(0);
    for (int base = kScanWaves; base < npm; base += kScanWaves) {
        load_window(base);
        window_pass(base);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        pm[t] = row16_max(pm[t]);
        if (n == 0) sm.pm[wave][4 * t + g] = pm[t];
    }
    __syncthreads();

    // ---- decide (Eq. 1): keep iff sigma >= m~ - delta; the kept list in LDS, in block order ----
    float thr[4 * NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float4 m = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
#pragma unroll
        for (int w = 0; w < kScanWaves; ++w) {
            const float4 p = reinterpret_cast<const float4*>(sm.pm[w])[t];
            m.x = fmaxf(m.x, p.x); m.y = fmaxf(m.y, p.y); m.z = fmaxf(m.z, p.z); m.w = fmaxf(m.w, p.w);
        }
        thr[4 * t] = m.x - a.delta;                 // -inf when both windows are empty
        thr[4 * t + 1] = m.y - a.delta;
        thr[4 * t + 2] = m.z - a.delta;
        thr[4 * t + 3] = m.w - a.delta;
    }
    if (a.m_tilde && s == 0 && tid < G) {
        float m = -INFINITY;
#pragma unroll
        for (int w = 0; w < kScanWaves; ++w) m = fmaxf(m, sm.pm[w][tid]);
        a.m_tilde[hrow0 + tid] = m;
    }
    // lane l of wave w decides share index 64 w + l (cnt <= kFfdMaxScanBlocks <= 64 kScanWaves)
    static_assert(kFfdMaxScanBlocks <= 64 * kScanWaves, "one decision per lane");
    uint32_t bits = 0;
    const int il = 64 * wave + lane;
    const int jl = s + S1 * il;
    if (il < cnt) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float4 sg = reinterpret_cast<const float4*>(sm.sig[il])[t];
            bits |= ((uint32_t)(sg.x >= thr[4 * t]) | (uint32_t)(sg.y >= thr[4 * t + 1]) << 1 |
                     (uint32_t)(sg.z >= thr[4 * t + 2]) << 2 | (uint32_t)(sg.w >= thr[4 * t + 3]) << 3) << (4 * t);
        }
        bits &= (1u << G) - 1u;                     // heads past G are never kept
        if (a.mask)
            for (int h = 0; h < G; ++h) a.mask[(hrow0 + h) * nblk_cap + jl] = (bits >> h) & 1u;
    }
    const uint64_t kept = __ballot(bits != 0);
    const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(kept >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)kept, 0u));
    if (lane == 0) sm.nkept[wave] = __popcll(kept);
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kScanWaves; ++w) {
        const int c = sm.nkept[w];
        before += w < wave ? c : 0;
        total += c;
    }
    if (bits != 0) sm.list[before + below] = (uint32_t)jl | (bits << 24);
    __syncthreads();

    // ---- refine (Eq. 4) and attend the kept blocks: wave w, tile T4 = w % 4, entries w / 4 + 2k --
    const int T4 = wave & 3, par = wave >> 2;
    const int mine = total > par ? (total - par + 1) / 2 : 0;
    const int8_t* resid_bh = a.resid + bh * (size_t)a.Lcap * kD;
    const uint16_t* v_bh = a.v + bh * (size_t)a.Lcap * kD;
    PvAcc<NT> pv;
    pv.zero();
    float m_run[NT], l_part[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { m_run[t] = -INFINITY; l_part[t] = 0.f; }
    TileP<NT>& tp = sm.tp[wave];
    auto entry = [&](int k) { return sm.list[par + 2 * min(k, mine - 1)]; };
    auto attend = [&](const RefineTile<NT, BITS>& rt, int j, uint32_t kb) {
        float z[NT];
        bool keep[NT];
        const float Mt = bf16_to_f32((uint16_t)rt.m);
        float shat[NT];                             // Eq. 4's first term: the scan scores, recomputed
        tile_scores<NT, BITS>(rt.cw, Mt, 64 * j + 16 * T4 + n < L, hc, shat);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], rt.r0, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], rt.r1, acc, 0, 0, 0);
            const float R = fmaf(65536.f, (float)acc.z, fmaf(256.f, (float)acc.y, (float)acc.x));
            const float sct = shat[t];
            z[t] = sct == -INFINITY ? -INFINITY : fmaf(R, Mt * hc.kap2[t], sct);
            keep[t] = (kb >> (4 * t + g)) & 1u;
        }
        softmax_tile<NT>(z, keep, m_run, l_part, tp, g, n);
        wave_lds_fence();
        pv_tile<NT>(pv, tp, rt.vt);
        wave_lds_fence();
    };
    if (mine > 0) {                                 // wave-uniform
        RefineTile<NT, BITS> rr[kRefineRing];
#pragma unroll
        for (int r = 0; r < kRefineRing; ++r)
            rr[r] = load_refine_tile<NT, BITS>(resid_bh, v_bh, codes_bh, absmax_bh,
                                               (int)(entry(r) & 0xffffffu), T4, lane, L);
        for (int k0 = 0; k0 < mine; k0 += kRefineRing) {
#pragma unroll
            for (int r = 0; r < kRefineRing; ++r) {
                const int k = k0 + r;
                if (k < mine) {
                    const uint32_t e = entry(k);
                    attend(rr[r], (int)(e & 0xffffffu), e >> 24);
                }
                // the last round's refills re-read the wave's last tile (clamped): still cached
                rr[r] = load_refine_tile<NT, BITS>(resid_bh, v_bh, codes_bh, absmax_bh,
                                                   (int)(entry(k + kRefineRing) & 0xffffffu), T4, lane, L);
            }
        }
    }

    write_partials<NT, kScanWaves>(sm.epi, pv, m_run, l_part, wave, lane, G, hrow0 * S1 + s, (size_t)S1,
                                   a.part_m, a.part_l, a.part_acc, out_h, lse_h);
}

// ================================================================================================
// Refinement: Eq. 4 on the kept blocks, online softmax and PV, one partial state per workgroup.
// Grid (W + B*Hkv). With N kept blocks in all and n_x in KV group x, group x gets
// W_x = ceil(n_x * min(W', N) / N) workgroups (1 if n_x = 0) in group order, W' = W or, with few
// splits, the largest W' found whose allocation still fits the grid (fill_grid); workgroup p of the
// group refines its kept blocks of rank [p n_x / W_x, (p + 1) n_x / W_x). Workgroups past the last
// group's exit.
// ================================================================================================
template <int NT, int RBITS>
__global__ __launch_bounds__(kRefineThreads, 1) void ffd_refine_kernel(RefineArgs a) {
    __shared__ RefineLds<NT> sm;
    const int wg = blockIdx.x;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int g = lane >> 4, n = lane & 15;
    constexpr int kPar = kRefineWaves / 4;          // waves per tile index
    const int T4 = wave & 3, par = wave >> 2;       // tile T4 of the share's entries par, par + kPar, ...
    const int G = a.G, S1 = a.S1, npairs = a.npairs;

    // ---- allocation: total kept N, then this workgroup's KV group ---------------------------
    // Usual case (at most 1024 scan counts and 256 KV groups): every wave computes the whole
    // allocation on its own, with no workgroup barrier. Lane l loads counts [16l, 16l + 16), one
    // wave prefix gives their exclusive prefix in (group, split) order, which every wave writes to
    // LDS (identical values, so each reads back its own writes), then lane l allocates groups
    // 4l .. 4l + 3 and a second wave prefix numbers their workgroups. Larger inputs: all scan counts
    // kept in LDS with workgroup scans (up to 4096), else summed per group in passes of kPairChunk
    // groups with LDS atomics.
    const int total = npairs * S1;
    const bool fast = total <= 16 * 64 && npairs <= 4 * 64;
    const bool cached = total <= kCountCache && npairs <= kPairChunk;
    int N = 0, running = 0, half = 0;
    auto scan = [&](int v, int* tot) {
        const int e = wg_exclusive_scan<kRefineWaves>(v, sm.wsum[half], tot);
        half ^= 1;
        return e;
    };
    const long long W = a.W;
    // ceil(n_x * We / N) workgroups for n_x > 0, We = min(W, N) or the grid-filling W' below; exact
    // in fp64 (the numerator stays below 2^52, and fl(u / N) cannot round up to an integer when
    // u < 2^52)
    auto alloc = [&](int nx, long long Weff) {
        return nx > 0 ? (int)floor(((double)nx * (double)Weff + (double)(N - 1)) / (double)N) : 1;
    };
    // The rounding up in alloc leaves up to one workgroup per group of the grid's W + B*Hkv unused.
    // When that can be a third of the grid or more (W <= 2 B*Hkv: many groups, few splits), grow
    // the effective W by the unused count while the allocation still fits the grid (at most three
    // steps, each halved once if it overshoots), so fewer CUs idle and the largest share shrinks
    // (the ragged batch of 16 sequences, 128 groups on 256 workgroups: refinement 422 -> 397 us).
    // With more splits the slack is small and the extra evaluations cost more than they save (4 x
    // 128K, delta 5: +2 us), so W is used as it is. total(We) is the allocation's workgroup count
    // for an effective We, the same value in every thread; the result depends only on the counts,
    // like the allocation itself.
    auto fill_grid = [&](auto total) {
        const long long grid = W + npairs;
        const long long cap = (long long)max(N, 1);
        long long We = min(W, cap);
        if (W > 2LL * npairs) return We;
        int used = total(We);
        for (int it = 0; it < 3 && used < grid && We < cap; ++it) {
            long long cand = min(We + (grid - used), cap);
            int uc = total(cand);
            if (uc > grid) {
                cand = We + (cand - We) / 2;
                if (cand == We) break;
                uc = total(cand);
                if (uc > grid) break;
            }
            We = cand;
            used = uc;
        }
        return We;
    };
    int x = 0, Qx = 0, Wx = 1, nx = 0;
    if (fast) {
        const int i0 = 16 * lane;
        int c[16], sum = 0;
#pragma unroll
        for (int k = 0; k < 16; k += 4) {
            // the counts region is padded to 256 bytes, so the last int4 stays inside it
            int4 v = make_int4(0, 0, 0, 0);
            if (i0 + k < total) v = *reinterpret_cast<const int4*>(a.counts + i0 + k);
            c[k] = v.x; c[k + 1] = v.y; c[k + 2] = v.z; c[k + 3] = v.w;
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            if (i0 + k >= total) c[k] = 0;
            sum += c[k];
        }
        const int incl = wave_inclusive_scan(sum);
        N = __builtin_amdgcn_readlane(incl, 63);
        int run = incl - sum;
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            if (i0 + k < total) sm.cnt[i0 + k] = run;
            run += c[k];
        }
        if (lane == 0) sm.cnt[total] = N;
        wave_lds_fence();
        int w4[4], n4[4], s4 = 0;                      // lane l: groups 4l .. 4l + 3
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int xi = 4 * lane + k;
            n4[k] = xi < npairs ? sm.cnt[(xi + 1) * S1] - sm.cnt[xi * S1] : 0;
        }
        const long long Weff = fill_grid([&](long long We) {
            int t = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) t += 4 * lane + k < npairs ? alloc(n4[k], We) : 0;
            return __builtin_amdgcn_readlane(wave_inclusive_scan(t), 63);
        });
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            w4[k] = 4 * lane + k < npairs ? alloc(n4[k], Weff) : 0;
            s4 += w4[k];
        }
        const int winc = wave_inclusive_scan(s4);
        running = __builtin_amdgcn_readlane(winc, 63);
        int q0 = winc - s4, hit = -1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (hit < 0 && wg >= q0 && wg < q0 + w4[k]) hit = k;
            if (hit < 0) q0 += w4[k];
        }
        const uint64_t hb = __ballot(hit >= 0);
        if (hb != 0) {                              // uniform; else wg >= running
            const int src = __builtin_amdgcn_readfirstlane((int)__builtin_ctzll(hb));
            const int kk = __builtin_amdgcn_readlane(hit, src);
            x = 4 * src + kk;
            Qx = __builtin_amdgcn_readlane(q0, src);
            int wsel = w4[0], nsel = n4[0];
#pragma unroll
            for (int k = 1; k < 4; ++k) if (kk == k) { wsel = w4[k]; nsel = n4[k]; }
            Wx = __builtin_amdgcn_readlane(wsel, src);
            nx = __builtin_amdgcn_readlane(nsel, src);
        }
    } else if (cached) {
        const int i0 = 16 * tid;
        int c[16], sum = 0;
#pragma unroll
        for (int k = 0; k < 16; k += 4) {
            int4 v = make_int4(0, 0, 0, 0);
            if (i0 + k < total) v = *reinterpret_cast<const int4*>(a.counts + i0 + k);
            c[k] = v.x; c[k + 1] = v.y; c[k + 2] = v.z; c[k + 3] = v.w;
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            if (i0 + k >= total) c[k] = 0;
            sum += c[k];
        }
        int run = scan(sum, &N);
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            if (i0 + k < total) sm.cnt[i0 + k] = run;
            run += c[k];
        }
        if (tid == 0) sm.cnt[total] = N;
        __syncthreads();
        int w4[4], n4[4], s4 = 0;                      // thread t: groups 4t .. 4t + 3
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int xi = 4 * tid + k;
            n4[k] = xi < npairs ? sm.cnt[(xi + 1) * S1] - sm.cnt[xi * S1] : 0;
        }
        const long long Weff = fill_grid([&](long long We) {
            int t = 0, tot = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) t += 4 * tid + k < npairs ? alloc(n4[k], We) : 0;
            (void)scan(t, &tot);
            return tot;
        });
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            w4[k] = 4 * tid + k < npairs ? alloc(n4[k], Weff) : 0;
            s4 += w4[k];
        }
        int q0 = scan(s4, &running);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (4 * tid + k < npairs && wg >= q0 && wg < q0 + w4[k]) {
                sm.sel[0] = 4 * tid + k;
                sm.sel[1] = q0;
                sm.sel[2] = w4[k];
                sm.sel[3] = n4[k];
            }
            q0 += w4[k];
        }
    } else {
        int part = 0;
        for (int i = tid; i < total; i += kRefineThreads) part += a.counts[i];
        (void)scan(part, &N);
        const long long Weff = min(W, (long long)max(N, 1));
        for (int c0 = 0; c0 < npairs; c0 += kPairChunk) {
            const int np = min(kPairChunk, npairs - c0);
            for (int i = tid; i < np; i += kRefineThreads) sm.pn[i] = 0;
            __syncthreads();
            for (int i = tid; i < np * S1; i += kRefineThreads) {
                const int c = a.counts[(size_t)c0 * S1 + i];
                if (c) atomicAdd(&sm.pn[i / S1], c);
            }
            __syncthreads();
            int w4[4], n4[4], s4 = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int xi = 4 * tid + k;
                n4[k] = xi < np ? sm.pn[xi] : 0;
                w4[k] = xi < np ? alloc(n4[k], Weff) : 0;
                s4 += w4[k];
            }
            int tot = 0;
            int q0 = running + scan(s4, &tot);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                if (4 * tid + k < np && wg >= q0 && wg < q0 + w4[k]) {
                    sm.sel[0] = c0 + 4 * tid + k;
                    sm.sel[1] = q0;
                    sm.sel[2] = w4[k];
                    sm.sel[3] = n4[k];
                }
                q0 += w4[k];
            }
            running += tot;
            __syncthreads();                           // pn is rewritten by the next pass
        }
    }
    if (wg >= running) return;                      // uniform: beyond the last group's workgroups
    if (!fast) {
        __syncthreads();
        x = sm.sel[0]; Qx = sm.sel[1]; Wx = sm.sel[2]; nx = sm.sel[3];
    }
    // uniform by construction; said explicitly so that the group's base addresses stay in scalar
    // registers
    x = __builtin_amdgcn_readfirstlane(x);
    Qx = __builtin_amdgcn_readfirstlane(Qx);
    Wx = __builtin_amdgcn_readfirstlane(Wx);
    nx = __builtin_amdgcn_readfirstlane(nx);
    const int b = x / a.Hkv, kvh = x % a.Hkv, hq0 = kvh * G;
    const int p = wg - Qx;
    const int r0 = (int)((long long)p * nx / Wx), r1 = (int)((long long)(p + 1) * nx / Wx);
    const size_t bh = (size_t)x;
    const int L = min(max(a.seq_lens[b], 0), a.Lcap);
    const int nblk = (L + kBlock - 1) / kBlock;
    const int nblk_cap = a.Lcap / kBlock;
    const int bps = (nblk + S1 - 1) / S1;
    if (p == 0 && tid == 0) a.table[x] = make_int2(Qx, Wx);

    const uint16_t* absmax_bh = a.absmax + bh * (size_t)a.Lcap;
    const int8_t* resid_bh = a.resid + bh * (size_t)a.Lcap * kD;
    const uint16_t* v_bh = a.v + bh * (size_t)a.Lcap * kD;
    const uint32_t* codes_bh = a.codes + bh * (size_t)a.Lcap * (4 * RBITS);
    const uint32_t* list_bh = a.lists + bh * (size_t)nblk_cap;

    // A share of at most kFastShare blocks (with the fast allocation) is staged by every wave on its
    // own, like the allocation; a longer one in chunks with workgroup barriers.
    constexpr int kFastShare = 256;
    const bool fast_share = fast && r1 - r0 <= kFastShare;
    uint32_t qw[NT];
    uint32_t qa[4 * NT];
    if (fast_share) {
#pragma unroll
        for (int h = 0; h < 4 * NT; ++h)
            qa[h] = reinterpret_cast<const uint32_t*>(a.q + ((size_t)b * a.Hq + hq0 + min(h, G - 1)) * kD)[lane];
    } else {
        load_query_words<NT>(a.q, b, a.Hq, hq0, G, wave, lane, qw);
    }
    // exclusive prefix of the group's per-split counts: rank r lies in split s with
    // pref(s) <= r < pref(s + 1), at list position s * bps + r - pref(s)
    if (!cached) {
        int run = 0;
        for (int c0 = 0; c0 < S1; c0 += kRefineThreads) {
            const int sidx = c0 + tid;
            const int c = sidx < S1 ? a.counts[bh * S1 + sidx] : 0;
            int tot = 0;
            const int e = scan(c, &tot);
            if (sidx < S1) sm.pref[sidx] = run + e;
            run += tot;
        }
        if (tid == 0) sm.pref[S1] = run;
        __syncthreads();
    }
    const int* pref = cached ? sm.cnt + x * S1 : sm.pref;
    const int pref0 = cached ? pref[0] : 0;
    auto list_entry = [&](int r) {                 // the kept block of rank r: j | keep bits << 24
        int lo = 0, hi = S1;                        // largest split with pref(split) <= r
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (pref[mid] - pref0 <= r) lo = mid; else hi = mid;
        }
        return list_bh[lo * bps + (r - (pref[lo] - pref0))];
    };
    HeadConsts<NT> hc;

    PvAcc<NT> pv;
    pv.zero();
    float m_run[NT], l_part[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) { m_run[t] = -INFINITY; l_part[t] = 0.f; }
    TileP<NT>& tp = sm.tp[wave];

    // refine (Eq. 4) and attend tile T4 of one kept block
    auto attend = [&](const RefineTile<NT, RBITS>& rt, int j, uint32_t bits) {
        float z[NT];
        bool keep[NT];
        const float Mt = bf16_to_f32((uint16_t)rt.m);
        float shat[NT];                             // Eq. 4's first term: the scan scores, recomputed
        tile_scores<NT, RBITS>(rt.cw, Mt, 64 * j + 16 * T4 + n < L, hc, shat);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            v4i acc = {0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][0], rt.r0, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(hc.A[t][1], rt.r1, acc, 0, 0, 0);
            const float R = fmaf(65536.f, (float)acc.z, fmaf(256.f, (float)acc.y, (float)acc.x));
            const float sct = shat[t];
            z[t] = sct == -INFINITY ? -INFINITY : fmaf(R, Mt * hc.kap2[t], sct);
            keep[t] = (bits >> (4 * t + g)) & 1u;
        }
        softmax_tile<NT>(z, keep, m_run, l_part, tp, g, n);
        wave_lds_fence();
        pv_tile<NT>(pv, tp, rt.vt);
        wave_lds_fence();
    };

    // the m list entries staged in LDS: this wave takes tile T4 of entries par, par + kPar, ... with
    // kRefineRing tiles in flight. The refill of the last round re-reads the wave's last tile
    // (clamped): it is still cached, and a conditional refill would cost more registers than it
    // saves. fast_consts: the query constants are built by this wave while its first tiles are in
    // flight.
    auto refine_entries = [&](int m, bool fast_consts) {
        const int mine = m > par ? (m - par + kPar - 1) / kPar : 0;
        if (mine == 0) {                            // wave-uniform
            if (fast_consts) build_query_consts_wave<NT>(sm.qs, qa, G, a.scale, a.top_level, lane, hc);
            return;
        }
        auto entry = [&](int k) { return sm.u.list[par + kPar * min(k, mine - 1)]; };
        RefineTile<NT, RBITS> ring[kRefineRing];
#pragma unroll
        for (int r = 0; r < kRefineRing; ++r)
            ring[r] = load_refine_tile<NT, RBITS>(resid_bh, v_bh, codes_bh, absmax_bh,
                                                  (int)(entry(r) & 0xffffffu), T4, lane, L);
        if (fast_consts) build_query_consts_wave<NT>(sm.qs, qa, G, a.scale, a.top_level, lane, hc);
        for (int k0 = 0; k0 < mine; k0 += kRefineRing) {
#pragma unroll
            for (int r = 0; r < kRefineRing; ++r) {
                const int k = k0 + r;
                if (k < mine) {
                    const uint32_t e = entry(k);
                    attend(ring[r], (int)(e & 0xffffffu), e >> 24);
                }
                ring[r] = load_refine_tile<NT, RBITS>(resid_bh, v_bh, codes_bh, absmax_bh,
                                                      (int)(entry(k + kRefineRing) & 0xffffffu), T4, lane, L);
            }
        }
    };

    if (fast_share) {
        // every wave loads the whole share's entries (lane i: ranks r0 + i + 64k) and writes them to
        // LDS: identical values, read back by the same wave
        const int m = r1 - r0;
        uint32_t ent[kFastShare / 64];
#pragma unroll
        for (int k = 0; k < kFastShare / 64; ++k) {
            const int i = lane + 64 * k;
            ent[k] = i < m ? list_entry(r0 + i) : 0u;
        }
#pragma unroll
        for (int k = 0; k < kFastShare / 64; ++k) {
            const int i = lane + 64 * k;
            if (i < m) sm.u.list[i] = ent[k];
        }
        wave_lds_fence();
        if (m > 0) refine_entries(m, true);
        else build_query_consts_wave<NT>(sm.qs, qa, G, a.scale, a.top_level, lane, hc);
        __syncthreads();                            // the list area becomes the epilogue's
    } else {
        bool consts_ready = false;
        for (int c = r0; c < r1; c += kChunk) {
            const int m = min(kChunk, r1 - c);
            for (int i = tid; i < m; i += kRefineThreads) sm.u.list[i] = list_entry(c + i);
            if (!consts_ready) {                    // the query loads and the list loads overlap
                build_query_consts<NT>(sm.qs, qw, G, a.scale, a.top_level, tid, hc);
                consts_ready = true;
            }
            __syncthreads();
            refine_entries(m, false);
            __syncthreads();                // the list is rewritten by the next chunk / the epilogue
        }
        if (!consts_ready) __syncthreads();
    }

    write_partials<NT, kRefineWaves>(sm.u.epi, pv, m_run, l_part, wave, lane, G, (size_t)wg * G, 1,
                                     a.part_m, a.part_l, a.part_acc);
}

template __global__ void ffd_scan_kernel<1, 2, kSelThumbnailPM>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 2, kSelThumbnailPM>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 4, kSelThumbnailPM>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 4, kSelThumbnailPM>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 8, kSelThumbnailPM>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 8, kSelThumbnailPM>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 2, kSelRefinedPM>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 2, kSelRefinedPM>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 4, kSelRefinedPM>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 4, kSelRefinedPM>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 8, kSelRefinedPM>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 8, kSelRefinedPM>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 2, kSelTopK>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 2, kSelTopK>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 4, kSelTopK>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 4, kSelTopK>(ScanArgs);
template __global__ void ffd_scan_kernel<1, 8, kSelTopK>(ScanArgs);
template __global__ void ffd_scan_kernel<2, 8, kSelTopK>(ScanArgs);
template __global__ void ffd_decode_kernel<1, 2, kSelThumbnailPM>(FusedArgs);
template __global__ void ffd_decode_kernel<2, 2, kSelThumbnailPM>(FusedArgs);
template __global__ void ffd_decode_kernel<1, 4, kSelThumbnailPM>(FusedArgs);
template __global__ void ffd_decode_kernel<2, 4, kSelThumbnailPM>(FusedArgs);
template __global__ void ffd_decode_kernel<1, 8, kSelThumbnailPM>(FusedArgs);
template __global__ void ffd_decode_kernel<2, 8, kSelThumbnailPM>(FusedArgs);
template __global__ void ffd_decode_kernel<1, 2, kSelRefinedPM>(FusedArgs);
template __global__ void ffd_decode_kernel<2, 2, kSelRefinedPM>(FusedArgs);
template __global__ void ffd_decode_kernel<1, 4, kSelRefinedPM>(FusedArgs);
template __global__ void ffd_decode_kernel<2, 4, kSelRefinedPM>(FusedArgs);
template __global__ void ffd_decode_kernel<1, 8, kSelRefinedPM>(FusedArgs);
template __global__ void ffd_decode_kernel<2, 8, kSelRefinedPM>(FusedArgs);
template __global__ void ffd_refine_kernel<1, 2>(RefineArgs);
template __global__ void ffd_refine_kernel<2, 2>(RefineArgs);
template __global__ void ffd_refine_kernel<1, 4>(RefineArgs);
template __global__ void ffd_refine_kernel<2, 4>(RefineArgs);
template __global__ void ffd_refine_kernel<1, 8>(RefineArgs);
template __global__ void ffd_refine_kernel<2, 8>(RefineArgs);

}  // namespace ffd
