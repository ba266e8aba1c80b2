// Fixed-budget (top-k) block selection: the rule the paper sets top-delta against (Sec. 1, Fig. 1 (a);
// the selection-rule overhead comparison of Table 3). Per query head, the k blocks with the largest
// block scores sigma (the maxima of the thumbnail scores over a block's valid tokens, as top-delta
// uses them) are kept; equal scores are taken in block order. Unlike top-delta, whose decision is a
// comparison with a per-head constant made while the scan streams, this needs every block score of
// the head first: the scan kernel writes them, and this kernel, one workgroup per (sequence, KV
// head), holds the group's scores in registers (as the order-preserving integer image of the fp32
// score; each wave holds whole 64-block runs of one head), finds each head's k-th largest score by a
// most-significant-digit radix select (four 8-bit digits counted in LDS histograms, stopping early
// once the digit bucket holds exactly the number still needed), marks the blocks above and equal to
// it in LDS bitmaps, then goes through the blocks in order, keeps those above the threshold and the
// first ones equal to it, and writes the group's kept list (block | keep bits << 24, the union over
// the group's heads) and its length in the scan's format, so the refinement kernel runs unchanged.
#include <climits>

#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

namespace {

constexpr int kBins = 256;
constexpr int kSelThreads = kTopkSelectThreads;      // 16 waves: 4 per SIMD hide each other's latency
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSlots = 8;                            // keys held per thread
constexpr int kTileKeys = kSlots * kSelThreads;      // (block, head) keys per tile

// Order-preserving image of a float: larger float, larger key. The scan writes +0 for a zero score.
__device__ __forceinline__ uint32_t order_key(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// hist[bin] += 1 for every active lane, with one LDS atomic per lane at most. Block scores of a head
// crowd into few buckets of the leading digit, so the two buckets of the first active lanes are
// counted by one leader lane each (adding the bucket's population in the wave); the remaining lanes
// add one each. Branch-free, so the cost per key stays a few instructions.
__device__ __forceinline__ void hist_add(int* hist, int bin, bool active, int lane) {
    const uint64_t act = __ballot(active);                              // wave-uniform
    const int l0 = act ? __ffsll((unsigned long long)act) - 1 : 0;
    const int b0 = __builtin_amdgcn_readlane(bin, l0);
    const uint64_t s0 = __ballot(active && bin == b0);
    const uint64_t rest = act & ~s0;
    const int l1 = rest ? __ffsll((unsigned long long)rest) - 1 : 0;
    const int b1 = __builtin_amdgcn_readlane(bin, l1);                  // != b0 when rest != 0
    const uint64_t s1 = __ballot(active && bin == b1) & rest;
    const bool lead0 = act != 0 && lane == l0;
    const bool lead1 = rest != 0 && lane == l1;
    const bool other = active && bin != b0 && bin != b1;
    const int at = lead0 ? b0 : (lead1 ? b1 : bin);
    const int val = lead0 ? (int)__popcll(s0) : (lead1 ? (int)__popcll(s1) : 1);
    if (lead0 || lead1 || other) atomicAdd(&hist[at], val);
}

// Which keys a thread holds. A tile is TB = kTileKeys / G blocks of every head. Register slot i of
// wave w (lane l) holds head w mod G at block 64 * (i * WPH + w / G) + l of the tile: each head's
// 64-block runs are spread over WPH = 16 / G waves.
template <int G>
struct Slots {
    static constexpr int TB = kTileKeys / G;
    static constexpr int WPH = kSelWaves / G;
    static constexpr int RUNS = TB / 64;             // 64-block runs per head per tile
    __device__ static int head(int wave) { return wave % G; }
    __device__ static int run(int wave, int i) { return i * WPH + wave / G; }
};

// Exclusive prefix sum over the workgroup (thread order) of x; *total receives the sum. One
// barrier: consecutive calls must alternate between the two halves of wsum[2][kSelWaves].
__device__ __forceinline__ int sel_exclusive_scan(int x, int* wsum, int* total) {
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
    for (int w = 0; w < kSelWaves; ++w) {
        const int v = wsum[w];
        before += w < wave ? v : 0;
        tot += v;
    }
    *total = tot;
    return before + incl - x;
}

template <int G>
struct TopkLds {
    int hist[2][G][kBins];
    uint64_t gtmap[G][Slots<G>::RUNS];    // per head and 64-block run: blocks above the threshold
    uint64_t eqmap[G][Slots<G>::RUNS];    // ... and equal to it
    uint32_t prefix[G];                   // digits of the k-th largest key found so far
    int rem[G];                           // keys still to take at or below the prefix
    int done[G];                          // the prefix's bucket holds exactly rem keys: all are taken
    int wsum[2][kSelWaves];
};

// This thread's keys of tile ti (blocks [ti * TB, ti * TB + nb)); slots past nb are not valid.
template <int G>
__device__ __forceinline__ void load_keys(uint32_t (&key)[kSlots], const float* __restrict__ sig, int ti,
                                          int nb, int wave, int lane) {
    using S = Slots<G>;
    float v[kSlots];
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
        const int jj = 64 * S::run(wave, i) + lane;
        v[i] = jj < nb ? sig[((size_t)ti * S::TB + jj) * G + S::head(wave)] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kSlots; ++i) key[i] = order_key(v[i]);
}

}  // namespace

// Grid (B * Hkv), kSelThreads threads; G query heads per KV head.
template <int G>
__global__ __launch_bounds__(kSelThreads) void ffd_topk_select_kernel(TopkArgs a) {
    using S = Slots<G>;
    constexpr int TB = S::TB;
    constexpr int BPT = TB / kSelThreads;            // blocks per thread in the keep pass (<= 8)
    __shared__ TopkLds<G> sm;
    const int x = blockIdx.x;
    const int b = x / a.Hkv, kvh = x % a.Hkv;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int L = min(max(a.seq_lens[b], 0), a.Lcap);
    const int nblk = (L + kBlock - 1) / kBlock;
    const int nblk_cap = a.Lcap / kBlock;
    const int keff = min(a.k, nblk);
    const int ntiles = (nblk + TB - 1) / TB;
    const float* sig = a.sigma + (size_t)x * nblk_cap * G;
    uint32_t key[kSlots];
    int loaded = -1;                                 // tile now in key[]
    auto use_tile = [&](int ti) {
        if (ti != loaded) load_keys<G>(key, sig, ti, min(TB, nblk - ti * TB), wave, lane);
        loaded = ti;
    };
    auto valid = [&](int ti, int i) { return 64 * S::run(wave, i) + lane < nblk - ti * TB; };

    // ---- the k-th largest key of each head ---------------------------------------------------
    if (tid < G) {
        sm.prefix[tid] = 0;
        sm.rem[tid] = keff;
        sm.done[tid] = 0;
    }
    for (int i = tid; i < G * kBins; i += kSelThreads) (&sm.hist[0][0][0])[i] = 0;
    __syncthreads();
    const int hw = S::head(wave);                    // this wave's head
    const bool select = keff < nblk;                 // else every block is kept
    if (select) {
        uint32_t pmask = 0;
        for (int pass = 0, shift = 24; shift >= 0; ++pass, shift -= 8) {
            int (*hist)[kBins] = sm.hist[pass & 1];
            const uint32_t pre = sm.prefix[hw];
            const bool live = !sm.done[hw];
            for (int ti = 0; ti < ntiles && live; ++ti) {  // uniform in the wave
                use_tile(ti);
#pragma unroll
                for (int i = 0; i < kSlots; ++i)
                    hist_add(hist[hw], (int)((key[i] >> shift) & 255u),
                             valid(ti, i) && (key[i] & pmask) == pre, lane);
            }
            __syncthreads();
            // wave w: heads w, w + 4. Lane l holds buckets 4l .. 4l + 3; "above" counts the keys in
            // higher buckets; the bucket where the count reaches rem holds the k-th largest key.
            for (int h = wave; h < G; h += kSelWaves) {
                if (sm.done[h]) continue;               // uniform in the wave
                int c[4], tot = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    c[i] = hist[h][4 * lane + i];
                    tot += c[i];
                }
                int incl = tot;                         // keys in buckets of lanes >= this one
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int y = __shfl_down(incl, o);
                    if (lane + o < 64) incl += y;
                }
                int above = incl - tot;
                const int rem = sm.rem[h];
#pragma unroll
                for (int i = 3; i >= 0; --i) {
                    if (above < rem && above + c[i] >= rem) {
                        sm.prefix[h] |= (uint32_t)(4 * lane + i) << shift;
                        sm.rem[h] = rem - above;
                        if (above + c[i] == rem) sm.done[h] = 1;
                    }
                    above += c[i];
                }
            }
            // the other buffer is next pass's histogram; its last reader finished before the barrier above
            int* other = &sm.hist[(pass + 1) & 1][0][0];
            for (int i = tid; i < G * kBins; i += kSelThreads) other[i] = 0;
            pmask |= 255u << shift;
            __syncthreads();
            bool all_done = true;
#pragma unroll
            for (int h = 0; h < G; ++h) all_done = all_done && sm.done[h];
            if (all_done) break;                        // uniform: read after the barrier
        }
    }

    // ---- keep: key > threshold, or key == threshold among the first `need` equal ones ----------
    // keep-all: threshold 0 with no limit on equal keys takes every key
    const uint32_t thr_w = select ? sm.prefix[hw] : 0u;
    int need[G], eq_run[G];                          // uniform: kept in scalar registers
#pragma unroll
    for (int h = 0; h < G; ++h) {
        need[h] = __builtin_amdgcn_readfirstlane(select && !sm.done[h] ? sm.rem[h] : INT_MAX);
        eq_run[h] = 0;
    }
    uint32_t* list_x = a.lists + (size_t)x * nblk_cap;
    uint8_t* mask_x = a.mask ? a.mask + ((size_t)b * a.Hq + (size_t)kvh * G) * nblk_cap : nullptr;
    int list_run = 0, half = 0;
    auto scan = [&](int v, int* tot) {
        const int e = sel_exclusive_scan(v, sm.wsum[half], tot);
        half ^= 1;
        return e;
    };
    for (int ti = 0; ti < ntiles; ++ti) {
        use_tile(ti);
#pragma unroll
        for (int i = 0; i < kSlots; ++i) {
            const bool ok = valid(ti, i);
            const uint64_t gb = __ballot(ok && key[i] > thr_w), eb = __ballot(ok && key[i] == thr_w);
            if (lane == 0) {
                sm.gtmap[hw][S::run(wave, i)] = gb;
                sm.eqmap[hw][S::run(wave, i)] = eb;
            }
        }
        __syncthreads();
        const int jt0 = ti * TB, nb = min(TB, nblk - jt0);
        const int jj0 = BPT * tid;                      // this thread's blocks jt0 + jj0 + i, i < BPT
        const uint32_t low = (1u << BPT) - 1u;
        uint32_t eqm[G], gtm[G];
#pragma unroll
        for (int h = 0; h < G; ++h) {
            gtm[h] = (uint32_t)(sm.gtmap[h][jj0 / 64] >> (jj0 % 64)) & low;
            eqm[h] = (uint32_t)(sm.eqmap[h][jj0 / 64] >> (jj0 % 64)) & low;
        }
        // equal keys of each head before this thread's blocks (two heads per scan in 16-bit fields:
        // a tile holds at most 8192 blocks)
        int eq_before[G];
#pragma unroll
        for (int h = 0; h < G; h += 2) {
            const int hi = h + 1 < G ? __popc(eqm[h + 1]) : 0;
            int tot = 0;
            const int e = scan(__popc(eqm[h]) | (hi << 16), &tot);
            tot = __builtin_amdgcn_readfirstlane(tot);
            eq_before[h] = eq_run[h] + (e & 0xffff);
            eq_run[h] += tot & 0xffff;
            if (h + 1 < G) {
                eq_before[h + 1] = eq_run[h + 1] + (e >> 16);
                eq_run[h + 1] += tot >> 16;
            }
        }
        uint32_t take[G], any = 0u;
#pragma unroll
        for (int h = 0; h < G; ++h) {
            take[h] = gtm[h];
            uint32_t e = eqm[h];
            int rank = eq_before[h];
            while (e != 0u && rank < need[h]) {         // the first `need` equal keys, in block order
                const uint32_t lowbit = e & (0u - e);
                take[h] |= lowbit;
                e ^= lowbit;
                ++rank;
            }
            any |= take[h];
        }
        int tot = 0;
        int pos = list_run + scan(__popc(any), &tot);
        list_run += __builtin_amdgcn_readfirstlane(tot);
#pragma unroll
        for (int i = 0; i < BPT; ++i) {
            const int j = jt0 + jj0 + i;
            if (jj0 + i < nb) {
                uint32_t bits = 0u;
#pragma unroll
                for (int h = 0; h < G; ++h) bits |= ((take[h] >> i) & 1u) << h;
                if (bits) list_x[pos++] = (uint32_t)j | (bits << 24);
                if (mask_x) {
#pragma unroll
                    for (int h = 0; h < G; ++h) mask_x[(size_t)h * nblk_cap + j] = (uint8_t)((bits >> h) & 1u);
                }
            }
        }
        __syncthreads();                                // the maps are rewritten for the next tile
    }
    int* counts_x = a.counts + (size_t)x * a.S1;
    for (int s = tid; s < a.S1; s += kSelThreads) counts_x[s] = s == 0 ? list_run : 0;
    if (mask_x) {
        for (int j = nblk + tid; j < nblk_cap; j += kSelThreads)
#pragma unroll
            for (int h = 0; h < G; ++h) mask_x[(size_t)h * nblk_cap + j] = 0;
    }
}

template __global__ void ffd_topk_select_kernel<1>(TopkArgs);
template __global__ void ffd_topk_select_kernel<2>(TopkArgs);
template __global__ void ffd_topk_select_kernel<4>(TopkArgs);
template __global__ void ffd_topk_select_kernel<8>(TopkArgs);

}  // namespace ffd
