// Kernel argument blocks and declarations of the library's HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ffd {

// Kept-block list entries staged in LDS per pass of the refinement kernel.
constexpr int kFfdChunk = 1024;
// Most blocks one scan workgroup covers (its kept list is staged in LDS), most scan workgroups per
// (sequence, KV head).
constexpr int kFfdMaxScanBlocks = 256;
constexpr int kScanWaves = 8;                  // waves per scan workgroup (one workgroup per CU)
constexpr int kScanThreads = 64 * kScanWaves;
// Waves per refinement workgroup (one workgroup per CU): 8 (two per SIMD) overlap one wave's waits
// with the other's work, which pays on long shares (the ragged 16-sequence batch, where half of the
// blocks are kept: 430 us of refinement against 503 us with 4 waves) and costs nothing at 4 x 128K.
constexpr int kRefineWaves = 8;
constexpr int kRefineThreads = 64 * kRefineWaves;
constexpr int kFfdMaxScanSplits = 1024;

// Thumbnail depth b (App. C: 2+8, 4+8, 8+8): 2^b levels c - Lv, Lv = (2^b - 1) / 2; a token's codes
// take 4b words.
__host__ __device__ constexpr float thumb_top_level(int bits) { return ((1 << bits) - 1) * 0.5f; }

struct ScanArgs {
    const uint16_t* q;          // bf16 [B, Hq, 128]
    const uint32_t* codes;      // [B, Hkv, Lcap/64, 64, 4b] (b = the kernel's thumbnail depth)
    const uint16_t* absmax;     // bf16 [B, Hkv, Lcap/64, 16, 4]
    const int8_t* resid;        // [B, Hkv, Lcap/16, 2, 64, 16]: read for the refined pseudo-max only
    const int32_t* seq_lens;    // [B]
    uint32_t* lists;            // [B*Hkv, Lcap/64]: kept blocks j | keep bits << 24, per scan split
    int* counts;                // [B*Hkv, S1]: kept blocks per scan split
    float* sigma;               // top-k selection: block scores [B*Hkv, Lcap/64, G]
    uint8_t* mask;              // [B, Hq, Lcap/64] or null
    float* m_tilde;             // [B, Hq] or null: the pseudo-max of each head
    int Hq, Hkv, Lcap, G, S1;
    float delta, scale;
    int n_sink, n_local;
};

struct RefineArgs {
    const uint16_t* q;          // bf16 [B, Hq, 128]
    const uint32_t* codes;      // thumbnail codes, from which the scan scores are recomputed
    const uint16_t* absmax;     // bf16 [B, Hkv, Lcap/64, 16, 4]
    const int8_t* resid;        // [B, Hkv, Lcap/16, 2, 64, 16]
    const uint16_t* v;          // bf16 [B, Hkv, Lcap, 128]
    const int32_t* seq_lens;    // [B]
    const uint32_t* lists;      // written by ffd_scan_kernel
    const int* counts;          // written by ffd_scan_kernel
    int2* table;                // [B*Hkv]: (first workgroup, workgroups) of each KV group
    float* part_m;              // [(W + B*Hkv) * G]
    float* part_l;
    float* part_acc;            // [(W + B*Hkv) * G, 128]
    int Hq, Hkv, Lcap, G, S1, W, npairs;
    float scale;
    float top_level;            // Lv of the thumbnail depth: the residual step is M / (254 Lv)
};

// The fused top-delta decode kernel: scan, pseudo-max, decisions, refinement and attention in one
// workgroup per (sequence, KV head, split), on an interleaved share of the group's blocks.
struct FusedArgs {
    const uint16_t* q;          // bf16 [B, Hq, 128]
    const uint32_t* codes;      // [B, Hkv, Lcap/64, 64, 4b]
    const uint16_t* absmax;     // bf16 [B, Hkv, Lcap/64, 16, 4]
    const int8_t* resid;        // [B, Hkv, Lcap/16, 2, 64, 16]
    const uint16_t* v;          // bf16 [B, Hkv, Lcap, 128]
    const int32_t* seq_lens;    // [B]
    uint8_t* mask;              // [B, Hq, Lcap/64] or null
    float* m_tilde;             // [B, Hq] or null: the pseudo-max of each head
    float* part_m;              // [B, Hq, S1] partial states (S1 > 1)
    float* part_l;
    float* part_acc;            // [B, Hq, S1, 128]
    uint16_t* out;              // bf16 [B, Hq, 128], written by the kernel itself when S1 == 1, else null
    float* lse;                 // [B, Hq] or null (S1 == 1 only)
    int Hq, Hkv, Lcap, G, S1;
    float delta, scale;
    int n_sink, n_local;
};

// Fixed-budget (top-k) selection over the block scores the scan kernel wrote; its output takes the
// place of the scan's kept lists and counts (each group's whole list in split 0).
struct TopkArgs {
    const float* sigma;         // [B*Hkv, Lcap/64, G]
    const int32_t* seq_lens;    // [B]
    uint32_t* lists;            // [B*Hkv, Lcap/64]: kept blocks j | keep bits << 24, in block order
    int* counts;                // [B*Hkv, S1]: the list length in split 0, zero elsewhere
    uint8_t* mask;              // [B, Hq, Lcap/64] or null
    int Hq, Hkv, Lcap, S1, k;
};

// Dense decode. Balanced mode (table != null, B <= kDenseBalanceMaxSeqs): a 1-D grid of
// (S + 1) * B * Hkv workgroups; sequence b (n_b blocks) gets W_b = ceil(n_b * min(W, N) / N)
// workgroups per KV head (W = S * B * Hkv, N = Hkv * sum n_b; 1 for an empty sequence), numbered in
// (sequence, KV head) order, each taking an equal run of the sequence's blocks and writing its
// partial rows at its own index (table[b * Hkv + kvh] = first workgroup, count). Otherwise a grid
// (S, Hkv, B) of equal runs per sequence with rows [B, Hq, S].
constexpr int kDenseBalanceMaxSeqs = 256;
struct DenseArgs {
    const uint16_t* q;          // bf16 [B, Hq, 128]
    const uint16_t* k;          // bf16 [B, Hkv, Lcap, 128]
    const uint16_t* v;          // bf16 [B, Hkv, Lcap, 128]
    const int32_t* seq_lens;
    float* part_m;
    float* part_l;
    float* part_acc;
    int2* table;                // balanced mode: [B * Hkv] (first workgroup, workgroups); else null
    int B, Hq, Hkv, Lcap, G, S;
    float scale;
};

struct QuantArgs {
    const uint16_t* k;          // bf16 [B, Hkv, Lcap, 128]
    uint32_t* codes;
    uint16_t* absmax;
    int8_t* resid;
    int Hkv, Lcap, t_begin, t_end;
};

struct AppendArgs {
    const uint16_t* k_new;      // bf16 [B, Hkv, 128]
    const uint16_t* v_new;      // bf16 [B, Hkv, 128]
    uint16_t* k_cache;          // bf16 [B, Hkv, Lcap, 128] or null
    uint16_t* v_cache;          // bf16 [B, Hkv, Lcap, 128] or null
    uint32_t* codes;
    uint16_t* absmax;
    int8_t* resid;
    int32_t* seq_lens;          // [B], read and advanced
    int Hkv, Lcap;
};

// What the scan kernel does after scoring a block:
//  kSelThumbnailPM  top-delta against the pseudo-max of the window tokens' thumbnail scores (Alg. 1);
//  kSelRefinedPM    top-delta against the pseudo-max of their refined logits (Eq. 3's reading);
//  kSelTopK         no decision: the block scores go to the workspace for ffd_topk_select_kernel.
// The first two write the kept lists and counts; no mode stores the scan scores.
enum ScanMode { kSelThumbnailPM = 0, kSelRefinedPM = 1, kSelTopK = 2 };
template <int NT, int BITS, int MODE> __global__ void ffd_scan_kernel(ScanArgs a);
// MODE kSelThumbnailPM or kSelRefinedPM; the scan scores of the kept tiles are recomputed from the
// codes the kernel has just streamed (bit for bit the values the decisions used).
template <int NT, int BITS, int MODE> __global__ void ffd_decode_kernel(FusedArgs a);
// The scan scores of the kept tiles (Eq. 4's first term) are recomputed from the RBITS-bit codes with
// the scan kernel's own integer MFMA and fp32 operations, so they equal the scan's bit for bit.
template <int NT, int RBITS> __global__ void ffd_refine_kernel(RefineArgs a);
template <int G> __global__ void ffd_topk_select_kernel(TopkArgs a);
constexpr int kTopkSelectThreads = 1024;
template <int NT> __global__ void dense_decode_kernel(DenseArgs a);
template <int BITS> __global__ void quantize_keys_kernel(QuantArgs a);
template <int BITS> __global__ void append_kv_kernel(AppendArgs a);
__global__ void lse_merge_kernel(const float* part_m, const float* part_l, const float* part_acc, int S,
                                 const int2* table, int G, uint16_t* out, float* lse);

}  // namespace ffd
