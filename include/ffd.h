/*
 * ffd.h — C ABI of the Faster Flash Decoding (FFD) decode-attention library for AMD MI355X (gfx950).
 *
 * One decode step of grouped-query attention for a batch of sequences:
 *
 *   ffd_quantize_keys           split each key into a b-bit thumbnail and an 8-bit residual
 *                               (Sec. 3.1; App. A formulation; Fig. 2 "K quantization"; b = 2, or
 *                               4 and 8 for the wider depths of App. C).
 *   ffd_append_kv               append one decode token per sequence to the bf16 and quantized
 *                               caches at its device-side length, and advance the length.
 *   ffd_decode_attention        pseudo-max over sink and local tokens (Alg. 1; Eq. 3), b-bit scan and
 *                               per-block top-delta selection (Alg. 1; Eq. 1), refinement of the kept
 *                               blocks' logits as the scan score plus the residual term (Eq. 4; the
 *                               scan score of a kept token is recomputed from its codes, bit for bit
 *                               the scan's value, rather than stored), online-softmax attention over
 *                               the kept blocks, split into partial states merged by log-sum-exp
 *                               (flash-decoding, Sec. 2 and Sec. 3.3). Kernels in order on `stream`:
 *                               either one fused kernel (scan, selection, refinement and attention
 *                               per interleaved slice of a sequence; short and mid contexts) plus
 *                               the merge when a head has more than one slice, or scan + selection,
 *                               refinement + attention spread over every CU, merge.
 *   ffd_dense_decode_attention  exact dense decode attention over the bf16 cache (the dense
 *                               comparator of Sec. 4.2), same split-and-merge scheme.
 *
 * Conventions for every entry point
 *  - Tensor arguments are DEVICE pointers to contiguous row-major buffers owned by the caller.
 *    The library never allocates, frees or retains them, never synchronises the host, and keeps no
 *    mutable global state apart from each device's compute-unit count, queried once and cached.
 *    Calls are asynchronous on `stream`; outputs are valid once it completes.
 *  - bf16 tensors are passed as `const void*` holding IEEE bfloat16 bit patterns.
 *  - Shapes: B sequences, Hq query heads, Hkv KV heads (Hq % Hkv == 0, G = Hq / Hkv in {1,2,4,8};
 *    query head h reads KV head h / G), head dimension D == 128, cache capacity Lcap tokens
 *    (a multiple of 64), KV block of 64 tokens.
 *  - seq_lens is a device int32 [B]; sequence b holds tokens [0, seq_lens[b]). Values are clamped
 *    to [0, Lcap] on the device (no host synchronisation to check them).
 *  - Pointers must be 16-byte aligned. Argument checks run before any launch; on failure nothing is
 *    enqueued and an ffd_status error is returned. A failed launch returns FFD_ERR_HIP.
 *
 * Thumbnail depth. `thumb_bits` b is 2 (the method's 2+8 format), 4 or 8 (the 4+8 and 8+8 depths of
 * App. C); any other positive value gives FFD_ERR_UNSUPPORTED. Code c in 0 .. 2^b - 1 stands for the
 * level c - Lv, Lv = (2^b - 1) / 2, on the step s = M / Lv. The same b must be used to write the
 * cache (ffd_quantize_keys, ffd_append_kv) and to read it (ffd_decode_attention).
 *
 * Quantized-key storage (this library's format; the paper fixes none). Per (b, kvh):
 *  - codes  uint32 [Lcap/64][b][64][4]: block j = tokens 64j..64j+63 holds 4b words for each lane
 *           l = n + 16g, word w of lane l at element [j][w / 4][l][w % 4] (so each group of four
 *           words is 1 KiB contiguous over the 64 lanes, one coalesced 16-byte load per lane). Lane
 *           l's words hold, for token 64j + 16*t4 + n and 64-dim chunk cc, the codes of dims
 *           64cc + 16g + e, e = 4k + i, in the b/2 words from (2*t4 + cc) * b/2: dim e in word
 *           (2*t4 + cc) * b/2 + k / (8/b) at bit 8i + b * (k % (8/b)). The field holds c for
 *           b = 2, 4 and the byte c - 128 (two's complement) for b = 8. For b = 2: word 2*t4 + cc,
 *           bit 8i + 2k.
 *  - absmax bf16 [Lcap/64][16][4]: element [j][n][t4] = M = max_i |k_i| of token 64j + 16*t4 + n.
 *  - resid  int8 [Lcap/16][2][64][16]: element [T][cc][n + 16g][e] is the residual of token 16T + n
 *           at dim 64cc + 16g + e.
 *  The reconstruction is k ~= M * n / (254 Lv) with n = 254 c + r - 254 Lv (thumbnail step M/Lv,
 *  residual step M/(254 Lv)); the thumbnail alone is k^quant = (c - Lv) * M / Lv. For b = 2:
 *  k ~= M * n / 381 and k^quant = (c - 1.5) * M / 1.5.
 */
#ifndef FFD_H
#define FFD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FFD_OK = 0,
    FFD_ERR_INVALID_ARGUMENT = 1,    /* null/misaligned pointer, bad shape, bad delta, bad range   */
    FFD_ERR_UNSUPPORTED = 2,         /* valid but not implemented: D != 128, block != 64, G > 8    */
    FFD_ERR_WORKSPACE_TOO_SMALL = 3, /* workspace_bytes < ffd_workspace_bytes(...)                 */
    FFD_ERR_HIP = 4,                 /* a HIP launch failed (hipGetLastError after the launch)     */
    FFD_ERR_SCRATCH_TOO_SMALL = 5    /* ffd_decode_attention_noalloc: the call needs more workspace
                                        than the library's fixed device scratch holds              */
} ffd_status;

#define FFD_HEAD_DIM 128
#define FFD_BLOCK 64
#define FFD_MAX_SPLITS 1024

/*
 * Key quantization (Sec. 3.1: k -> {k^quant, k^res}; App. A: symmetric mid-rise 2-bit codebook
 * {-1.5,-0.5,0.5,1.5}, s = max|k|/1.5, nearest level; ties at bin edges go to the upper level;
 * App. C: the same scheme with 2^b levels for b = 4, 8). Residual: r = rint(254 Lv k / M) - 254 c
 * + 254 Lv in [-127, 127] (round half to even; for b = 2, rint(381 k / M) - 254 c + 381); M = 0
 * gives code 2^(b-1) (level +0.5) and residual 0. Exact for every finite bf16 key.
 *
 *   k         bf16  [B, Hkv, Lcap, D]      keys (read)
 *   k_codes   uint32 codes layout above    (written for tokens [t_begin, t_end) only)
 *   k_absmax  bf16  absmax layout above    (written for tokens [t_begin, t_end) only)
 *   k_resid   int8  resid layout above     (written for tokens [t_begin, t_end) only)
 *   0 <= t_begin <= t_end <= Lcap. Tokens outside the range are left untouched, so appending one
 *   decode-step token is t_begin = L, t_end = L + 1.
 */
int ffd_quantize_keys(const void* k, void* k_codes, void* k_absmax, void* k_resid,
                      int B, int Hkv, int Lcap, int D, int thumb_bits, int t_begin, int t_end,
                      hipStream_t stream);

/*
 * Decode-step append, the cache update before attention in each step of a decode loop (the cache
 * grows by one token per step; the key is split as by ffd_quantize_keys, Sec. 3.1 and App. A). For
 * every sequence b with L = seq_lens[b] < Lcap: k_new[b] and v_new[b] are written at position L of
 * the bf16 caches (each cache pointer may be NULL to skip it), k_new[b] is quantized into codes,
 * absmax and residual at position L, and seq_lens[b] becomes L + 1. A sequence with L >= Lcap (or
 * L < 0) is left unchanged. Everything happens on the device, so the call can be captured in a HIP
 * graph together with ffd_decode_attention and the graph replayed as the cache grows (the kernels
 * read the lengths from seq_lens and size their grids from Lcap).
 *
 *   k_new, v_new   bf16 [B, Hkv, D]          the new token's key and value (read)
 *   k_cache, v_cache  bf16 [B, Hkv, Lcap, D]  or NULL
 *   k_codes, k_absmax, k_resid                quantized key layouts above, b = thumb_bits
 *   seq_lens       int32 [B] (device, read and written)
 */
int ffd_append_kv(const void* k_new, const void* v_new, void* k_cache, void* v_cache, void* k_codes,
                  void* k_absmax, void* k_resid, int32_t* seq_lens, int B, int Hkv, int Lcap, int D,
                  int thumb_bits, hipStream_t stream);

/*
 * FFD decode attention (Alg. 1 with Eq. 1-4), one query per head.
 *
 *   q            bf16  [B, Hq, D]
 *   k_codes, k_absmax, k_resid   quantized keys (from ffd_quantize_keys with the same thumb_bits)
 *   v            bf16  [B, Hkv, Lcap, D]
 *   thumb_bits   thumbnail depth b of the codes (2, 4 or 8); the scan reads 16b bytes per token
 *   seq_lens     int32 [B] (device)
 *   block_size   must be 64
 *   delta        top-delta margin >= 0 (+inf keeps every block); a block j is kept for head h iff
 *                max over its valid tokens of the thumbnail score >= m~_h - delta, where
 *                m~_h is the max thumbnail score over tokens [0, n_sink) U [L - n_local, L).
 *                All scores carry softmax_scale. With n_sink = n_local = 0, m~ = -inf and every
 *                block is kept.
 *   num_splits   refinement workgroups per KV group on average (1..FFD_MAX_SPLITS), or 0 for
 *                automatic: the call uses W = num_splits * B * Hkv refinement workgroups in all,
 *                given to the KV groups in proportion to their kept blocks (at least one each),
 *                each refining an equal run of its group's kept blocks in block order; their
 *                partial states are merged by log-sum-exp.
 *   softmax_scale  > 0, or 0 for 1/sqrt(D).
 *   out          bf16  [B, Hq, D]  softmax(z over kept tokens) . V, z the refined logits;
 *                                   0 for a head with no kept token (empty sequence).
 *   lse          float [B, Hq] or NULL: ln sum exp(z) over kept tokens (-inf if none).
 *   block_mask   uint8 [B, Hq, Lcap/64] or NULL: 1 iff head h kept block j; 0 at/after the end.
 *   workspace    device scratch of at least ffd_workspace_bytes(B, Hq, Hkv, Lcap, D, num_splits)
 *                bytes: the partials, a per-KV-group table locating them, the scan's kept-block
 *                lists and counts, and the per-head block scores the top-k rule selects from
 *                (4 * G bytes per block of the capacity). It needs no initialisation and is
 *                clobbered. Calls that overlap in time (different streams) need separate workspaces.
 *  Limits: B * Hkv <= 2^20 and Lcap <= 2^24 tokens, else FFD_ERR_UNSUPPORTED.
 */
int ffd_decode_attention(const void* q, const void* k_codes, const void* k_absmax,
                         const void* k_resid, const void* v, const int32_t* seq_lens,
                         int B, int Hq, int Hkv, int Lcap, int D, int thumb_bits, int block_size,
                         float delta, int n_sink, int n_local, int num_splits, float softmax_scale,
                         void* out, float* lse, uint8_t* block_mask,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Pseudo-max sources (ffd_decode_extras.pseudo_max). */
#define FFD_PSEUDO_MAX_THUMBNAIL 0   /* m~ over the window tokens' thumbnail scores (Alg. 1; default) */
#define FFD_PSEUDO_MAX_REFINED 1     /* m~ over their refined logits, thumbnail + residual (Eq. 3's
                                        window scores read with the 8-bit residual, Eq. 4) */

/* Kernels of the top-delta rule (ffd_decode_extras.kernels). */
#define FFD_KERNELS_AUTO 0    /* FFD_KERNELS_FUSED while each of its workgroups covers at most 64 blocks
                                 of the capacity (128 when there is at most one workgroup per compute
                                 unit), or a sequence fits one workgroup (ffd_select_kernels), else
                                 FFD_KERNELS_SPLIT */
#define FFD_KERNELS_FUSED 1   /* one kernel: each of S1 = ffd_fused_splits(...) workgroups per
                                 (sequence, KV head) scans the blocks j = s + S1 i, decides, refines and
                                 attends its own kept blocks; then the merge of the S1 partial states
                                 per head (no merge when S1 == 1: the kernel writes the outputs) */
#define FFD_KERNELS_SPLIT 2   /* scan + selection kernel (contiguous block ranges), refinement kernel
                                 (the kept blocks of all groups spread evenly over about one
                                 workgroup per CU), merge */

/*
 * Optional inputs and outputs of ffd_decode_attention_ex, for measurement and diagnostics
 * (Sec. 5.1, Sec. 5.2). A NULL pointer field, or a NULL extras pointer, leaves that feature off.
 *   stage_events  four events created by the caller (hipEventCreate), recorded on `stream`: before
 *                 the first kernel; after the selection (the scan kernel, or the top-k selection
 *                 kernel; with the fused kernel: after it); after the refinement (with the fused
 *                 kernel: the same point); after the merge (the same point again when no merge runs).
 *   m_tilde       float [B, Hq] (device): the pseudo-max m~ of each head (-inf for an empty
 *                 sequence or when both windows are empty), for the gap m - m~ of Sec. 5.2.
 *   pseudo_max    FFD_PSEUDO_MAX_THUMBNAIL or FFD_PSEUDO_MAX_REFINED (other values:
 *                 FFD_ERR_INVALID_ARGUMENT). The refined source reads the window blocks' residuals
 *                 as well; the selection still compares thumbnail block scores with m~ - delta.
 *   top_k         0: the top-delta rule. k > 0: the fixed-budget rule the paper compares top-delta
 *                 with (Sec. 1 and Fig. 1 (a); Table 3's selection-rule overhead): each head keeps
 *                 the min(k, blocks) blocks with the largest thumbnail block scores, equal scores
 *                 taken in block order; delta, n_sink, n_local and pseudo_max are then unused and
 *                 m_tilde must be NULL. The call then launches four kernels: the scan (writing every
 *                 block score), a per-(sequence, KV head) selection kernel, the refinement
 *                 (recomputing the kept blocks' thumbnail scores from the codes) and the merge; the
 *                 second stage event follows the selection kernel. Negative: FFD_ERR_INVALID_ARGUMENT.
 */
typedef struct ffd_decode_extras {
    hipEvent_t* stage_events;
    float* m_tilde;
    int pseudo_max;
    int top_k;
    int kernels;        /* FFD_KERNELS_AUTO, _FUSED or _SPLIT (top-delta only; with top_k > 0 the
                           split kernels run and FFD_KERNELS_FUSED is FFD_ERR_INVALID_ARGUMENT) */
} ffd_decode_extras;

/*
 * ffd_decode_attention with the extras above; ffd_decode_attention is this call with extras = NULL.
 * Everything else is as for ffd_decode_attention.
 */
int ffd_decode_attention_ex(const void* q, const void* k_codes, const void* k_absmax,
                            const void* k_resid, const void* v, const int32_t* seq_lens,
                            int B, int Hq, int Hkv, int Lcap, int D, int thumb_bits, int block_size,
                            float delta, int n_sink, int n_local, int num_splits, float softmax_scale,
                            void* out, float* lse, uint8_t* block_mask,
                            void* workspace, size_t workspace_bytes, hipStream_t stream,
                            const ffd_decode_extras* extras);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): ffd_decode_attention without a workspace argument. The
 * workspace is a fixed device array of FFD_NOALLOC_SCRATCH_BYTES inside the library, one per device,
 * which the device holds from the first call on it until the process ends (that first call resolves
 * its address; no call allocates). Arguments, outputs and kernels are those of ffd_decode_attention.
 *  - A call whose ffd_workspace_bytes(B, Hq, Hkv, Lcap, D, num_splits) exceeds the scratch returns
 *    FFD_ERR_SCRATCH_TOO_SMALL before any launch (16 MiB covers, for example, B * Hkv = 128 KV
 *    groups at Lcap = 131072 and G = 4).
 *  - Every call on a device uses that device's one scratch array, and the array keeps the last
 *    call's contents (nothing in it needs to start at zero). Calls that overlap in time on one
 *    device (different streams, or different host threads) race on it and give undefined results:
 *    serialise them, or use ffd_decode_attention with separate workspaces.
 */
#define FFD_NOALLOC_SCRATCH_BYTES (16u << 20)
int ffd_decode_attention_noalloc(const void* q, const void* k_codes, const void* k_absmax,
                                 const void* k_resid, const void* v, const int32_t* seq_lens,
                                 int B, int Hq, int Hkv, int Lcap, int D, int thumb_bits, int block_size,
                                 float delta, int n_sink, int n_local, int num_splits, float softmax_scale,
                                 void* out, float* lse, uint8_t* block_mask, hipStream_t stream);

/*
 * Exact dense decode attention over bf16 keys and values (the FlashAttention-2 comparator of
 * Sec. 4.2): out = softmax(softmax_scale * q K^T) V over tokens [0, seq_lens[b]).
 * Arguments as above; k is bf16 [B, Hkv, Lcap, D]; num_splits splits each sequence's blocks into
 * equal runs; the workspace needs ffd_dense_workspace_bytes(...) bytes.
 */
int ffd_dense_decode_attention(const void* q, const void* k, const void* v, const int32_t* seq_lens,
                               int B, int Hq, int Hkv, int Lcap, int D, int num_splits,
                               float softmax_scale, void* out, float* lse,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Number of splits an ffd_decode_attention call with this num_splits (0 = automatic) will use: the
 * automatic count gives the refinement (S + 1) * B * Hkv workgroups, at most one per compute unit of
 * the current device (its CU count is queried once per device and cached; 256, an MI355X's, if the
 * query fails). The workspace size depends on it, so size and call on the same device.
 * 0 on invalid input. */
int ffd_resolve_splits(int B, int Hkv, int Lcap, int num_splits);

/* Workgroups per (sequence, KV head) of the fused top-delta kernel for this num_splits: num_splits
 * itself, or automatically 1 when the capacity has at most 64 blocks, else about 16 blocks of the
 * capacity per workgroup with at most two workgroups per compute unit in all, or one per compute
 * unit when that cap would leave 64 or more blocks per workgroup and one per unit leaves at most
 * 128; raised to ceil((Lcap / 64) / 256) when smaller (a workgroup covers at most 256 blocks).
 * 0 on invalid input. */
int ffd_fused_splits(int B, int Hkv, int Lcap, int num_splits);

/* The kernels FFD_KERNELS_AUTO uses for these arguments: FFD_KERNELS_FUSED or FFD_KERNELS_SPLIT;
 * 0 on invalid input. */
int ffd_select_kernels(int B, int Hkv, int Lcap, int num_splits);

/* The same for ffd_dense_decode_attention, whose automatic count allows two workgroups per compute
 * unit (B * Hkv * S). */
int ffd_dense_resolve_splits(int B, int Hkv, int Lcap, int num_splits);

/* Workspace bytes needed by ffd_decode_attention for these arguments: the larger of the layout below
 * and ffd_dense_workspace_bytes(...), so it serves the dense entry point too. With
 * S = ffd_resolve_splits(...), P = B * Hkv KV groups, G = Hq / Hkv, C = Lcap / 64
 * blocks and S1 scan splits per group (chosen by the library from B, Hkv, Lcap), the regions, each
 * starting on a 256-byte boundary, are: partials (S * P + P) * G * (D + 2) * 4 bytes, table P * 8,
 * kept counts P * S1 * 4, kept lists P * C * 4, block scores P * C * G * 4.
 * 0 on invalid or unsupported input. */
size_t ffd_workspace_bytes(int B, int Hq, int Hkv, int Lcap, int D, int num_splits);

/* Workspace bytes needed by ffd_dense_decode_attention: B * Hq * S * (D + 2) * 4 (fp32 partials
 * m, l, acc) with S = ffd_dense_resolve_splits(...). 0 on invalid input. */
size_t ffd_dense_workspace_bytes(int B, int Hq, int Hkv, int Lcap, int D, int num_splits);

/* Static, human-readable name of a status code. */
const char* ffd_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* FFD_H */
