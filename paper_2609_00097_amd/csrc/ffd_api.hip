// C ABI of the FFD decode-attention library: argument checks, split choice, kernel launches.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <mutex>

#include "ffd.h"
#include "ffd_device.h"
#include "ffd_kernels.h"

using namespace ffd;

namespace {

// Compute units of the current device, queried once per device and cached (with the no-alloc
// entry point's per-device scratch address below, the only state the library keeps). kFallbackCus
// (an MI355X's count) is used if the query fails.
constexpr int kFallbackCus = 256;
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];

int device_cus() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return kFallbackCus;
    int n = g_cus[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        n = kFallbackCus;
    g_cus[dev].store(n, std::memory_order_relaxed);
    return n;
}

// Device scratch of ffd_decode_attention_noalloc: one array per device, held until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: the array is only ever
// reached through the address hipGetSymbolAddress returns for the current device, cached per device.
constexpr size_t kNoallocScratchBytes = (size_t)FFD_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

// The current device's scratch address (resolved on the first call on that device), or null.
void* device_scratch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (p) return p;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch[dev].store(p, std::memory_order_release);
    }
    return p;
}

// Automatic split counts. The FFD refinement grid has W + B*Hkv = (S + 1) * B*Hkv workgroups of
// equal work; it should not exceed one per CU, because a CU serves its older workgroup's memory
// requests first, so a second workgroup on a CU finishes its share about 3 us later (at 4 x 128K on
// 256 CUs, delta 5: S = 7 (256 workgroups) 60.0 us per step; S = 8 (288) 65.2 us; S = 15 (512)
// 62.2 us; S = 6 (224) 62.3 us). The dense path keeps two workgroups per CU for up to 63 KV groups
// (4 x 128K: S = 15, 512 workgroups, against S = 23 or 31 about 2 % slower; B = 1: more splits are
// slower still) and three from 64 groups on (the ragged batch of 16 sequences, 128 groups: 512
// workgroups 873 us, 768 workgroups 833 us, 1024 workgroups 832 us).
int ffd_target_workgroups() { return device_cus(); }
int dense_target_workgroups(long long pairs) { return (pairs >= 64 ? 3 : 2) * device_cus(); }
constexpr int kMinBlocksPerSplit = 8;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int resolve_splits(int B, int Hkv, int Lcap, int num_splits, bool dense = false) {
    if (B <= 0 || Hkv <= 0 || Lcap <= 0 || num_splits < 0 || num_splits > FFD_MAX_SPLITS) return 0;
    if (num_splits > 0) return num_splits;
    const long long pairs = (long long)B * Hkv;
    const int target = dense ? dense_target_workgroups(pairs) : ffd_target_workgroups();
    long long s = target / pairs - 1;
    const long long cap = (long long)(Lcap / FFD_BLOCK) / kMinBlocksPerSplit;
    if (s > cap) s = cap;
    if (s < 1) s = 1;
    if (s > FFD_MAX_SPLITS) s = FFD_MAX_SPLITS;
    return (int)s;
}

int check_shapes(int B, int Hq, int Hkv, int Lcap, int D) {
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Lcap < FFD_BLOCK || Lcap % FFD_BLOCK) return FFD_ERR_INVALID_ARGUMENT;
    if (Hq % Hkv) return FFD_ERR_INVALID_ARGUMENT;
    if (B > 65535 || Hkv > 65535) return FFD_ERR_UNSUPPORTED;
    const int G = Hq / Hkv;
    if (G != 1 && G != 2 && G != 4 && G != 8) return FFD_ERR_UNSUPPORTED;
    if (D != FFD_HEAD_DIM) return FFD_ERR_UNSUPPORTED;
    // element counts must fit the kernels' size_t indexing and the per-sequence int token index
    if ((long long)Lcap > (1LL << 30)) return FFD_ERR_UNSUPPORTED;
    return FFD_OK;
}

// Thumbnail depths with kernels: 2+8 (App. A), 4+8 and 8+8 (App. C).
int check_bits(int bits) {
    if (bits == 2 || bits == 4 || bits == 8) return FFD_OK;
    return bits > 0 ? FFD_ERR_UNSUPPORTED : FFD_ERR_INVALID_ARGUMENT;
}

int launch_status() {
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? FFD_OK : FFD_ERR_HIP;
}

// Workspace: split partials m [B,Hq,S], l [B,Hq,S], acc [B,Hq,S,D] (fp32); the FFD path adds the
// scan kernel's kept lists and counts and the top-k rule's block scores.
struct Partials {
    float* m;
    float* l;
    float* acc;
};

constexpr size_t kAlign = 256;
size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

size_t partials_bytes(int B, int Hq, int S, int D) { return (size_t)B * Hq * S * (D + 2) * sizeof(float); }

Partials carve(void* ws, int B, int Hq, int S) {
    const size_t rows = (size_t)B * Hq * S;
    float* base = static_cast<float*>(ws);
    return Partials{base, base + rows, base + 2 * rows};
}

int head_tiles(int G) { return G <= 4 ? 1 : 2; }

// Workgroups of the scan kernel per (sequence, KV head): about one per CU in all (one 8-wave
// workgroup per CU: 8 waves x 4 blocks of 2 KiB in flight cover a CU's share of the HBM bandwidth at
// its load latency; 512 or 1024 workgroups of 8 or 4 waves measured 0.6-1.1 us slower at 4 x 128K),
// each scanning at least kMinScanBlocks blocks so the pseudo-max and query setup stay a small part
// of its work, and at most kFfdMaxScanBlocks (their maxima are staged in LDS).
constexpr int kMinScanBlocks = 16;

int scan_splits(int B, int Hkv, int Lcap) {
    const long long pairs = (long long)B * Hkv;
    const long long nblk_cap = Lcap / FFD_BLOCK;
    const long long target = device_cus();
    long long s = (target + pairs - 1) / pairs;
    const long long cap = nblk_cap / kMinScanBlocks;
    if (s > cap) s = cap;
    const long long need = (nblk_cap + kFfdMaxScanBlocks - 1) / kFfdMaxScanBlocks;
    if (s < need) s = need;
    if (s < 1) s = 1;
    return (int)s;
}

// Workgroups per (sequence, KV head) of the fused top-delta kernel, S1: num_splits when given;
// automatically one for a group of at most kFusedAloneBlocks blocks (the kernel then writes the
// outputs itself, with no merge launch), else about kFusedTargetBlocks blocks per workgroup with
// at most two workgroups per CU in all. Never fewer than ceil(blocks / kFfdMaxScanBlocks) (a
// workgroup's block scores are staged in LDS). Measured at B = 1, 32q/8kv, delta 5 (layer-averaged
// us per step, best split count per length): 4K 13.7 (S1 = 1; 15.0 with a merge), 8K 14.5 (8),
// 16K 14.6 (16), 32K 15.7 (16..32), 64K 25.0 (64), 128K 29.8 (64).
constexpr int kFusedAloneBlocks = 64;
constexpr int kFusedTargetBlocks = 16;
constexpr int kFusedMaxBlocks = 64;            // blocks per workgroup the fused kernel takes ...
constexpr int kFusedWideMaxBlocks = 128;       // ... or this many with at most one workgroup per CU

int decode_splits(int B, int Hkv, int Lcap, int num_splits) {
    if (B <= 0 || Hkv <= 0 || Lcap <= 0 || num_splits < 0 || num_splits > FFD_MAX_SPLITS) return 0;
    const long long pairs = (long long)B * Hkv;
    const long long nblk_cap = Lcap / FFD_BLOCK;
    const long long need = (nblk_cap + kFfdMaxScanBlocks - 1) / kFfdMaxScanBlocks;
    long long s = num_splits;
    if (s == 0) {
        if (nblk_cap <= kFusedAloneBlocks) {
            s = 1;
        } else {
            s = (nblk_cap + kFusedTargetBlocks - 1) / kFusedTargetBlocks;
            const long long cap = 2LL * device_cus() / pairs;
            if (s > cap) {
                s = cap;
                // where the two-per-CU cap leaves kFusedMaxBlocks or more blocks per workgroup, one
                // workgroup per CU with up to twice the blocks streams better (its waves do not
                // queue behind another workgroup's on the CU): at 1 x 256K, 32q/8kv, delta 5, 32
                // workgroups of 128 blocks per group 31.1 us (the clustered workload: 29.6 us)
                // against 32.7 (31.6) us for 64 of 64 blocks; at 1 x 128K the 64 workgroups of 32
                // blocks stay ahead (29.5 against 34.0 us)
                const long long one = std::max(1LL, (long long)device_cus() / pairs);
                if (s > 0 && (nblk_cap + s - 1) / s >= kFusedMaxBlocks &&
                    (nblk_cap + one - 1) / one <= kFusedWideMaxBlocks)
                    s = one;
            }
        }
    }
    if (s < need) s = need;
    if (s < 1) s = 1;
    if (s > kFfdMaxScanSplits) return 0;
    return (int)s;
}

// The top-delta kernels FFD_KERNELS_AUTO picks: the fused kernel while its workgroups cover at
// most kFusedMaxBlocks blocks of the capacity each (or a group fits one workgroup), else scan +
// refinement + merge, whose refinement spreads the kept blocks over every CU. (The fused kernel
// refines each workgroup's own kept blocks, so its time follows the workgroup with the most: at
// 4 x 128K, 32q/8kv, delta 5, its best split count gave 66.9 us against 58.9 us for the split
// kernels; at 1 x 256K, 32 workgroups of 128 blocks per group gave 31.1 us against 34.3 us.) With
// at most one workgroup per CU the fused kernel takes up to kFusedWideMaxBlocks blocks each.
int auto_kernels(int B, int Hkv, int Lcap, int S1f) {
    const int nblk_cap = Lcap / FFD_BLOCK;
    const int bps = (nblk_cap + S1f - 1) / S1f;
    const bool one_per_cu = (long long)S1f * B * Hkv <= device_cus();
    return bps <= kFusedMaxBlocks || nblk_cap <= kFusedAloneBlocks || (one_per_cu && bps <= kFusedWideMaxBlocks)
               ? FFD_KERNELS_FUSED : FFD_KERNELS_SPLIT;
}

// FFD workspace: partial states (for the fused top-delta kernel's B * Hq * S1f rows, or for the
// top-k path's W + B*Hkv refinement workgroups (W = S * B * Hkv) of G heads each), and for the
// top-k path the per-group (first workgroup, count) table, the scan's per-split kept counts and
// kept lists, and the block scores [P, C, G] it selects from.
struct FfdWorkspace {
    size_t rows;                      // partial rows
    size_t table_off, counts_off, lists_off, sigma_off, total;
};

FfdWorkspace ffd_layout(int B, int Hq, int Hkv, int Lcap, int D, int S, int S1f) {
    FfdWorkspace w;
    const size_t pairs = (size_t)B * Hkv;
    const size_t nblk_cap = (size_t)(Lcap / FFD_BLOCK);
    // the top-k path's refinement rows, or the fused kernel's [B, Hq, S1f] rows
    w.rows = std::max(((size_t)S * pairs + pairs) * (size_t)(Hq / Hkv), (size_t)B * Hq * (size_t)S1f);
    w.table_off = round_up(w.rows * (D + 2) * sizeof(float), kAlign);
    w.counts_off = w.table_off + round_up(pairs * 2 * sizeof(int), kAlign);
    w.lists_off = w.counts_off + round_up(pairs * (size_t)scan_splits(B, Hkv, Lcap) * sizeof(int), kAlign);
    w.sigma_off = w.lists_off + round_up(pairs * nblk_cap * sizeof(uint32_t), kAlign);
    w.total = w.sigma_off + pairs * nblk_cap * (size_t)(Hq / Hkv) * sizeof(float);
    return w;
}

int attention_common_checks(const void* q, const void* v, const int32_t* seq_lens, int B, int Hq,
                            int Hkv, int Lcap, int D, int num_splits, float softmax_scale,
                            const void* out, const float* lse, const void* ws, size_t ws_bytes,
                            bool dense, int* S_out, bool check_ws = true) {
    int st = check_shapes(B, Hq, Hkv, Lcap, D);
    if (st != FFD_OK) return st;
    if (num_splits < 0 || num_splits > FFD_MAX_SPLITS) return FFD_ERR_INVALID_ARGUMENT;
    if (!(softmax_scale >= 0.f) || std::isinf(softmax_scale)) return FFD_ERR_INVALID_ARGUMENT;
    if (B == 0) { *S_out = 0; return FFD_OK; }
    if (!q || !v || !seq_lens || !out || (check_ws && !ws)) return FFD_ERR_INVALID_ARGUMENT;
    if (!aligned16(q) || !aligned16(v) || !aligned16(out) || (check_ws && !aligned16(ws)))
        return FFD_ERR_INVALID_ARGUMENT;
    if ((reinterpret_cast<uintptr_t>(seq_lens) & 3u) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)))
        return FFD_ERR_INVALID_ARGUMENT;
    const int S = resolve_splits(B, Hkv, Lcap, num_splits, dense);
    if (S <= 0) return FFD_ERR_INVALID_ARGUMENT;
    *S_out = S;
    return FFD_OK;
}

// The scan kernel for this depth, head tiling and selection mode (ScanMode).
template <int NT, int BITS>
void launch_scan_nt(int mode, dim3 grid, hipStream_t stream, const ScanArgs& sa) {
    if (mode == kSelRefinedPM)
        hipLaunchKernelGGL((ffd_scan_kernel<NT, BITS, kSelRefinedPM>), grid, dim3(kScanThreads), 0, stream, sa);
    else if (mode == kSelTopK)
        hipLaunchKernelGGL((ffd_scan_kernel<NT, BITS, kSelTopK>), grid, dim3(kScanThreads), 0, stream, sa);
    else
        hipLaunchKernelGGL((ffd_scan_kernel<NT, BITS, kSelThumbnailPM>), grid, dim3(kScanThreads), 0, stream, sa);
}

template <int BITS>
void launch_scan_bits(int nt, int mode, dim3 grid, hipStream_t stream, const ScanArgs& sa) {
    if (nt == 1) launch_scan_nt<1, BITS>(mode, grid, stream, sa);
    else launch_scan_nt<2, BITS>(mode, grid, stream, sa);
}

void launch_scan(int bits, int nt, int mode, dim3 grid, hipStream_t stream, const ScanArgs& sa) {
    if (bits == 2) launch_scan_bits<2>(nt, mode, grid, stream, sa);
    else if (bits == 4) launch_scan_bits<4>(nt, mode, grid, stream, sa);
    else launch_scan_bits<8>(nt, mode, grid, stream, sa);
}

// The fused top-delta kernel for this depth, head tiling and pseudo-max source.
template <int NT, int BITS>
void launch_fused_nt(int mode, dim3 grid, hipStream_t stream, const FusedArgs& fa) {
    if (mode == kSelRefinedPM)
        hipLaunchKernelGGL((ffd_decode_kernel<NT, BITS, kSelRefinedPM>), grid, dim3(kScanThreads), 0, stream, fa);
    else
        hipLaunchKernelGGL((ffd_decode_kernel<NT, BITS, kSelThumbnailPM>), grid, dim3(kScanThreads), 0, stream, fa);
}

void launch_fused(int bits, int nt, int mode, dim3 grid, hipStream_t stream, const FusedArgs& fa) {
    if (bits == 2) nt == 1 ? launch_fused_nt<1, 2>(mode, grid, stream, fa) : launch_fused_nt<2, 2>(mode, grid, stream, fa);
    else if (bits == 4) nt == 1 ? launch_fused_nt<1, 4>(mode, grid, stream, fa) : launch_fused_nt<2, 4>(mode, grid, stream, fa);
    else nt == 1 ? launch_fused_nt<1, 8>(mode, grid, stream, fa) : launch_fused_nt<2, 8>(mode, grid, stream, fa);
}

// The refinement kernel, recomputing the scan scores from rbits-bit codes.
template <int NT>
void launch_refine_nt(int rbits, dim3 grid, hipStream_t stream, const RefineArgs& ra) {
    if (rbits == 2) hipLaunchKernelGGL((ffd_refine_kernel<NT, 2>), grid, dim3(kRefineThreads), 0, stream, ra);
    else if (rbits == 4) hipLaunchKernelGGL((ffd_refine_kernel<NT, 4>), grid, dim3(kRefineThreads), 0, stream, ra);
    else hipLaunchKernelGGL((ffd_refine_kernel<NT, 8>), grid, dim3(kRefineThreads), 0, stream, ra);
}

// Every argument check of ffd_decode_attention_ex, in its order, with nothing launched; with
// check_ws false the workspace pointer is not checked (the no-alloc entry point brings its own).
// *S_out receives the split count (0 when B == 0).
int decode_checks(const void* q, const void* k_codes, const void* k_absmax, const void* k_resid,
                  const void* v, const int32_t* seq_lens, int B, int Hq, int Hkv, int Lcap, int D,
                  int thumb_bits, int block_size, float delta, int n_sink, int n_local, int num_splits,
                  float softmax_scale, const void* out, const float* lse, const void* workspace,
                  const ffd_decode_extras* extras, bool check_ws, int* S_out) {
    const float* m_tilde = extras ? extras->m_tilde : nullptr;
    const int pm_source = extras ? extras->pseudo_max : FFD_PSEUDO_MAX_THUMBNAIL;
    const int top_k = extras ? extras->top_k : 0;
    const int kernels = extras ? extras->kernels : FFD_KERNELS_AUTO;
    if (pm_source != FFD_PSEUDO_MAX_THUMBNAIL && pm_source != FFD_PSEUDO_MAX_REFINED)
        return FFD_ERR_INVALID_ARGUMENT;
    if (kernels != FFD_KERNELS_AUTO && kernels != FFD_KERNELS_FUSED && kernels != FFD_KERNELS_SPLIT)
        return FFD_ERR_INVALID_ARGUMENT;
    if (top_k > 0 && kernels == FFD_KERNELS_FUSED) return FFD_ERR_INVALID_ARGUMENT;
    if (top_k < 0 || (top_k > 0 && m_tilde)) return FFD_ERR_INVALID_ARGUMENT;
    if (block_size != FFD_BLOCK) return block_size > 0 ? FFD_ERR_UNSUPPORTED : FFD_ERR_INVALID_ARGUMENT;
    if (std::isnan(delta) || delta < 0.f || n_sink < 0 || n_local < 0) return FFD_ERR_INVALID_ARGUMENT;
    int st = check_bits(thumb_bits);
    if (st != FFD_OK) return st;
    st = attention_common_checks(q, v, seq_lens, B, Hq, Hkv, Lcap, D, num_splits, softmax_scale, out,
                                 lse, workspace, 0, false, S_out, check_ws);
    if (st != FFD_OK || B == 0) return st;
    if (!k_codes || !k_absmax || !k_resid) return FFD_ERR_INVALID_ARGUMENT;
    if (!aligned16(k_codes) || !aligned16(k_absmax) || !aligned16(k_resid)) return FFD_ERR_INVALID_ARGUMENT;
    if (m_tilde && (reinterpret_cast<uintptr_t>(m_tilde) & 3u)) return FFD_ERR_INVALID_ARGUMENT;
    if ((long long)B * Hkv > (1LL << 20)) return FFD_ERR_UNSUPPORTED;
    if (Lcap / FFD_BLOCK > kFfdMaxScanBlocks * kFfdMaxScanSplits) return FFD_ERR_UNSUPPORTED;
    return FFD_OK;
}

}  // namespace

extern "C" {

int ffd_resolve_splits(int B, int Hkv, int Lcap, int num_splits) {
    return resolve_splits(B, Hkv, Lcap, num_splits);
}

int ffd_fused_splits(int B, int Hkv, int Lcap, int num_splits) {
    return decode_splits(B, Hkv, Lcap, num_splits);
}

int ffd_select_kernels(int B, int Hkv, int Lcap, int num_splits) {
    const int S1f = decode_splits(B, Hkv, Lcap, num_splits);
    if (S1f <= 0) return 0;
    return auto_kernels(B, Hkv, Lcap, S1f);
}

int ffd_dense_resolve_splits(int B, int Hkv, int Lcap, int num_splits) {
    return resolve_splits(B, Hkv, Lcap, num_splits, true);
}

size_t ffd_dense_workspace_bytes(int B, int Hq, int Hkv, int Lcap, int D, int num_splits) {
    if (check_shapes(B, Hq, Hkv, Lcap, D) != FFD_OK) return 0;
    const int S = resolve_splits(B > 0 ? B : 1, Hkv, Lcap, num_splits, true);
    if (S <= 0) return 0;
    if (B > kDenseBalanceMaxSeqs) return partials_bytes(B, Hq, S, D);
    // balanced mode: (S + 1) partial rows per head, then the per-(sequence, KV head) table
    return round_up(partials_bytes(B, Hq, S + 1, D), kAlign) + (size_t)B * Hkv * sizeof(int2);
}

size_t ffd_workspace_bytes(int B, int Hq, int Hkv, int Lcap, int D, int num_splits) {
    if (check_shapes(B, Hq, Hkv, Lcap, D) != FFD_OK) return 0;
    const int S = resolve_splits(B > 0 ? B : 1, Hkv, Lcap, num_splits);
    const int S1f = decode_splits(B > 0 ? B : 1, Hkv, Lcap, num_splits);
    if (S <= 0 || S1f <= 0) return 0;
    if ((long long)B * Hkv > (1LL << 20) || Lcap / FFD_BLOCK > kFfdMaxScanBlocks * kFfdMaxScanSplits) return 0;
    // enough for the dense entry point with the same num_splits too
    return std::max(ffd_layout(B, Hq, Hkv, Lcap, D, S, S1f).total,
                    ffd_dense_workspace_bytes(B, Hq, Hkv, Lcap, D, num_splits));
}

const char* ffd_status_string(int status) {
    switch (status) {
        case FFD_OK: return "FFD_OK";
        case FFD_ERR_INVALID_ARGUMENT: return "FFD_ERR_INVALID_ARGUMENT";
        case FFD_ERR_UNSUPPORTED: return "FFD_ERR_UNSUPPORTED";
        case FFD_ERR_WORKSPACE_TOO_SMALL: return "FFD_ERR_WORKSPACE_TOO_SMALL";
        case FFD_ERR_HIP: return "FFD_ERR_HIP";
        case FFD_ERR_SCRATCH_TOO_SMALL: return "FFD_ERR_SCRATCH_TOO_SMALL";
        default: return "FFD_ERR_UNKNOWN";
    }
}

int ffd_quantize_keys(const void* k, void* k_codes, void* k_absmax, void* k_resid, int B, int Hkv,
                      int Lcap, int D, int thumb_bits, int t_begin, int t_end, hipStream_t stream) {
    int st = check_shapes(B, Hkv, Hkv, Lcap, D);
    if (st == FFD_OK) st = check_bits(thumb_bits);
    if (st != FFD_OK) return st;
    if (t_begin < 0 || t_end < t_begin || t_end > Lcap) return FFD_ERR_INVALID_ARGUMENT;
    if (B == 0 || t_end == t_begin) return FFD_OK;
    if (!k || !k_codes || !k_absmax || !k_resid) return FFD_ERR_INVALID_ARGUMENT;
    if (!aligned16(k) || !aligned16(k_codes) || !aligned16(k_absmax) || !aligned16(k_resid))
        return FFD_ERR_INVALID_ARGUMENT;
    QuantArgs a{static_cast<const uint16_t*>(k), static_cast<uint32_t*>(k_codes),
                static_cast<uint16_t*>(k_absmax), static_cast<int8_t*>(k_resid), Hkv, Lcap, t_begin, t_end};
    const dim3 grid((unsigned)((t_end - (t_begin & ~63) + 63) / 64), (unsigned)Hkv, (unsigned)B);
    if (thumb_bits == 2)
        hipLaunchKernelGGL(quantize_keys_kernel<2>, grid, dim3(kThreads), 0, stream, a);
    else if (thumb_bits == 4)
        hipLaunchKernelGGL(quantize_keys_kernel<4>, grid, dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(quantize_keys_kernel<8>, grid, dim3(kThreads), 0, stream, a);
    return launch_status();
}

int ffd_append_kv(const void* k_new, const void* v_new, void* k_cache, void* v_cache, void* k_codes,
                  void* k_absmax, void* k_resid, int32_t* seq_lens, int B, int Hkv, int Lcap, int D,
                  int thumb_bits, hipStream_t stream) {
    int st = check_shapes(B, Hkv, Hkv, Lcap, D);
    if (st == FFD_OK) st = check_bits(thumb_bits);
    if (st != FFD_OK) return st;
    if (B == 0) return FFD_OK;
    if (!k_new || !v_new || !k_codes || !k_absmax || !k_resid || !seq_lens) return FFD_ERR_INVALID_ARGUMENT;
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_codes) || !aligned16(k_absmax) ||
        !aligned16(k_resid) || (k_cache && !aligned16(k_cache)) || (v_cache && !aligned16(v_cache)) ||
        (reinterpret_cast<uintptr_t>(seq_lens) & 3u))
        return FFD_ERR_INVALID_ARGUMENT;
    AppendArgs a{static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                 static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache),
                 static_cast<uint32_t*>(k_codes), static_cast<uint16_t*>(k_absmax),
                 static_cast<int8_t*>(k_resid), seq_lens, Hkv, Lcap};
    if (thumb_bits == 2)
        hipLaunchKernelGGL(append_kv_kernel<2>, dim3((unsigned)B), dim3(kThreads), 0, stream, a);
    else if (thumb_bits == 4)
        hipLaunchKernelGGL(append_kv_kernel<4>, dim3((unsigned)B), dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(append_kv_kernel<8>, dim3((unsigned)B), dim3(kThreads), 0, stream, a);
    return launch_status();
}

int ffd_decode_attention_ex(const void* q, const void* k_codes, const void* k_absmax,
                            const void* k_resid, const void* v, const int32_t* seq_lens, int B, int Hq,
                            int Hkv, int Lcap, int D, int thumb_bits, int block_size, float delta, int n_sink,
                            int n_local, int num_splits, float softmax_scale, void* out, float* lse,
                            uint8_t* block_mask, void* workspace, size_t workspace_bytes,
                            hipStream_t stream, const ffd_decode_extras* extras) {
    hipEvent_t* stage_events = extras ? extras->stage_events : nullptr;
    float* m_tilde = extras ? extras->m_tilde : nullptr;
    const int pm_source = extras ? extras->pseudo_max : FFD_PSEUDO_MAX_THUMBNAIL;
    const int top_k = extras ? extras->top_k : 0;
    const int kernels_req = extras ? extras->kernels : FFD_KERNELS_AUTO;
    int S = 0;
    int st = decode_checks(q, k_codes, k_absmax, k_resid, v, seq_lens, B, Hq, Hkv, Lcap, D, thumb_bits,
                           block_size, delta, n_sink, n_local, num_splits, softmax_scale, out, lse,
                           workspace, extras, true, &S);
    if (st != FFD_OK || B == 0) return st;
    if (workspace_bytes < ffd_workspace_bytes(B, Hq, Hkv, Lcap, D, num_splits)) return FFD_ERR_WORKSPACE_TOO_SMALL;
    const int G = Hq / Hkv;
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt((float)D);
    const int S1f = decode_splits(B, Hkv, Lcap, num_splits);
    const FfdWorkspace W = ffd_layout(B, Hq, Hkv, Lcap, D, S, S1f);
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    float* part_m = reinterpret_cast<float*>(ws);
    float* part_l = part_m + W.rows;
    float* part_acc = part_l + W.rows;
    int2* table = reinterpret_cast<int2*>(ws + W.table_off);
    int* counts = reinterpret_cast<int*>(ws + W.counts_off);
    uint32_t* lists = reinterpret_cast<uint32_t*>(ws + W.lists_off);
    float* sigma = reinterpret_cast<float*>(ws + W.sigma_off);
    const int S1 = scan_splits(B, Hkv, Lcap);
    const int npairs = B * Hkv;
    const int Wr = S * npairs;
    ScanArgs sa{static_cast<const uint16_t*>(q), static_cast<const uint32_t*>(k_codes),
                static_cast<const uint16_t*>(k_absmax), static_cast<const int8_t*>(k_resid), seq_lens, lists,
                counts, sigma, block_mask, m_tilde, Hq, Hkv, Lcap, G, S1, delta, scale, n_sink, n_local};
    RefineArgs ra{static_cast<const uint16_t*>(q), static_cast<const uint32_t*>(k_codes),
                  static_cast<const uint16_t*>(k_absmax),
                  static_cast<const int8_t*>(k_resid), static_cast<const uint16_t*>(v), seq_lens, lists,
                  counts, table, part_m, part_l, part_acc, Hq, Hkv, Lcap, G, S1, Wr, npairs, scale,
                  thumb_top_level(thumb_bits)};
    TopkArgs ta{sigma, seq_lens, lists, counts, block_mask, Hq, Hkv, Lcap, S1, top_k};
    const dim3 scan_grid((unsigned)S1, (unsigned)Hkv, (unsigned)B);
    const dim3 refine_grid((unsigned)(Wr + npairs));
    auto mark = [&](int i) {
        return stage_events && hipEventRecord(stage_events[i], stream) != hipSuccess ? FFD_ERR_HIP : FFD_OK;
    };

    const int mode = top_k > 0 ? kSelTopK : (pm_source == FFD_PSEUDO_MAX_REFINED ? kSelRefinedPM : kSelThumbnailPM);
    if ((st = mark(0)) != FFD_OK) return st;
    const int kernels = kernels_req == FFD_KERNELS_AUTO ? auto_kernels(B, Hkv, Lcap, S1f) : kernels_req;
    if (top_k == 0 && kernels == FFD_KERNELS_FUSED) {
        // top-delta, fused: one kernel, then the merge of its S1f partial states per head (none when
        // S1f == 1: the kernel writes the outputs itself)
        const bool direct = S1f == 1;
        FusedArgs fa{static_cast<const uint16_t*>(q), static_cast<const uint32_t*>(k_codes),
                     static_cast<const uint16_t*>(k_absmax), static_cast<const int8_t*>(k_resid),
                     static_cast<const uint16_t*>(v), seq_lens, block_mask, m_tilde, part_m, part_l, part_acc,
                     direct ? static_cast<uint16_t*>(out) : nullptr, direct ? lse : nullptr,
                     Hq, Hkv, Lcap, G, S1f, delta, scale, n_sink, n_local};
        launch_fused(thumb_bits, G <= 4 ? 1 : 2, mode, dim3((unsigned)S1f, (unsigned)Hkv, (unsigned)B), stream, fa);
        if ((st = launch_status()) != FFD_OK || (st = mark(1)) != FFD_OK || (st = mark(2)) != FFD_OK) return st;
        if (!direct) {
            hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)(B * Hq)), dim3(kThreads), 0, stream, part_m,
                               part_l, part_acc, S1f, nullptr, 1, static_cast<uint16_t*>(out), lse);
            if ((st = launch_status()) != FFD_OK) return st;
        }
        return mark(3);
    }
    launch_scan(thumb_bits, G <= 4 ? 1 : 2, mode, scan_grid, stream, sa);
    if ((st = launch_status()) != FFD_OK) return st;
    if (top_k > 0) {
        const dim3 grid((unsigned)npairs);
        const dim3 block(kTopkSelectThreads);
        if (G == 1) hipLaunchKernelGGL(ffd_topk_select_kernel<1>, grid, block, 0, stream, ta);
        else if (G == 2) hipLaunchKernelGGL(ffd_topk_select_kernel<2>, grid, block, 0, stream, ta);
        else if (G == 4) hipLaunchKernelGGL(ffd_topk_select_kernel<4>, grid, block, 0, stream, ta);
        else hipLaunchKernelGGL(ffd_topk_select_kernel<8>, grid, block, 0, stream, ta);
        if ((st = launch_status()) != FFD_OK) return st;
    }
    if ((st = mark(1)) != FFD_OK) return st;
    if (G <= 4) launch_refine_nt<1>(thumb_bits, refine_grid, stream, ra);
    else launch_refine_nt<2>(thumb_bits, refine_grid, stream, ra);
    if ((st = launch_status()) != FFD_OK || (st = mark(2)) != FFD_OK) return st;
    hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)(B * Hq)), dim3(kThreads), 0, stream, part_m, part_l,
                       part_acc, 0, table, G, static_cast<uint16_t*>(out), lse);
    if ((st = launch_status()) != FFD_OK) return st;
    return mark(3);
}

int ffd_decode_attention(const void* q, const void* k_codes, const void* k_absmax, const void* k_resid,
                         const void* v, const int32_t* seq_lens, int B, int Hq, int Hkv, int Lcap, int D,
                         int thumb_bits, int block_size, float delta, int n_sink, int n_local, int num_splits,
                         float softmax_scale, void* out, float* lse, uint8_t* block_mask,
                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return ffd_decode_attention_ex(q, k_codes, k_absmax, k_resid, v, seq_lens, B, Hq, Hkv, Lcap, D,
                                   thumb_bits, block_size, delta, n_sink, n_local, num_splits, softmax_scale, out,
                                   lse, block_mask, workspace, workspace_bytes, stream, nullptr);
}

int ffd_decode_attention_noalloc(const void* q, const void* k_codes, const void* k_absmax,
                                 const void* k_resid, const void* v, const int32_t* seq_lens, int B, int Hq,
                                 int Hkv, int Lcap, int D, int thumb_bits, int block_size, float delta,
                                 int n_sink, int n_local, int num_splits, float softmax_scale, void* out,
                                 float* lse, uint8_t* block_mask, hipStream_t stream) {
    int S = 0;
    const int st = decode_checks(q, k_codes, k_absmax, k_resid, v, seq_lens, B, Hq, Hkv, Lcap, D, thumb_bits,
                                 block_size, delta, n_sink, n_local, num_splits, softmax_scale, out, lse,
                                 nullptr, nullptr, false, &S);
    if (st != FFD_OK || B == 0) return st;
    if (ffd_workspace_bytes(B, Hq, Hkv, Lcap, D, num_splits) > kNoallocScratchBytes)
        return FFD_ERR_SCRATCH_TOO_SMALL;
    void* ws = device_scratch();
    if (!ws) return FFD_ERR_HIP;
    return ffd_decode_attention_ex(q, k_codes, k_absmax, k_resid, v, seq_lens, B, Hq, Hkv, Lcap, D,
                                   thumb_bits, block_size, delta, n_sink, n_local, num_splits, softmax_scale,
                                   out, lse, block_mask, ws, kNoallocScratchBytes, stream, nullptr);
}

int ffd_dense_decode_attention(const void* q, const void* k, const void* v, const int32_t* seq_lens, int B,
                               int Hq, int Hkv, int Lcap, int D, int num_splits, float softmax_scale,
                               void* out, float* lse, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
    int S = 0;
    int st = attention_common_checks(q, v, seq_lens, B, Hq, Hkv, Lcap, D, num_splits, softmax_scale, out,
                                     lse, workspace, workspace_bytes, true, &S);
    if (st != FFD_OK || B == 0) return st;
    if (!k || !aligned16(k)) return FFD_ERR_INVALID_ARGUMENT;
    if (workspace_bytes < ffd_dense_workspace_bytes(B, Hq, Hkv, Lcap, D, num_splits))
        return FFD_ERR_WORKSPACE_TOO_SMALL;
    const int G = Hq / Hkv;
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt((float)D);
    const bool balanced = B <= kDenseBalanceMaxSeqs;
    const Partials P = carve(workspace, B, Hq, balanced ? S + 1 : S);
    int2* table = balanced ? reinterpret_cast<int2*>(static_cast<uint8_t*>(workspace) +
                                                     round_up(partials_bytes(B, Hq, S + 1, D), kAlign))
                           : nullptr;
    DenseArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                static_cast<const uint16_t*>(v), seq_lens, P.m, P.l, P.acc, table, B, Hq, Hkv, Lcap, G, S, scale};
    const dim3 grid = balanced ? dim3((unsigned)((S + 1) * B * Hkv)) : dim3((unsigned)S, (unsigned)Hkv, (unsigned)B);
    if (G <= 4)
        hipLaunchKernelGGL(dense_decode_kernel<1>, grid, dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(dense_decode_kernel<2>, grid, dim3(kThreads), 0, stream, a);
    st = launch_status();
    if (st != FFD_OK) return st;
    hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)(B * Hq)), dim3(kThreads), 0, stream, P.m, P.l,
                       P.acc, S, table, balanced ? G : 1, static_cast<uint16_t*>(out), lse);
    return launch_status();
}

}  // extern "C"
