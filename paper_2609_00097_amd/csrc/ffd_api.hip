// C ABI of the FFD decode-attention library: argument checks, split choice, kernel launches.
#include <cmath>
#include <cstdint>

#include "ffd.h"
#include "ffd_device.h"
#include "ffd_kernels.h"

using namespace ffd;

namespace {

constexpr int kTargetWorkgroups = 2048;   // ~8 per CU on 256 CUs
constexpr int kMinBlocksPerSplit = 8;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int resolve_splits(int B, int Hkv, int Lcap, int num_splits) {
    if (B <= 0 || Hkv <= 0 || Lcap <= 0 || num_splits < 0 || num_splits > FFD_MAX_SPLITS) return 0;
    if (num_splits > 0) return num_splits;
    const long long pairs = (long long)B * Hkv;
    long long s = (kTargetWorkgroups + pairs - 1) / pairs;
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

int launch_status() {
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? FFD_OK : FFD_ERR_HIP;
}

// Workspace: split partials m [B,Hq,S], l [B,Hq,S], acc [B,Hq,S,D] (fp32).
struct Partials {
    float* m;
    float* l;
    float* acc;
};

size_t partials_bytes(int B, int Hq, int S, int D) { return (size_t)B * Hq * S * (D + 2) * sizeof(float); }

Partials carve(void* ws, int B, int Hq, int S) {
    const size_t rows = (size_t)B * Hq * S;
    float* base = static_cast<float*>(ws);
    return Partials{base, base + rows, base + 2 * rows};
}

int attention_common_checks(const void* q, const void* v, const int32_t* seq_lens, int B, int Hq,
                            int Hkv, int Lcap, int D, int num_splits, float softmax_scale,
                            const void* out, const float* lse, const void* ws, size_t ws_bytes,
                            int* S_out) {
    int st = check_shapes(B, Hq, Hkv, Lcap, D);
    if (st != FFD_OK) return st;
    if (num_splits < 0 || num_splits > FFD_MAX_SPLITS) return FFD_ERR_INVALID_ARGUMENT;
    if (!(softmax_scale >= 0.f) || std::isinf(softmax_scale)) return FFD_ERR_INVALID_ARGUMENT;
    if (B == 0) { *S_out = 0; return FFD_OK; }
    if (!q || !v || !seq_lens || !out || !ws) return FFD_ERR_INVALID_ARGUMENT;
    if (!aligned16(q) || !aligned16(v) || !aligned16(out) || !aligned16(ws)) return FFD_ERR_INVALID_ARGUMENT;
    if ((reinterpret_cast<uintptr_t>(seq_lens) & 3u) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)))
        return FFD_ERR_INVALID_ARGUMENT;
    const int S = resolve_splits(B, Hkv, Lcap, num_splits);
    if (S <= 0) return FFD_ERR_INVALID_ARGUMENT;
    if (ws_bytes < ffd_workspace_bytes(B, Hq, Hkv, Lcap, D, num_splits)) return FFD_ERR_WORKSPACE_TOO_SMALL;
    *S_out = S;
    return FFD_OK;
}

}  // namespace

extern "C" {

int ffd_resolve_splits(int B, int Hkv, int Lcap, int num_splits) {
    return resolve_splits(B, Hkv, Lcap, num_splits);
}

size_t ffd_workspace_bytes(int B, int Hq, int Hkv, int Lcap, int D, int num_splits) {
    if (check_shapes(B, Hq, Hkv, Lcap, D) != FFD_OK) return 0;
    const int S = resolve_splits(B > 0 ? B : 1, Hkv, Lcap, num_splits);
    if (S <= 0) return 0;
    return partials_bytes(B, Hq, S, D);
}

const char* ffd_status_string(int status) {
    switch (status) {
        case FFD_OK: return "FFD_OK";
        case FFD_ERR_INVALID_ARGUMENT: return "FFD_ERR_INVALID_ARGUMENT";
        case FFD_ERR_UNSUPPORTED: return "FFD_ERR_UNSUPPORTED";
        case FFD_ERR_WORKSPACE_TOO_SMALL: return "FFD_ERR_WORKSPACE_TOO_SMALL";
        case FFD_ERR_HIP: return "FFD_ERR_HIP";
        default: return "FFD_ERR_UNKNOWN";
    }
}

int ffd_quantize_keys(const void* k, void* k_codes, void* k_absmax, void* k_resid, int B, int Hkv,
                      int Lcap, int D, int t_begin, int t_end, hipStream_t stream) {
    int st = check_shapes(B, Hkv, Hkv, Lcap, D);
    if (st != FFD_OK) return st;
    if (t_begin < 0 || t_end < t_begin || t_end > Lcap) return FFD_ERR_INVALID_ARGUMENT;
    if (B == 0 || t_end == t_begin) return FFD_OK;
    if (!k || !k_codes || !k_absmax || !k_resid) return FFD_ERR_INVALID_ARGUMENT;
    if (!aligned16(k) || !aligned16(k_codes) || !aligned16(k_absmax) || !aligned16(k_resid))
        return FFD_ERR_INVALID_ARGUMENT;
    QuantArgs a{static_cast<const uint16_t*>(k), static_cast<uint32_t*>(k_codes),
                static_cast<uint16_t*>(k_absmax), static_cast<int8_t*>(k_resid), Hkv, Lcap, t_begin, t_end};
    const dim3 grid((unsigned)((t_end - t_begin + 15) / 16), (unsigned)Hkv, (unsigned)B);
    hipLaunchKernelGGL(quantize_keys_kernel, grid, dim3(kThreads), 0, stream, a);
    return launch_status();
}

int ffd_decode_attention(const void* q, const void* k_codes, const void* k_absmax, const void* k_resid,
                         const void* v, const int32_t* seq_lens, int B, int Hq, int Hkv, int Lcap, int D,
                         int block_size, float delta, int n_sink, int n_local, int num_splits,
                         float softmax_scale, void* out, float* lse, uint8_t* block_mask,
                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (block_size != FFD_BLOCK) return block_size > 0 ? FFD_ERR_UNSUPPORTED : FFD_ERR_INVALID_ARGUMENT;
    if (std::isnan(delta) || delta < 0.f || n_sink < 0 || n_local < 0) return FFD_ERR_INVALID_ARGUMENT;
    int S = 0;
    int st = attention_common_checks(q, v, seq_lens, B, Hq, Hkv, Lcap, D, num_splits, softmax_scale, out,
                                     lse, workspace, workspace_bytes, &S);
    if (st != FFD_OK || B == 0) return st;
    if (!k_codes || !k_absmax || !k_resid) return FFD_ERR_INVALID_ARGUMENT;
    if (!aligned16(k_codes) || !aligned16(k_absmax) || !aligned16(k_resid)) return FFD_ERR_INVALID_ARGUMENT;
    const int G = Hq / Hkv;
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt((float)D);
    const Partials P = carve(workspace, B, Hq, S);
    DecodeArgs a{static_cast<const uint16_t*>(q), static_cast<const uint32_t*>(k_codes),
                 static_cast<const uint16_t*>(k_absmax), static_cast<const int8_t*>(k_resid),
                 static_cast<const uint16_t*>(v), seq_lens, P.m, P.l, P.acc, block_mask, Hq, Hkv,
                 Lcap, G, S, delta, scale, n_sink, n_local};
    const dim3 grid((unsigned)S, (unsigned)Hkv, (unsigned)B);
    if (G <= 4)
        hipLaunchKernelGGL(ffd_decode_kernel<1>, grid, dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(ffd_decode_kernel<2>, grid, dim3(kThreads), 0, stream, a);
    st = launch_status();
    if (st != FFD_OK) return st;
    hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)(B * Hq)), dim3(kThreads), 0, stream, P.m, P.l,
                       P.acc, S, static_cast<uint16_t*>(out), lse);
    return launch_status();
}

int ffd_dense_decode_attention(const void* q, const void* k, const void* v, const int32_t* seq_lens, int B,
                               int Hq, int Hkv, int Lcap, int D, int num_splits, float softmax_scale,
                               void* out, float* lse, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
    int S = 0;
    int st = attention_common_checks(q, v, seq_lens, B, Hq, Hkv, Lcap, D, num_splits, softmax_scale, out,
                                     lse, workspace, workspace_bytes, &S);
    if (st != FFD_OK || B == 0) return st;
    if (!k || !aligned16(k)) return FFD_ERR_INVALID_ARGUMENT;
    const int G = Hq / Hkv;
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt((float)D);
    const Partials P = carve(workspace, B, Hq, S);
    DenseArgs a{static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                static_cast<const uint16_t*>(v), seq_lens, P.m, P.l, P.acc, Hq, Hkv, Lcap, G, S, scale};
    const dim3 grid((unsigned)S, (unsigned)Hkv, (unsigned)B);
    if (G <= 4)
        hipLaunchKernelGGL(dense_decode_kernel<1>, grid, dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(dense_decode_kernel<2>, grid, dim3(kThreads), 0, stream, a);
    st = launch_status();
    if (st != FFD_OK) return st;
    hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)(B * Hq)), dim3(kThreads), 0, stream, P.m, P.l,
                       P.acc, S, static_cast<uint16_t*>(out), lse);
    return launch_status();
}

}  // extern "C"
