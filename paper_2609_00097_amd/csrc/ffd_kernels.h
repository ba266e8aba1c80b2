// Kernel argument blocks and declarations of the library's HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ffd {

struct DecodeArgs {
    const uint16_t* q;          // bf16 [B, Hq, 128]
    const uint32_t* codes;      // [B, Hkv, Lcap/16, 64, 2]
    const uint16_t* absmax;     // bf16 [B, Hkv, Lcap]
    const int8_t* resid;        // [B, Hkv, Lcap/16, 2, 64, 16]
    const uint16_t* v;          // bf16 [B, Hkv, Lcap, 128]
    const int32_t* seq_lens;    // [B]
    float* part_m;              // [B, Hq, S]
    float* part_l;              // [B, Hq, S]
    float* part_acc;            // [B, Hq, S, 128]
    uint8_t* mask;              // [B, Hq, Lcap/64] or null
    int Hq, Hkv, Lcap, G, S;
    float delta, scale;
    int n_sink, n_local;
};

struct DenseArgs {
    const uint16_t* q;          // bf16 [B, Hq, 128]
    const uint16_t* k;          // bf16 [B, Hkv, Lcap, 128]
    const uint16_t* v;          // bf16 [B, Hkv, Lcap, 128]
    const int32_t* seq_lens;
    float* part_m;
    float* part_l;
    float* part_acc;
    int Hq, Hkv, Lcap, G, S;
    float scale;
};

struct QuantArgs {
    const uint16_t* k;          // bf16 [B, Hkv, Lcap, 128]
    uint32_t* codes;
    uint16_t* absmax;
    int8_t* resid;
    int Hkv, Lcap, t_begin, t_end;
};

template <int NT> __global__ void ffd_decode_kernel(DecodeArgs a);
template <int NT> __global__ void dense_decode_kernel(DenseArgs a);
__global__ void quantize_keys_kernel(QuantArgs a);
__global__ void lse_merge_kernel(const float* part_m, const float* part_l, const float* part_acc, int S,
                                 uint16_t* out, float* lse);

}  // namespace ffd
