// Log-sum-exp merge of split partials (the flash-decoding reduction, Sec. 2): for each (sequence,
// query head), M* = max_s m_s, l* = sum_s e^{m_s - M*} l_s, out = sum_s e^{m_s - M*} acc_s / l*,
// lse = M* + ln l*. Splits that kept nothing carry m = -inf and are skipped; a head with no split
// gets out = 0 and lse = -inf.
//
// Partial rows of head bh = b * Hq + h: without a table, rows bh * S + s for s < S (the dense path's
// fixed splits); with a table (the FFD path), rows (first + i) * G + bh % G for i < count, where
// (first, count) = table[bh / G] describes the refinement workgroups given to that KV group.
//
// Mapping: one workgroup per (sequence, query head), running merge_partial_rows.
#include "ffd_device.h"
#include "ffd_kernels.h"

namespace ffd {

__global__ __launch_bounds__(kThreads) void lse_merge_kernel(const float* __restrict__ part_m,
                                                             const float* __restrict__ part_l,
                                                             const float* __restrict__ part_acc, int S,
                                                             const int2* __restrict__ table, int G,
                                                             uint16_t* __restrict__ out, float* __restrict__ lse) {
    size_t row0 = (size_t)blockIdx.x * S, stride = 1;      // blockIdx.x = b * Hq + h
    if (table) {
        const int2 fc = table[blockIdx.x / G];
        row0 = (size_t)fc.x * G + blockIdx.x % G;
        stride = (size_t)G;
        S = fc.y;
    }
    merge_partial_rows(part_m, part_l, part_acc, row0, stride, S, out + (size_t)blockIdx.x * kD,
                       lse ? lse + blockIdx.x : nullptr);
}

}  // namespace ffd
