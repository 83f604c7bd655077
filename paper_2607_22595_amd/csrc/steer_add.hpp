// The steering sum of one 16-byte slice of a row (internal), shared by the
// steering kernel and the fused probe + steering pass so that both add in
// the same order: acc (the slice, widened to fp64) += alpha[s] * v_s for
// every set bit s of sel, ascending, one fp64 FMA per element.  The
// vectors are fetched four at a time before their adds, so the loads of a
// group are in flight together.
#pragma once

#include "common.hpp"

namespace xmix {

template <bool BF16>
__device__ __forceinline__ void steer_accumulate(double (&acc)[BF16 ? 8 : 4], uint32_t sel,
                                                 const float* __restrict__ a_row,
                                                 const uint4* __restrict__ V, int32_t nvec,
                                                 int32_t i) {
    for (uint32_t rest = sel; rest != 0;) {
        uint4 vv[4];
        double a[4];
        int n = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            vv[j] = make_uint4(0u, 0u, 0u, 0u);
            a[j] = 0.0;
            if (rest != 0) {
                const int s = __builtin_ctz(rest);
                rest &= rest - 1;
                a[j] = a_row[s];
                vv[j] = V[static_cast<int64_t>(s) * nvec + i];
                n = j + 1;
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (j >= n) break;
            const uint32_t vw[4] = {vv[j].x, vv[j].y, vv[j].z, vv[j].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if constexpr (BF16) {
                    acc[2 * e] = fma(a[j], static_cast<double>(lo_bf16(vw[e])), acc[2 * e]);
                    acc[2 * e + 1] =
                        fma(a[j], static_cast<double>(hi_bf16(vw[e])), acc[2 * e + 1]);
                } else {
                    acc[e] = fma(a[j], static_cast<double>(__uint_as_float(vw[e])), acc[e]);
                }
            }
        }
    }
}

}  // namespace xmix
