// The steering sum of one 16-byte slice of a row (internal), shared by the
// steering kernel and the fused probe + steering pass so that both add in
// the same order: acc (the slice, widened to fp64) += alpha[s] * v_s for
// every set bit s of sel, ascending, one fp64 FMA per element.  The
// vectors are fetched four at a time before their adds, so the loads of a
// group are in flight together; a kernel may fetch the first group together
// with the row it adds to (steer_fetch), add it (steer_add_group) and pass
// the remaining bits to steer_accumulate.
#pragma once

#include "common.hpp"

namespace xmix {

// Up to four vectors of the steering sum, fetched before their adds: the
// next set bits of `rest` (ascending; they are cleared from it), with their
// alphas widened to fp64.
struct SteerGroup {
    uint4 v[4];
    double a[4];
    int n;
};

__device__ __forceinline__ void steer_fetch(SteerGroup& g, uint32_t& rest,
                                            const float* __restrict__ a_row,
                                            const uint4* __restrict__ V, int32_t nvec,
                                            int32_t i) {
    g.n = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        g.v[j] = make_uint4(0u, 0u, 0u, 0u);
        g.a[j] = 0.0;
        if (rest != 0) {
            const int s = __builtin_ctz(rest);
            rest &= rest - 1;
            g.a[j] = a_row[s];
            g.v[j] = V[static_cast<int64_t>(s) * nvec + i];
            g.n = j + 1;
        }
    }
}

// acc += a[j] * v_j for the group's vectors in order, one fp64 FMA per element.
template <bool BF16>
__device__ __forceinline__ void steer_add_group(double (&acc)[BF16 ? 8 : 4],
                                                const SteerGroup& g) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (j >= g.n) break;
        const uint32_t vw[4] = {g.v[j].x, g.v[j].y, g.v[j].z, g.v[j].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (BF16) {
                acc[2 * e] = fma(g.a[j], static_cast<double>(lo_bf16(vw[e])), acc[2 * e]);
                acc[2 * e + 1] = fma(g.a[j], static_cast<double>(hi_bf16(vw[e])), acc[2 * e + 1]);
            } else {
                acc[e] = fma(g.a[j], static_cast<double>(__uint_as_float(vw[e])), acc[e]);
            }
        }
    }
}

// The whole steering sum of the set bits of sel, four vectors at a time.
template <bool BF16>
__device__ __forceinline__ void steer_accumulate(double (&acc)[BF16 ? 8 : 4], uint32_t sel,
                                                 const float* __restrict__ a_row,
                                                 const uint4* __restrict__ V, int32_t nvec,
                                                 int32_t i) {
    for (uint32_t rest = sel; rest != 0;) {
        SteerGroup g;
        steer_fetch(g, rest, a_row, V, nvec, i);
        steer_add_group<BF16>(acc, g);
    }
}

}  // namespace xmix
