// Linear probes: per-token logit/sigmoid, and mean-pooled per request.
//
// Token pass: one workgroup per token slot reads the row once in 16-byte
// slices and accumulates one partial dot product per subscribed probe in
// registers; partials are reduced with fixed DPP moves inside each wave
// and a fixed-order sum over the waves (bit-reproducible, no atomics).
//
// Mean pooling is a segmented reduction in two launches: the token pass
// writes each token's dot products (without bias) to the workspace, then one
// workgroup per request sums its contiguous span in a fixed order.  Whether
// a request is pooled is decided at the first token of its span, so in this
// mode the token pass finds each token's span and takes the subscription of
// the span's first token: every token of a pooled span gets its dots, also
// where its own mask lacks the bit (a conditional filter narrowed it, or the
// span runs past T_valid).
//
// Last-token mode runs the token pass with one workgroup per request on the
// last token of its span, writing [n_probe][R_max].
#include "common.hpp"
#include "kernels.hpp"
#include "launch.hpp"

namespace xmix {

constexpr int kProbeThreads = 512;  // the fused probe + steering pass slices rows the same way
constexpr int kProbeWaves = kProbeThreads / kWave;

// The request whose span [cu[r], cu[r+1]) holds token t, or -1: with cu
// non-decreasing, r + 1 is the number of entries cu[0..R] that are <= t.
// Called by every thread of the workgroup (the count is a barrier).
__device__ __forceinline__ int32_t span_of_token(const int32_t* __restrict__ cu, int32_t R,
                                                 int32_t t) {
    int c = 0;
    for (int32_t i0 = 0; i0 <= R; i0 += kProbeThreads) {
        const int32_t i = i0 + static_cast<int32_t>(threadIdx.x);
        c += __syncthreads_count(i <= R && cu[i] <= t);
    }
    const int32_t r = c - 1;
    if (r < 0 || r >= R) return -1;
    return t < cu[r + 1] ? r : -1;
}

template <bool BF16, int MAXP>
__global__ void __launch_bounds__(kProbeThreads)
probe_token_kernel(const void* __restrict__ h, int32_t d, int32_t T_max,
                   const uint32_t* __restrict__ tok_mask, const void* __restrict__ w,
                   const float* __restrict__ b, BitList bits, int32_t n_probe,
                   const int32_t* __restrict__ cu, int32_t R, int32_t mode,
                   float* __restrict__ logit, float* __restrict__ score,
                   float* __restrict__ dots) {
    __shared__ float red[kProbeWaves][MAXP];
    // token mode: slot = token; last-token mode: slot = request, reading the
    // last token of its span (subscription of its first token); mean mode:
    // slot = token, subscription of the first token of its span
    int32_t t = blockIdx.x;
    int32_t out_len = T_max;
    uint32_t mask;
    if (mode == 2) {
        const int32_t lo = cu[blockIdx.x], hi = cu[blockIdx.x + 1];
        if (hi <= lo || lo < 0 || hi > T_max) return;
        t = hi - 1;
        mask = tok_mask[lo];
        out_len = static_cast<int32_t>(gridDim.x);
    } else if (mode == 1) {
        const int32_t r = span_of_token(cu, R, t);
        if (r < 0) return;
        const int32_t lo = cu[r], hi = cu[r + 1];
        if (lo < 0 || hi > T_max) return;  // the pooling skips such a span too
        mask = tok_mask[lo];
    } else {
        mask = tok_mask[t];
    }
    uint32_t sel = 0;
    for (int p = 0; p < n_probe; ++p) sel |= ((mask >> bits.bit[p]) & 1u) << p;
    if (sel == 0) return;

    constexpr int EPV = BF16 ? 8 : 4;
    const int32_t nvec = d / EPV;
    const uint4* row = reinterpret_cast<const uint4*>(h) + static_cast<int64_t>(t) * nvec;
    const uint4* W = reinterpret_cast<const uint4*>(w);
    float part[MAXP];
#pragma unroll
    for (int p = 0; p < MAXP; ++p) part[p] = 0.0f;

    // weights fetched together with the row (the rest, for more than eight
    // probes, when used)
    constexpr int AP = MAXP < 8 ? MAXP : 8;
    for (int32_t i = threadIdx.x; i < nvec; i += kProbeThreads) {
        // the row and the weights of the token's probes, all loaded before the
        // first use, so that the slice waits for one memory round trip
        const uint4 hv = row[i];
        uint4 wv[AP];
#pragma unroll
        for (int p = 0; p < AP; ++p)
            wv[p] = ((sel >> p) & 1u) ? W[static_cast<int64_t>(p) * nvec + i]
                                      : make_uint4(0u, 0u, 0u, 0u);
        const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
        float x[EPV];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (BF16) {
                x[2 * e] = lo_bf16(hw[e]);
                x[2 * e + 1] = hi_bf16(hw[e]);
            } else {
                x[e] = __uint_as_float(hw[e]);
            }
        }
#pragma unroll
        for (int p = 0; p < MAXP; ++p) {
            if (!((sel >> p) & 1u)) continue;
            const uint4 w4 = p < AP ? wv[p < AP ? p : 0] : W[static_cast<int64_t>(p) * nvec + i];
            const uint32_t ww[4] = {w4.x, w4.y, w4.z, w4.w};
            float acc = part[p];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if constexpr (BF16) {
                    acc = fmaf(lo_bf16(ww[e]), x[2 * e], acc);
                    acc = fmaf(hi_bf16(ww[e]), x[2 * e + 1], acc);
                } else {
                    acc = fmaf(__uint_as_float(ww[e]), x[e], acc);
                }
            }
            part[p] = acc;
        }
    }

    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int p = 0; p < MAXP; ++p) {
        if (!((sel >> p) & 1u)) continue;
        const float s = wave_sum(part[p]);
        if (lane_id() == 0) red[wave][p] = s;
    }
    __syncthreads();
    const int p = threadIdx.x;
    if (p < n_probe && ((sel >> p) & 1u)) {
        float dot = 0.0f;
#pragma unroll
        for (int wv = 0; wv < kProbeWaves; ++wv) dot += red[wv][p];
        const int64_t o = static_cast<int64_t>(p) * out_len + blockIdx.x;
        if (dots) {
            dots[o] = dot;
        } else {
            const float l = b[p] + dot;
            logit[o] = l;
            score[o] = logistic(l);
        }
    }
}

// One workgroup per request: pooled logit of every probe whose bit the
// request carries.  Threads sum strided tokens of the span in order, then a
// fixed DPP pattern and a fixed-order sum over the waves combine them.
__global__ void __launch_bounds__(kProbeThreads)
probe_pool_kernel(const float* __restrict__ dots, int32_t T_max,
                  const uint32_t* __restrict__ tok_mask, const int32_t* __restrict__ cu,
                  const float* __restrict__ b, BitList bits, int32_t n_probe, int32_t R_max,
                  float* __restrict__ logit, float* __restrict__ score) {
    __shared__ float red[kProbeWaves];
    const int32_t r = blockIdx.x;
    const int32_t lo = cu[r], hi = cu[r + 1];
    if (hi <= lo || lo < 0 || hi > T_max) return;
    const uint32_t mask = tok_mask[lo];
    const int wave = threadIdx.x / kWave;
    for (int p = 0; p < n_probe; ++p) {
        if (!((mask >> bits.bit[p]) & 1u)) continue;  // uniform over the block
        const float* dp = dots + static_cast<int64_t>(p) * T_max;
        float s = 0.0f;
        for (int32_t t = lo + threadIdx.x; t < hi; t += kProbeThreads) s += dp[t];
        s = wave_sum(s);
        if (lane_id() == 0) red[wave] = s;
        __syncthreads();
        if (threadIdx.x == 0) {
            float tot = 0.0f;
#pragma unroll
            for (int wv = 0; wv < kProbeWaves; ++wv) tot += red[wv];
            const float l = b[p] + tot / static_cast<float>(hi - lo);
            const int64_t o = static_cast<int64_t>(p) * R_max + r;
            logit[o] = l;
            score[o] = logistic(l);
        }
        __syncthreads();
    }
}

template <bool BF16>
static hipError_t launch_probe_t(const void* h, int32_t d, int32_t T_max,
                                 const uint32_t* tok_mask, const void* w, const float* b,
                                 const BitList& bits, int32_t n_probe, const int32_t* cu,
                                 int32_t R, int32_t mode, int32_t slots, float* logit,
                                 float* score, float* dots, hipStream_t stream) {
    dim3 g(slots), blk(kProbeThreads);
    if (n_probe <= 4)
        hipLaunchKernelGGL((probe_token_kernel<BF16, 4>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, w, b, bits, n_probe, cu, R, mode, logit, score, dots);
    else if (n_probe <= 8)
        hipLaunchKernelGGL((probe_token_kernel<BF16, 8>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, w, b, bits, n_probe, cu, R, mode, logit, score, dots);
    else if (n_probe <= 16)
        hipLaunchKernelGGL((probe_token_kernel<BF16, 16>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, w, b, bits, n_probe, cu, R, mode, logit, score, dots);
    else
        hipLaunchKernelGGL((probe_token_kernel<BF16, 32>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, w, b, bits, n_probe, cu, R, mode, logit, score, dots);
    return hipGetLastError();
}

hipError_t launch_probe(const void* h, bool bf16, int32_t d, int32_t T_max,
                        const uint32_t* tok_mask, const void* w, const float* b,
                        const BitList& bits, int32_t n_probe, int32_t mode,
                        const int32_t* cu_seqlens, int32_t R_max, float* logit, float* score,
                        float* ws, hipStream_t stream) {
    float* dots = mode == 1 ? ws : nullptr;
    const int32_t* cu = mode == 0 ? nullptr : cu_seqlens;
    const int32_t slots = mode == 2 ? R_max : T_max;
    hipError_t e = bf16 ? launch_probe_t<true>(h, d, T_max, tok_mask, w, b, bits, n_probe, cu,
                                               R_max, mode, slots, logit, score, dots, stream)
                        : launch_probe_t<false>(h, d, T_max, tok_mask, w, b, bits, n_probe, cu,
                                                R_max, mode, slots, logit, score, dots, stream);
    if (e != hipSuccess || mode != 1) return e;
    hipLaunchKernelGGL(probe_pool_kernel, dim3(R_max), dim3(kProbeThreads), 0, stream, ws, T_max,
                       tok_mask, cu_seqlens, b, bits, n_probe, R_max, logit, score);
    return hipGetLastError();
}

void add_probe_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(probe_token_kernel<true, 4>));
    t.push_back(kernel_info(probe_token_kernel<true, 8>));
    t.push_back(kernel_info(probe_token_kernel<true, 16>));
    t.push_back(kernel_info(probe_token_kernel<true, 32>));
    t.push_back(kernel_info(probe_token_kernel<false, 4>));
    t.push_back(kernel_info(probe_token_kernel<false, 8>));
    t.push_back(kernel_info(probe_token_kernel<false, 16>));
    t.push_back(kernel_info(probe_token_kernel<false, 32>));
    t.push_back(kernel_info(probe_pool_kernel));
}

}  // namespace xmix
