// SAE clamp-decode: h[t] += sum_q (c_q - z_q) * W_dec[id_q] for the tokens of
// one app, fp32 accumulation and one RNE rounding.  Only the n_clamp decoder
// rows are read; the dense m x d decode is never formed.  One workgroup per
// slot of the app's token list (slots past the live count return at once).
#include <stddef.h>
#include <string.h>

#include "common.hpp"
#include "kernels.hpp"
#include "launch.hpp"

namespace xmix {

constexpr int kClampThreads = 256;
constexpr int kClampMax = 16;

__global__ void __launch_bounds__(kClampThreads)
clamp_decode_kernel(uint16_t* __restrict__ h, int32_t d, const int32_t* __restrict__ app_count,
                    const int32_t* __restrict__ tok_list, const int32_t* __restrict__ idx,
                    const uint16_t* __restrict__ val, int32_t k,
                    const uint16_t* __restrict__ W_dec, int32_t m,
                    const int32_t* __restrict__ clamp_ids, const float* __restrict__ clamp_vals,
                    int32_t n_clamp, float* __restrict__ delta_out) {
    __shared__ float coef[kClampMax];
    __shared__ int32_t cid[kClampMax];
    const int n = blockIdx.x;
    if (n >= *app_count) return;
    const int32_t t = tok_list[n];
    const int tid = threadIdx.x;
    if (tid < n_clamp) {
        const int32_t j = clamp_ids[tid];
        const bool ok = j >= 0 && j < m;  // an id outside [0, m) clamps nothing
        cid[tid] = ok ? j : 0;
        coef[tid] = ok ? clamp_vals[tid] : 0.0f;
    }
    __syncthreads();
    if (tid < k) {  // z of a clamped feature = its encoded value if selected
        const int32_t j = idx[static_cast<int64_t>(t) * k + tid];
        const float z = bf16_to_f32(val[static_cast<int64_t>(t) * k + tid]);
        for (int q = 0; q < n_clamp; ++q)
            if (j == clamp_ids[q] && j >= 0 && j < m) coef[q] = clamp_vals[q] - z;
    }
    __syncthreads();

    const int32_t nvec = d / 8;
    uint4* row = reinterpret_cast<uint4*>(h) + static_cast<int64_t>(t) * nvec;
    for (int32_t i = tid; i < nvec; i += kClampThreads) {
        float delta[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) delta[e] = 0.0f;
        for (int q = 0; q < n_clamp; ++q) {
            const float c = coef[q];
            const uint4 wv = reinterpret_cast<const uint4*>(W_dec)[static_cast<int64_t>(cid[q]) * nvec + i];
            const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                delta[2 * e] = fmaf(c, lo_bf16(ww[e]), delta[2 * e]);
                delta[2 * e + 1] = fmaf(c, hi_bf16(ww[e]), delta[2 * e + 1]);
            }
        }
        const uint4 hv = row[i];
        const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
        uint32_t out[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            out[e] = pack_bf16(lo_bf16(hw[e]) + delta[2 * e], hi_bf16(hw[e]) + delta[2 * e + 1]);
        row[i] = make_uint4(out[0], out[1], out[2], out[3]);
        if (delta_out) {
            float4* dp = reinterpret_cast<float4*>(delta_out + static_cast<int64_t>(t) * d) + 2 * i;
            dp[0] = make_float4(delta[0], delta[1], delta[2], delta[3]);
            dp[1] = make_float4(delta[4], delta[5], delta[6], delta[7]);
        }
    }
}

// Several clamp apps in one launch (the apps of one hook, in app order): one
// workgroup per token slot reads its row once, applies every app whose bit
// the token carries in the given order, each with its own fp32 delta and RNE
// rounding exactly as clamp_decode_kernel does, and writes the row once.
struct ClampApps {
    ClampAppIn a[kMultiMax];
    int32_t n;
};

__global__ void __launch_bounds__(kClampThreads)
clamp_multi_kernel(uint16_t* __restrict__ h, int32_t d, const uint32_t* __restrict__ tok_mask,
                   ClampApps apps) {
    __shared__ float coef[kMultiMax][kClampMax];
    __shared__ int32_t cid[kMultiMax][kClampMax];  // the row read for each clamp (0 if invalid)
    __shared__ int32_t rid[kMultiMax][kClampMax];  // the id a selected latent must match (-1: none)
    const int32_t t = blockIdx.x;
    const uint32_t mask = tok_mask[t];
    uint32_t sel = 0;
    for (int a = 0; a < apps.n; ++a) sel |= ((mask >> apps.a[a].bit) & 1u) << a;
    if (sel == 0) return;  // uniform
    const int tid = threadIdx.x;
    // every selected app's clamp table, the loads of all apps in flight together
#pragma unroll
    for (int a = 0; a < kMultiMax; ++a) {
        if (!((sel >> a) & 1u)) continue;
        const ClampAppIn& p = apps.a[a];
        if (tid < p.n_clamp) {
            const int32_t j = p.clamp_ids[tid];
            const bool ok = j >= 0 && j < p.m;  // an id outside [0, m) clamps nothing
            cid[a][tid] = ok ? j : 0;
            rid[a][tid] = ok ? j : -1;
            coef[a][tid] = ok ? p.clamp_vals[tid] : 0.0f;
        }
    }
    __syncthreads();
#pragma unroll
    for (int a = 0; a < kMultiMax; ++a) {
        if (!((sel >> a) & 1u)) continue;
        const ClampAppIn& p = apps.a[a];
        if (tid < p.k) {  // z of a clamped feature = its encoded value if selected
            const int32_t j = p.idx[static_cast<int64_t>(t) * p.k + tid];
            const float z = bf16_to_f32(p.val[static_cast<int64_t>(t) * p.k + tid]);
            for (int q = 0; q < p.n_clamp; ++q)
                if (j == rid[a][q]) coef[a][q] = p.clamp_vals[q] - z;
        }
    }
    __syncthreads();

    const int32_t nvec = d / 8;
    uint4* row = reinterpret_cast<uint4*>(h) + static_cast<int64_t>(t) * nvec;
    for (int32_t i = tid; i < nvec; i += kClampThreads) {
        // the deltas of every selected app first (their loads in flight
        // together), then each rounded into the row in app order
        float delta[kMultiMax][8];
#pragma unroll
        for (int a = 0; a < kMultiMax; ++a) {
#pragma unroll
            for (int e = 0; e < 8; ++e) delta[a][e] = 0.0f;
            if (!((sel >> a) & 1u)) continue;
            const ClampAppIn& p = apps.a[a];
#pragma unroll 4
            for (int q = 0; q < p.n_clamp; ++q) {
                const float c = coef[a][q];
                const uint4 wv =
                    reinterpret_cast<const uint4*>(p.W_dec)[static_cast<int64_t>(cid[a][q]) * nvec + i];
                const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    delta[a][2 * e] = fmaf(c, lo_bf16(ww[e]), delta[a][2 * e]);
                    delta[a][2 * e + 1] = fmaf(c, hi_bf16(ww[e]), delta[a][2 * e + 1]);
                }
            }
        }
        const uint4 hv = row[i];
        uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
        for (int a = 0; a < kMultiMax; ++a) {
            if (!((sel >> a) & 1u)) continue;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                hw[e] = pack_bf16(lo_bf16(hw[e]) + delta[a][2 * e],
                                  hi_bf16(hw[e]) + delta[a][2 * e + 1]);
            float* dout = apps.a[a].delta_out;
            if (dout) {
                float4* dp = reinterpret_cast<float4*>(dout + static_cast<int64_t>(t) * d) + 2 * i;
                dp[0] = make_float4(delta[a][0], delta[a][1], delta[a][2], delta[a][3]);
                dp[1] = make_float4(delta[a][4], delta[a][5], delta[a][6], delta[a][7]);
            }
        }
        row[i] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
    }
}

hipError_t launch_clamp_multi(uint16_t* h, int32_t d, int32_t T_max, const uint32_t* tok_mask,
                              int32_t n, const ClampAppIn* apps, hipStream_t stream) {
    for (int32_t c0 = 0; c0 < n; c0 += kMultiMax) {
        ClampApps ca;
        memset(&ca, 0, sizeof(ca));
        ca.n = n - c0 < kMultiMax ? n - c0 : kMultiMax;
        for (int32_t i = 0; i < ca.n; ++i) ca.a[i] = apps[c0 + i];
        hipLaunchKernelGGL(clamp_multi_kernel, dim3(T_max), dim3(kClampThreads), 0, stream, h, d,
                           tok_mask, ca);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_clamp_decode(uint16_t* h, int32_t d, const int32_t* app_count,
                               const int32_t* tok_list, int32_t T_max, const int32_t* idx,
                               const uint16_t* val, int32_t k, const uint16_t* W_dec, int32_t m,
                               const int32_t* clamp_ids, const float* clamp_vals,
                               int32_t n_clamp, float* delta_out, hipStream_t stream) {
    hipLaunchKernelGGL(clamp_decode_kernel, dim3(T_max), dim3(kClampThreads), 0, stream, h, d,
                       app_count, tok_list, idx, val, k, W_dec, m, clamp_ids, clamp_vals,
                       n_clamp, delta_out);
    return hipGetLastError();
}

// Where the batched descriptor holds device pointers (for the graph
// executor's redirection).
template <>
struct ArgPointers<ClampApps> {
    static std::vector<uint16_t> offsets() {
        std::vector<uint16_t> o;
        for (int i = 0; i < kMultiMax; ++i)
            for (const size_t f : {offsetof(ClampAppIn, idx), offsetof(ClampAppIn, val),
                                   offsetof(ClampAppIn, W_dec), offsetof(ClampAppIn, clamp_ids),
                                   offsetof(ClampAppIn, clamp_vals),
                                   offsetof(ClampAppIn, delta_out)})
                o.push_back(
                    static_cast<uint16_t>(offsetof(ClampApps, a) + i * sizeof(ClampAppIn) + f));
        return o;
    }
};

void add_clamp_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(clamp_decode_kernel));
    t.push_back(kernel_info(clamp_multi_kernel));
}

}  // namespace xmix
