// SAE clamp-decode: h[t] += sum_q (c_q - z_q) * W_dec[id_q] for the tokens of
// one app, fp32 accumulation and one RNE rounding.  Only the n_clamp decoder
// rows are read; the dense m x d decode is never formed.  One workgroup per
// slot of the app's token list (slots past the live count return at once).
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

void add_clamp_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(clamp_decode_kernel));
}

}  // namespace xmix
