// Steering add: h[t] += sum over the token's steering bits of alpha * v,
// accumulated in fp64 and rounded once.  The products alpha (fp32) x v
// (bf16/fp32) are exact in fp64 and the few-term sum carries ~1e-16
// relative error, so the single rounding to the storage type is correct even
// when h and the steering terms nearly cancel (fp32 accumulation can be off
// by an ulp of the small result there).  The kernel is bound by HBM, so the
// fp64 arithmetic costs nothing measurable.  One workgroup per token slot; each
// thread owns 16-byte slices of the row, so every global access is a
// coalesced 16-byte load or store.  Rows without a steering bit return
// before touching memory beyond their mask word.
#include "common.hpp"
#include "kernels.hpp"
#include "launch.hpp"
#include "steer_add.hpp"

namespace xmix {

constexpr int kSteerThreads = 256;

template <bool BF16>
__global__ void __launch_bounds__(kSteerThreads)
steer_kernel(void* __restrict__ h, int32_t d, const uint32_t* __restrict__ tok_mask,
             const int32_t* __restrict__ req, const void* __restrict__ vecs, BitList bits,
             const float* __restrict__ alpha, int32_t n_steer) {
    const int32_t t = blockIdx.x;
    const uint32_t mask = tok_mask[t];
    uint32_t sel = 0;
    for (int s = 0; s < n_steer; ++s) sel |= ((mask >> bits.bit[s]) & 1u) << s;
    if (sel == 0) return;
    const float* a_row = alpha + static_cast<int64_t>(req[t]) * n_steer;

    constexpr int EPV = BF16 ? 8 : 4;  // elements per 16-byte vector
    const int32_t nvec = d / EPV;
    uint4* row = reinterpret_cast<uint4*>(h) + static_cast<int64_t>(t) * nvec;
    const uint4* V = reinterpret_cast<const uint4*>(vecs);
    for (int32_t i = threadIdx.x; i < nvec; i += kSteerThreads) {
        // the row and the first four vectors with their alphas, loaded
        // together (one memory round trip before the first add)
        const uint4 hv = row[i];
        uint32_t rest = sel;
        SteerGroup g0;
        steer_fetch(g0, rest, a_row, V, nvec, i);
        const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
        double acc[EPV];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (BF16) {
                acc[2 * e] = lo_bf16(hw[e]);
                acc[2 * e + 1] = hi_bf16(hw[e]);
            } else {
                acc[e] = __uint_as_float(hw[e]);
            }
        }
        steer_add_group<BF16>(acc, g0);
        if (rest) steer_accumulate<BF16>(acc, rest, a_row, V, nvec, i);
        uint4 out;
        if constexpr (BF16) {
            out.x = pack_bf16_from_f64(acc[0], acc[1]);
            out.y = pack_bf16_from_f64(acc[2], acc[3]);
            out.z = pack_bf16_from_f64(acc[4], acc[5]);
            out.w = pack_bf16_from_f64(acc[6], acc[7]);
        } else {
            out.x = __float_as_uint(static_cast<float>(acc[0]));
            out.y = __float_as_uint(static_cast<float>(acc[1]));
            out.z = __float_as_uint(static_cast<float>(acc[2]));
            out.w = __float_as_uint(static_cast<float>(acc[3]));
        }
        row[i] = out;
    }
}

hipError_t launch_steer(void* h, bool bf16, int32_t d, int32_t T_max, const uint32_t* tok_mask,
                        const int32_t* req, const void* vecs, const BitList& bits,
                        const float* alpha, int32_t n_steer, hipStream_t stream) {
    if (bf16)
        hipLaunchKernelGGL(steer_kernel<true>, dim3(T_max), dim3(kSteerThreads), 0, stream, h, d,
                           tok_mask, req, vecs, bits, alpha, n_steer);
    else
        hipLaunchKernelGGL(steer_kernel<false>, dim3(T_max), dim3(kSteerThreads), 0, stream, h,
                           d, tok_mask, req, vecs, bits, alpha, n_steer);
    return hipGetLastError();
}

void add_steer_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(steer_kernel<true>));
    t.push_back(kernel_info(steer_kernel<false>));
}

}  // namespace xmix
