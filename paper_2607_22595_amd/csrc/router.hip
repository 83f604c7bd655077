// Router-logit write for mixture-of-experts models: expert (de)activation
// on the router's logits (Table 1, App-7).  For a token with router bits,
//   logits[t,e] <- round( logits[t,e] + offsets[s1,e] + offsets[s2,e] + ... )
// over its subscribed router apps in ascending app order, added in fp64 and
// rounded once; -inf in an offset removes the expert.  The logits are a few
// KB ([T, n_experts], n_experts of 8 to a few hundred), so the kernel is
// launch-latency bound: one thread per (token slot, expert), tokens without a
// router bit leave after reading their mask word.
#include "common.hpp"
#include "kernels.hpp"
#include "launch.hpp"

namespace xmix {

constexpr int kRouterThreads = 256;

template <bool BF16>
__global__ void __launch_bounds__(kRouterThreads)
router_kernel(void* __restrict__ logits, int32_t n_experts, int32_t n_elem,
              const uint32_t* __restrict__ tok_mask, BitList bits,
              const float* __restrict__ offsets, int32_t n_router) {
    const int32_t i = blockIdx.x * kRouterThreads + threadIdx.x;
    if (i >= n_elem) return;
    const int32_t t = i / n_experts, e = i - t * n_experts;
    const uint32_t mask = tok_mask[t];
    uint32_t sel = 0;
    for (int s = 0; s < n_router; ++s) sel |= ((mask >> bits.bit[s]) & 1u) << s;
    if (sel == 0) return;
    double acc = BF16 ? static_cast<double>(bf16_to_f32(static_cast<const uint16_t*>(logits)[i]))
                      : static_cast<double>(static_cast<const float*>(logits)[i]);
    for (uint32_t rest = sel; rest; rest &= rest - 1)
        acc += static_cast<double>(offsets[__builtin_ctz(rest) * n_experts + e]);
    if constexpr (BF16) static_cast<uint16_t*>(logits)[i] = f64_to_bf16_rne(acc);
    else static_cast<float*>(logits)[i] = static_cast<float>(acc);
}

hipError_t launch_router_write(void* logits, bool bf16, int32_t n_experts, int32_t T_max,
                               const uint32_t* tok_mask, const BitList& bits,
                               const float* offsets, int32_t n_router, hipStream_t stream) {
    const int32_t n_elem = T_max * n_experts;
    const dim3 grid((n_elem + kRouterThreads - 1) / kRouterThreads);
    if (bf16)
        hipLaunchKernelGGL(router_kernel<true>, grid, dim3(kRouterThreads), 0, stream, logits,
                           n_experts, n_elem, tok_mask, bits, offsets, n_router);
    else
        hipLaunchKernelGGL(router_kernel<false>, grid, dim3(kRouterThreads), 0, stream, logits,
                           n_experts, n_elem, tok_mask, bits, offsets, n_router);
    return hipGetLastError();
}

void add_router_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(router_kernel<true>));
    t.push_back(kernel_info(router_kernel<false>));
}

}  // namespace xmix
