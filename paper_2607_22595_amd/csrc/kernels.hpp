// Argument layout of the library's kernels, read off their signatures, so
// that the graph executor can decode and rewrite the arguments of captured
// kernel nodes (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <vector>

namespace xmix {

struct KernelInfo {
    const void* func;             // the address hipLaunchKernelGGL records
    std::vector<uint16_t> size;   // bytes of each argument, in order
    std::vector<uint8_t> is_ptr;  // 1 for a pointer argument
};

// Top-level qualifiers (const, __restrict__) are not part of a function
// type, so A... are the plain parameter types.
template <typename... A>
KernelInfo kernel_info(void (*f)(A...)) {
    return KernelInfo{reinterpret_cast<const void*>(f),
                      {static_cast<uint16_t>(sizeof(A))...},
                      {static_cast<uint8_t>(std::is_pointer<A>::value)...}};
}

// One per kernel source: appends the kernels that file launches.
void add_route_kernels(std::vector<KernelInfo>& t);
void add_steer_kernels(std::vector<KernelInfo>& t);
void add_steer_probe_kernels(std::vector<KernelInfo>& t);
void add_probe_kernels(std::vector<KernelInfo>& t);
void add_router_kernels(std::vector<KernelInfo>& t);
void add_sae_kernels(std::vector<KernelInfo>& t);
void add_clamp_kernels(std::vector<KernelInfo>& t);
void add_compact_kernels(std::vector<KernelInfo>& t);

}  // namespace xmix
