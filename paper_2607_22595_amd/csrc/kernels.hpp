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
    const void* func;                           // the address hipLaunchKernelGGL records
    std::vector<uint16_t> size;                 // bytes of each argument, in order
    std::vector<std::vector<uint16_t>> ptr_at;  // device pointers inside each argument
};

// Byte offsets of the device pointers inside an argument of type T: the
// argument itself when it is a pointer, none otherwise.  A struct passed by
// value that holds pointers (the batched calls' app descriptors) lists them
// in a specialization beside its definition, before its kernels' table.
template <typename T>
struct ArgPointers {
    static std::vector<uint16_t> offsets() {
        return std::is_pointer<T>::value ? std::vector<uint16_t>{0} : std::vector<uint16_t>{};
    }
};

// Top-level qualifiers (const, __restrict__) are not part of a function
// type, so A... are the plain parameter types.
template <typename... A>
KernelInfo kernel_info(void (*f)(A...)) {
    return KernelInfo{reinterpret_cast<const void*>(f),
                      {static_cast<uint16_t>(sizeof(A))...},
                      {ArgPointers<A>::offsets()...}};
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
