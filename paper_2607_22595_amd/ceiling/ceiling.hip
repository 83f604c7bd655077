// Measured ceilings of the device: how fast a plain stream of HBM reads and
// a stream of register-only MFMAs actually run on the GPU at hand.  These
// are measurement aids for the benchmark (they put the encode kernels'
// rates beside what the hardware reaches, next to the published peaks); no
// kernel of the hook step uses them.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "xmix_ceiling.h"

namespace {

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

constexpr int kReadThreads = 256;
constexpr int kReadUnroll = 4;        // 16-byte pieces per thread per round
constexpr int kReadBlocksPerCU = 2;
constexpr uint32_t kNever = 0x9E3779B9u;  // xor of the data is compared to it

// Grid-stride stream of nontemporal 16-byte loads: in each round the grid
// reads one contiguous span, each wave-wide load 1 KB contiguous.  The xor
// of everything read feeds a store that a real buffer never triggers, so
// the loads cannot be dropped.
__global__ void __launch_bounds__(kReadThreads)
ceiling_read_kernel(const u32x4_t* __restrict__ p, uint64_t n, uint32_t* __restrict__ sink) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kReadThreads * kReadUnroll;
    uint32_t acc = 0;
    for (uint64_t base = static_cast<uint64_t>(blockIdx.x) * kReadThreads * kReadUnroll + threadIdx.x;
         base < n; base += stride) {
        u32x4_t v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) {
            const uint64_t i = base + static_cast<uint64_t>(u) * kReadThreads;
            v[u] = i < n ? __builtin_nontemporal_load(p + i) : u32x4_t{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    if (acc == kNever) atomicOr(sink, acc);
}

// Eight independent 32x32x16 bf16 MFMA chains per wave, operands in
// registers: the matrix unit's sustained rate with nothing else to wait for.
__global__ void __launch_bounds__(256)
ceiling_mfma_kernel(int32_t iters, float* __restrict__ sink) {
    f32x16_t acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.0f;
    bf16x8_t a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = static_cast<__bf16>(static_cast<float>(threadIdx.x & 7) * 0.125f + i);
        b[i] = static_cast<__bf16>(1.0f - 0.0625f * i);
    }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[i][r];
    if (s == -1.0f) *sink = s;  // the sums are never negative
}

int cu_count() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return cus;
}

}  // namespace

extern "C" {

int xmix_ceiling_read(const void* buf, uint64_t bytes, uint32_t* sink, void* stream) {
    if (!buf || !sink || bytes == 0 || bytes % 16 != 0 ||
        reinterpret_cast<uintptr_t>(buf) % 16 != 0)
        return 1;
    const int cus = cu_count();
    if (cus <= 0) return 4;
    hipLaunchKernelGGL(ceiling_read_kernel, dim3(cus * kReadBlocksPerCU), dim3(kReadThreads), 0,
                       static_cast<hipStream_t>(stream), static_cast<const u32x4_t*>(buf),
                       bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

int xmix_ceiling_mfma(int32_t iters, float* sink, double* flops, void* stream) {
    if (!sink || iters <= 0) return 1;
    const int cus = cu_count();
    if (cus <= 0) return 4;
    hipLaunchKernelGGL(ceiling_mfma_kernel, dim3(cus), dim3(256), 0,
                       static_cast<hipStream_t>(stream), iters, sink);
    if (flops)  // 4 waves x 8 chains x iters MFMAs of 32 x 32 x 16 per workgroup
        *flops = static_cast<double>(cus) * 4.0 * 8.0 * iters * (2.0 * 32 * 32 * 16);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

}  // extern "C"
