// Readback compaction into a fixed-capacity device ring.  One wave per row of
// the app's token list (the list is already ascending and compact, built by
// the routing kernel's ballot/prefix pass); slot = (head + i) mod capacity.
// Every workgroup that holds a row reads head[0] before it takes a ticket
// from head[1]; the one drawing the last ticket has therefore seen every
// other read, and it alone advances head[0] and returns the ticket counter
// to zero.  Workgroups without a row take no ticket, so a step with no
// subscriber costs no atomics.
#include "common.hpp"
#include "kernels.hpp"
#include "launch.hpp"

namespace xmix {

constexpr int kCompactThreads = 256;
constexpr int kRowsPerBlock = kCompactThreads / kWave;

// Row copies move U-sized units (uint32_t when every row and segment size
// is a multiple of 4 bytes, else uint16_t, so that rows of any even size are
// written with aligned stores).
template <typename U>
__global__ void __launch_bounds__(kCompactThreads)
compact_kernel(Segments segs, const int32_t* __restrict__ app_count,
               const int32_t* __restrict__ tok_list, const int32_t* __restrict__ req,
               int32_t layer_id, int32_t app_id, uint8_t* __restrict__ slots,
               uint64_t* __restrict__ head, int32_t capacity, int32_t row_bytes) {
    __shared__ uint64_t h0_s;
    __shared__ int32_t cnt_s;
    if (threadIdx.x == 0) {
        h0_s = __atomic_load_n(&head[0], __ATOMIC_RELAXED);
        cnt_s = *app_count;
    }
    __syncthreads();
    const uint64_t h0 = h0_s;
    const int32_t cnt = cnt_s;
    const int32_t n_active = (cnt + kRowsPerBlock - 1) / kRowsPerBlock;
    if (static_cast<int32_t>(blockIdx.x) >= n_active) return;  // uniform

    constexpr int kU = static_cast<int>(sizeof(U));
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int32_t i = blockIdx.x * kRowsPerBlock + wave;
    // rows older than the last `capacity` of this call would be overwritten
    if (i < cnt && static_cast<int64_t>(i) >= static_cast<int64_t>(cnt) - capacity) {
        const int32_t t = tok_list[i];
        U* dst = reinterpret_cast<U*>(
            slots + static_cast<int64_t>((h0 + static_cast<uint64_t>(i)) % static_cast<uint64_t>(capacity)) * row_bytes);
        // header {token, request, layer, app}: 16 bytes in 16 / kU units
        if (lane < 16 / kU) {
            const int f = lane * kU / 4;
            const int32_t hdr = f == 0 ? t : f == 1 ? req[t] : f == 2 ? layer_id : app_id;
            const uint32_t hv = static_cast<uint32_t>(hdr);
            dst[lane] = static_cast<U>(kU == 4 ? hv : (lane & 1) ? (hv >> 16) : (hv & 0xFFFFu));
        }
        int32_t off = 16 / kU;
        for (int s = 0; s < segs.n; ++s) {
            const int32_t nu = segs.bytes[s] / kU;
            const U* src = reinterpret_cast<const U*>(segs.ptr[s]) + static_cast<int64_t>(t) * nu;
            for (int32_t w = lane; w < nu; w += kWave) dst[off + w] = src[w];
            off += nu;
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        // no fence: the rows and the head are read by work ordered after the
        // kernel, which its completion makes visible
        const uint64_t ticket = atomicAdd(reinterpret_cast<unsigned long long*>(&head[1]), 1ull);
        if (ticket == static_cast<uint64_t>(n_active) - 1u) {
            __atomic_store_n(&head[0], h0 + static_cast<uint64_t>(cnt), __ATOMIC_RELAXED);
            atomicExch(reinterpret_cast<unsigned long long*>(&head[1]), 0ull);
        }
    }
}

hipError_t launch_compact(const Segments& segs, const int32_t* app_count,
                          const int32_t* tok_list, int32_t T_max, const int32_t* req,
                          int32_t layer_id, int32_t app_id, uint8_t* slots, uint64_t* head,
                          int32_t capacity, int32_t row_bytes, hipStream_t stream) {
    const int blocks = (T_max + kRowsPerBlock - 1) / kRowsPerBlock;
    bool words = row_bytes % 4 == 0;
    for (int s = 0; s < segs.n; ++s)
        words = words && segs.bytes[s] % 4 == 0 &&
                (reinterpret_cast<uintptr_t>(segs.ptr[s]) & 3u) == 0;
    if (words)
        hipLaunchKernelGGL(compact_kernel<uint32_t>, dim3(blocks), dim3(kCompactThreads), 0,
                           stream, segs, app_count, tok_list, req, layer_id, app_id, slots,
                           head, capacity, row_bytes);
    else
        hipLaunchKernelGGL(compact_kernel<uint16_t>, dim3(blocks), dim3(kCompactThreads), 0,
                           stream, segs, app_count, tok_list, req, layer_id, app_id, slots,
                           head, capacity, row_bytes);
    return hipGetLastError();
}

void add_compact_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(compact_kernel<uint32_t>));
    t.push_back(kernel_info(compact_kernel<uint16_t>));
}

}  // namespace xmix
