// Routing table: token -> request -> app bitmask, plus one ascending token
// list per app (per-request toggling inside one continuous batch).
//
// One workgroup per app walks the token slots in chunks of 1024.  Inside a
// chunk each wave turns "token has bit a" into a 64-bit ballot; a lane's
// place in the list is the popcount of the ballot below it (mbcnt) plus the
// totals of the waves before it (an exclusive scan over 16 wave counts in
// LDS) plus the running total of earlier chunks.  Workgroup 0 also writes
// the token masks and the error word.
#include "common.hpp"
#include "launch.hpp"

namespace xmix {

constexpr int kRouteThreads = 1024;
constexpr int kRouteWaves = kRouteThreads / kWave;

__global__ void __launch_bounds__(kRouteThreads)
route_build_kernel(const int32_t* __restrict__ req, const int32_t* __restrict__ T_valid_p,
                   const uint32_t* __restrict__ sub, int32_t R_max, int32_t T_max,
                   int32_t n_apps, uint32_t* __restrict__ tok_mask,
                   int32_t* __restrict__ app_count, int32_t* __restrict__ app_tokens,
                   uint32_t* __restrict__ err_word) {
    __shared__ int32_t wave_tot[kRouteWaves];
    const int a = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const uint32_t keep = n_apps >= 32 ? 0xFFFFFFFFu : ((1u << n_apps) - 1u);

    int32_t tv = *T_valid_p;
    uint32_t err = 0;
    if (tv < 0 || tv > T_max) {
        err |= 2u;
        tv = tv < 0 ? 0 : T_max;
    }

    int32_t* list = app_tokens + static_cast<int64_t>(a) * T_max;
    int32_t base = 0;
    for (int32_t c0 = 0; c0 < T_max; c0 += kRouteThreads) {
        const int32_t t = c0 + tid;
        uint32_t mask = 0;
        if (t < tv) {
            const int32_t r = req[t];
            if (r >= R_max) err |= 1u;
            else if (r >= 0) mask = sub[r] & keep;
        }
        if (a == 0 && t < T_max) tok_mask[t] = mask;

        const bool has = (mask >> a) & 1u;
        const uint64_t bal = wave_ballot(has);
        if (lane_id() == 0) wave_tot[wave] = __popcll(bal);
        __syncthreads();
        int32_t before = 0, total = 0;
#pragma unroll
        for (int w = 0; w < kRouteWaves; ++w) {
            const int32_t c = wave_tot[w];
            before += (w < wave) ? c : 0;
            total += c;
        }
        if (has) list[base + before + lanes_below(bal)] = t;
        base += total;
        __syncthreads();  // wave_tot is rewritten by the next chunk
    }
    for (int32_t i = base + tid; i < T_max; i += kRouteThreads) list[i] = -1;
    if (tid == 0) app_count[a] = base;

    if (a == 0) {  // uniform over the workgroup: every lane takes part
        uint32_t e = err;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) e |= __shfl_xor(e, off, kWave);
        if (lane_id() == 0 && e != 0) atomicOr(err_word, e);
    }
}

hipError_t launch_route_build(const int32_t* req, const int32_t* T_valid, const uint32_t* sub,
                              int32_t R_max, int32_t T_max, int32_t n_apps, uint32_t* tok_mask,
                              int32_t* app_count, int32_t* app_tokens, uint32_t* err_word,
                              hipStream_t stream) {
    hipLaunchKernelGGL(route_build_kernel, dim3(n_apps), dim3(kRouteThreads), 0, stream, req,
                       T_valid, sub, R_max, T_max, n_apps, tok_mask, app_count, app_tokens,
                       err_word);
    return hipGetLastError();
}

}  // namespace xmix
