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
#include "kernels.hpp"
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

// ------------------------------------------------------- conditional writes
// Narrow one app's routing entry in place to the tokens that satisfy a
// device-side condition: one workgroup walks the app's token list in chunks
// of 1024, evaluates the condition per listed token, clears the app bit of
// the tokens that fail, and compacts the survivors to the front of the list
// (ballot + wave-total scan, as in the build).  A chunk's entries are all
// read before any is written, and a survivor never moves to a later slot, so
// the compaction can run in place.
struct GateArgs {
    const float* signal;       // activation-driven: the signal
    const int32_t* req;        //   per-request index (nullable: per token)
    int32_t n_signal;          //   entries of `signal`
    int32_t signal_bit;        //   bit the token must carry (< 0: none)
    const float* threshold;    //   device scalar
    const int32_t* token_ids;  // token-driven: id per token slot
    const uint32_t* vocab_bits;  //   trigger bitmap
    int32_t vocab_size;
};

template <bool BY_TOKEN_ID>
__global__ void __launch_bounds__(kRouteThreads)
route_filter_kernel(int32_t T_max, int32_t app_bit, uint32_t* __restrict__ tok_mask,
                    int32_t* __restrict__ app_count, int32_t* __restrict__ app_tokens,
                    GateArgs g) {
    __shared__ int32_t wave_tot[kRouteWaves];
    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int32_t cnt = app_count[app_bit];
    int32_t* list = app_tokens + static_cast<int64_t>(app_bit) * T_max;
    const float thr = BY_TOKEN_ID ? 0.0f : *g.threshold;
    int32_t base = 0;
    for (int32_t c0 = 0; c0 < cnt; c0 += kRouteThreads) {
        const int32_t i = c0 + tid;
        const int32_t t = i < cnt ? list[i] : -1;
        bool keep = false;
        if (t >= 0 && t < T_max) {
            const uint32_t m = tok_mask[t];
            if constexpr (BY_TOKEN_ID) {
                const int32_t v = g.token_ids[t];
                keep = v >= 0 && v < g.vocab_size && ((g.vocab_bits[v >> 5] >> (v & 31)) & 1u);
            } else {
                keep = g.signal_bit < 0 || ((m >> g.signal_bit) & 1u);
                if (keep) {
                    const int32_t si = g.req ? g.req[t] : t;
                    keep = si >= 0 && si < g.n_signal && g.signal[si] >= thr;  // NaN fails
                }
            }
            if (!keep) tok_mask[t] = m & ~(1u << app_bit);
        }
        const uint64_t bal = wave_ballot(keep);
        if (lane_id() == 0) wave_tot[wave] = __popcll(bal);
        __syncthreads();  // also: every entry of the chunk has been read
        int32_t before = 0, total = 0;
#pragma unroll
        for (int w = 0; w < kRouteWaves; ++w) {
            const int32_t c = wave_tot[w];
            before += (w < wave) ? c : 0;
            total += c;
        }
        if (keep) list[base + before + lanes_below(bal)] = t;
        base += total;
        __syncthreads();  // wave_tot is rewritten by the next chunk
    }
    for (int32_t i = base + tid; i < cnt; i += kRouteThreads) list[i] = -1;
    if (tid == 0) app_count[app_bit] = base;
}

hipError_t launch_route_gate(int32_t T_max, int32_t app_bit, uint32_t* tok_mask,
                             int32_t* app_count, int32_t* app_tokens, const float* signal,
                             const int32_t* req, int32_t n_signal, int32_t signal_bit,
                             const float* threshold, hipStream_t stream) {
    GateArgs g{};
    g.signal = signal;
    g.req = req;
    g.n_signal = n_signal;
    g.signal_bit = signal_bit;
    g.threshold = threshold;
    hipLaunchKernelGGL(route_filter_kernel<false>, dim3(1), dim3(kRouteThreads), 0, stream, T_max,
                       app_bit, tok_mask, app_count, app_tokens, g);
    return hipGetLastError();
}

hipError_t launch_route_trigger(int32_t T_max, int32_t app_bit, uint32_t* tok_mask,
                                int32_t* app_count, int32_t* app_tokens,
                                const int32_t* token_ids, const uint32_t* vocab_bits,
                                int32_t vocab_size, hipStream_t stream) {
    GateArgs g{};
    g.token_ids = token_ids;
    g.vocab_bits = vocab_bits;
    g.vocab_size = vocab_size;
    hipLaunchKernelGGL(route_filter_kernel<true>, dim3(1), dim3(kRouteThreads), 0, stream, T_max,
                       app_bit, tok_mask, app_count, app_tokens, g);
    return hipGetLastError();
}

void add_route_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(route_build_kernel));
    t.push_back(kernel_info(route_filter_kernel<false>));
    t.push_back(kernel_info(route_filter_kernel<true>));
}

}  // namespace xmix
