// In-kernel route build for a kernel that takes the place of the route-build
// launch (internal).  The rules are the route-build kernel's: T_valid is
// clamped to [0, T_max] (error value XMIX_ERR_T_VALID = 2); a request id >=
// R_max routes nowhere (XMIX_ERR_REQUEST_RANGE = 1); a negative id is
// padding.
#pragma once

#include "common.hpp"

namespace xmix {

constexpr int kRouteMaxT = 1024;    // most token slots a kernel routes itself
constexpr int kStageSubMax = 2048;  // most request-table entries staged in LDS

// T_valid clamped to [0, T_max]; XMIX_ERR_T_VALID (2) when it was outside.
__device__ __forceinline__ int32_t clamp_t_valid(int32_t tv, int32_t T_max, uint32_t& err) {
    if (tv < 0 || tv > T_max) {
        err |= 2u;
        tv = tv < 0 ? 0 : T_max;
    }
    return tv;
}

// The mask of token slot t, whose request id r the caller loaded (0 past
// T_valid, or for a bad id with XMIX_ERR_REQUEST_RANGE (1)).  The table
// entry is fetched without waiting for T_valid.
__device__ __forceinline__ uint32_t request_mask(int32_t r, int32_t t, int32_t tv,
                                                 const uint32_t* __restrict__ sub,
                                                 int32_t R_max, uint32_t keep, uint32_t& err) {
    const bool in_range = r >= 0 && r < R_max;
    const uint32_t m = in_range ? sub[r] : 0u;
    if (t >= tv) return 0u;
    if (r >= R_max) err |= 1u;
    return m & keep;
}

// The routing inputs staged in LDS for the list builds below: req[0, T_max)
// into req_s (T_max <= kRouteMaxT) and, when R_max <= kStageSubMax, the
// request table into sub_s; every global load is issued before the first
// wait, so the staging costs one memory round trip.  The caller places a
// barrier between this and the first build.  Returns whether a request this
// thread staged subscribes to an app of `bits` (true when the table was too
// large to stage): no token can carry those bits unless some thread saw one.
template <int THREADS>
__device__ __forceinline__ bool stage_route(const int32_t* __restrict__ req, int32_t T_max,
                                            const uint32_t* __restrict__ sub, int32_t R_max,
                                            int32_t* req_s, uint32_t* sub_s,
                                            uint32_t bits = 0u) {
    constexpr int kT = (kRouteMaxT + THREADS - 1) / THREADS;
    constexpr int kR = (kStageSubMax + THREADS - 1) / THREADS;
    const int tid = threadIdx.x;
    const bool fits = R_max <= kStageSubMax;
    int32_t rv[kT];
    uint32_t sv[kR];
#pragma unroll
    for (int j = 0; j < kT; ++j) {
        const int32_t i = tid + j * THREADS;
        rv[j] = i < T_max ? req[i] : -1;
    }
#pragma unroll
    for (int j = 0; j < kR; ++j) {
        const int32_t i = tid + j * THREADS;
        sv[j] = (fits && i < R_max) ? sub[i] : 0u;
    }
#pragma unroll
    for (int j = 0; j < kT; ++j)
        if (tid + j * THREADS < T_max) req_s[tid + j * THREADS] = rv[j];
    bool seen = !fits;
#pragma unroll
    for (int j = 0; j < kR; ++j) {
        if (fits && tid + j * THREADS < R_max) sub_s[tid + j * THREADS] = sv[j];
        seen = seen || (sv[j] & bits) != 0u;
    }
    return seen;
}

// slot_mask on the staged inputs (the request table from global memory when
// it was too large to stage).
__device__ __forceinline__ uint32_t slot_mask_staged(const int32_t* req_s, int32_t t, int32_t tv,
                                                     const uint32_t* sub_s,
                                                     const uint32_t* __restrict__ sub,
                                                     int32_t R_max, uint32_t keep,
                                                     uint32_t& err) {
    if (t >= tv) return 0u;
    const int32_t r = req_s[t];
    if (r >= R_max) {
        err |= 1u;
        return 0u;
    }
    if (r < 0) return 0u;
    return (R_max <= kStageSubMax ? sub_s[r] : sub[r]) & keep;
}

// The ascending list of the token slots that carry `bit`, into list_s (LDS),
// by a workgroup of THREADS threads from the staged inputs; returns its
// length.  `mask_out`, if given, receives every slot's mask.  Every thread
// takes part (two barriers per THREADS slots); wtot holds THREADS / 64 ints
// of LDS.
template <int THREADS>
__device__ int32_t build_token_list(const int32_t* req_s, int32_t tv, const uint32_t* sub_s,
                                    const uint32_t* __restrict__ sub, int32_t R_max,
                                    uint32_t keep, int bit, int32_t T_max, int32_t* list_s,
                                    int32_t* wtot, uint32_t* __restrict__ mask_out,
                                    uint32_t& err) {
    constexpr int kWaves = THREADS / kWave;
    const int tid = threadIdx.x, wave = tid / kWave;
    int32_t base = 0;
    for (int32_t c0 = 0; c0 < T_max; c0 += THREADS) {
        const int32_t t = c0 + tid;
        const uint32_t mask =
            t < T_max ? slot_mask_staged(req_s, t, tv, sub_s, sub, R_max, keep, err) : 0u;
        if (mask_out && t < T_max) mask_out[t] = mask;
        const bool has = (mask >> bit) & 1u;
        const uint64_t bal = wave_ballot(has);
        if (lane_id() == 0) wtot[wave] = __popcll(bal);
        __syncthreads();
        int32_t before = 0, total = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const int32_t c = wtot[w];
            before += (w < wave) ? c : 0;
            total += c;
        }
        if (has) list_s[base + before + lanes_below(bal)] = t;
        base += total;
        __syncthreads();  // wtot is rewritten by the next chunk
    }
    return base;
}

// Publishes one app's list (padded with -1) and count, as the route build does.
template <int THREADS>
__device__ void publish_token_list(const int32_t* list_s, int32_t n, int32_t T_max,
                                   int32_t* __restrict__ list_g, int32_t* __restrict__ count_g) {
    for (int32_t i = threadIdx.x; i < T_max; i += THREADS) list_g[i] = i < n ? list_s[i] : -1;
    if (threadIdx.x == 0) *count_g = n;
}

// ORs the workgroup's error bits into the error word (every lane takes part).
__device__ __forceinline__ void publish_error(uint32_t err, uint32_t* __restrict__ err_word) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) err |= __shfl_xor(err, off, kWave);
    if (lane_id() == 0 && err != 0) atomicOr(err_word, err);
}

}  // namespace xmix
