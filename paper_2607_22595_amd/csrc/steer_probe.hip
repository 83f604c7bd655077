// Per-token probes and the steering add in one pass over each row: a hook
// where apps read and write (probes and steering vectors composed at one
// layer).  The row is read once in 16-byte slices; the probes take their
// dot products from the values as read (the activation as the model
// produced it), the steering sum is added in fp64 and the row written back
// rounded once.  The arithmetic and its order are those of the separate
// probe and steering kernels (same slicing, same per-thread accumulation,
// same reductions), so the results are bit-identical to a token-mode probe
// call followed by a steering call.  One workgroup of 512 threads per
// token slot (a 4096-wide bf16 row is one slice per thread, so every load
// of the pass goes out at once); a row with neither kind of bit returns
// after reading its mask word.
//
// With r_tvalid given, the kernel also builds the step's routing (in place
// of a route-build launch): n_apps more workgroups, dispatched first, each
// build one app's token list from the routing inputs staged in LDS and
// publish it with its count (the first also the error word), and each token
// workgroup computes its token's mask itself and writes it.
#include "common.hpp"
#include "kernels.hpp"
#include "launch.hpp"
#include "route_list.hpp"
#include "steer_add.hpp"

namespace xmix {

constexpr int kFuseThreads = 512;  // a 4096-wide bf16 row is one 16-byte slice per thread
constexpr int kFuseWaves = kFuseThreads / kWave;

template <bool BF16, int MAXP>
__global__ void __launch_bounds__(kFuseThreads)
steer_probe_kernel(void* __restrict__ h, int32_t d, int32_t T_max,
                   const uint32_t* __restrict__ tok_mask, const int32_t* __restrict__ req,
                   const void* __restrict__ vecs, BitList sbits, const float* __restrict__ alpha,
                   int32_t n_steer, const void* __restrict__ w, const float* __restrict__ b,
                   BitList pbits, int32_t n_probe, float* __restrict__ logit,
                   float* __restrict__ score, const int32_t* __restrict__ r_tvalid,
                   const uint32_t* __restrict__ r_sub, int32_t r_Rmax, int32_t r_napps,
                   uint32_t* __restrict__ r_mask, int32_t* __restrict__ r_count,
                   int32_t* __restrict__ r_lists, uint32_t* __restrict__ r_err) {
    __shared__ float red[kFuseWaves][MAXP];
    const int n_list = r_tvalid ? r_napps : 0;  // route-list workgroups
    if (static_cast<int>(blockIdx.x) < n_list) {  // uniform
        __shared__ int32_t list_s[kRouteMaxT];
        __shared__ int32_t rtot_s[kFuseWaves];
        __shared__ int32_t req_s[kRouteMaxT];
        __shared__ uint32_t sub_s[kStageSubMax];
        const int a = blockIdx.x;
        stage_route<kFuseThreads>(req, T_max, r_sub, r_Rmax, req_s, sub_s);
        uint32_t err = 0;
        const int32_t tv = clamp_t_valid(*r_tvalid, T_max, err);
        const uint32_t keep = r_napps >= 32 ? 0xFFFFFFFFu : ((1u << r_napps) - 1u);
        __syncthreads();  // the staged inputs
        const int32_t n = build_token_list<kFuseThreads>(req_s, tv, sub_s, r_sub, r_Rmax, keep, a,
                                                         T_max, list_s, rtot_s, nullptr, err);
        publish_token_list<kFuseThreads>(list_s, n, T_max,
                                         r_lists + static_cast<int64_t>(a) * T_max, r_count + a);
        if (a == 0) publish_error(err, r_err);  // its pass saw every slot
        return;
    }
    const int32_t t = static_cast<int32_t>(blockIdx.x) - n_list;
    const int32_t rq = req[t];  // loaded beside the mask (alpha's row depends on it)
    uint32_t mask;
    if (r_tvalid) {  // uniform
        uint32_t unused = 0;
        const int32_t tv = clamp_t_valid(*r_tvalid, T_max, unused);
        const uint32_t keep = r_napps >= 32 ? 0xFFFFFFFFu : ((1u << r_napps) - 1u);
        mask = request_mask(rq, t, tv, r_sub, r_Rmax, keep, unused);
        if (threadIdx.x == 0) r_mask[t] = mask;
    } else {
        mask = tok_mask[t];
    }
    uint32_t ss = 0, sp = 0;
    for (int s = 0; s < n_steer; ++s) ss |= ((mask >> sbits.bit[s]) & 1u) << s;
    for (int p = 0; p < n_probe; ++p) sp |= ((mask >> pbits.bit[p]) & 1u) << p;
    if ((ss | sp) == 0) return;
    const float* a_row = ss ? alpha + static_cast<int64_t>(rq) * n_steer : alpha;

    constexpr int EPV = BF16 ? 8 : 4;  // elements per 16-byte vector
    const int32_t nvec = d / EPV;
    uint4* row = reinterpret_cast<uint4*>(h) + static_cast<int64_t>(t) * nvec;
    const uint4* V = reinterpret_cast<const uint4*>(vecs);
    const uint4* W = reinterpret_cast<const uint4*>(w);
    float part[MAXP];
#pragma unroll
    for (int p = 0; p < MAXP; ++p) part[p] = 0.0f;

    // probe weights fetched together with the row (the rest, for more than
    // eight probes, when used)
    constexpr int AP = MAXP < 8 ? MAXP : 8;
    for (int32_t i = threadIdx.x; i < nvec; i += kFuseThreads) {
        // Every load of the slice before its first use: the row, the weights
        // of the token's probes and its first four steering vectors with
        // their alphas, so that the slice waits for one memory round trip,
        // not one per operand.
        const uint4 hv = row[i];
        uint4 wv[AP];
#pragma unroll
        for (int p = 0; p < AP; ++p)
            wv[p] = ((sp >> p) & 1u) ? W[static_cast<int64_t>(p) * nvec + i]
                                     : make_uint4(0u, 0u, 0u, 0u);
        uint32_t rest = ss;
        SteerGroup g0;
        steer_fetch(g0, rest, a_row, V, nvec, i);
        const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
        // probes, on the row as read
        float x[EPV];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if constexpr (BF16) {
                x[2 * e] = lo_bf16(hw[e]);
                x[2 * e + 1] = hi_bf16(hw[e]);
            } else {
                x[e] = __uint_as_float(hw[e]);
            }
        }
#pragma unroll
        for (int p = 0; p < MAXP; ++p) {
            if (!((sp >> p) & 1u)) continue;
            const uint4 w4 = p < AP ? wv[p < AP ? p : 0] : W[static_cast<int64_t>(p) * nvec + i];
            const uint32_t ww[4] = {w4.x, w4.y, w4.z, w4.w};
            float acc = part[p];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if constexpr (BF16) {
                    acc = fmaf(lo_bf16(ww[e]), x[2 * e], acc);
                    acc = fmaf(hi_bf16(ww[e]), x[2 * e + 1], acc);
                } else {
                    acc = fmaf(__uint_as_float(ww[e]), x[e], acc);
                }
            }
            part[p] = acc;
        }
        // steering, written back: the first four vectors as fetched, then
        // the rest (more than four steering apps) four at a time
        if (ss) {
            double acc[EPV];
#pragma unroll
            for (int e = 0; e < EPV; ++e) acc[e] = x[e];
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
    if (sp == 0) return;  // uniform over the block

    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int p = 0; p < MAXP; ++p) {
        if (!((sp >> p) & 1u)) continue;
        const float s = wave_sum(part[p]);
        if (lane_id() == 0) red[wave][p] = s;
    }
    __syncthreads();
    const int p = threadIdx.x;
    if (p < n_probe && ((sp >> p) & 1u)) {
        float dot = 0.0f;
#pragma unroll
        for (int wv = 0; wv < kFuseWaves; ++wv) dot += red[wv][p];
        const int64_t o = static_cast<int64_t>(p) * T_max + t;
        const float l = b[p] + dot;
        logit[o] = l;
        score[o] = logistic(l);
    }
}

template <bool BF16>
static hipError_t launch_steer_probe_t(void* h, int32_t d, int32_t T_max,
                                       const uint32_t* tok_mask, const int32_t* req,
                                       const void* vecs, const BitList& sbits,
                                       const float* alpha, int32_t n_steer, const void* w,
                                       const float* b, const BitList& pbits, int32_t n_probe,
                                       float* logit, float* score, const RouteIn& r,
                                       hipStream_t stream) {
    dim3 g(T_max + (r.T_valid ? r.n_apps : 0)), blk(kFuseThreads);
    if (n_probe <= 4)
        hipLaunchKernelGGL((steer_probe_kernel<BF16, 4>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, req, vecs, sbits, alpha, n_steer, w, b, pbits, n_probe,
                           logit, score, r.T_valid, r.sub, r.R_max, r.n_apps, r.tok_mask,
                           r.app_count, r.app_tokens, r.err_word);
    else if (n_probe <= 8)
        hipLaunchKernelGGL((steer_probe_kernel<BF16, 8>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, req, vecs, sbits, alpha, n_steer, w, b, pbits, n_probe,
                           logit, score, r.T_valid, r.sub, r.R_max, r.n_apps, r.tok_mask,
                           r.app_count, r.app_tokens, r.err_word);
    else if (n_probe <= 16)
        hipLaunchKernelGGL((steer_probe_kernel<BF16, 16>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, req, vecs, sbits, alpha, n_steer, w, b, pbits, n_probe,
                           logit, score, r.T_valid, r.sub, r.R_max, r.n_apps, r.tok_mask,
                           r.app_count, r.app_tokens, r.err_word);
    else
        hipLaunchKernelGGL((steer_probe_kernel<BF16, 32>), g, blk, 0, stream, h, d, T_max,
                           tok_mask, req, vecs, sbits, alpha, n_steer, w, b, pbits, n_probe,
                           logit, score, r.T_valid, r.sub, r.R_max, r.n_apps, r.tok_mask,
                           r.app_count, r.app_tokens, r.err_word);
    return hipGetLastError();
}

hipError_t launch_steer_probe(void* h, bool bf16, int32_t d, int32_t T_max,
                              const uint32_t* tok_mask, const int32_t* req, const void* vecs,
                              const BitList& sbits, const float* alpha, int32_t n_steer,
                              const void* w, const float* b, const BitList& pbits,
                              int32_t n_probe, float* logit, float* score, hipStream_t stream,
                              const RouteIn* route) {
    RouteIn r{};
    if (route) {
        if (T_max > kRouteMaxT || T_max < route->n_apps) {
            // the kernel cannot route this batch: the route-build launch first
            const hipError_t e = launch_route_build(route->req, route->T_valid, route->sub,
                                                    route->R_max, T_max, route->n_apps,
                                                    route->tok_mask, route->app_count,
                                                    route->app_tokens, route->err_word, stream);
            if (e != hipSuccess) return e;
        } else {
            r = *route;
        }
    }
    return bf16 ? launch_steer_probe_t<true>(h, d, T_max, tok_mask, req, vecs, sbits, alpha,
                                             n_steer, w, b, pbits, n_probe, logit, score, r,
                                             stream)
                : launch_steer_probe_t<false>(h, d, T_max, tok_mask, req, vecs, sbits, alpha,
                                              n_steer, w, b, pbits, n_probe, logit, score, r,
                                              stream);
}

void add_steer_probe_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(steer_probe_kernel<true, 4>));
    t.push_back(kernel_info(steer_probe_kernel<true, 8>));
    t.push_back(kernel_info(steer_probe_kernel<true, 16>));
    t.push_back(kernel_info(steer_probe_kernel<true, 32>));
    t.push_back(kernel_info(steer_probe_kernel<false, 4>));
    t.push_back(kernel_info(steer_probe_kernel<false, 8>));
    t.push_back(kernel_info(steer_probe_kernel<false, 16>));
    t.push_back(kernel_info(steer_probe_kernel<false, 32>));
}

}  // namespace xmix
