// SAE encode with TopK: pre = W_enc . h + c_fold for the tokens subscribed
// to one app, then the k largest pre-activations per token.
//
// Stage 1 (sae_stream_kernel) is an MFMA bf16 GEMM with fp32 accumulation.
// A workgroup (8 waves, two per SIMD so one wave's waits overlap the other's
// MFMAs) owns 256 latents x 128 subscribed tokens and walks K = d in chunks
// of 64:
//   - the dictionary (operand A) streams from HBM straight into registers
//     from the tiled layout below (each wave-wide load is 1 KB contiguous,
//     each workgroup reads its 2 MiB slice front to back; nontemporal
//     loads, as nothing reads it again), each wave owning 32 latents,
//     through a four-deep register ring (three chunks in flight);
//   - the token rows (operand B) are gathered through the app's token list
//     into LDS (double buffered; the 16-byte chunk c of row n is stored at
//     c ^ ((n >> 1) & 7), so the 16 rows one MFMA-layout read touches per
//     LDS cycle land in 16 distinct bank groups) and shared by the 8 waves.
// Epilogue, per token of the tile: a threshold tau is chosen so that the
// number of latents with pre >= tau lies in a small window (first guess
// mean + z * stdev of the tile's 256 values, then bisection on the value if
// needed); every latent with pre >= tau is emitted as a candidate, and the
// count and the tile's bound are recorded: a value that every latent left
// out lies below (the decode kernels: the next value above the largest one
// left out; the prefill GEMM: tau, or the next value above the tile's
// maximum when nothing is emitted).  This costs O(1) work per value.
// The decode kernel writes the tile to LDS token-major, and eight lanes of
// one wave select for each token with no barrier or LDS atomic between the
// waves.  The prefill kernel (one wave per SIMD, values in accumulator
// registers) runs the four token groups of a wave through each phase
// together; a wave alone on its SIMD has no other wave to hide its
// latencies, and the LDS path measured slower there.
//
// Stage 2 (sae_merge_kernel): one workgroup per subscribed token gathers the
// candidates of all tiles and selects the exact top-k of that pool (a radix
// select over (value, latent) composites, ties to the lower latent).  The result is the exact top-k of
// all m latents whenever the k-th selected value is >= every tile's bound,
// because a latent that was not emitted lies below its tile's bound.  When
// that certificate fails (only for inputs whose best latents crowd into a
// few tiles or tie across whole tiles), the workgroup recomputes tiles'
// 256 pre-activations with plain fp32 dot products, in descending order of
// their bounds, until no tile left can hold a winner.  The
// decode kernel's first threshold guess leaves a tile's outlying values
// out of the statistics (beyond mean +- 5 stdev), so that a few strong
// latents, such as features clamped high by a steering app, or rows of a
// much larger norm than the others, do not lift it: with a decode
// dictionary's ratio of k to m the certificate has little slack.  The
// prefill kernel keeps the plain statistics (a GEMM epilogue
// pays for every extra pass, and the repair covers the rare failure).
//
// The workgroup-to-tile map is XCD-aware: launch slots are dealt round-robin
// to the 8 XCDs, so consecutive tiles of one XCD share a dictionary slice in
// that XCD's L2.
#include <math.h>
#include <stddef.h>
#include <string.h>

#include <atomic>

#include "common.hpp"
#include "kernels.hpp"
#include "launch.hpp"
#include "route_list.hpp"

namespace xmix {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;

constexpr int kBM = 256;  // latents per workgroup
constexpr int kBN = 128;  // tokens per workgroup
constexpr int kBK = 64;   // K chunk
constexpr int kEncWaves = 8;
constexpr int kEncThreads = kEncWaves * kWave;
constexpr int kRefineIters = 24;
constexpr int kMaxCap = 64;  // most candidate pairs one slice may emit
// Values beyond mean +- kTrimZ * stdev of a tile's 256 pre-activations are
// left out of the statistics behind the decode kernel's first threshold
// guess (one strong latent, or one of a large norm on either side, would
// otherwise raise the guess for its whole tile).
constexpr float kTrimZ = 5.0f;
constexpr int kLatentFastTiles = 4;  // token tiles up to which the latent tile runs fastest
constexpr int kBlkTok = 8;           // prefill block: token tiles
constexpr int kBlkLat = 4;           // prefill block: latent tiles

// v[r] for a lane-varying r in [0, 16), by a select tree on the bits of r
// (registers cannot be indexed per lane)
__device__ __forceinline__ float pick16(const f32x16_t& v, int r) {
    const bool b0 = r & 1, b1 = r & 2, b2 = r & 4, b3 = r & 8;
    const float a0 = b0 ? v[1] : v[0], a1 = b0 ? v[3] : v[2], a2 = b0 ? v[5] : v[4],
                a3 = b0 ? v[7] : v[6], a4 = b0 ? v[9] : v[8], a5 = b0 ? v[11] : v[10],
                a6 = b0 ? v[13] : v[12], a7 = b0 ? v[15] : v[14];
    const float c0 = b1 ? a1 : a0, c1 = b1 ? a3 : a2, c2 = b1 ? a5 : a4, c3 = b1 ? a7 : a6;
    const float d0 = b2 ? c1 : c0, d1 = b2 ? c3 : c2;
    return b3 ? d1 : d0;
}

// mean + z * stdev of n values with sum s1 and sum of squares s2
__device__ __forceinline__ float trimmed_guess(float s1, float s2, int n, float z) {
    const float inv = 1.0f / static_cast<float>(n > 0 ? n : 1);
    const float mu = s1 * inv;
    return mu + z * sqrtf(fmaxf(s2 * inv - mu * mu, 0.0f));
}

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) {
    return __builtin_bit_cast(bf16x8_t, v);
}

// ------------------------------------------------------- dictionary layout
// W_enc is kept in HBM in a tiled layout matched to the encode GEMMs, built
// once when an SAE app is loaded.  The unit is a 16-byte piece (8 bf16 of
// one latent row).  Latent j = 256*mt + 32*w + r and row element
// i = 64*kc + 16*s + 8*g + e (e < 8) live in piece
//     (kc*n_mt + mt)*2048 + w*256 + s*64 + (r + 32*g)
// so the 32 KB of a 256-latent slice per K chunk of 64 are contiguous,
// every wave-wide 16-byte load is 1 KB contiguous (the A operand of one
// 32x32x16 MFMA step s: lane r + 32*g holds elements 16*s + 8*g .. + 7),
// each half chunk (steps 0-1, steps 2-3) is 2 KB contiguous per 32
// latents, and at each K step the whole grid streams one contiguous region
// (chunk-major order spreads concurrent workgroups over all HBM channels).
__device__ __forceinline__ int64_t packed_piece(int32_t j, int32_t i, int32_t n_mt) {
    const int32_t mt = j >> 8, jr = j & 255;
    const int32_t w = jr >> 5, r = jr & 31;
    const int32_t kc = i >> 6, s = (i >> 4) & 3, g = (i >> 3) & 1;
    return (static_cast<int64_t>(kc) * n_mt + mt) * 2048 + w * 256 + s * 64 + r + 32 * g;
}

__global__ void __launch_bounds__(256)
sae_pack_kernel(const uint16_t* __restrict__ W, int32_t m, int32_t d, uint16_t* __restrict__ Wp) {
    const int32_t pieces_per_row = d / 8;
    const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (q >= static_cast<int64_t>(m) * pieces_per_row) return;
    const int32_t j = static_cast<int32_t>(q / pieces_per_row);
    const int32_t i = static_cast<int32_t>(q % pieces_per_row) * 8;
    reinterpret_cast<uint4*>(Wp)[packed_piece(j, i, m / kBM)] =
        reinterpret_cast<const uint4*>(W)[q];
}

// c_fold[j] = b_enc[j] - W_enc[j,:] . b_dec (packed W_enc), one wave per latent.
__global__ void __launch_bounds__(256)
sae_fold_kernel(const uint16_t* __restrict__ Wp, const uint16_t* __restrict__ b_enc,
                const uint16_t* __restrict__ b_dec, int32_t m, int32_t d,
                float* __restrict__ c_fold) {
    const int32_t j = blockIdx.x * 4 + threadIdx.x / kWave;
    if (j >= m) return;
    const int32_t n_mt = m / kBM;
    const uint4* P = reinterpret_cast<const uint4*>(Wp);
    const uint4* bd = reinterpret_cast<const uint4*>(b_dec);
    float acc = 0.0f;
    for (int32_t p = lane_id(); p < d / 8; p += kWave) {
        const uint4 wv = P[packed_piece(j, p * 8, n_mt)], bv = bd[p];
        const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
        const uint32_t bw[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc = fmaf(lo_bf16(ww[e]), lo_bf16(bw[e]), acc);
            acc = fmaf(hi_bf16(ww[e]), hi_bf16(bw[e]), acc);
        }
    }
    acc = wave_sum(acc);
    if (lane_id() == 0) c_fold[j] = bf16_to_f32(b_enc[j]) - acc;
}

// ------------------------------------------------ wave-local slice selection
// After a tile's K loop, its values are written to LDS token-major (one row
// of kSelStride floats per token, 256 latents each) and the 256 values of a
// token are taken by 8 lanes of one wave, 32 contiguous latents per lane.
// The threshold search, the counts and the emission prefix then reduce over
// those 8 lanes with DPP moves: no barrier and no LDS atomic between the
// waves.  Each lane works on NT tokens at once (independent chains that
// fill each other's latencies).  The row stride is 4 words past a multiple
// of the 64 LDS banks, so the 16-byte reads of the 64 lanes at one step
// spread over every bank.
constexpr int kSelStride = 260;  // floats per token row

// Reductions inside groups of 8 lanes on DPP moves (quad_perm, row_half_mirror)
__device__ __forceinline__ float sum8(float v) {
    v += dpp_f<kDppXor1>(v);
    v += dpp_f<kDppXor2>(v);
    return v + dpp_f<kDppHalfMirror>(v);
}
__device__ __forceinline__ int isum8(int v) {
    v += dpp_i<kDppXor1>(v);
    v += dpp_i<kDppXor2>(v);
    return v + dpp_i<kDppHalfMirror>(v);
}
__device__ __forceinline__ float max8(float v) {
    v = fmaxf(v, dpp_f<kDppXor1>(v));
    v = fmaxf(v, dpp_f<kDppXor2>(v));
    return fmaxf(v, dpp_f<kDppHalfMirror>(v));
}
// sum over the lanes q' < q of the group of 8 (q = lane & 7)
__device__ __forceinline__ int excl_scan8(int v, int q) {
    int incl = v;
    int y = dpp_i<0x111>(incl);  // row_shr:1
    incl += q >= 1 ? y : 0;
    y = dpp_i<0x112>(incl);      // row_shr:2
    incl += q >= 2 ? y : 0;
    y = dpp_i<0x114>(incl);      // row_shr:4
    incl += q >= 4 ? y : 0;
    return incl - v;
}

// The selection of NT tokens over one 256-latent slice each: per token a
// threshold tau with lo_cnt <= count(pre >= tau) <= cap (first guess
// mean + z * stdev of the 256 values, then bisection on the value), and
// every latent with pre >= tau written to dst[t][0 .. count) as (fp32 bits,
// latent), with the count and the slice's bound beside it.  vrow[t]: token
// t's LDS row; q = lane & 7 takes latents [32q, 32q + 32); lat0: the slice's first
// latent.  Every lane of the wave calls it (the cross-lane steps are
// wave-wide); the lanes of a token with valid[t] == false take part in them
// and write nothing.  With TRIM, the values beyond mean +- 5 stdev are left
// out of the statistics behind the first guess (a few outlying latents would
// otherwise lift it for the whole slice).
template <bool TRIM, int NT>
__device__ __forceinline__ void select_slices(const float* const (&vrow)[NT], int q,
                                              const bool (&valid)[NT], float z, int lo_cnt,
                                              int cap, int32_t lat0, uint2* const (&dst)[NT],
                                              int32_t* const (&cnt_out)[NT],
                                              float* const (&tau_out)[NT]) {
    float x[NT][32];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const float4* src = reinterpret_cast<const float4*>(vrow[t]);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float4 v = src[8 * q + i];
            x[t][4 * i] = v.x;
            x[t][4 * i + 1] = v.y;
            x[t][4 * i + 2] = v.z;
            x[t][4 * i + 3] = v.w;
        }
    }
    // ax[t]: the largest magnitude among the token's values
    float tau[NT], s1[NT], s2[NT], ax[NT], mu[NT], sd[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float a = 0.0f, b = 0.0f, c = 0.0f;
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            a += x[t][i];
            b = fmaf(x[t][i], x[t][i], b);
            if (TRIM) c = fmaxf(c, fabsf(x[t][i]));
        }
        s1[t] = a;
        s2[t] = b;
        ax[t] = c;
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        s1[t] = sum8(s1[t]);
        s2[t] = sum8(s2[t]);
        if (TRIM) ax[t] = max8(ax[t]);
        mu[t] = s1[t] * (1.0f / kBM);
        sd[t] = sqrtf(fmaxf(s2[t] * (1.0f / kBM) - mu[t] * mu[t], 0.0f));
        tau[t] = mu[t] + z * sd[t];
    }
    if (TRIM) {
        // values more than kTrimZ stdev from the mean on either side: a large
        // value lifts the mean and the spread, a large negative one the
        // spread.  A value that far out has a magnitude above
        // kTrimZ * stdev - |mean|; the pass below leaves out exactly the
        // values beyond the two cuts, so a token it finds none for keeps its
        // guess.
        bool trim[NT], any = false;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            trim[t] = valid[t] && ax[t] + fabsf(mu[t]) > kTrimZ * sd[t];
            any = any || trim[t];
        }
        if (wave_ballot(any)) {  // uniform
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const float cut = mu[t] + kTrimZ * sd[t], cut_lo = mu[t] - kTrimZ * sd[t];
                float e1 = 0.0f, e2 = 0.0f;
                int ne = 0;
#pragma unroll
                for (int i = 0; i < 32; ++i) {
                    const bool o = x[t][i] > cut || x[t][i] < cut_lo;
                    ne += o ? 1 : 0;
                    e1 += o ? x[t][i] : 0.0f;
                    e2 = fmaf(o ? x[t][i] : 0.0f, x[t][i], e2);
                }
                e1 = sum8(e1);
                e2 = sum8(e2);
                ne = isum8(ne);
                if (trim[t]) tau[t] = trimmed_guess(s1[t] - e1, s2[t] - e2, kBM - ne, z);
            }
        }
    }
    float lo[NT], hi[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        lo[t] = -INFINITY;
        hi[t] = INFINITY;
    }
    // m[t]: this lane's latents at or above tau[t], one bit each; the count
    // is its population, so the emission below reuses the last round's masks
    uint32_t m[NT];
    auto masks = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            uint32_t b = 0;
#pragma unroll
            for (int i = 0; i < 32; ++i) b |= (x[t][i] >= tau[t] ? 1u : 0u) << i;
            m[t] = b;
        }
    };
    bool settled = false;
    for (int it = 0; it < kRefineIters; ++it) {
        masks();
        int c[NT];
        bool bad[NT], any = false;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            c[t] = isum8(__popc(m[t]));
            bad[t] = valid[t] && (c[t] > cap || c[t] < lo_cnt);
            any = any || bad[t];
        }
        if (!wave_ballot(any)) {  // uniform
            settled = true;
            break;
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (!bad[t]) continue;
            if (c[t] > cap) lo[t] = tau[t];
            else hi[t] = tau[t];
            if (it == kRefineIters - 1) {
                // out of rounds: a threshold whose count is known to be below
                // lo_cnt (or +inf, count 0); the merge then checks exactness
                tau[t] = hi[t];
            } else if (isfinite(lo[t]) && isfinite(hi[t])) {
                tau[t] = 0.5f * (lo[t] + hi[t]);
            } else {
                // step away from the bad side by a growing fraction of |tau| + 1
                const float step = ldexpf(0.25f * (fabsf(tau[t]) + 1.0f), it);
                tau[t] = isfinite(hi[t]) ? tau[t] - step : tau[t] + step;
            }
        }
    }
    // out of rounds: the final thresholds were set after the last masks
    if (!settled) masks();
    // emission: this lane's selected latents go to the slots after those of
    // the lanes before it in the token's group of 8; nk[t]: the largest of
    // the token's values that are not kept (NaN never counts: it compares
    // below everything)
    int base[NT], total[NT];
    float nk[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int cl = __popc(m[t]);
        base[t] = excl_scan8(cl, q);
        total[t] = isum8(cl);
        float l = -INFINITY;
#pragma unroll
        for (int i = 0; i < 32; ++i) l = fmaxf(l, x[t][i] >= tau[t] ? -INFINITY : x[t][i]);
        nk[t] = max8(l);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (!valid[t]) continue;
        uint32_t b = m[t];
        int slot = base[t];
        while (b != 0) {
            const int i = __builtin_ctz(b);
            b &= b - 1;
            if (slot < cap)
                dst[t][slot] = make_uint2(__float_as_uint(vrow[t][32 * q + i]),
                                          static_cast<uint32_t>(lat0 + 32 * q + i));
            ++slot;
        }
        if (q == 0) {
            *cnt_out[t] = min(total[t], cap);
            // the slice's bound: the next value above the largest one it
            // does not keep (at most tau, and the tightest bound there is;
            // with nothing kept, the next value above its maximum)
            *tau_out[t] = key_f32(f32_key(nk[t]) + 1u);
        }
    }
}

// ---------------------------------------------- GEMM + candidate emission
// The dictionary stream of one workgroup: the first piece of a slice's K
// chunk 0, and the pieces from one K chunk to the next (both the same for
// every lane; each lane adds its own offset when it loads).
struct SliceSrc {
    const uint4* base;
    int64_t stride;
};
__device__ __forceinline__ SliceSrc slice_src(const uint16_t* W, int32_t n_mt, int mt) {
    return {reinterpret_cast<const uint4*>(W) + static_cast<int64_t>(mt) * 2048,
            static_cast<int64_t>(n_mt) * 2048};
}
// operand A of one K chunk at p: this wave's 32 latents of the packed
// slice.  The dictionary is read once per launch: nontemporal loads stream
// it past the caches (about 4 % faster than cached loads at 65536 x 4096).
__device__ __forceinline__ void load_chunk(uint4 (&a)[4], const uint4* p) {
    const uint32_t off = threadIdx.x & 511;  // wave * 256 + lane: pieces 4 x 64 apart
    const u32x4_t* q = reinterpret_cast<const u32x4_t*>(p) + ((off >> 6) * 256 + (off & 63));
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const u32x4_t v = __builtin_nontemporal_load(q + s * 64);
        a[s] = make_uint4(v.x, v.y, v.z, v.w);
    }
}
// the folded bias of this lane's 16 latents of slice mt
__device__ __forceinline__ void load_bias(float (&cfv)[16], const float* c_fold, int mt) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float* cf = c_fold + mt * kBM + 32 * wave + 4 * (lane >> 5);
#pragma unroll
    for (int r = 0; r < 16; ++r) cfv[r] = cf[8 * (r / 4) + (r % 4)];
}

// Where one app's slices put their candidates, and how they select them.
struct SliceSink {
    uint2* cand;
    int32_t* tile_cnt;
    float* tile_tau;
    int32_t n_mt, lo_cnt, cap;
    float z;
};

// The GEMM and candidate emission of latent slice mt over the token tiles
// nt, nt + 1, ... of the app's list tl[0, cnt) (only tile nt unless
// in_turn); the caller has checked nt * kBN < cnt.  On entry wa0..wa2 hold
// the slice's K chunks 0-2 and cfv its folded bias when `issued`.  The K
// loop fetches three chunks ahead; past the slice's last chunk it fetches
// the first chunks of what runs next: the same slice again for the next
// token tile, else slice `nxt` when has_nxt (then also its bias from
// nxt_cf, after this tile's selection), else nothing new (the last chunk
// again, unused).  Returns has_nxt: whether wa0..wa2 and cfv now hold nxt's
// first chunks and bias.  lds_main is the workgroup's token-chunk and
// selection space.
__device__ __forceinline__ bool slice_tiles(
    uint4* lds_main, const uint16_t* __restrict__ h, int32_t d, const int32_t* tl, int cnt,
    int nt, bool in_turn, int mt, const SliceSrc cur, const SliceSink sink, bool issued,
    const SliceSrc nxt, bool has_nxt, int nxt_mt, const float* __restrict__ nxt_cf,
    const float* __restrict__ c_fold, uint4 (&wa0)[4], uint4 (&wa1)[4], uint4 (&wa2)[4],
    uint4 (&wa3)[4], float (&cfv)[16]) {
    uint4 (*xs)[kBN * 8] = reinterpret_cast<uint4 (*)[kBN * 8]>(lds_main);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 5, j32 = lane & 31;
    const int nK = d / kBK;  // a multiple of 4 (d % 256 == 0)

    // operand B: gathered token rows; padding rows read a valid row and are
    // zeroed when written to LDS
    const int xr = tid >> 3, xc = tid & 7;
    const uint16_t* xrow[2];
    uint32_t xmask[2];
    f32x16_t acc[4];
    uint4 xv0[2], xv1[2];                   // token ring: 2 chunks in flight
    auto load_x = [&](uint4 (&xv)[2], int kc) {
        kc = min(kc, nK - 1);
#pragma unroll
        for (int p = 0; p < 2; ++p) xv[p] = *reinterpret_cast<const uint4*>(xrow[p] + kc * kBK);
    };
    auto store_x = [&](const uint4 (&xv)[2], int buf) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int n = xr + 64 * p;
            const uint4 v = make_uint4(xv[p].x & xmask[p], xv[p].y & xmask[p],
                                       xv[p].z & xmask[p], xv[p].w & xmask[p]);
            xs[buf][n * 8 + (xc ^ ((n >> 1) & 7))] = v;
        }
    };
    auto compute = [&](const uint4 (&a)[4], int buf) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const bf16x8_t A = as_bf16x8(a[s]);
            uint4 bop[4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int n = 32 * nb + j32;
                const int chunk = 2 * s + g;
                bop[nb] = xs[buf][n * 8 + (chunk ^ ((n >> 1) & 7))];
            }
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
                acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, as_bf16x8(bop[nb]), acc[nb],
                                                                  0, 0, 0);
        }
    };
    // One K chunk (branch-free): issue the token chunk two ahead and the W
    // chunk three ahead (at wp), multiply the current chunk, then publish
    // the next token chunk to the other LDS buffer.  Loads are issued
    // oldest-needed first, so the in-order vmcnt wait for the next token
    // chunk never waits on a W prefetch.
    auto step = [&](int kc, const uint4 (&cur_w)[4], uint4 (&wnext)[4], const uint4* wp,
                    uint4 (&xload)[2], const uint4 (&xstore)[2]) {
        load_x(xload, kc + 2);
        __builtin_amdgcn_sched_barrier(0);  // keep the token loads ahead of the W loads
        load_chunk(wnext, wp);
        __syncthreads();
        compute(cur_w, kc & 1);
        store_x(xstore, (kc + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
    };

    if (!issued) load_bias(cfv, c_fold, mt);  // the slice's bias serves every token tile
    for (;; ++nt) {
        const int n0 = nt * kBN;
        const int ntok = min(kBN, cnt - n0);
        const bool last = !in_turn || n0 + kBN >= cnt;
        // the stream past this slice's last chunk: the next token tile's
        // first chunks, nxt's, or the last chunk again (unused)
        const uint4* after = !last ? cur.base : has_nxt ? nxt.base : cur.base + (nK - 1) * cur.stride;
        const int64_t after_stride = !last ? cur.stride : has_nxt ? nxt.stride : 0;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int n = xr + 64 * p;
            const bool ok = n < ntok;
            xmask[p] = ok ? 0xFFFFFFFFu : 0u;
            xrow[p] = h + static_cast<int64_t>(tl[n0 + (ok ? n : 0)]) * d + 8 * xc;
        }
        // the accumulators start from the folded bias
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[b][r] = cfv[r];

        load_x(xv0, 0);
        load_x(xv1, 1);
        if (!issued) {
            load_chunk(wa0, cur.base);
            load_chunk(wa1, cur.base + cur.stride);
            load_chunk(wa2, cur.base + 2 * cur.stride);
        }
        store_x(xv0, 0);
        // four chunks per round (the W registers rotate); the last round
        // fetches what follows the slice
        auto round4 = [&](int kc, const uint4* p0, const uint4* p1, const uint4* p2,
                          const uint4* p3) {
            step(kc + 0, wa0, wa3, p0, xv0, xv1);
            step(kc + 1, wa1, wa0, p1, xv1, xv0);
            step(kc + 2, wa2, wa1, p2, xv0, xv1);
            step(kc + 3, wa3, wa2, p3, xv1, xv0);
        };
        const uint4* wp = cur.base + 3 * cur.stride;
        const int64_t ws = cur.stride;
        if (nK > 4) {
            // The first round runs apart from the loop: its loads follow the
            // prologue's (whose W chunks may have been issued long before),
            // while every round of the loop follows a round.  So the loop's
            // waits count only a round's loads, and a step waits for its
            // token chunk without waiting for the W chunk issued a step ago.
            round4(0, wp, wp + ws, wp + 2 * ws, wp + 3 * ws);
            wp += 4 * ws;
            for (int kc = 4; kc < nK - 4; kc += 4) {
                round4(kc, wp, wp + ws, wp + 2 * ws, wp + 3 * ws);
                wp += 4 * ws;
            }
        }
        round4(nK - 4, wp, after, after + after_stride, after + 2 * after_stride);
        // wa0..wa2 now hold the first three chunks of what runs next
        issued = !last || has_nxt;

        // ------------------------------------------------------ epilogue
        // acc[nb][r] holds latent 32*wave + 8*(r/4) + 4*g + r%4 of token
        // 32*nb + j32 (the 32x32 MFMA output layout).  Every lane writes its
        // values to the tile's 128 token rows in LDS; then wave w selects for
        // rows 16w .. 16w + 15, eight lanes per row, two rows per lane.
        __syncthreads();  // every wave is done with the token chunks
        float* V = reinterpret_cast<float*>(lds_main);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
            float* rowp = V + (32 * nb + j32) * kSelStride + 32 * wave + 4 * g;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                *reinterpret_cast<float4*>(rowp + 8 * j) =
                    make_float4(acc[nb][4 * j], acc[nb][4 * j + 1], acc[nb][4 * j + 2],
                                acc[nb][4 * j + 3]);
        }
        __syncthreads();
        const int q = lane & 7;
        const int r0 = 16 * wave + (lane >> 3), r1 = r0 + 8;
        const int64_t row0 = static_cast<int64_t>(n0 + r0) * sink.n_mt + mt;
        const int64_t row1 = static_cast<int64_t>(n0 + r1) * sink.n_mt + mt;
        const float* const vr[2] = {V + r0 * kSelStride, V + r1 * kSelStride};
        const bool ok[2] = {r0 < ntok, r1 < ntok};
        uint2* const dst[2] = {sink.cand + row0 * sink.cap, sink.cand + row1 * sink.cap};
        int32_t* const co[2] = {sink.tile_cnt + row0, sink.tile_cnt + row1};
        float* const to[2] = {sink.tile_tau + row0, sink.tile_tau + row1};
        select_slices<true, 2>(vr, q, ok, sink.z, sink.lo_cnt, sink.cap, mt * kBM, dst, co, to);
        if (last) {
            if (has_nxt && nxt_cf) load_bias(cfv, nxt_cf, nxt_mt);
            return has_nxt;
        }
        __syncthreads();  // the tile rows are read before the next tile's token chunks land
    }
}

// One workgroup's tile: L is the tile's launch slot within its app's grid,
// own the workgroup's index in the launch (its route-publishing duty).
__device__ __forceinline__ void stream_tile(
    int L, int own, const uint16_t* __restrict__ h, int32_t d,
    const int32_t* __restrict__ app_count, const int32_t* __restrict__ tok_list,
    const uint16_t* __restrict__ W, const float* __restrict__ c_fold, int32_t n_mt, int32_t n_nt,
    float z_guess, int32_t lo_cnt, int32_t cap, uint2* __restrict__ cand,
    int32_t* __restrict__ tile_cnt, float* __restrict__ tile_tau,
    const int32_t* __restrict__ r_req, const int32_t* __restrict__ r_tvalid,
    const uint32_t* __restrict__ r_sub, int32_t r_Rmax, int32_t r_Tmax, int32_t r_napps,
    int32_t r_bit, uint32_t* __restrict__ r_mask, int32_t* __restrict__ r_count,
    int32_t* __restrict__ r_lists, uint32_t* __restrict__ r_err) {
    // K loop: two 16 KiB token chunks; epilogue: the tile's 128 token rows
    __shared__ uint4 lds_main[kBN * kSelStride / 4];
    static_assert(kBN * kSelStride / 4 >= 2 * kBN * 8, "token chunks fit");
    __shared__ int32_t list_s[kRouteMaxT];    // the app's token list (in-kernel route build)
    __shared__ int32_t rtot_s[kEncWaves];
    __shared__ int32_t seen_s[kEncWaves];

    // Tile order.  Few token tiles (decode): one workgroup per latent tile,
    // which takes the live token tiles of its slice in turn (no workgroup
    // is launched for a tile past the live count; the first tile, the one
    // every live token count reaches, spreads over every CU).
    // Many token tiles (prefill): launch slot L runs on XCD L % 8; XCD x
    // owns the latent tiles [x*M8, (x+1)*M8) and walks them in blocks of 8
    // token tiles x 4 latent tiles, 32 consecutive slots per block, token
    // blocks fastest.  The 32 workgroups of a block run together on the
    // XCD's 32 CUs, so each K chunk of 8 token tiles and 4 dictionary
    // slices is fetched into the XCD's L2 once and read by 4 and 8
    // workgroups; consecutive blocks reuse the same 4 slices.
    int nt, mt;
    bool live;  // the tile exists (its tokens are counted below)
    if (n_nt <= kLatentFastTiles) {
        nt = L / n_mt;
        mt = L % n_mt;
        live = nt < n_nt;
    } else {
        const int xcd = L % 8, slot = L / 8;
        const int m8 = (n_mt + 7) / 8;              // latent tiles per XCD
        const int nbt = (n_nt + kBlkTok - 1) / kBlkTok;
        const int b = slot / (kBlkTok * kBlkLat), p = slot % (kBlkTok * kBlkLat);
        const int bt = b % nbt, bl = b / nbt;
        const int lt = kBlkLat * bl + p / kBlkTok;
        nt = kBlkTok * bt + p % kBlkTok;
        mt = xcd * m8 + lt;
        live = nt < n_nt && lt < m8;
    }
    live = live && mt < n_mt;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const SliceSrc src = slice_src(W, n_mt, mt);
    uint4 wa0[4], wa1[4], wa2[4], wa3[4];   // W ring: 4 chunks, 3 in flight
    float cfv[16];

    // With r_req given, the kernel also builds the step's routing (in place
    // of a route-build launch): every workgroup builds its app's token list
    // in LDS from the routing inputs staged there (in the space of the K
    // loop's token chunks); workgroup a < n_apps publishes app a's list and
    // count, and workgroup 0 the token masks and the error word.  A
    // workgroup of the first token tile starts its first dictionary chunks
    // as soon as the staged table shows a request subscribed to the app, so
    // that the stream runs while the list is built (without a subscriber it
    // reads nothing).
    const int32_t* tl = tok_list;
    int cnt = 0;
    bool w_issued = false;
    if (r_req) {  // uniform
        static_assert(sizeof(lds_main) >= (kRouteMaxT + kStageSubMax) * 4, "staging fits");
        int32_t* req_s = reinterpret_cast<int32_t*>(lds_main);
        uint32_t* sub_s = reinterpret_cast<uint32_t*>(lds_main) + kRouteMaxT;
        const bool seen = stage_route<kEncThreads>(r_req, r_Tmax, r_sub, r_Rmax, req_s, sub_s,
                                                   1u << r_bit);
        const uint64_t seen_b = wave_ballot(seen);
        if (lane == 0) seen_s[wave] = seen_b != 0;
        uint32_t err = 0;
        const int32_t tv = clamp_t_valid(*r_tvalid, r_Tmax, err);
        const uint32_t keep = r_napps >= 32 ? 0xFFFFFFFFu : ((1u << r_napps) - 1u);
        uint32_t* masks = own == 0 ? r_mask : nullptr;
        __syncthreads();  // the staged inputs
        bool any = false;
#pragma unroll
        for (int w = 0; w < kEncWaves; ++w) any = any || seen_s[w] != 0;
        // no request subscribes to the app: no token is listed, and a
        // workgroup with nothing to publish is done
        if (!any && own >= r_napps) return;  // uniform
        if (live && nt == 0 && any) {  // uniform
            load_chunk(wa0, src.base);
            load_chunk(wa1, src.base + src.stride);
            load_chunk(wa2, src.base + 2 * src.stride);
            load_bias(cfv, c_fold, mt);
            w_issued = true;
        }
        if (own < r_napps && own != r_bit) {
            const int32_t n = build_token_list<kEncThreads>(req_s, tv, sub_s, r_sub, r_Rmax, keep,
                                                            own, r_Tmax, list_s, rtot_s, masks,
                                                            err);
            masks = nullptr;
            publish_token_list<kEncThreads>(list_s, n, r_Tmax,
                                            r_lists + static_cast<int64_t>(own) * r_Tmax,
                                            r_count + own);
            __syncthreads();  // list_s is rebuilt below
        }
        cnt = build_token_list<kEncThreads>(req_s, tv, sub_s, r_sub, r_Rmax, keep, r_bit, r_Tmax,
                                            list_s, rtot_s, masks, err);
        if (own == r_bit)
            publish_token_list<kEncThreads>(list_s, cnt, r_Tmax,
                                            r_lists + static_cast<int64_t>(r_bit) * r_Tmax,
                                            r_count + r_bit);
        if (own == 0) publish_error(err, r_err);
        tl = list_s;
    } else {
        cnt = *app_count;
    }
    if (!live || nt * kBN >= cnt) return;
    const SliceSink sink{cand, tile_cnt, tile_tau, n_mt, lo_cnt, cap, z_guess};
    slice_tiles(lds_main, h, d, tl, cnt, nt, n_nt <= kLatentFastTiles, mt, src, sink, w_issued,
                src, false, 0, nullptr, c_fold, wa0, wa1, wa2, wa3, cfv);
}

__global__ void __launch_bounds__(kEncThreads, 1)
sae_stream_kernel(const uint16_t* __restrict__ h, int32_t d,
                  const int32_t* __restrict__ app_count, const int32_t* __restrict__ tok_list,
                  const uint16_t* __restrict__ W, const float* __restrict__ c_fold,
                  int32_t n_mt, int32_t n_nt, float z_guess, int32_t lo_cnt, int32_t cap,
                  uint2* __restrict__ cand, int32_t* __restrict__ tile_cnt,
                  float* __restrict__ tile_tau, const int32_t* __restrict__ r_req,
                  const int32_t* __restrict__ r_tvalid, const uint32_t* __restrict__ r_sub,
                  int32_t r_Rmax, int32_t r_Tmax, int32_t r_napps, int32_t r_bit,
                  uint32_t* __restrict__ r_mask, int32_t* __restrict__ r_count,
                  int32_t* __restrict__ r_lists, uint32_t* __restrict__ r_err) {
    stream_tile(blockIdx.x, blockIdx.x, h, d, app_count, tok_list, W, c_fold, n_mt, n_nt,
                z_guess, lo_cnt, cap, cand, tile_cnt, tile_tau, r_req, r_tvalid, r_sub, r_Rmax,
                r_Tmax, r_napps, r_bit, r_mask, r_count, r_lists, r_err);
}

// Several SAE apps of one hook in one launch: the apps' grids follow each
// other (app i owns launch slots [grid0[i], grid0[i + 1])), so a CU that
// finishes its slice of one app takes a slice of the next, and the step
// pays one launch for every app's candidates.
struct EncApp {
    const int32_t* app_count;
    const int32_t* tok_list;
    const uint16_t* W;
    const float* c_fold;
    uint2* cand;
    int32_t* tile_cnt;
    float* tile_tau;
    int32_t n_mt, lo_cnt, cap, bit, grid0;
    float z;
};
struct EncApps {
    EncApp a[kMultiMax];
    int32_t n, grid_end;
};

__global__ void __launch_bounds__(kEncThreads, 1)
sae_stream_multi_kernel(const uint16_t* __restrict__ h, int32_t d, int32_t n_nt, EncApps apps,
                        const int32_t* __restrict__ r_req, const int32_t* __restrict__ r_tvalid,
                        const uint32_t* __restrict__ r_sub, int32_t r_Rmax, int32_t r_Tmax,
                        int32_t r_napps, uint32_t* __restrict__ r_mask,
                        int32_t* __restrict__ r_count, int32_t* __restrict__ r_lists,
                        uint32_t* __restrict__ r_err) {
    const int g = blockIdx.x;
    int i = 0;
    for (int j = 1; j < apps.n; ++j) i = g >= apps.a[j].grid0 ? j : i;  // uniform
    const EncApp& a = apps.a[i];
    stream_tile(g - a.grid0, g, h, d, a.app_count, a.tok_list, a.W, a.c_fold, a.n_mt, n_nt, a.z,
                a.lo_cnt, a.cap, a.cand, a.tile_cnt, a.tile_tau, r_req, r_tvalid, r_sub, r_Rmax,
                r_Tmax, r_napps, a.bit, r_mask, r_count, r_lists, r_err);
}

// The same batch with few token tiles, on a persistent grid: workgroup w
// runs slices w, w + G, w + 2G, ... of the apps' slices laid end to end (G
// the grid, at most one workgroup per CU), each over its app's live token
// tiles in turn, and skips the slices of an app without a token.  The
// routing inputs are staged once per workgroup, in LDS of their own; the
// dictionary stream runs on from one slice into the next, so the next
// slice's first chunks load while this one's candidates are selected.
__global__ void __launch_bounds__(kEncThreads, 1)
sae_stream_apps_kernel(const uint16_t* __restrict__ h, int32_t d, EncApps apps,
                       const int32_t* __restrict__ r_req, const int32_t* __restrict__ r_tvalid,
                       const uint32_t* __restrict__ r_sub, int32_t r_Rmax, int32_t r_Tmax,
                       int32_t r_napps, uint32_t* __restrict__ r_mask,
                       int32_t* __restrict__ r_count, int32_t* __restrict__ r_lists,
                       uint32_t* __restrict__ r_err) {
    __shared__ uint4 lds_main[kBN * kSelStride / 4];
    __shared__ int32_t list_s[kRouteMaxT];
    __shared__ int32_t rtot_s[kEncWaves];
    __shared__ int32_t stage_s[kRouteMaxT + kStageSubMax];
    __shared__ uint32_t bits_s;
    const int tid = threadIdx.x, lane = tid & 63;
    const int own = blockIdx.x, G = gridDim.x, U = apps.grid_end;

    // the batch's apps with at least one token (bit i for apps.a[i])
    uint32_t live = 0;
    int32_t* req_s = stage_s;
    uint32_t* sub_s = reinterpret_cast<uint32_t*>(stage_s + kRouteMaxT);
    int32_t tv = 0;
    uint32_t keep = 0;
    if (r_req) {  // uniform
        if (tid == 0) bits_s = 0u;
        stage_route<kEncThreads>(r_req, r_Tmax, r_sub, r_Rmax, req_s, sub_s);
        uint32_t err = 0;
        tv = clamp_t_valid(*r_tvalid, r_Tmax, err);
        keep = r_napps >= 32 ? 0xFFFFFFFFu : ((1u << r_napps) - 1u);
        __syncthreads();  // the staged inputs
        // every app bit some token slot carries
        uint32_t any = 0u;
        for (int32_t t = tid; t < r_Tmax; t += kEncThreads)
            any |= slot_mask_staged(req_s, t, tv, sub_s, r_sub, r_Rmax, keep, err);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) any |= __shfl_xor(any, off, kWave);
        if (lane == 0 && any != 0u) atomicOr(&bits_s, any);
        if (own < r_napps) {
            const int32_t n = build_token_list<kEncThreads>(
                req_s, tv, sub_s, r_sub, r_Rmax, keep, own, r_Tmax, list_s, rtot_s,
                own == 0 ? r_mask : nullptr, err);
            publish_token_list<kEncThreads>(list_s, n, r_Tmax,
                                            r_lists + static_cast<int64_t>(own) * r_Tmax,
                                            r_count + own);
        }
        if (own == 0) publish_error(err, r_err);
        __syncthreads();  // bits_s complete; list_s free
        const uint32_t bits = bits_s;
        for (int i = 0; i < apps.n; ++i) live |= ((bits >> apps.a[i].bit) & 1u) << i;
    } else {
        for (int i = 0; i < apps.n; ++i) live |= (*apps.a[i].app_count > 0 ? 1u : 0u) << i;
    }

    auto app_of = [&](int u) {
        int i = 0;
        for (int j = 1; j < apps.n; ++j) i = u >= apps.a[j].grid0 ? j : i;
        return i;
    };
    // the first of u, u + G, ... whose app has a token (U if none)
    auto live_from = [&](int u) {
        for (; u < U; u += G)
            if ((live >> app_of(u)) & 1u) break;
        return u;
    };
    int u = live_from(own);
    if (u >= U) return;  // uniform
    int i = app_of(u);
    int mt = u - apps.a[i].grid0;
    SliceSrc src = slice_src(apps.a[i].W, apps.a[i].n_mt, mt);
    uint4 wa0[4], wa1[4], wa2[4], wa3[4];
    float cfv[16];
    load_chunk(wa0, src.base);
    load_chunk(wa1, src.base + src.stride);
    load_chunk(wa2, src.base + 2 * src.stride);
    load_bias(cfv, apps.a[i].c_fold, mt);
    int list_app = -1, cnt = 0;
    const int32_t* tl = nullptr;
    for (;;) {
        const EncApp& a = apps.a[i];
        if (i != list_app) {  // uniform
            if (r_req) {
                uint32_t e = 0;
                cnt = build_token_list<kEncThreads>(req_s, tv, sub_s, r_sub, r_Rmax, keep, a.bit,
                                                    r_Tmax, list_s, rtot_s, nullptr, e);
                tl = list_s;
            } else {
                cnt = *a.app_count;
                tl = a.tok_list;
            }
            list_app = i;
        }
        const int un = live_from(u + G);
        const bool has_nxt = un < U;
        const int in = has_nxt ? app_of(un) : i;
        const int mtn = has_nxt ? un - apps.a[in].grid0 : mt;
        const SliceSrc nsrc = has_nxt ? slice_src(apps.a[in].W, apps.a[in].n_mt, mtn) : src;
        const SliceSink sink{a.cand, a.tile_cnt, a.tile_tau, a.n_mt, a.lo_cnt, a.cap, a.z};
        slice_tiles(lds_main, h, d, tl, cnt, 0, true, mt, src, sink, true, nsrc, has_nxt, mtn,
                    apps.a[in].c_fold, a.c_fold, wa0, wa1, wa2, wa3, cfv);
        if (!has_nxt) return;
        __syncthreads();  // the tile rows and list_s are read before they are rewritten
        u = un;
        i = in;
        mt = mtn;
        src = nsrc;
    }
}

// ------------------------------------------ prefill GEMM + candidate emission
// Many subscribed tokens make the encode MFMA-bound.  The token rows are
// first gathered into a staged layout (sae_xstage_kernel): plane j holds
// elements [32j, 32j+32) of every listed token, 64 contiguous bytes per
// token, zero past the subscribed count.  sae_gemm_kernel then runs 4 waves
// (one per SIMD) on a 256-latent x 256-token tile, each wave a 128 x 128
// quarter held in 256 accumulator registers.  Both operands of each K
// stage of 32 (a 16 KB dictionary half chunk, 2 KB contiguous per 32
// latents, and a 16 KB token plane slice) are copied by the load unit
// straight into LDS (global_load_lds, no register staging) into a ring of
// 4 stages.  Per pair of stages a wave waits for its own copies of the
// pair, meets the others at a barrier, refills the pair of buffers freed by
// the previous step, and runs 64 MFMAs whose operands come from LDS; the
// operands of the last step are read before the next barrier and
// multiplied after it, so the matrix unit has work while the waves meet.  The epilogue is the same threshold emission as the decode kernel,
// per token over the tile's 256 latents.
constexpr int kGemmThreads = 256;
constexpr int kGemmTok = 256;       // tokens per tile
constexpr int kStagePieces = 1024;  // 16-byte pieces per operand per stage
constexpr int kPrefillMinT = 1025;  // token slots from which the prefill GEMM runs
constexpr int kGBlkTok = 8;         // XCD block: token tiles
constexpr int kGBlkLat = 4;         // XCD block: latent tiles

// Stage-plane LDS swizzle: the 16-byte piece c of token n sits at
// n*4 + (c ^ gsw(n)); with it the MFMA-layout reads of 16 tokens x 4
// pieces hit distinct banks.
__device__ __forceinline__ int gsw(int n) { return ((n >> 3) ^ (n >> 4)) & 3; }

// Word 3 of a raw buffer resource (32-bit element format, no swizzle).
constexpr int kBufferDword3 = 0x00020000;

// s_waitcnt: at most n vector-memory operations of this wave outstanding
// and no LDS operation.
#define XMIX_WAIT_VM_LGKM0(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 15) | (7 << 4) | (((n) >> 4) << 14))

__global__ void __launch_bounds__(256)
sae_xstage_kernel(const uint16_t* __restrict__ h, int32_t d, const int32_t* __restrict__ app_count,
                  const int32_t* __restrict__ tok_list, int32_t n_pad, uint16_t* __restrict__ xs) {
    // one 16-byte piece per thread, output order (plane, token, piece)
    const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    const int64_t total = static_cast<int64_t>(n_pad) * (d / 8);
    if (q >= total) return;
    const int32_t c = static_cast<int32_t>(q & 3);
    const int64_t jn = q >> 2;
    const int32_t n = static_cast<int32_t>(jn % n_pad);
    const int32_t j = static_cast<int32_t>(jn / n_pad);
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (n < *app_count)
        v = *reinterpret_cast<const uint4*>(h + static_cast<int64_t>(tok_list[n]) * d + 32 * j + 8 * c);
    reinterpret_cast<uint4*>(xs)[q] = v;
}

__global__ void __launch_bounds__(kGemmThreads, 1)
sae_gemm_kernel(const uint16_t* __restrict__ xs_g, int32_t d, int32_t n_pad,
                const int32_t* __restrict__ app_count, const uint16_t* __restrict__ W,
                const float* __restrict__ c_fold, int32_t n_mt, int32_t n_nt, float z_guess,
                int32_t lo_cnt, int32_t cap, uint2* __restrict__ cand,
                int32_t* __restrict__ tile_cnt, float* __restrict__ tile_tau) {
    __shared__ uint4 wsA[kStagePieces], wsB[kStagePieces], wsC[kStagePieces], wsD[kStagePieces];
    __shared__ uint4 xsA[kStagePieces], xsB[kStagePieces], xsC[kStagePieces], xsD[kStagePieces];
    __shared__ float red1[2][kGemmTok];
    __shared__ float red2[2][kGemmTok];
    __shared__ int cnt_s[kGemmTok];
    __shared__ int cnt2_s[2][kGemmTok];
    __shared__ float red3[2][kGemmTok];  // per-token maxima

    // Tile order: launch slot L runs on XCD L % 8, which owns the latent
    // tiles [x*M8, (x+1)*M8) and walks them in blocks of 8 token tiles x 4
    // latent tiles (32 consecutive slots, one per CU of the XCD), token
    // blocks fastest, so each stage of a block's operands is fetched into
    // the XCD's L2 once and read by 4 and 8 workgroups.
    const int L = blockIdx.x;
    const int xcd = L % 8, slot = L / 8;
    const int m8 = (n_mt + 7) / 8;
    const int nbt = (n_nt + kGBlkTok - 1) / kGBlkTok;
    const int b = slot / (kGBlkTok * kGBlkLat), p = slot % (kGBlkTok * kGBlkLat);
    const int bt = b % nbt, bl = b / nbt;
    const int lt = kGBlkLat * bl + p / kGBlkTok;
    const int nt = kGBlkTok * bt + p % kGBlkTok;
    if (nt >= n_nt || lt >= m8) return;
    const int mt = xcd * m8 + lt;
    if (mt >= n_mt) return;
    const int cnt = *app_count;
    const int n0 = nt * kGemmTok;
    if (n0 >= cnt) return;
    const int ntok = min(kGemmTok, cnt - n0);

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;  // latent half, token half
    const int g = lane >> 5, j32 = lane & 31;
    const int nS = d / 32;                    // stages, a multiple of 8

    const uint4* W4 = reinterpret_cast<const uint4*>(W);
    const uint4* X4 = reinterpret_cast<const uint4*>(xs_g);
    const int64_t wstride = static_cast<int64_t>(n_mt) * 2048;  // pieces per K chunk of 64
    const int64_t xplane = static_cast<int64_t>(n_pad) * 4;     // pieces per stage plane
    // copy sources, in pieces from the start of the stage's operand block
    // (lane-contiguous LDS destinations q*256 + wave*64 + lane)
    int wsrc[4], xsrc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int P = q * 256 + wave * 64 + lane;
        wsrc[q] = (P >> 7) * 256 + (P & 127);
        const int n = P >> 2;
        xsrc[q] = n * 4 + ((P & 3) ^ gsw(n));
    }
    W4 += static_cast<int64_t>(mt) * 2048;  // this tile's latent slice
    X4 += static_cast<int64_t>(n0) * 4;     // this tile's tokens
    // issue the 8 copies of stage j (past the end: the last stage again,
    // which keeps the loop free of branches that would split the schedule).
    // Each copy is a buffer load whose resource covers exactly the stage's
    // operand block (its base and size are scalar), so the per-lane offset is
    // a fixed 32-bit value and an offset outside the block would read zeros.
    auto copy_stage = [&](int j, uint4* wdst, uint4* xdst) __attribute__((always_inline)) {
        j = min(j, nS - 1);
        const int kc = j >> 1, hh = j & 1;
        const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint4*>(W4 + kc * wstride + hh * 128), 0, 2048 * 16, kBufferDword3);
        const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint4*>(X4 + j * xplane), 0, kStagePieces * 16, kBufferDword3);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                wr, (__attribute__((address_space(3))) void*)(wdst + q * 256 + wave * 64),
                16, static_cast<unsigned>(wsrc[q]) * 16u, 0, 0, 0);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                xr, (__attribute__((address_space(3))) void*)(xdst + q * 256 + wave * 64),
                16, static_cast<unsigned>(xsrc[q]) * 16u, 0, 0, 0);
    };

    // accumulators start at the folded bias of their latent:
    // acc[a][nb][r] holds latent 128*wm + 32*a + 8*(r/4) + 4*g + r%4
    f32x16_t acc[4][4];
    {
        const float* cf = c_fold + mt * 256 + 128 * wm + 4 * g;
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 c4 = *reinterpret_cast<const float4*>(cf + 32 * a + 8 * q);
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) {
                    acc[a][nb][4 * q + 0] = c4.x;
                    acc[a][nb][4 * q + 1] = c4.y;
                    acc[a][nb][4 * q + 2] = c4.z;
                    acc[a][nb][4 * q + 3] = c4.w;
                }
            }
    }

    uint4 FA[4], FB[4], PA[4], PB[4];
    auto read_step = [&](const uint4* wb, const uint4* xb, int s, uint4 (&A)[4], uint4 (&B)[4])
        __attribute__((always_inline)) {
#pragma unroll
        for (int a = 0; a < 4; ++a) A[a] = wb[(4 * wm + a) * 128 + s * 64 + lane];
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
            const int n = 128 * wn + 32 * nb + j32;
            B[nb] = xb[n * 4 + ((2 * s + g) ^ gsw(n))];
        }
    };
    auto mfma_step = [&](const uint4 (&A)[4], const uint4 (&B)[4]) __attribute__((always_inline)) {
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
                acc[a][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(A[a]),
                                                                     as_bf16x8(B[nb]), acc[a][nb],
                                                                     0, 0, 0);
    };
    // Two stages per barrier.  Wait for this wave's copies of stages j and
    // j + 1 and its LDS reads, then meet at the barrier: every copy of the
    // pair has landed and every wave is done with the pair before it, whose
    // buffers are refilled with stages j + 2 and j + 3 while this pair is
    // multiplied.  In each stage: read step 0, multiply the carried step,
    // read step 1 (carried on), multiply step 0.
    auto stage_pair = [&](int j, const uint4* w0, const uint4* x0, const uint4* w1,
                          const uint4* x1, uint4* wf0, uint4* xf0, uint4* wf1, uint4* xf1,
                          bool first) __attribute__((always_inline)) {
        XMIX_WAIT_VM_LGKM0(0);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        copy_stage(j + 2, wf0, xf0);
        read_step(w0, x0, 0, FA, FB);
        if (!first) mfma_step(PA, PB);
        read_step(w0, x0, 1, PA, PB);
        mfma_step(FA, FB);
        copy_stage(j + 3, wf1, xf1);
        read_step(w1, x1, 0, FA, FB);
        mfma_step(PA, PB);
        read_step(w1, x1, 1, PA, PB);
        mfma_step(FA, FB);
        // instruction order: first stage's step-0 reads; carried MFMAs with
        // the first refill between them; step-0 MFMAs with step-1 reads;
        // second stage's step-0 reads and the second refill between the
        // carried MFMAs; step-0 MFMAs with step-1 reads
        __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
        if (!first) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            }
        } else {
            __builtin_amdgcn_sched_group_barrier(0x020, 8, 0);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
    };

    copy_stage(0, wsA, xsA);
    copy_stage(1, wsB, xsB);
    stage_pair(0, wsA, xsA, wsB, xsB, wsC, xsC, wsD, xsD, true);
    stage_pair(2, wsC, xsC, wsD, xsD, wsA, xsA, wsB, xsB, false);
    for (int j = 4; j < nS; j += 4) {
        stage_pair(j + 0, wsA, xsA, wsB, xsB, wsC, xsC, wsD, xsD, false);
        stage_pair(j + 2, wsC, xsC, wsD, xsD, wsA, xsA, wsB, xsB, false);
    }
    mfma_step(PA, PB);
    // every wave's trailing copies have landed and its reads are done before
    // the stage buffers are reused below
    XMIX_WAIT_VM_LGKM0(0);
    __syncthreads();

    // ---------------------------------------------------------- epilogue
    // acc[a][nb][r] holds latent 128*wm + 32*a + 8*(r/4) + 4*g + r%4 of
    // token 128*wn + 32*nb + j32; lanes j32 and j32 + 32 of waves (0, wn)
    // and (1, wn) together hold the 256 latents of one token.  The four
    // token groups nb of a wave go through each phase together, so the
    // waves meet once for the statistics and twice per refinement round
    // (not once per group) and the groups' independent work fills the gaps
    // of a wave that has its SIMD to itself.  Each token's threshold follows
    // the same sequence of guesses as when its group is finished alone: the
    // rounds go on while any token of the tile is outside the window, and a
    // token inside it keeps its threshold.  The count pass keeps a bit mask
    // of the lane's values >= tau; for the emission a group's values are
    // parked in the wave's own part of the (now idle) stage buffers, so that
    // the few selected ones are fetched by index.
    cnt_s[tid] = 0;
    float* park[2] = {reinterpret_cast<float*>(wave == 0 ? wsA : wave == 1 ? wsB : wave == 2 ? wsC : wsD),
                      reinterpret_cast<float*>(wave == 0 ? xsA : wave == 1 ? xsB : wave == 2 ? xsC : xsD)};
    // park the values of group nb in buffer nb % 2 (16-byte groups,
    // lane-contiguous, so the stores are conflict-free)
    auto park_group = [&](int nb) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < 16; ++q)
            reinterpret_cast<float4*>(park[nb & 1])[q * 64 + lane] =
                make_float4(acc[q >> 2][nb][4 * (q & 3)], acc[q >> 2][nb][4 * (q & 3) + 1],
                            acc[q >> 2][nb][4 * (q & 3) + 2], acc[q >> 2][nb][4 * (q & 3) + 3]);
    };
    park_group(0);
    park_group(1);
    // mean and variance over the tile's 256 latents, per token, and the
    // largest value
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        float s1 = 0.0f, s2 = 0.0f, mx = -INFINITY;
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                s1 += acc[a][nb][r];
                s2 = fmaf(acc[a][nb][r], acc[a][nb][r], s2);
                mx = fmaxf(mx, acc[a][nb][r]);
            }
        s1 += __shfl_xor(s1, 32, kWave);
        s2 += __shfl_xor(s2, 32, kWave);
        mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
        if (g == 0) {
            red1[wm][128 * wn + 32 * nb + j32] = s1;
            red2[wm][128 * wn + 32 * nb + j32] = s2;
            red3[wm][128 * wn + 32 * nb + j32] = mx;
        }
    }
    __syncthreads();
    float tau[4], lo_b[4], hi_b[4], mxv[4];
    uint32_t m0[4], m1[4];  // bit i: value i >= tau (m1: value 32 + i)
    bool bad[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        const int n = 128 * wn + 32 * nb + j32;
        const float s1 = red1[0][n] + red1[1][n], s2 = red2[0][n] + red2[1][n];
        const float mu = s1 * (1.0f / 256.0f);
        const float sd = sqrtf(fmaxf(s2 * (1.0f / 256.0f) - mu * mu, 0.0f));
        const float mx = fmaxf(red3[0][n], red3[1][n]);
        mxv[nb] = mx;
        // a strong latent (above mean + 5 stdev, such as a feature clamped
        // high at an earlier layer) would lift the guess for its whole
        // slice: the guess leaves the slice's largest value out then (the
        // decode kernel leaves out every value above the cut; here a second
        // pass over the accumulators would not fit the register file)
        tau[nb] = mx > mu + kTrimZ * sd ? trimmed_guess(s1 - mx, s2 - mx * mx, kBM - 1, z_guess)
                                        : mu + z_guess * sd;
        lo_b[nb] = -INFINITY;
        hi_b[nb] = INFINITY;
        bad[nb] = false;
    }
    auto count_at = [&](int nb) __attribute__((always_inline)) {
        uint32_t b0 = 0, b1 = 0;
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            b0 |= (acc[i >> 4][nb][i & 15] >= tau[nb] ? 1u : 0u) << i;
            b1 |= (acc[2 + (i >> 4)][nb][i & 15] >= tau[nb] ? 1u : 0u) << i;
        }
        m0[nb] = b0;
        m1[nb] = b1;
        return __popc(b0) + __popc(b1);
    };
    // count(pre >= tau) per token; refine tau until lo_cnt <= count <= cap.
    // cnt2_s is written before the round's first barrier and read before its
    // second, so one buffer serves every round.
    bool gave_up = false;
    for (int it = 0; it < kRefineIters; ++it) {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
            const int c_lane = count_at(nb);
            const int c = c_lane + __shfl_xor(c_lane, 32, kWave);
            if (g == 0) cnt2_s[wm][128 * wn + 32 * nb + j32] = c;
        }
        __syncthreads();
        bool any_bad = false;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
            const int n = 128 * wn + 32 * nb + j32;
            const int cn = cnt2_s[0][n] + cnt2_s[1][n];
            bad[nb] = false;
            if (n < ntok) {
                if (cn > cap) {
                    lo_b[nb] = tau[nb];
                    bad[nb] = true;
                } else if (cn < lo_cnt) {
                    hi_b[nb] = tau[nb];
                    bad[nb] = true;
                }
            }
            if (bad[nb]) {
                if (isfinite(lo_b[nb]) && isfinite(hi_b[nb])) {
                    tau[nb] = 0.5f * (lo_b[nb] + hi_b[nb]);
                } else {
                    const float step = ldexpf(0.25f * (fabsf(tau[nb]) + 1.0f), it);
                    tau[nb] = isfinite(hi_b[nb]) ? tau[nb] - step : tau[nb] + step;
                }
            }
            any_bad = any_bad || bad[nb];
        }
        if (!__syncthreads_or(any_bad)) break;
        // out of rounds: a threshold whose count is known to be <= cap
        if (it == kRefineIters - 1) {
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
                if (bad[nb]) tau[nb] = hi_b[nb];
            gave_up = true;
        }
    }
    if (gave_up) {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) count_at(nb);
    }
    // emit every latent with pre >= tau: reserve the lane's slots with one
    // LDS atomic, then write one selected (value, latent) pair per round,
    // the value read back from where it was parked
    const int lat0 = mt * 256 + 128 * wm + 4 * g;
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        const int n = 128 * wn + 32 * nb + j32;
        const float* pk = park[nb & 1];
        uint32_t b0 = n < ntok ? m0[nb] : 0u, b1 = n < ntok ? m1[nb] : 0u;
        const int c = __popc(b0) + __popc(b1);
        int slot = 0;
        if (c > 0) slot = atomicAdd(&cnt_s[n], c);
        const int64_t row = static_cast<int64_t>(n0 + n) * n_mt + mt;
        uint2* dst = cand + row * cap;
        while (__builtin_amdgcn_read_exec() & wave_ballot((b0 | b1) != 0)) {
            if ((b0 | b1) != 0) {
                const int i = b0 ? __builtin_ctz(b0) : 32 + __builtin_ctz(b1);
                if (b0) b0 &= b0 - 1;
                else b1 &= b1 - 1;
                const float val = pk[((i >> 2) * 64 + lane) * 4 + (i & 3)];
                if (slot < cap)
                    dst[slot] = make_uint2(__float_as_uint(val),
                                           static_cast<uint32_t>(lat0 + 32 * (i >> 4) +
                                                                 8 * ((i >> 2) & 3) + (i & 3)));
                ++slot;
            }
        }
        // the slice's bound: tau, or with nothing at or above it the next
        // value above the slice's maximum (the tighter of the two)
        if (n < ntok && wm == 0 && g == 0)
            tile_tau[row] = mxv[nb] < tau[nb] ? key_f32(f32_key(mxv[nb]) + 1u) : tau[nb];
        // the wave's reads of this buffer precede these stores in its LDS queue
        if (nb < 2) park_group(nb + 2);
    }
    __syncthreads();
    if (tid < ntok) tile_cnt[static_cast<int64_t>(n0 + tid) * n_mt + mt] = min(cnt_s[tid], cap);
}

// ------------------------------------------------------------- final merge
// Keys are order-preserving integer images of the fp32 values and the
// selection order is (key descending, latent ascending).

// Makes this wave's LDS writes visible to its other lanes.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int wave_count(bool p) { return __popcll(wave_ballot(p)); }

// Selects the k best of the pool key[0..n) / idx[0..n) (this wave's LDS
// region, n <= 64 * R) and moves them to lanes 0..k-1 (returned in wk/wi,
// in pool order; other lanes get key 0).  The selection is
//   { i : key[i] > tau  or  (key[i] == tau and idx[i] <= cut) }
// with exactly k entries (requires n >= k); tau is returned.  The keys stay
// in registers for the whole selection; the latents are read from LDS only
// where needed (entries tied at tau, and the k taken).  tau is found by
// bisection on the key bits below the highest bit in which the pool's keys
// differ (counts are ballot popcounts), stopping as soon as the count hits k.
template <int R>
__device__ __forceinline__ void wave_select_take(const uint32_t* key, const int32_t* idx, int n,
                                                 int k, uint32_t* stage_k, int32_t* stage_i,
                                                 uint32_t* tau_out, uint32_t* wk, int32_t* wi) {
    const int lane = lane_id();
    uint32_t kr[R];
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = lane + kWave * r;
        kr[r] = i < n ? key[i] : 0u;  // real keys are >= 1; 0 never counts
        if (i < n) {
            kmin = min(kmin, kr[r]);
            kmax = max(kmax, kr[r]);
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        kmin = min(kmin, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmin), off, kWave)));
        kmax = max(kmax, static_cast<uint32_t>(__shfl_xor(static_cast<int>(kmax), off, kWave)));
    }
    // every key shares the bits of kmin above the highest differing bit, so
    // the k-th largest does too: start the bisection below it
    const uint32_t diff = kmin ^ kmax;
    const int top = diff ? 31 - __builtin_clz(diff) : -1;
    uint32_t tau = top < 31 ? (kmin & ~((2u << top) - 1u)) : 0u;
    if (top < 0) tau = kmin;
    bool exact = false;
    for (int bit = top; bit >= 0; --bit) {
        const uint32_t c = tau | (1u << bit);
        int ge = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) ge += wave_count(kr[r] >= c);
        if (ge >= k) {
            tau = c;
            if (ge == k) {  // the k best are exactly the keys >= c
                exact = true;
                break;
            }
        }
    }
    int32_t cut = 0x7FFFFFFF;
    if (!exact) {
        int gt = 0, eq = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            gt += wave_count(kr[r] > tau);
            eq += wave_count(kr[r] == tau);
        }
        const int need = k - gt;
        if (eq > need) {
            // smallest I with #{key == tau and idx <= I} >= need; the tied
            // latents are read from LDS, only in rounds that hold a tie
            int32_t lo = 0;
            for (int bit = 30; bit >= 0; --bit) {
                const int32_t probe = lo | ((1 << bit) - 1);
                int c = 0;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const bool tie = kr[r] == tau;
                    if (wave_ballot(tie)) c += wave_count(tie && idx[lane + kWave * r] <= probe);
                }
                if (c < need) lo |= (1 << bit);
            }
            cut = lo;
        }
    }
    // compact the selection to the front of the stage area
    int base = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = lane + kWave * r;
        bool take = i < n && kr[r] >= tau;
        const uint64_t cand = wave_ballot(take);
        if (cand) {
            int32_t ir = 0;
            if (take) ir = idx[i];
            take = take && (kr[r] > tau || ir <= cut);
            const uint64_t b = wave_ballot(take);
            if (take) {
                stage_k[base + lanes_below(b)] = kr[r];
                stage_i[base + lanes_below(b)] = ir;
            }
            base += __popcll(b);
        }
    }
    wave_sync();
    *tau_out = tau;
    *wk = lane < base ? stage_k[lane] : 0u;
    *wi = lane < base ? stage_i[lane] : 0x7FFFFFFF;
}

// Optional readback of the merged rows into a ring (same row format and
// head protocol as the readback compaction).
struct RingOut {
    uint8_t* slots;     // null: no readback
    uint64_t* head;     // [2]: head, ticket counter (zero between calls)
    int32_t capacity, row_bytes;
    const int32_t* req;
    int32_t layer_id, app_id;
};

// The workgroup's ticket; the last of the `cnt` workgroups that hold a token
// advances the head by `cnt` (each read the head before its ticket) and
// resets the counter.  Workgroups without a token take no ticket, so a step
// with no subscriber costs no atomics.  No fence before the ticket: the rows
// and the head are read by work ordered after the kernel, which its
// completion makes visible.
__device__ __forceinline__ void ring_ticket(const RingOut& ring, uint64_t h0, int cnt) {
    const uint64_t ticket = atomicAdd(reinterpret_cast<unsigned long long*>(&ring.head[1]), 1ull);
    if (ticket == static_cast<uint64_t>(cnt) - 1u) {
        __atomic_store_n(&ring.head[0], h0 + static_cast<uint64_t>(cnt), __ATOMIC_RELAXED);
        atomicExch(reinterpret_cast<unsigned long long*>(&ring.head[1]), 0ull);
    }
}

constexpr int kMergeThreads = 256;
constexpr int kMergeWaves = kMergeThreads / kWave;
constexpr int kMergeR = 32;                        // pool entries per lane
constexpr int kPoolMax = kMergeR * kWave;          // 2048
constexpr int kRepairR = 6;                        // repair pool entries per lane
constexpr int kRepairPool = kRepairR * kWave;      // 384 >= k + one slice
constexpr int kFloorRounds = 3;                    // pool refills above a raised floor

// Wave-wide scans and reductions on DPP lane moves (every lane active):
// within each row of 16 lanes, then across the four rows (row_bcast for the
// scan, lane reads for the reductions, whose results are uniform).
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_rows(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xF, false);
}
// inclusive prefix sum over the lanes: row_shr 1, 2, 4, 8 inside each row
// (a lane with no source adds 0), then row_bcast:15 adds row 0's total to
// row 1 and row 2's to row 3, and row_bcast:31 the total of rows 0-1 to
// rows 2 and 3
__device__ __forceinline__ int wave_incl_sum(int v) {
    v += dpp_rows<0x111, 0xF>(v);
    v += dpp_rows<0x112, 0xF>(v);
    v += dpp_rows<0x114, 0xF>(v);
    v += dpp_rows<0x118, 0xF>(v);
    v += dpp_rows<0x142, 0xA>(v);
    v += dpp_rows<0x143, 0xC>(v);
    return v;
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
    const uint32_t lo = static_cast<uint32_t>(dpp_i<CTRL>(static_cast<int>(v)));
    const uint32_t hi = static_cast<uint32_t>(dpp_i<CTRL>(static_cast<int>(v >> 32)));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(v), l);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(v >> 32), l);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}
template <bool MAX>
__device__ __forceinline__ uint32_t wave_minmax_u32(uint32_t v) {
    auto op = [](uint32_t a, uint32_t b) { return MAX ? max(a, b) : min(a, b); };
    v = op(v, static_cast<uint32_t>(dpp_i<kDppXor1>(static_cast<int>(v))));
    v = op(v, static_cast<uint32_t>(dpp_i<kDppXor2>(static_cast<int>(v))));
    v = op(v, static_cast<uint32_t>(dpp_i<kDppHalfMirror>(static_cast<int>(v))));
    v = op(v, static_cast<uint32_t>(dpp_i<kDppMirror>(static_cast<int>(v))));
    const int iv = static_cast<int>(v);
    return op(op(__builtin_amdgcn_readlane(iv, 0), __builtin_amdgcn_readlane(iv, 16)),
              op(__builtin_amdgcn_readlane(iv, 32), __builtin_amdgcn_readlane(iv, 48)));
}
template <bool MAX>
__device__ __forceinline__ uint64_t wave_minmax_u64(uint64_t v) {
    auto op = [](uint64_t a, uint64_t b) { return MAX ? max(a, b) : min(a, b); };
    v = op(v, dpp_u64<kDppXor1>(v));
    v = op(v, dpp_u64<kDppXor2>(v));
    v = op(v, dpp_u64<kDppHalfMirror>(v));
    v = op(v, dpp_u64<kDppMirror>(v));
    return op(op(readlane_u64(v, 0), readlane_u64(v, 16)),
              op(readlane_u64(v, 32), readlane_u64(v, 48)));
}

// The pre-activation without bias of latent 256*mt + threadIdx.x for one
// token: a plain fp32 dot product of the packed dictionary row with the
// token row, the whole workgroup computing the 256 latents of slice mt
// together.  The slice's K chunks of 64 (32 KB contiguous each in the
// packed layout) are read with coalesced 16-byte loads: thread tid reads
// pieces tid + 256 w (w = 0..7), elements 16 s + 8 g .. + 7 (s = tid >> 6,
// g = (tid >> 5) & 1) of latent 32 w + (tid & 31), and keeps one partial
// sum per latent; the 8 partials of a latent are added in a fixed order,
// in pairs across lanes and then through LDS (part: 4 * 256 floats).
__device__ __forceinline__ float slice_dot(const uint16_t* __restrict__ Wp,
                                           const uint16_t* __restrict__ hrow, int32_t mt,
                                           int32_t n_mt, int32_t d, float* part) {
    const int tid = threadIdx.x;
    const int sg = tid >> 5;  // 2 s + g
    const uint4* P = reinterpret_cast<const uint4*>(Wp) + static_cast<int64_t>(mt) * 2048 + tid;
    const int64_t stride = static_cast<int64_t>(n_mt) * 2048;  // pieces per K chunk
    const uint4* hr = reinterpret_cast<const uint4*>(hrow) + sg;
    float acc[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) acc[w] = 0.0f;
    const int nK = d / 64;
#pragma unroll 1
    for (int kc = 0; kc < nK; ++kc) {
        const uint4 hv = hr[kc * 8];
        uint4 wv[8];
#pragma unroll
        for (int w = 0; w < 8; ++w) wv[w] = P[kc * stride + w * 256];
        const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
        for (int w = 0; w < 8; ++w) {
            const uint32_t ww[4] = {wv[w].x, wv[w].y, wv[w].z, wv[w].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[w] = fmaf(lo_bf16(ww[e]), lo_bf16(hw[e]), acc[w]);
                acc[w] = fmaf(hi_bf16(ww[e]), hi_bf16(hw[e]), acc[w]);
            }
        }
    }
    // lanes r and r + 32 hold the two halves g of one latent's elements
    const int s = tid >> 6;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
        const float both = acc[w] + __shfl_xor(acc[w], 32, kWave);
        if ((tid & 32) == 0) part[s * kBM + 32 * w + (tid & 31)] = both;
    }
    __syncthreads();
    const float dot = (part[tid] + part[kBM + tid]) + (part[2 * kBM + tid] + part[3 * kBM + tid]);
    __syncthreads();  // part is free for the next slice
    return dot;
}

// One workgroup per subscribed token.  Every thread gathers the candidates
// of the slices it owns (count, threshold and the slice's pair block are
// loaded together, so the gather costs one memory round trip), a prefix
// over the workgroup places them in an LDS pool, the workgroup selects the
// k best of it (radix select) and wave 0 checks the certificate; a failed
// check is repaired by the whole workgroup; wave 0 then writes each winner
// at its rank.  When the candidates exceed the pool, the k-th best of the
// first kPoolMax of them is a lower bound of the k-th best of all: the pool
// is filled again with the candidates at or above it (a little below, so
// that a repair finds what it needs; when exact ties leave that value floor
// where it was, the k-th composite (value, latent) itself), up to
// kFloorRounds times.  n: the workgroup's slot of the app's token list.
__device__ __forceinline__ void merge_token(
    int n, const uint2* __restrict__ cand, const int32_t* __restrict__ tile_cnt,
    const float* __restrict__ tile_tau, int32_t n_mt, int32_t cap,
    const int32_t* __restrict__ app_count, const int32_t* __restrict__ tok_list, int32_t k,
    const uint16_t* __restrict__ h, int32_t d, const uint16_t* __restrict__ Wp,
    const float* __restrict__ c_fold, int32_t* __restrict__ idx_out,
    uint16_t* __restrict__ val_out, const RingOut& ring) {
    __shared__ uint32_t K[kPoolMax + kWave];
    __shared__ int32_t I[kPoolMax + kWave];
    __shared__ __align__(16) uint32_t K2[kWave];  // the selected k entries (k <= 64)
    __shared__ __align__(16) int32_t I2[kWave];
    __shared__ __align__(16) int hist_s[3][256];  // radix digit counts, 3 rounds in flight
    __shared__ float part_s[4 * kBM];  // partial sums of a slice recompute
    __shared__ uint64_t cmin_s[kMergeWaves], cmax_s[kMergeWaves];
    __shared__ int sel_n_s;
    __shared__ int scan_s[2][kMergeWaves];  // gather rounds alternate between the two
    __shared__ uint32_t tmax_s[2][kMergeWaves];
    __shared__ int pool_n_s;
    __shared__ uint32_t floor_s;
    __shared__ uint64_t rbest_s[kMergeWaves], kth_s;  // repair: next slice, k-th composite
    const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
    const int64_t row0 = static_cast<int64_t>(n) * n_mt;
    // The first round of the gather below does not depend on the token
    // count: its loads go out before the count is read (the slot's area
    // exists for every slot below T_max; a slot past the count leaves
    // without using them).
    const int last = cap / 2 - 1;
    uint4 v0[4];
    int c0 = 0;
    float tf0 = 0.0f;
    {
        const bool own = tid < n_mt;
        const int64_t row = row0 + (own ? tid : 0);
        const uint4* src = reinterpret_cast<const uint4*>(cand + row * cap);
#pragma unroll
        for (int u = 0; u < 4; ++u) v0[u] = src[min(u, last)];
        if (own) {
            c0 = tile_cnt[row];
            tf0 = tile_tau[row];
        }
    }
    // readback ring (optional): each workgroup with a token reads the head
    // before it takes a ticket; the one drawing the last ticket advances it.
    // Read with the loads above (after them, so that no wait for those
    // waits for this one); the head was last written by an earlier call.
    uint64_t h0 = 0;
    if (ring.slots && tid == 0) h0 = ring.head[0];
    const int32_t t = tok_list[n];
    const int cnt = *app_count;
    if (n >= cnt) return;  // uniform: no token, no ring row, no ticket

    // Gather: the candidates whose composite (key, ~latent) is >= floor, in
    // slice order, into the pool
    // (the first kPoolMax of them; the rest are counted only).  Returns their
    // number; tau_tiles receives the largest slice bound, and each
    // wave's smallest and largest pool composite go to cmin_s / cmax_s (read
    // after the caller's barrier, with the first radix histogram cleared).
    uint32_t tau_tiles = 0;
    auto gather = [&](uint64_t floor) __attribute__((always_inline)) {
        int total = 0;
        uint64_t cmn = ~0ull, cmx = 0ull;
        for (int t0 = 0; t0 < n_mt; t0 += kMergeThreads) {
            const int tl = t0 + tid;
            const bool own = tl < n_mt;
            const int64_t row = row0 + (own ? tl : 0);
            // count, threshold and the first 8 pairs of the slice, in one round
            // (a slice holds about 2-3 candidates; more are fetched below)
            const uint4* src = reinterpret_cast<const uint4*>(cand + row * cap);
            uint4 v[4];
            int c;
            uint32_t tk;
            if (t0 == 0 && floor == 0) {
#pragma unroll
                for (int u = 0; u < 4; ++u) v[u] = v0[u];
                c = c0;
                tk = own ? f32_key(tf0) : 0u;
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u) v[u] = src[min(u, last)];
                c = own ? tile_cnt[row] : 0;
                tk = own ? f32_key(tile_tau[row]) : 0u;
            }
            // with a floor, only the candidates at or above it are kept
            int kept = c;
            if (floor != 0) {  // uniform
                kept = 0;
                for (int q0 = 0; q0 < c; q0 += 8) {
                    uint4 x[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) x[u] = q0 == 0 ? v[u] : src[min(q0 / 2 + u, last)];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int q = q0 + 2 * u;
                        const uint64_t ca =
                            (static_cast<uint64_t>(f32_key(__uint_as_float(x[u].x))) << 32) |
                            ~x[u].y;
                        const uint64_t cb =
                            (static_cast<uint64_t>(f32_key(__uint_as_float(x[u].z))) << 32) |
                            ~x[u].w;
                        kept += (q < c && ca >= floor) ? 1 : 0;
                        kept += (q + 1 < c && cb >= floor) ? 1 : 0;
                    }
                }
            }
            // workgroup prefix of the kept counts (the slots of a round were
            // last read before the previous round's barrier)
            const int incl = wave_incl_sum(kept);
            const uint32_t tm = wave_minmax_u32<true>(tk);
            const int par = (t0 / kMergeThreads) & 1;
            if (lane == kWave - 1) scan_s[par][wave] = incl;
            if (lane == 0) tmax_s[par][wave] = tm;
            __syncthreads();
            int base = total, round = 0;
#pragma unroll
            for (int w = 0; w < kMergeWaves; ++w) {
                base += (w < wave) ? scan_s[par][w] : 0;
                round += scan_s[par][w];
                tau_tiles = max(tau_tiles, tmax_s[par][w]);
            }
            int pos = base + incl - kept;
            total += round;
            if (pos >= kPoolMax) continue;  // nothing of this slice fits
            // the entries of this slice, in order (the first kPoolMax overall)
            for (int q0 = 0; q0 < c; q0 += 8) {
                uint4 x[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) x[u] = q0 == 0 ? v[u] : src[min(q0 / 2 + u, last)];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int q = q0 + 2 * u;
                    const uint32_t ka = f32_key(__uint_as_float(x[u].x));
                    const uint32_t kb = f32_key(__uint_as_float(x[u].z));
                    if (q < c && ((static_cast<uint64_t>(ka) << 32) | ~x[u].y) >= floor) {
                        if (pos < kPoolMax) {
                            K[pos] = ka;
                            I[pos] = static_cast<int32_t>(x[u].y);
                            const uint64_t cc = (static_cast<uint64_t>(ka) << 32) | ~x[u].y;
                            cmn = min(cmn, cc);
                            cmx = max(cmx, cc);
                        }
                        ++pos;
                    }
                    if (q + 1 < c && ((static_cast<uint64_t>(kb) << 32) | ~x[u].w) >= floor) {
                        if (pos < kPoolMax) {
                            K[pos] = kb;
                            I[pos] = static_cast<int32_t>(x[u].w);
                            const uint64_t cc = (static_cast<uint64_t>(kb) << 32) | ~x[u].w;
                            cmn = min(cmn, cc);
                            cmx = max(cmx, cc);
                        }
                        ++pos;
                    }
                }
            }
        }
        cmn = wave_minmax_u64<false>(cmn);
        cmx = wave_minmax_u64<true>(cmx);
        if (lane == 0) {
            cmin_s[wave] = cmn;
            cmax_s[wave] = cmx;
        }
        hist_s[0][tid] = 0;
        return total;
    };

    // Radix select of the k-th best pool entry (entries 0 .. np - 1, np >= k)
    // by the whole workgroup.  An entry's rank is its 64-bit composite
    // (key, ~latent), so the order key descending, latent ascending has no
    // ties and exactly k entries lie at or above the k-th composite.
    // Starting at the 8-bit digit that holds the highest bit in which the
    // composites differ (from the gather's smallest and largest), each round
    // counts (LDS atomics) the digits of the entries that match the prefix
    // found so far, and every wave finds the digit that holds the k-th entry
    // from the same counts (one barrier per round; the three count buffers
    // rotate, so a buffer is cleared two barriers after its last read); the
    // rounds end as soon as that digit's whole bin is needed.  Returns the
    // prefix (the k best are the entries whose composite >> *shift_out is
    // >= prefix >> *shift_out).
    auto comp = [&](int i) __attribute__((always_inline)) {
        return (static_cast<uint64_t>(K[i]) << 32) | static_cast<uint32_t>(~I[i]);
    };
    auto radix_kth = [&](int np, int* shift_out) __attribute__((always_inline)) {
        uint64_t cmin = cmin_s[0], cmax = cmax_s[0];
#pragma unroll
        for (int w = 1; w < kMergeWaves; ++w) {
            cmin = min(cmin, cmin_s[w]);
            cmax = max(cmax, cmax_s[w]);
        }
        const uint64_t diff = cmin ^ cmax;
        int shift = diff ? ((63 - __clzll(static_cast<long long>(diff))) & ~7) : 0;
        // bits above the first digit are common to every entry
        uint64_t prefix = shift < 56 ? cmin & ~((1ull << (shift + 8)) - 1ull) : 0ull;
        int need = k;
        for (int round = 0;; ++round) {
            int* hc = hist_s[round % 3];
            const uint64_t hi = shift < 56 ? prefix >> (shift + 8) : 0ull;
            for (int i = tid; i < np; i += kMergeThreads) {
                const uint64_t c = comp(i);
                if (shift >= 56 || (c >> (shift + 8)) == hi)
                    atomicAdd(&hc[static_cast<int>(c >> shift) & 255], 1);
            }
            // for the next round; its last reads (two rounds ago) came
            // before the previous round's barrier
            hist_s[(round + 1) % 3][tid] = 0;
            __syncthreads();
            const int4 h4v = reinterpret_cast<const int4*>(hc)[lane];  // bins 4 lane .. + 3
            const int h4[4] = {h4v.x, h4v.y, h4v.z, h4v.w};
            const int ls = (h4[0] + h4[1]) + (h4[2] + h4[3]);
            const int incl = wave_incl_sum(ls);
            // entries in the bins of every higher lane
            int above = __builtin_amdgcn_readlane(incl, kWave - 1) - incl, dl = 0, gl = 0, hl = 0;
            bool found = false;
#pragma unroll
            for (int j = 3; j >= 0; --j) {
                if (above < need && need <= above + h4[j]) {
                    dl = 4 * lane + j;
                    gl = above;
                    hl = h4[j];
                    found = true;
                }
                above += h4[j];
            }
            // exactly one bin holds the need-th entry
            const uint64_t fb = wave_ballot(found);
            const int src = fb ? __ffsll(static_cast<long long>(fb)) - 1 : 0;
            const int D = __builtin_amdgcn_readlane(dl, src),
                      gt = __builtin_amdgcn_readlane(gl, src),
                      hb = __builtin_amdgcn_readlane(hl, src);
            need -= gt;
            prefix |= static_cast<uint64_t>(D) << shift;
            if (hb == need || shift == 0) break;  // uniform
            shift -= 8;
        }
        *shift_out = shift;
        return prefix;
    };

    // Gather, then selection of the k best of the pool (the pool itself is
    // left as it was: the repair below reads it).  While the candidates
    // overflow the pool, the k-th best of its first kPoolMax entries gives
    // the floor of a refill (one gather and one radix select serve every
    // round).
    uint32_t wk = 0;
    int32_t wi = 0x7FFFFFFF;
    uint64_t floor_c = 0;  // composite floor of the refills
    int total = 0;
    bool fits = false;
    for (int fr = 0;; ++fr) {
        total = gather(floor_c);
        __syncthreads();  // the pool is written
        const bool refill = total > kPoolMax && fr < kFloorRounds;  // uniform
        fits = total <= kPoolMax && total >= k;
        if (!refill && !fits) break;
        if (tid == 0) sel_n_s = 0;
        int shift;
        const uint64_t prefix = radix_kth(refill ? kPoolMax : total, &shift);
        if (refill) {
            // the k-th key is >= the prefix's key bits (the bits below its
            // last digit are zero); step a little below it, as the repair's
            // floor does
            const float fv = key_f32(static_cast<uint32_t>(prefix >> 32));
            uint64_t fl = static_cast<uint64_t>(f32_key(fv - fabsf(fv) * 0x1p-11f)) << 32;
            if (fl <= floor_c) {
                // no progress on the value (exact ties at the floor): the
                // k-th composite of the first kPoolMax itself, with exactly k
                // of them at or above it (the latent breaks the ties)
                fl = prefix;
                if (fl <= floor_c) {  // uniform: no progress at all
                    fits = false;
                    break;
                }
            }
            floor_c = fl;
            __syncthreads();  // every read of the pool is done
            continue;
        }
        const uint64_t cut = prefix >> shift;
        for (int i = tid; i < total; i += kMergeThreads) {
            const uint64_t c = comp(i);
            if ((c >> shift) >= cut) {
                const int pos = atomicAdd(&sel_n_s, 1);  // exactly k entries
                if (pos < kWave) {
                    K2[pos] = static_cast<uint32_t>(c >> 32);
                    I2[pos] = static_cast<int32_t>(~static_cast<uint32_t>(c));
                }
            }
        }
        __syncthreads();
        if (lane < k) {
            wk = K2[lane];
            wi = I2[lane];
        }
        break;
    }
    // every wave: the k-th key (the smallest of the selected) and whether
    // the selection stands (0), fails its certificate (1) or was not made (2)
    const uint32_t sel_tau = wave_minmax_u32<false>(lane < k ? wk : 0xFFFFFFFFu);
    const int fix = !fits ? 2 : (tau_tiles <= sel_tau ? 0 : 1);
    if (fix != 0) {  // uniform
        // Repair: whole slices are recomputed exactly (fp32 dot products,
        // the workgroup streaming each slice once).  A slice hides only
        // values below its threshold, none of them at a latent below its
        // first: that composite bound says whether it can hide a winner.
        // The pool is cut down to what can still reach the top k; then the
        // slices are redone in descending order of their bound, each one's
        // pool entries replaced by its recomputed values above the floor,
        // wave 0 keeping the k best (at most kRepairPool entries) and raising
        // the floor and the k-th composite; the first slice whose bound lies
        // at or below the k-th composite ends the repair, since no later one
        // can hold a winner.  So tied or crowded slices cost the slices that
        // hold the top k, not every slice.  When the pool misses candidates
        // (more than kPoolMax after the refills) or keeps too many entries,
        // every slice is redone from an empty pool.
        const uint16_t* hrow = h + static_cast<int64_t>(t) * d;
        // the k-th selected composite (0: no selection yet)
        uint64_t kth = fix == 1 ? wave_minmax_u64<false>(
                                      lane < k ? (static_cast<uint64_t>(wk) << 32) |
                                                     static_cast<uint32_t>(~wi)
                                               : ~0ull)
                                : 0ull;
        // pool entries of slice q leave the pool (wave 0; q < 0: none), the
        // others from `fl` up stay
        auto cut_pool = [&](int np, uint32_t fl, int q) __attribute__((always_inline)) {
            int out = 0;
            for (int b0 = 0; b0 < np; b0 += kWave) {
                const int i = b0 + lane;
                const uint32_t kk = i < np ? K[i] : 0u;
                const int32_t ii = i < np ? I[i] : 0;
                const bool keep = i < np && kk >= fl && ii / kBM != q;
                const uint64_t bal = wave_ballot(keep);
                wave_sync();  // this round's reads come before its writes
                if (keep) {
                    K[out + lanes_below(bal)] = kk;
                    I[out + lanes_below(bal)] = ii;
                }
                out += __popcll(bal);
            }
            wave_sync();
            return out;
        };
        bool all = total > kPoolMax;  // uniform: the pool misses candidates
        if (!all && wave == 0) {
            // with a selection, a little below its k-th value, so that a
            // value whose recomputed rounding differs from the GEMM's still
            // enters; without one, the whole pool
            uint32_t fl = 0u;
            if (fix == 1) {
                const float tv = key_f32(sel_tau);
                fl = f32_key(tv - fabsf(tv) * 0x1p-12f);
            }
            const int out = cut_pool(total, fl, -1);
            if (lane == 0) {
                pool_n_s = out;
                floor_s = fl;
            }
        }
        __syncthreads();
        if (!all && pool_n_s > kRepairPool - kBM) all = true;
        if (!all) {
            uint64_t prev = ~0ull;  // the slices with bounds below it are left
            for (;;) {
                uint64_t best = 0ull;
                for (int q = tid; q < n_mt; q += kMergeThreads) {
                    const uint32_t tk = f32_key(tile_tau[row0 + q]);
                    const uint64_t bq = tk == 0u ? 0ull
                                                 : (static_cast<uint64_t>(tk - 1u) << 32) |
                                                       static_cast<uint32_t>(~(q * kBM));
                    if (bq < prev) best = max(best, bq);
                }
                best = wave_minmax_u64<true>(best);
                if (lane == 0) rbest_s[wave] = best;
                __syncthreads();
                best = max(max(rbest_s[0], rbest_s[1]), max(rbest_s[2], rbest_s[3]));
                if (best <= kth) break;  // uniform: no slice left can hold a winner
                prev = best;
                const int32_t q = static_cast<int32_t>(~static_cast<uint32_t>(best)) / kBM;
                if (wave == 0) {
                    const int out = cut_pool(pool_n_s, 0u, q);
                    if (lane == 0) pool_n_s = out;
                }
                __syncthreads();
                const int32_t j = q * kBM + tid;
                const float dot = slice_dot(Wp, hrow, q, n_mt, d, part_s);
                const uint32_t key = f32_key(dot + c_fold[j]);
                if (key >= floor_s) {
                    const int pos = atomicAdd(&pool_n_s, 1);
                    K[pos] = key;
                    I[pos] = j;
                }
                __syncthreads();
                const int pn = pool_n_s;
                __syncthreads();  // every thread has read the pool size
                if (pn >= k) {
                    if (wave == 0) {
                        uint32_t tk, a;
                        int32_t b;
                        if (pn > k) {
                            wave_select_take<kRepairR>(K, I, pn, k, K + kPoolMax, I + kPoolMax,
                                                       &tk, &a, &b);
                            if (lane < k) {
                                K[lane] = a;
                                I[lane] = b;
                            }
                        } else {
                            a = lane < k ? K[lane] : 0xFFFFFFFFu;
                            b = lane < k ? I[lane] : 0;
                            tk = wave_minmax_u32<false>(a);
                        }
                        const uint64_t kc = wave_minmax_u64<false>(
                            lane < k ? (static_cast<uint64_t>(a) << 32) | static_cast<uint32_t>(~b)
                                     : ~0ull);
                        if (lane == 0) {
                            pool_n_s = k;
                            floor_s = max(floor_s, tk);
                            kth_s = kc;
                        }
                    }
                    __syncthreads();
                    kth = kth_s;
                }
            }
            // the pool holds the k best unless no slice was redone after the cut
            const int pn = pool_n_s;
            if (pn > k && wave == 0) {
                uint32_t tk, a;
                int32_t b;
                wave_select_take<kRepairR>(K, I, pn, k, K + kPoolMax, I + kPoolMax, &tk, &a, &b);
                if (lane < k) {
                    K[lane] = a;
                    I[lane] = b;
                }
            }
            all = pn < k;  // (rounding) redo every slice
        }
        if (all) {  // uniform
            __syncthreads();  // every thread has read the pool size
            if (tid == 0) {
                pool_n_s = 0;
                floor_s = 0u;
            }
            __syncthreads();
            for (int q = 0; q < n_mt; ++q) {
                const int32_t j = q * kBM + tid;
                const float dot = slice_dot(Wp, hrow, q, n_mt, d, part_s);
                const uint32_t key = f32_key(dot + c_fold[j]);
                if (key >= floor_s) {
                    const int pos = atomicAdd(&pool_n_s, 1);
                    K[pos] = key;
                    I[pos] = j;
                }
                __syncthreads();
                const int pn = pool_n_s;
                __syncthreads();  // every thread has read the pool size
                if (pn > k) {
                    if (wave == 0) {
                        uint32_t tk, a;
                        int32_t b;
                        wave_select_take<kRepairR>(K, I, pn, k, K + kPoolMax, I + kPoolMax, &tk,
                                                   &a, &b);
                        if (lane < k) {
                            K[lane] = a;
                            I[lane] = b;
                        }
                        if (lane == 0) {
                            pool_n_s = k;
                            floor_s = max(floor_s, tk);
                        }
                    }
                    __syncthreads();
                }
            }
        }
        if (wave == 0) {
            wk = lane < k ? K[lane] : 0u;
            wi = lane < k ? I[lane] : 0x7FFFFFFF;
        }
    }
    if (wave != 0) return;
    // write the k winners in the order (value desc, index asc): each lane
    // counts the winners that come before its own (the entries are
    // distinct), reading them back from LDS in broadcast
    if (lane < k) {
        K2[lane] = wk;
        I2[lane] = wi;
    }
    wave_sync();
    const uint64_t mine = (static_cast<uint64_t>(wk) << 32) | static_cast<uint32_t>(~wi);
    int rank = 0;
    for (int j = 0; j < k; ++j) {
        const uint64_t other = (static_cast<uint64_t>(K2[j]) << 32) | static_cast<uint32_t>(~I2[j]);
        rank += other > mine ? 1 : 0;
    }
    const uint16_t vb = f32_to_bf16_rne(fmaxf(key_f32(wk), 0.0f));
    if (lane < k) {
        const int64_t o = static_cast<int64_t>(t) * k + rank;
        idx_out[o] = wi;
        val_out[o] = vb;
    }
    if (ring.slots) {
        // ring row {token, request, layer, app} + idx[k] + val[k]; only the
        // last `capacity` rows of this call are written
        h0 = static_cast<uint64_t>(__shfl(static_cast<long long>(h0), 0, kWave));
        if (static_cast<int64_t>(n) >= static_cast<int64_t>(cnt) - ring.capacity) {
            uint8_t* row = ring.slots + static_cast<int64_t>((h0 + static_cast<uint64_t>(n)) %
                                                             static_cast<uint64_t>(ring.capacity)) *
                                            ring.row_bytes;
            // 16-bit stores: with k odd, every other row starts 2 bytes
            // past a 4-byte boundary
            uint16_t* row16 = reinterpret_cast<uint16_t*>(row);
            if (lane < 8) {
                const int f = lane >> 1;
                const uint32_t hdr = static_cast<uint32_t>(
                    f == 0 ? t : f == 1 ? ring.req[t] : f == 2 ? ring.layer_id : ring.app_id);
                row16[lane] = static_cast<uint16_t>((lane & 1) ? hdr >> 16 : hdr & 0xFFFFu);
            }
            if (lane < k) {
                const uint32_t iv = static_cast<uint32_t>(wi);
                row16[8 + 2 * rank] = static_cast<uint16_t>(iv & 0xFFFFu);
                row16[8 + 2 * rank + 1] = static_cast<uint16_t>(iv >> 16);
                row16[8 + 2 * k + rank] = vb;
            }
        }
        if (lane == 0) ring_ticket(ring, h0, cnt);
    }
}

__global__ void __launch_bounds__(kMergeThreads) __attribute__((amdgpu_waves_per_eu(4)))
sae_merge_kernel(const uint2* __restrict__ cand, const int32_t* __restrict__ tile_cnt,
                 const float* __restrict__ tile_tau, int32_t n_mt, int32_t cap,
                 const int32_t* __restrict__ app_count, const int32_t* __restrict__ tok_list,
                 int32_t k, const uint16_t* __restrict__ h, int32_t d,
                 const uint16_t* __restrict__ Wp, const float* __restrict__ c_fold,
                 int32_t* __restrict__ idx_out, uint16_t* __restrict__ val_out,
                 RingOut ring) {
    merge_token(blockIdx.x, cand, tile_cnt, tile_tau, n_mt, cap, app_count, tok_list, k, h, d,
                Wp, c_fold, idx_out, val_out, ring);
}

// One app's merge inputs and outputs in a batched launch.
struct MergeApp {
    const uint2* cand;
    const int32_t* tile_cnt;
    const float* tile_tau;
    const int32_t* app_count;
    const int32_t* tok_list;
    const uint16_t* Wp;
    const float* c_fold;
    int32_t* idx_out;
    uint16_t* val_out;
    RingOut ring;
    int32_t n_mt, cap, k;
};
struct MergeApps {
    MergeApp a[kMultiMax];
};

// The merges of a batch of apps on a persistent grid: the pairs (app, slot
// of its token list) of every app's listed tokens, app by app, are dealt to
// the workgroups in turn, so a slot past its app's count costs nothing (no
// workgroup, no gather) and an empty batch costs one read of the counts.
__global__ void __launch_bounds__(kMergeThreads) __attribute__((amdgpu_waves_per_eu(4)))
sae_merge_apps_kernel(const uint16_t* __restrict__ h, int32_t d, int32_t T_max, int32_t n_apps,
                      MergeApps apps) {
    __shared__ int32_t cnt_s[kMultiMax];
    for (int i = 0; i < n_apps; ++i)
        if (threadIdx.x == i) cnt_s[i] = min(max(*apps.a[i].app_count, 0), T_max);
    __syncthreads();
    int32_t start[kMultiMax + 1];
    start[0] = 0;
#pragma unroll
    for (int i = 0; i < kMultiMax; ++i) start[i + 1] = start[i] + (i < n_apps ? cnt_s[i] : 0);
    const int32_t P = start[kMultiMax];
    for (int32_t p = blockIdx.x; p < P; p += gridDim.x) {  // uniform
        int i = 0;
#pragma unroll
        for (int j = 1; j < kMultiMax; ++j) i = j < n_apps && p >= start[j] ? j : i;
        const MergeApp& a = apps.a[i];
        merge_token(p - start[i], a.cand, a.tile_cnt, a.tile_tau, a.n_mt, a.cap, a.app_count,
                    a.tok_list, a.k, h, d, a.Wp, a.c_fold, a.idx_out, a.val_out, a.ring);
        __syncthreads();  // the token's LDS is read before the next token's gather
    }
}

// ------------------------------------------------------------------ launch
static int enc_grid(int32_t n_mt, int32_t n_nt) {
    if (n_nt <= kLatentFastTiles) return n_mt;  // one workgroup per slice, tiles in turn
    const int m8 = (n_mt + 7) / 8;
    const int nbt = (n_nt + kBlkTok - 1) / kBlkTok;
    const int nbl = (m8 + kBlkLat - 1) / kBlkLat;
    return 8 * nbt * nbl * kBlkTok * kBlkLat;
}

// Candidate emission parameters for a dictionary of m latents and top-k:
// target emitted per tile (so that m/256 tiles together hold about twice
// the k needed, plus slack), the per-tile capacity, the lower count bound
// (non-zero only when few tiles must supply all k), and the standard normal
// quantile that aims the first threshold guess at the target.
struct EmitPlan {
    int target, cap, lo;
    float z;
};

static EmitPlan emit_plan(int32_t m, int32_t k) {
    const int n_mt = m / kBM;
    EmitPlan e;
    e.target = (2 * k * kBM + m - 1) / m + 1;
    e.target = e.target < 2 ? 2 : (e.target > 64 ? 64 : e.target);
    e.cap = 4 * e.target;
    e.cap = e.cap < 8 ? 8 : (e.cap > kMaxCap ? kMaxCap : e.cap);
    e.lo = (n_mt * e.target >= 4 * k) ? 0 : (k < e.cap ? k : e.cap);
    const double want = e.lo ? 0.5 * (e.lo + e.cap) : e.target;
    // upper-tail quantile: 0.5 * erfc(z / sqrt 2) = want / 256, by bisection
    const double f = want / kBM;
    double a = -8.0, b = 8.0;
    for (int i = 0; i < 100; ++i) {
        const double mid = 0.5 * (a + b);
        if (0.5 * erfc(mid / sqrt(2.0)) > f) a = mid;
        else b = mid;
    }
    e.z = static_cast<float>(0.5 * (a + b));
    return e;
}

struct CandArea {
    uint2* cand;   // (fp32 bits, latent) pairs, [T_max][n_mt][cap]
    int32_t* cnt;  // [T_max][n_mt]
    float* tau;    // [T_max][n_mt]
};

static CandArea cand_area(void* base, int32_t T_max, int32_t n_mt, int cap) {
    const size_t slots = static_cast<size_t>(T_max) * n_mt;
    CandArea a;
    a.cand = static_cast<uint2*>(base);
    a.cnt = reinterpret_cast<int32_t*>(a.cand + slots * cap);
    a.tau = reinterpret_cast<float*>(a.cnt + slots);
    return a;
}

static int32_t stage_tokens(int32_t T_max) {
    return (T_max + kGemmTok - 1) / kGemmTok * kGemmTok;
}

static size_t candidate_bytes(int32_t T_max, int32_t m, int32_t k) {
    const EmitPlan e = emit_plan(m, k);
    const size_t slots = static_cast<size_t>(T_max) * (m / kBM);
    return slots * (static_cast<size_t>(e.cap) * 8u + 8u);
}

size_t sae_candidate_bytes(int32_t T_max, int32_t d, int32_t m, int32_t k) {
    size_t bytes = (candidate_bytes(T_max, m, k) + 255u) / 256u * 256u;
    if (T_max >= kPrefillMinT)  // staged token rows of the prefill GEMM
        bytes += static_cast<size_t>(stage_tokens(T_max)) * d * sizeof(uint16_t);
    return bytes;
}

hipError_t launch_sae_pack(const uint16_t* W_enc, int32_t m, int32_t d, uint16_t* W_packed,
                           hipStream_t stream) {
    const int64_t pieces = static_cast<int64_t>(m) * (d / 8);
    hipLaunchKernelGGL(sae_pack_kernel, dim3(static_cast<uint32_t>((pieces + 255) / 256)),
                       dim3(256), 0, stream, W_enc, m, d, W_packed);
    return hipGetLastError();
}

hipError_t launch_sae_fold(const uint16_t* W_enc, const uint16_t* b_enc, const uint16_t* b_dec,
                           int32_t m, int32_t d, float* c_fold, hipStream_t stream) {
    hipLaunchKernelGGL(sae_fold_kernel, dim3((m + 3) / 4), dim3(256), 0, stream, W_enc, b_enc,
                       b_dec, m, d, c_fold);
    return hipGetLastError();
}

hipError_t launch_sae_candidates(const uint16_t* h, int32_t d, int32_t T_max,
                                 const int32_t* app_count, const int32_t* tok_list,
                                 const uint16_t* W_enc, const float* c_fold, int32_t m,
                                 int32_t k, void* cand, hipStream_t stream,
                                 const RouteIn* route) {
    const int32_t n_mt = m / kBM;
    const EmitPlan e = emit_plan(m, k);
    const CandArea a = cand_area(cand, T_max, n_mt, e.cap);
    // the decode kernel routes when the batch fits its LDS list and its grid
    // has a workgroup for every app to publish
    if (route && (T_max > kRouteMaxT ||
                  enc_grid(n_mt, (T_max + kBN - 1) / kBN) < route->n_apps)) {
        const hipError_t r = launch_route_build(route->req, route->T_valid, route->sub,
                                                route->R_max, T_max, route->n_apps,
                                                route->tok_mask, route->app_count,
                                                route->app_tokens, route->err_word, stream);
        if (r != hipSuccess) return r;
        route = nullptr;
    }
    if (T_max >= kPrefillMinT) {
        const int32_t n_pad = stage_tokens(T_max);
        uint16_t* xs = reinterpret_cast<uint16_t*>(
            static_cast<char*>(cand) + (candidate_bytes(T_max, m, k) + 255u) / 256u * 256u);
        const int64_t pieces = static_cast<int64_t>(n_pad) * (d / 8);
        hipLaunchKernelGGL(sae_xstage_kernel, dim3(static_cast<uint32_t>((pieces + 255) / 256)),
                           dim3(256), 0, stream, h, d, app_count, tok_list, n_pad, xs);
        const int32_t n_nt = n_pad / kGemmTok;
        const int m8 = (n_mt + 7) / 8;
        const int nbt = (n_nt + kGBlkTok - 1) / kGBlkTok;
        const int nbl = (m8 + kGBlkLat - 1) / kGBlkLat;
        hipLaunchKernelGGL(sae_gemm_kernel, dim3(8 * nbt * nbl * kGBlkTok * kGBlkLat),
                           dim3(kGemmThreads), 0, stream, xs, d, n_pad, app_count, W_enc, c_fold,
                           n_mt, n_nt, e.z, e.lo, e.cap, a.cand, a.cnt, a.tau);
        return hipGetLastError();
    }
    const int32_t n_nt = (T_max + kBN - 1) / kBN;
    const RouteIn none{};
    const RouteIn& ri = route ? *route : none;
    hipLaunchKernelGGL(sae_stream_kernel, dim3(enc_grid(n_mt, n_nt)), dim3(kEncThreads), 0,
                       stream, h, d, app_count, tok_list, W_enc, c_fold, n_mt, n_nt, e.z, e.lo,
                       e.cap, a.cand, a.cnt, a.tau, ri.req, ri.T_valid, ri.sub, ri.R_max, T_max,
                       ri.n_apps, ri.app_bit, ri.tok_mask, ri.app_count, ri.app_tokens,
                       ri.err_word);
    return hipGetLastError();
}

hipError_t launch_sae_merge(const uint16_t* h, int32_t d, int32_t T_max,
                            const int32_t* app_count, const int32_t* tok_list,
                            const uint16_t* W_enc, const float* c_fold, int32_t m, int32_t k,
                            int32_t* idx_out, uint16_t* val_out, void* cand,
                            const MergeRing* ring, hipStream_t stream) {
    const int32_t n_mt = m / kBM;
    const EmitPlan e = emit_plan(m, k);
    const CandArea a = cand_area(cand, T_max, n_mt, e.cap);
    RingOut r{};
    if (ring) {
        r.slots = ring->slots;
        r.head = ring->head;
        r.capacity = ring->capacity;
        r.row_bytes = ring->row_bytes;
        r.req = ring->req;
        r.layer_id = ring->layer_id;
        r.app_id = ring->app_id;
    }
    hipLaunchKernelGGL(sae_merge_kernel, dim3(T_max), dim3(kMergeThreads), 0, stream, a.cand,
                       a.cnt, a.tau, n_mt, e.cap, app_count, tok_list, k, h, d, W_enc,
                       c_fold, idx_out, val_out, r);
    return hipGetLastError();
}

bool sae_multi_supported(int32_t T_max) { return T_max < kPrefillMinT; }

// CUs of the current device (256 if the query fails), looked up once per device.
static int32_t cu_count() {
    constexpr int kDevs = 64;
    static std::atomic<int32_t> cache[kDevs];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevs) return 256;
    int32_t n = cache[dev].load(std::memory_order_relaxed);
    if (n <= 0) {
        int v = 0;
        n = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                    v > 0
                ? v
                : 256;
        cache[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

hipError_t launch_sae_encode_multi(const uint16_t* h, int32_t d, int32_t T_max, int32_t n,
                                   const SaeAppIn* apps, hipStream_t stream,
                                   const RouteIn* route) {
    const int32_t n_nt = (T_max + kBN - 1) / kBN;
    for (int32_t c0 = 0; c0 < n; c0 += kMultiMax) {
        const int32_t nc = n - c0 < kMultiMax ? n - c0 : kMultiMax;
        EncApps ea;
        MergeApps ma;
        memset(&ea, 0, sizeof(ea));
        memset(&ma, 0, sizeof(ma));
        int32_t grid = 0;
        for (int32_t i = 0; i < nc; ++i) {
            const SaeAppIn& in = apps[c0 + i];
            const int32_t n_mt = in.m / kBM;
            const EmitPlan e = emit_plan(in.m, in.k);
            const CandArea a = cand_area(in.cand, T_max, n_mt, e.cap);
            ea.a[i] = EncApp{in.app_count, in.tok_list, in.W, in.c_fold, a.cand, a.cnt, a.tau,
                             n_mt, e.lo, e.cap, in.bit, grid, e.z};
            grid += enc_grid(n_mt, n_nt);
            RingOut r{};
            if (in.ring) {
                r.slots = in.ring->slots;
                r.head = in.ring->head;
                r.capacity = in.ring->capacity;
                r.row_bytes = in.ring->row_bytes;
                r.req = in.ring->req;
                r.layer_id = in.ring->layer_id;
                r.app_id = in.ring->app_id;
            }
            ma.a[i] = MergeApp{a.cand, a.cnt, a.tau, in.app_count, in.tok_list, in.W, in.c_fold,
                               in.idx_out, in.val_out, r, n_mt, e.cap, in.k};
        }
        ea.n = nc;
        ea.grid_end = grid;
        // the first launch builds the routing when the batch fits its LDS list
        // and its grid has a workgroup for every app to publish
        const RouteIn* ri = c0 == 0 ? route : nullptr;
        if (ri && (T_max > kRouteMaxT || grid < ri->n_apps)) {
            const hipError_t r = launch_route_build(ri->req, ri->T_valid, ri->sub, ri->R_max,
                                                    T_max, ri->n_apps, ri->tok_mask,
                                                    ri->app_count, ri->app_tokens,
                                                    ri->err_word, stream);
            if (r != hipSuccess) return r;
            ri = nullptr;
        }
        const RouteIn none{};
        const RouteIn& rr = ri ? *ri : none;
        if (n_nt <= kLatentFastTiles) {
            // persistent: one workgroup per CU (and one per app to publish)
            int32_t g = grid < cu_count() ? grid : cu_count();
            if (ri && g < ri->n_apps) g = ri->n_apps;
            hipLaunchKernelGGL(sae_stream_apps_kernel, dim3(g), dim3(kEncThreads), 0, stream, h,
                               d, ea, rr.req, rr.T_valid, rr.sub, rr.R_max, T_max, rr.n_apps,
                               rr.tok_mask, rr.app_count, rr.app_tokens, rr.err_word);
        } else {
            hipLaunchKernelGGL(sae_stream_multi_kernel, dim3(grid), dim3(kEncThreads), 0, stream,
                               h, d, n_nt, ea, rr.req, rr.T_valid, rr.sub, rr.R_max, T_max,
                               rr.n_apps, rr.tok_mask, rr.app_count, rr.app_tokens, rr.err_word);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        // persistent merges: up to four workgroups per CU
        const int32_t mg = nc * T_max < 4 * cu_count() ? nc * T_max : 4 * cu_count();
        hipLaunchKernelGGL(sae_merge_apps_kernel, dim3(mg), dim3(kMergeThreads), 0, stream, h, d,
                           T_max, nc, ma);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Where the by-value descriptors hold device pointers (for the graph
// executor's redirection).
template <>
struct ArgPointers<RingOut> {
    static std::vector<uint16_t> offsets() {
        return {offsetof(RingOut, slots), offsetof(RingOut, head), offsetof(RingOut, req)};
    }
};
template <>
struct ArgPointers<EncApps> {
    static std::vector<uint16_t> offsets() {
        std::vector<uint16_t> o;
        for (int i = 0; i < kMultiMax; ++i)
            for (const size_t f : {offsetof(EncApp, app_count), offsetof(EncApp, tok_list),
                                   offsetof(EncApp, W), offsetof(EncApp, c_fold),
                                   offsetof(EncApp, cand), offsetof(EncApp, tile_cnt),
                                   offsetof(EncApp, tile_tau)})
                o.push_back(static_cast<uint16_t>(offsetof(EncApps, a) + i * sizeof(EncApp) + f));
        return o;
    }
};
template <>
struct ArgPointers<MergeApps> {
    static std::vector<uint16_t> offsets() {
        std::vector<uint16_t> o;
        for (int i = 0; i < kMultiMax; ++i) {
            const size_t b = offsetof(MergeApps, a) + i * sizeof(MergeApp);
            for (const size_t f : {offsetof(MergeApp, cand), offsetof(MergeApp, tile_cnt),
                                   offsetof(MergeApp, tile_tau), offsetof(MergeApp, app_count),
                                   offsetof(MergeApp, tok_list), offsetof(MergeApp, Wp),
                                   offsetof(MergeApp, c_fold), offsetof(MergeApp, idx_out),
                                   offsetof(MergeApp, val_out)})
                o.push_back(static_cast<uint16_t>(b + f));
            for (const uint16_t f : ArgPointers<RingOut>::offsets())
                o.push_back(static_cast<uint16_t>(b + offsetof(MergeApp, ring) + f));
        }
        return o;
    }
};

void add_sae_kernels(std::vector<KernelInfo>& t) {
    t.push_back(kernel_info(sae_pack_kernel));
    t.push_back(kernel_info(sae_fold_kernel));
    t.push_back(kernel_info(sae_stream_kernel));
    t.push_back(kernel_info(sae_xstage_kernel));
    t.push_back(kernel_info(sae_gemm_kernel));
    t.push_back(kernel_info(sae_merge_kernel));
    t.push_back(kernel_info(sae_stream_multi_kernel));
    t.push_back(kernel_info(sae_merge_apps_kernel));
    t.push_back(kernel_info(sae_stream_apps_kernel));
}

}  // namespace xmix
