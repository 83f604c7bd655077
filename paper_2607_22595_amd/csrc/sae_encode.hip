// SAE encode with TopK: pre = W_enc . h + c_fold for the tokens subscribed
// to one app, then the k largest pre-activations per token.
//
// Stage 1 (sae_stream_topk_kernel) is an MFMA bf16 GEMM with fp32
// accumulation.  A workgroup owns 256 latents x 128 subscribed tokens and
// walks K = d in chunks of 64:
//   - the W_enc rows (operand A) stream from HBM straight into registers,
//     each wave owning 64 latents, with a three-deep register ring so two
//     chunks are in flight while one is multiplied;
//   - the token rows (operand B) are gathered through the app's token list
//     into LDS (double buffered, 16-byte chunks XOR-swizzled by row so the
//     MFMA-layout reads are conflict-free) and shared by the four waves.
// The epilogue adds the folded bias, stages 32 tokens at a time in LDS and
// lets each wave pick, per token, the local top-k of its 256 latents with a
// 32-step bisection on order-preserving integer keys (ballot counts; equal
// keys are taken in ascending latent order).  Candidates go to the
// workspace as (fp32 pre, latent index).
//
// Stage 2 (sae_merge_kernel): one workgroup per subscribed token selects the
// exact top-k among the (m / 256) * k candidates with the same bisection over
// the whole workgroup, breaks remaining ties by latent index, ranks the k
// winners by (value desc, index asc) and writes idx / bf16(ReLU(pre)).
//
// The workgroup-to-tile map is XCD-aware: launch slots are dealt round-robin
// to the 8 XCDs, so consecutive tiles of one XCD share a W_enc slice in that
// XCD's L2.
#include "common.hpp"
#include "launch.hpp"

namespace xmix {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

constexpr int kBM = 256;  // latents per workgroup
constexpr int kBN = 128;  // tokens per workgroup
constexpr int kBK = 64;   // K chunk
constexpr int kEncThreads = 256;
constexpr int kMergeThreads = 256;
constexpr int kMaxCPT = 64;  // merge candidates per thread
constexpr int kMaxTopK = 64;

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) {
    return __builtin_bit_cast(bf16x8_t, v);
}

// ---------------------------------------------------------------- bias fold
// c_fold[j] = b_enc[j] - W_enc[j,:] . b_dec, one wave per latent.
__global__ void __launch_bounds__(256)
sae_fold_kernel(const uint16_t* __restrict__ W, const uint16_t* __restrict__ b_enc,
                const uint16_t* __restrict__ b_dec, int32_t m, int32_t d,
                float* __restrict__ c_fold) {
    const int32_t j = blockIdx.x * 4 + threadIdx.x / kWave;
    if (j >= m) return;
    const uint4* row = reinterpret_cast<const uint4*>(W + static_cast<int64_t>(j) * d);
    const uint4* bd = reinterpret_cast<const uint4*>(b_dec);
    float acc = 0.0f;
    for (int32_t i = lane_id(); i < d / 8; i += kWave) {
        const uint4 wv = row[i], bv = bd[i];
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

// ------------------------------------------------------ GEMM + local top-k
__global__ void __launch_bounds__(kEncThreads, 1)
sae_stream_topk_kernel(const uint16_t* __restrict__ h, int32_t d,
                       const int32_t* __restrict__ app_count,
                       const int32_t* __restrict__ tok_list, const uint16_t* __restrict__ W,
                       const float* __restrict__ c_fold, int32_t k, int32_t n_mt, int32_t n_nt,
                       float* __restrict__ cand_val, int32_t* __restrict__ cand_idx) {
    __shared__ uint4 xs[2][kBN * 8];         // 2 x 16 KiB
    __shared__ float pre[32][kBM + 1];       // one 32-token pass of the epilogue

    // XCD-aware tile order: slot L runs on XCD L % 8; give each XCD a
    // contiguous range of tiles, token tile fastest.
    const int L = blockIdx.x;
    const int per_xcd = gridDim.x / 8;
    const int u = (L % 8) * per_xcd + (L / 8);
    const int nt = u % n_nt;
    const int mt = u / n_nt;
    if (mt >= n_mt) return;
    const int cnt = *app_count;
    const int n0 = nt * kBN;
    if (n0 >= cnt) return;
    const int ntok = min(kBN, cnt - n0);

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 5, i32 = lane & 31;

    // operand A: rows of W_enc, 64 contiguous bytes of each row per chunk
    const uint16_t* wp0 = W + static_cast<int64_t>(mt * kBM + 64 * wave + i32) * d + 32 * g;
    const uint16_t* wp1 = wp0 + static_cast<int64_t>(32) * d;

    // operand B: gathered token rows; padding rows read a valid row and zero it
    const int xr = tid >> 3, xc = tid & 7;
    const uint16_t* xrow[4];
    bool xok[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const int n = xr + 32 * p;
        xok[p] = n < ntok;
        const int32_t tok = tok_list[n0 + (xok[p] ? n : 0)];
        xrow[p] = h + static_cast<int64_t>(tok) * d + 8 * xc;
    }

    f32x16_t acc[2][4];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

    uint4 wa0[8], wa1[8], wa2[8];
    uint4 xv[4];
    const int nK = d / kBK;

    auto load_w = [&](uint4 (&a)[8], int kc) {
        const uint4* p0 = reinterpret_cast<const uint4*>(wp0 + kc * kBK);
        const uint4* p1 = reinterpret_cast<const uint4*>(wp1 + kc * kBK);
#pragma unroll
        for (int s = 0; s < 4; ++s) a[s] = p0[s];
#pragma unroll
        for (int s = 0; s < 4; ++s) a[4 + s] = p1[s];
    };
    auto load_x = [&](int kc) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            uint4 v = *reinterpret_cast<const uint4*>(xrow[p] + kc * kBK);
            if (!xok[p]) v = make_uint4(0, 0, 0, 0);
            xv[p] = v;
        }
    };
    auto store_x = [&](int buf) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int n = xr + 32 * p;
            xs[buf][n * 8 + (xc ^ (n & 7))] = xv[p];
        }
    };
    auto compute = [&](const uint4 (&a)[8], int buf) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const bf16x8_t A0 = as_bf16x8(a[s]);
            const bf16x8_t A1 = as_bf16x8(a[4 + s]);
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int n = 32 * nb + i32;
                const int chunk = 4 * g + s;
                const bf16x8_t B = as_bf16x8(xs[buf][n * 8 + (chunk ^ (n & 7))]);
                acc[0][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A0, B, acc[0][nb], 0, 0, 0);
                acc[1][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A1, B, acc[1][nb], 0, 0, 0);
            }
        }
    };
    // One K chunk: issue the next token chunk and the W chunk two ahead,
    // multiply the current chunk, then publish the next token chunk.
    auto step = [&](int kc, const uint4 (&cur)[8], uint4 (&nxt)[8]) {
        if (kc + 1 < nK) load_x(kc + 1);
        if (kc + 2 < nK) load_w(nxt, kc + 2);
        __syncthreads();
        compute(cur, kc & 1);
        if (kc + 1 < nK) store_x((kc + 1) & 1);
    };

    load_x(0);
    load_w(wa0, 0);
    if (nK > 1) load_w(wa1, 1);
    store_x(0);
    for (int kc = 0; kc < nK; kc += 3) {
        step(kc, wa0, wa2);
        if (kc + 1 < nK) step(kc + 1, wa1, wa0);
        if (kc + 2 < nK) step(kc + 2, wa2, wa1);
    }

    // ---------------------------------------------------------- epilogue
    // acc[mb][nb][r] holds latent 64*wave + 32*mb + 8*(r/4) + 4*g + r%4 of
    // token 32*nb + i32 (the 32x32 MFMA output layout).
    const float* cf = c_fold + mt * kBM + 64 * wave + 4 * g;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float c = cf[32 * mb + 8 * (r / 4) + (r % 4)];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) acc[mb][nb][r] += c;
        }

#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        if (32 * nb >= ntok) continue;  // uniform; unrolled so acc stays in registers
        __syncthreads();
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                pre[i32][64 * wave + 32 * mb + 8 * (r / 4) + 4 * g + (r % 4)] = acc[mb][nb][r];
        __syncthreads();
        for (int q = 0; q < 8; ++q) {
            const int nl = 8 * wave + q;
            const int n = 32 * nb + nl;
            if (n >= ntok) break;  // uniform over the wave
            uint32_t key[4];
            float v[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                v[s] = pre[nl][lane + 64 * s];
                key[s] = f32_key(v[s]);
            }
            // largest tau with #{key >= tau} >= k
            uint32_t tau = 0;
            for (int bit = 31; bit >= 0; --bit) {
                const uint32_t c = tau | (1u << bit);
                int ge = 0;
#pragma unroll
                for (int s = 0; s < 4; ++s) ge += __popcll(wave_ballot(key[s] >= c));
                if (ge >= k) tau = c;
            }
            int c_gt = 0;
#pragma unroll
            for (int s = 0; s < 4; ++s) c_gt += __popcll(wave_ballot(key[s] > tau));
            const int need_eq = k - c_gt;
            const int64_t base = (static_cast<int64_t>(n0 + n) * n_mt + mt) * k;
            int gt_base = 0, eq_seen = 0;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const bool gt = key[s] > tau, eq = key[s] == tau;
                const uint64_t bg = wave_ballot(gt), be = wave_ballot(eq);
                int pos = -1;
                if (gt) pos = gt_base + lanes_below(bg);
                if (eq) {
                    const int er = eq_seen + lanes_below(be);
                    if (er < need_eq) pos = c_gt + er;
                }
                if (pos >= 0) {
                    cand_val[base + pos] = v[s];
                    cand_idx[base + pos] = mt * kBM + lane + 64 * s;
                }
                gt_base += __popcll(bg);
                eq_seen += __popcll(be);
            }
        }
    }
}

// ------------------------------------------------------------- final merge
__device__ __forceinline__ int block_sum_int(int v, int* red) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    __syncthreads();
    if (lane_id() == 0) red[threadIdx.x / kWave] = v;
    __syncthreads();
    int tot = 0;
#pragma unroll
    for (int w = 0; w < kMergeThreads / kWave; ++w) tot += red[w];
    return tot;
}

template <int CPT>
__global__ void __launch_bounds__(kMergeThreads)
sae_merge_kernel(const float* __restrict__ cand_val, const int32_t* __restrict__ cand_idx,
                 int32_t n_cand, const int32_t* __restrict__ app_count,
                 const int32_t* __restrict__ tok_list, int32_t k, int32_t* __restrict__ idx_out,
                 uint16_t* __restrict__ val_out) {
    __shared__ int red[kMergeThreads / kWave];
    __shared__ uint32_t sel_key[kMaxTopK];
    __shared__ int32_t sel_idx[kMaxTopK];
    __shared__ float sel_val[kMaxTopK];
    __shared__ int n_sel;

    const int n = blockIdx.x;
    if (n >= *app_count) return;
    const int32_t t = tok_list[n];
    const float* cv = cand_val + static_cast<int64_t>(n) * n_cand;
    const int32_t* ci = cand_idx + static_cast<int64_t>(n) * n_cand;

    uint32_t key[CPT];
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
        const int e = threadIdx.x + kMergeThreads * c;
        key[c] = e < n_cand ? f32_key(cv[e]) : 0u;
    }
    uint32_t tau = 0;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t c = tau | (1u << bit);
        int ge = 0;
#pragma unroll
        for (int q = 0; q < CPT; ++q) ge += key[q] >= c ? 1 : 0;
        if (block_sum_int(ge, red) >= k) tau = c;
    }
    int gt = 0, eq = 0;
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        gt += key[q] > tau ? 1 : 0;
        eq += key[q] == tau ? 1 : 0;
    }
    const int c_gt = block_sum_int(gt, red);
    const int c_eq = block_sum_int(eq, red);
    const int need_eq = k - c_gt;
    // Ties at the threshold: keep the need_eq lowest latent indices.
    int32_t idx_cut = 0x7FFFFFFF;
    if (c_eq > need_eq) {
        // smallest I with #{key == tau and idx <= I} >= need_eq
        int32_t lo = 0;
        for (int bit = 30; bit >= 0; --bit) {
            const int32_t probe = lo | ((1 << bit) - 1);  // candidate upper bound
            int c = 0;
#pragma unroll
            for (int q = 0; q < CPT; ++q) {
                const int e = threadIdx.x + kMergeThreads * q;
                if (key[q] == tau && e < n_cand && ci[e] <= probe) ++c;
            }
            if (block_sum_int(c, red) < need_eq) lo |= (1 << bit);
        }
        idx_cut = lo;
    }
    if (threadIdx.x == 0) n_sel = 0;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
        const int e = threadIdx.x + kMergeThreads * q;
        if (e >= n_cand) continue;
        bool take = key[q] > tau;
        if (key[q] == tau) take = ci[e] <= idx_cut;
        if (take) {
            const int slot = atomicAdd(&n_sel, 1);
            if (slot >= kMaxTopK) continue;  // cannot happen: exactly k are taken
            sel_key[slot] = key[q];
            sel_idx[slot] = ci[e];
            sel_val[slot] = cv[e];
        }
    }
    __syncthreads();
    // rank by (value desc, index asc); keys are distinct as (key, idx) pairs
    const int q = threadIdx.x;
    if (q < k) {
        const uint32_t kq = sel_key[q];
        const int32_t iq = sel_idx[q];
        int rank = 0;
        for (int j = 0; j < k; ++j) {
            const uint32_t kj = sel_key[j];
            rank += (kj > kq || (kj == kq && sel_idx[j] < iq)) ? 1 : 0;
        }
        const int64_t o = static_cast<int64_t>(t) * k + rank;
        idx_out[o] = iq;
        val_out[o] = f32_to_bf16_rne(fmaxf(sel_val[q], 0.0f));
    }
}

// ------------------------------------------------------------------ launch
static int enc_grid(int32_t n_mt, int32_t n_nt) {
    const int tiles = n_mt * n_nt;
    return (tiles + 7) / 8 * 8;
}

size_t sae_candidate_bytes(int32_t T_max, int32_t m, int32_t k) {
    const size_t n_mt = static_cast<size_t>(m) / kBM;
    return static_cast<size_t>(T_max) * n_mt * static_cast<size_t>(k) * 8u;
}

hipError_t launch_sae_fold(const uint16_t* W_enc, const uint16_t* b_enc, const uint16_t* b_dec,
                           int32_t m, int32_t d, float* c_fold, hipStream_t stream) {
    hipLaunchKernelGGL(sae_fold_kernel, dim3((m + 3) / 4), dim3(256), 0, stream, W_enc, b_enc,
                       b_dec, m, d, c_fold);
    return hipGetLastError();
}

hipError_t launch_sae_encode(const uint16_t* h, int32_t d, int32_t T_max,
                             const int32_t* app_count, const int32_t* tok_list,
                             const uint16_t* W_enc, const float* c_fold, int32_t m, int32_t k,
                             int32_t* idx_out, uint16_t* val_out, void* cand,
                             hipStream_t stream) {
    const int32_t n_mt = m / kBM;
    const int32_t n_nt = (T_max + kBN - 1) / kBN;
    const int32_t n_cand = n_mt * k;
    float* cand_val = static_cast<float*>(cand);
    int32_t* cand_idx = reinterpret_cast<int32_t*>(
        static_cast<char*>(cand) + static_cast<size_t>(T_max) * n_cand * sizeof(float));
    hipLaunchKernelGGL(sae_stream_topk_kernel, dim3(enc_grid(n_mt, n_nt)), dim3(kEncThreads), 0,
                       stream, h, d, app_count, tok_list, W_enc, c_fold, k, n_mt, n_nt,
                       cand_val, cand_idx);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int cpt = (n_cand + kMergeThreads - 1) / kMergeThreads;
    dim3 g(T_max), b(kMergeThreads);
    if (cpt <= 8)
        hipLaunchKernelGGL(sae_merge_kernel<8>, g, b, 0, stream, cand_val, cand_idx, n_cand,
                           app_count, tok_list, k, idx_out, val_out);
    else if (cpt <= 16)
        hipLaunchKernelGGL(sae_merge_kernel<16>, g, b, 0, stream, cand_val, cand_idx, n_cand,
                           app_count, tok_list, k, idx_out, val_out);
    else if (cpt <= 32)
        hipLaunchKernelGGL(sae_merge_kernel<32>, g, b, 0, stream, cand_val, cand_idx, n_cand,
                           app_count, tok_list, k, idx_out, val_out);
    else
        hipLaunchKernelGGL(sae_merge_kernel<kMaxCPT>, g, b, 0, stream, cand_val, cand_idx,
                           n_cand, app_count, tok_list, k, idx_out, val_out);
    return hipGetLastError();
}

}  // namespace xmix
