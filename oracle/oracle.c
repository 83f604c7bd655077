/*
 * CPU oracle for the per-layer, multi-tenant MI hook step of xMIx
 * (arXiv 2607.22595).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header or constant with the
 * HIP library.
 *
 * Rules followed throughout:
 *  - every input is widened exactly (bf16 and fp32 values are exact doubles);
 *  - every floating-point result is computed in fp64 with plain loops, in the
 *    order the definition is written;
 *  - a result stored as bf16 is rounded once, to nearest with ties to even,
 *    directly from the fp64 value; a result stored as fp32 is rounded once.
 *
 * The paper states the problem (MI functions that consume the activation at
 * a hook plus per-app runtime parameters and produce a signal and/or an
 * activation update, toggled per request; Sec. 4.2, "Executable units",
 * "Toggling semantics", "Composition model"; Sec. 4.3, "Graph-level toggling
 * and continuous batching") but prints no formula for the individual MI
 * functions.  The definitions below are the textbook ones: additive steering
 * (Sec. 3, the Write primitive), a logistic-regression probe (Sec. 3, the Read
 * primitive; Table 1 App-4), a TopK sparse autoencoder encoder, and an
 * error-preserving feature clamp.  Every reading taken where the paper is
 * silent is listed in the repository's design notes.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- numbers */

static double bf16_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* Round-to-nearest-even of a double onto the bf16 grid (8 significant bits,
 * fp32 exponent range, subnormal quantum 2^-133), returned as bits. */
uint16_t oracle_round_bf16(double x) {
    if (x != x) return 0x7FC0;
    uint16_t sign = (x < 0.0 || (x == 0.0 && 1.0 / x < 0.0)) ? 0x8000 : 0;
    double a = fabs(x);
    if (a == 0.0) return sign;
    int e;
    (void)frexp(a, &e);            /* a in [2^(e-1), 2^e) */
    int q = e - 8;                 /* weight of the last kept bit */
    if (q < -133) q = -133;
    double scaled = ldexp(a, -q);  /* exact */
    double fl = floor(scaled);
    double rem = scaled - fl;      /* exact */
    double r = fl;
    if (rem > 0.5 || (rem == 0.5 && fmod(fl, 2.0) != 0.0)) r = fl + 1.0;
    double v = ldexp(r, q);
    if (v >= 0x1p128) return sign | 0x7F80;
    float f = (float)v;            /* exact */
    uint32_t u;
    memcpy(&u, &f, 4);
    return sign | (uint16_t)(u >> 16);
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the parallel loops below (n < 1: leave unchanged); for timing
 * the oracle single-threaded beside its all-core runs. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ----------------------------------------------------------------- routing
 * Token -> request -> app bitmask (Sec. 4.2 "Toggling semantics": an app is
 * deployed for every request but active only for the requests that turned it
 * on; Sec. 4.3: inactive apps are bypassed per request inside one batch).
 *
 *   tok_mask[t] = sub[req[t]] & (2^n_apps - 1)   if t < T_valid and
 *                                                 0 <= req[t] < R_max
 *               = 0                               otherwise
 *   app_tokens[a][0 .. count[a]) = the tokens t with bit a of tok_mask[t]
 *                                  set, ascending; the rest of the row is -1.
 *   err bit 0: some t < T_valid has req[t] >= R_max.
 *   err bit 1: T_valid outside [0, T_max] (it is then clamped).
 * A negative request id marks a padding token and is not an error. */
void oracle_route(const int32_t *req, int32_t T_valid, int32_t T_max,
                  const uint32_t *sub, int32_t R_max, int32_t n_apps,
                  uint32_t *tok_mask, int32_t *count, int32_t *app_tokens,
                  uint32_t *err) {
    uint32_t e = 0;
    if (T_valid < 0) { T_valid = 0; e |= 2u; }
    if (T_valid > T_max) { T_valid = T_max; e |= 2u; }
    uint32_t keep = (n_apps >= 32) ? 0xFFFFFFFFu : ((1u << n_apps) - 1u);
    for (int32_t t = 0; t < T_max; ++t) {
        uint32_t mask = 0;
        if (t < T_valid) {
            int32_t r = req[t];
            if (r >= R_max) e |= 1u;
            else if (r >= 0) mask = sub[r] & keep;
        }
        tok_mask[t] = mask;
    }
    for (int32_t a = 0; a < n_apps; ++a) {
        int32_t c = 0;
        for (int32_t t = 0; t < T_max; ++t)
            if ((tok_mask[t] >> a) & 1u) app_tokens[(int64_t)a * T_max + c++] = t;
        count[a] = c;
        for (int32_t i = c; i < T_max; ++i) app_tokens[(int64_t)a * T_max + i] = -1;
    }
    *err = e;
}

/* ------------------------------------------------------ conditional writes
 * A conditional write is a write that applies only where a device-side
 * condition holds (Sec. 4.1, `.cond(...)`; Sec. 4.2, condition classes):
 * activation-driven (a probe's signal from an earlier layer against a
 * threshold) or token-driven (the token id is in a trigger list).  Both
 * narrow one app's routing entry: a token keeps bit `app_bit` only if the
 * condition holds for it, and the app's token list is rebuilt from the
 * narrowed masks (ascending, -1 after the count).  Other apps are untouched.
 *
 * Activation-driven: the condition is  s >= threshold  with
 *   s = signal[t]                  (signal_per_request == 0), or
 *   s = signal[req_of_token[t]]    (signal_per_request != 0, ids in [0, n_signal)),
 * and, when signal_bit >= 0, the token must also carry bit signal_bit (the
 * signal exists only where the probe app ran).  NaN never passes. */
void oracle_route_gate(int32_t T_max, uint32_t *tok_mask, int32_t *app_count,
                       int32_t *app_tokens, int32_t app_bit, const float *signal,
                       int32_t signal_per_request, const int32_t *req_of_token,
                       int32_t n_signal, int32_t signal_bit, float threshold) {
    int32_t *list = app_tokens + (int64_t)app_bit * T_max;
    int32_t n = 0;
    for (int32_t t = 0; t < T_max; ++t) {
        if (!((tok_mask[t] >> app_bit) & 1u)) continue;
        int pass = 1;
        if (signal_bit >= 0 && !((tok_mask[t] >> signal_bit) & 1u)) pass = 0;
        double sv = 0.0;
        if (pass) {
            int32_t i = signal_per_request ? req_of_token[t] : t;
            if (i < 0 || i >= n_signal) pass = 0;
            else sv = (double)signal[i];
        }
        if (pass && !(sv >= (double)threshold)) pass = 0;
        if (pass) list[n++] = t;
        else tok_mask[t] &= ~(1u << app_bit);
    }
    for (int32_t i = n; i < T_max; ++i) list[i] = -1;
    app_count[app_bit] = n;
}

/* Token-driven: the condition is that token_ids[t] lies in [0, vocab_size)
 * and its bit is set in the trigger bitmap vocab_bits (bit v of word v/32). */
void oracle_route_trigger(int32_t T_max, uint32_t *tok_mask, int32_t *app_count,
                          int32_t *app_tokens, int32_t app_bit, const int32_t *token_ids,
                          const uint32_t *vocab_bits, int32_t vocab_size) {
    int32_t *list = app_tokens + (int64_t)app_bit * T_max;
    int32_t n = 0;
    for (int32_t t = 0; t < T_max; ++t) {
        if (!((tok_mask[t] >> app_bit) & 1u)) continue;
        int32_t v = token_ids[t];
        int pass = v >= 0 && v < vocab_size && ((vocab_bits[v >> 5] >> (v & 31)) & 1u);
        if (pass) list[n++] = t;
        else tok_mask[t] &= ~(1u << app_bit);
    }
    for (int32_t i = n; i < T_max; ++i) list[i] = -1;
    app_count[app_bit] = n;
}

/* ---------------------------------------------------------------- steering
 * Additive steering, the Write primitive (Sec. 3: add or subtract a vector on
 * the activation).  For every token t that has at least one steering bit:
 *   h'[t,i] = round( h[t,i] + sum_{s : bit app_bits[s] of tok_mask[t]}
 *                               alpha[req[t], s] * v[s,i] )
 * with the sum taken in fp64 and one rounding to the storage type.  A
 * subtraction is a negative alpha.  Tokens without a steering bit are left
 * untouched.  `is_bf16` selects bf16 (uint16 bits) or fp32 storage of h and
 * v. */
void oracle_steer(void *h, int is_bf16, int32_t T_max, int32_t d,
                  const uint32_t *tok_mask, const int32_t *req,
                  const void *v, const int32_t *app_bits, const float *alpha,
                  int32_t n_steer) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t t = 0; t < T_max; ++t) {
        uint32_t mask = tok_mask[t];
        int any = 0;
        for (int32_t s = 0; s < n_steer; ++s)
            if ((mask >> app_bits[s]) & 1u) any = 1;
        if (!any) continue;
        int32_t r = req[t];
        for (int32_t i = 0; i < d; ++i) {
            int64_t at = (int64_t)t * d + i;
            double acc = is_bf16 ? bf16_to_double(((const uint16_t *)h)[at])
                                 : (double)((const float *)h)[at];
            for (int32_t s = 0; s < n_steer; ++s) {
                if (!((mask >> app_bits[s]) & 1u)) continue;
                int64_t vi = (int64_t)s * d + i;
                double vv = is_bf16 ? bf16_to_double(((const uint16_t *)v)[vi])
                                    : (double)((const float *)v)[vi];
                acc += (double)alpha[(int64_t)r * n_steer + s] * vv;
            }
            if (is_bf16) ((uint16_t *)h)[at] = oracle_round_bf16(acc);
            else ((float *)h)[at] = (float)acc;
        }
    }
}

/* ------------------------------------------------------ router-logit write
 * Expert (de)activation on a mixture-of-experts router (Table 1, App-7: a
 * conditional write whose locus is the router logits).  For every token with
 * at least one of the router apps' bits:
 *   logits[t,e] = round( logits[t,e] + offsets[s1,e] + offsets[s2,e] + ... )
 * over the token's subscribed router apps s1 < s2 < ... (their index in the
 * app list), added in that order in fp64 and rounded once to the storage
 * type.  An offset of -inf removes expert e for that app's tokens; a large
 * finite offset forces it into the router's selection.  Non-finite values
 * follow IEEE arithmetic.  Other rows are untouched. */
void oracle_router_write(void *logits, int is_bf16, int32_t T_max, int32_t n_experts,
                         const uint32_t *tok_mask, const int32_t *app_bits,
                         const float *offsets, int32_t n_router) {
    for (int32_t t = 0; t < T_max; ++t) {
        uint32_t mask = tok_mask[t];
        int any = 0;
        for (int32_t s = 0; s < n_router; ++s)
            if ((mask >> app_bits[s]) & 1u) any = 1;
        if (!any) continue;
        for (int32_t e = 0; e < n_experts; ++e) {
            int64_t at = (int64_t)t * n_experts + e;
            double acc = is_bf16 ? bf16_to_double(((const uint16_t *)logits)[at])
                                 : (double)((const float *)logits)[at];
            for (int32_t s = 0; s < n_router; ++s)
                if ((mask >> app_bits[s]) & 1u) acc += (double)offsets[(int64_t)s * n_experts + e];
            if (is_bf16) ((uint16_t *)logits)[at] = oracle_round_bf16(acc);
            else ((float *)logits)[at] = (float)acc;
        }
    }
}

/* ------------------------------------------------------------------ probes
 * Linear read-out with a logistic link, the Read primitive (Sec. 3: a
 * linear probe that turns activations into a score; Table 1 App-4,
 * logistic regression on activations).
 *   logit[p][t] = b[p] + sum_i w[p,i] * h[t,i],  score = 1 / (1 + exp(-logit))
 * for every token with bit app_bits[p] set.  Entries of unsubscribed tokens
 * are left untouched. */
static double dot_row(const void *h, int is_bf16, int64_t row, int32_t d,
                      const void *w, int64_t wrow) {
    double acc = 0.0;
    for (int32_t i = 0; i < d; ++i) {
        double hv = is_bf16 ? bf16_to_double(((const uint16_t *)h)[row * d + i])
                            : (double)((const float *)h)[row * d + i];
        double wv = is_bf16 ? bf16_to_double(((const uint16_t *)w)[wrow * d + i])
                            : (double)((const float *)w)[wrow * d + i];
        acc += wv * hv;
    }
    return acc;
}

static double logistic(double x) { return 1.0 / (1.0 + exp(-x)); }

void oracle_probe_token(const void *h, int is_bf16, int32_t T_max, int32_t d,
                        const uint32_t *tok_mask, const void *w, const float *b,
                        const int32_t *app_bits, int32_t n_probe,
                        double *logit, double *score) {
#pragma omp parallel for schedule(dynamic, 4)
    for (int32_t t = 0; t < T_max; ++t) {
        for (int32_t p = 0; p < n_probe; ++p) {
            if (!((tok_mask[t] >> app_bits[p]) & 1u)) continue;
            double l = (double)b[p] + dot_row(h, is_bf16, t, d, w, p);
            logit[(int64_t)p * T_max + t] = l;
            score[(int64_t)p * T_max + t] = logistic(l);
        }
    }
}

/* Mean-pooled probe over each request's contiguous token span
 * [cu[r], cu[r+1]):
 *   pooled[p][r] = b[p] + (1/n_r) * sum_{t in span} sum_i w[p,i] * h[t,i]
 * which is the probe applied to the span's mean activation.  A request is
 * subscribed when the first token of its span has bit app_bits[p]; requests
 * with an empty span are not written. */
void oracle_probe_mean(const void *h, int is_bf16, int32_t T_max, int32_t d,
                       const uint32_t *tok_mask, const void *w, const float *b,
                       const int32_t *app_bits, int32_t n_probe,
                       const int32_t *cu_seqlens, int32_t R,
                       double *logit, double *score) {
    (void)T_max;
#pragma omp parallel for schedule(dynamic, 1) collapse(2)
    for (int32_t r = 0; r < R; ++r) {
        for (int32_t p = 0; p < n_probe; ++p) {
            int32_t lo = cu_seqlens[r], hi = cu_seqlens[r + 1];
            if (hi <= lo) continue;
            if (!((tok_mask[lo] >> app_bits[p]) & 1u)) continue;
            double sum = 0.0;
            for (int32_t t = lo; t < hi; ++t) sum += dot_row(h, is_bf16, t, d, w, p);
            double l = (double)b[p] + sum / (double)(hi - lo);
            logit[(int64_t)p * R + r] = l;
            score[(int64_t)p * R + r] = logistic(l);
        }
    }
}

/* Last-token probe of each request (the "last token" activation condition
 * of a read, Sec. 4.1): for each request r with a non-empty span
 * [cu[r], cu[r+1]) whose first token has bit app_bits[p],
 *   logit[p][r] = b[p] + sum_i w[p,i] * h[cu[r+1]-1, i]
 * i.e. the per-token probe of the span's last token. */
void oracle_probe_last(const void *h, int is_bf16, int32_t T_max, int32_t d,
                       const uint32_t *tok_mask, const void *w, const float *b,
                       const int32_t *app_bits, int32_t n_probe,
                       const int32_t *cu_seqlens, int32_t R,
                       double *logit, double *score) {
    (void)T_max;
    for (int32_t r = 0; r < R; ++r) {
        for (int32_t p = 0; p < n_probe; ++p) {
            int32_t lo = cu_seqlens[r], hi = cu_seqlens[r + 1];
            if (hi <= lo) continue;
            if (!((tok_mask[lo] >> app_bits[p]) & 1u)) continue;
            double l = (double)b[p] + dot_row(h, is_bf16, hi - 1, d, w, p);
            logit[(int64_t)p * R + r] = l;
            score[(int64_t)p * R + r] = logistic(l);
        }
    }
}

/* --------------------------------------------------------- SAE encode+TopK
 * TopK sparse-autoencoder encoder on one token (the paper names sparse
 * autoencoders and feature dictionaries as app artefacts, Sec. 3, and
 * feature activations as a gate signal, Sec. 4.2):
 *   u     = h - b_dec                                  (exact)
 *   pre_j = b_enc[j] + sum_i W_enc[j,i] * u_i          for all j < m
 *   S     = the k indices with the largest pre_j; equal values keep the
 *           lower index first
 *   val_j = bf16( max(pre_j, 0) )                      for j in S
 * Output rows are ordered by pre descending, then index ascending. */
void oracle_sae_pre(const uint16_t *h_row, int32_t d, const uint16_t *W_enc,
                    const uint16_t *b_enc, const uint16_t *b_dec, int32_t m,
                    double *pre) {
    double *u = (double *)malloc(sizeof(double) * (size_t)d);
    for (int32_t i = 0; i < d; ++i)
        u[i] = bf16_to_double(h_row[i]) - bf16_to_double(b_dec[i]);
    for (int32_t j = 0; j < m; ++j) {
        const uint16_t *wr = W_enc + (int64_t)j * d;
        double acc = bf16_to_double(b_enc[j]);
        for (int32_t i = 0; i < d; ++i) acc += bf16_to_double(wr[i]) * u[i];
        pre[j] = acc;
    }
    free(u);
}

typedef struct { double v; int32_t j; } scored;

static int by_value_desc_index_asc(const void *pa, const void *pb) {
    const scored *a = (const scored *)pa, *b = (const scored *)pb;
    if (a->v > b->v) return -1;
    if (a->v < b->v) return 1;
    return (a->j > b->j) - (a->j < b->j);
}

/* Select the k best of pre[0..m) by a full sort (library qsort). */
void oracle_topk(const double *pre, int32_t m, int32_t k, int32_t *idx,
                 double *val_exact, uint16_t *val_bf16) {
    scored *all = (scored *)malloc(sizeof(scored) * (size_t)m);
    for (int32_t j = 0; j < m; ++j) { all[j].v = pre[j]; all[j].j = j; }
    qsort(all, (size_t)m, sizeof(scored), by_value_desc_index_asc);
    for (int32_t q = 0; q < k; ++q) {
        double z = all[q].v > 0.0 ? all[q].v : 0.0;
        idx[q] = all[q].j;
        if (val_exact) val_exact[q] = z;
        if (val_bf16) val_bf16[q] = oracle_round_bf16(z);
    }
    free(all);
}

/* Encode the listed tokens.  tokens[0..n_tok) are row numbers of h; output
 * row q belongs to tokens[q].  If `pre_out` is non-null it receives the full
 * [n_tok, m] pre-activation matrix (used to judge near-ties). */
void oracle_sae_encode(const uint16_t *h, int32_t d, const int32_t *tokens,
                       int32_t n_tok, const uint16_t *W_enc,
                       const uint16_t *b_enc, const uint16_t *b_dec, int32_t m,
                       int32_t k, int32_t *idx_out, uint16_t *val_out,
                       double *val_exact_out, double *pre_out) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t q = 0; q < n_tok; ++q) {
        double *pre = pre_out ? pre_out + (int64_t)q * m
                              : (double *)malloc(sizeof(double) * (size_t)m);
        oracle_sae_pre(h + (int64_t)tokens[q] * d, d, W_enc, b_enc, b_dec, m, pre);
        oracle_topk(pre, m, k, idx_out + (int64_t)q * k,
                    val_exact_out ? val_exact_out + (int64_t)q * k : NULL,
                    val_out + (int64_t)q * k);
        if (!pre_out) free(pre);
    }
}

/* -------------------------------------------------------- SAE clamp-decode
 * Feature clamp with the decoded delta written back (a Write whose payload is
 * computed from a read of the same hook).  For every token t with bit
 * `app_bit`:
 *   z_j   = the token's encoded value of feature j if j is among its selected
 *           indices idx[t,*], else 0
 *   delta = sum_{q < n_clamp} (c_q - z_{C_q}) * W_dec[C_q, :]
 *   h'[t] = bf16( h[t] + delta )
 * i.e. decode(z') - decode(z) for z' = z with the clamped features set, which
 * leaves the SAE reconstruction error in place.  `delta_out` (nullable)
 * receives delta for every processed token. */
void oracle_clamp_decode(uint16_t *h, int32_t T_max, int32_t d,
                         const uint32_t *tok_mask, int32_t app_bit,
                         const int32_t *idx, const uint16_t *val, int32_t k,
                         const uint16_t *W_dec, int32_t m,
                         const int32_t *clamp_ids, const float *clamp_vals,
                         int32_t n_clamp, double *delta_out) {
    (void)m;
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t t = 0; t < T_max; ++t) {
        if (!((tok_mask[t] >> app_bit) & 1u)) continue;
        double coef[64];
        for (int32_t q = 0; q < n_clamp; ++q) {
            double z = 0.0;
            for (int32_t s = 0; s < k; ++s)
                if (idx[(int64_t)t * k + s] == clamp_ids[q])
                    z = bf16_to_double(val[(int64_t)t * k + s]);
            coef[q] = (double)clamp_vals[q] - z;
        }
        for (int32_t i = 0; i < d; ++i) {
            double delta = 0.0;
            for (int32_t q = 0; q < n_clamp; ++q)
                delta += coef[q] * bf16_to_double(W_dec[(int64_t)clamp_ids[q] * d + i]);
            if (delta_out) delta_out[(int64_t)t * d + i] = delta;
            int64_t at = (int64_t)t * d + i;
            h[at] = oracle_round_bf16(bf16_to_double(h[at]) + delta);
        }
    }
}

/* ------------------------------------------------------ readback to a ring
 * Read results land in a buffer that CPU code reads later (Sec. 1 and
 * Sec. 4.2 "State and dataflow").  The tokens with bit `app_bit`, ascending,
 * are appended to a ring of `capacity` slots of `row_bytes` bytes:
 *   slot (head + i) mod capacity <- { t, req[t], layer_id, app_id } (4 x
 *                                   int32) followed by the payload bytes of
 *                                   row t, the concatenation of the given
 *                                   segments
 * then head += count.  A later row overwrites an older one in the same slot.
 * Segment s of row t starts at seg[s] + t * seg_bytes[s]. */
void oracle_compact(const uint8_t *const *seg, const int32_t *seg_bytes,
                    int32_t n_seg, const uint32_t *tok_mask, int32_t T_max,
                    int32_t app_bit, const int32_t *req, int32_t layer_id,
                    int32_t app_id, uint8_t *slots, int32_t capacity,
                    int32_t row_bytes, uint64_t *head) {
    uint64_t h0 = *head;
    uint64_t i = 0;
    for (int32_t t = 0; t < T_max; ++t) {
        if (!((tok_mask[t] >> app_bit) & 1u)) continue;
        uint8_t *dst = slots + (int64_t)((h0 + i) % (uint64_t)capacity) * row_bytes;
        int32_t hdr[4] = { t, req[t], layer_id, app_id };
        memcpy(dst, hdr, 16);
        int64_t off = 16;
        for (int32_t s = 0; s < n_seg; ++s) {
            memcpy(dst + off, seg[s] + (int64_t)t * seg_bytes[s], (size_t)seg_bytes[s]);
            off += seg_bytes[s];
        }
        ++i;
    }
    *head = h0 + i;
}
