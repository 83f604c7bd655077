/*
 * xmix.h - C ABI of the per-layer, multi-tenant MI hook step on one MI355X
 * (gfx950), after xMIx (arXiv 2607.22595).
 *
 * The paper's contract for an MI function (Sec. 4.2, "Executable units"):
 * it consumes the activation slice at a hook plus the runtime parameters of
 * one app, and yields a derived signal, an update of the activation, or
 * both.  Read results go to buffers that later GPU work or the CPU consume
 * (Sec. 4.2, "State and dataflow").  Apps are deployed once and toggled per
 * request, and a request that does not use an app must not pay for it
 * (Sec. 4.2, "Toggling semantics"; Sec. 4.3, "Graph-level toggling and
 * continuous batching").  Graph replay needs a fixed structure whose
 * arguments can change between launches (Sec. 4.3, "CUDA-graph-safe kernel
 * design").
 *
 * Conventions shared by every call
 * --------------------------------
 * - All data pointers are DEVICE pointers unless the comment says "host".
 *   The caller allocates and owns every buffer; the library keeps no
 *   per-call state and allocates nothing (the one exception is the step
 *   graph executor, xmix_graph_*, which owns the graphs it instantiates).
 * - bf16 values travel as their raw 16-bit patterns (uint16_t).
 * - Activations are row-major [T_max, d]: one row per token slot of the
 *   continuous batch.  T_max is the static batch capacity; the number of
 *   live tokens, T_valid, lives in device memory, so one captured graph
 *   serves every batch.
 * - Every hook-step call is asynchronous on `stream` (a hipStream_t; NULL =
 *   the null stream), never synchronises, never copies between host and
 *   device, and can be captured into a HIP graph.  Per-step data (T_valid, subscription
 *   masks, alpha, clamp values, ring heads) is read from device memory at
 *   run time, so a graph can be replayed with new requests without
 *   recapture.
 * - Host-side argument checks return a status immediately and launch
 *   nothing.  Data errors found on the device never abort: they are ORed
 *   into a caller-owned error word (xmix_route_build) and the offending
 *   token is routed to no app.
 * - Rows of unsubscribed tokens or requests are never written in any
 *   output ("don't use, don't pay").
 * - No C++ exception crosses this interface.
 *
 * Calls, in the order of one layer's step: routing (xmix_route_build) and
 * its conditional filters (xmix_route_gate, xmix_route_trigger); the reads
 * (xmix_probe_score, xmix_sae_encode_topk and its stages); the writes
 * (xmix_steer_apply, xmix_sae_clamp_decode, xmix_router_write); readback
 * (xmix_readback_compact, or fused into the SAE merge with the _ring
 * variants).  Step graphs (xmix_graph_*) capture and replay such a
 * sequence.
 */
#ifndef XMIX_H
#define XMIX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    XMIX_OK = 0,
    XMIX_E_INVAL = 1,        /* bad pointer, size or combination of sizes */
    XMIX_E_UNSUPPORTED = 2,  /* valid request outside what the library supports */
    XMIX_E_WORKSPACE = 3,    /* workspace missing or smaller than required */
    XMIX_E_LAUNCH = 4        /* the HIP runtime rejected a launch */
} xmix_status;

typedef enum { XMIX_F32 = 0, XMIX_BF16 = 1 } xmix_dtype;

enum { XMIX_PROBE_TOKEN = 0, XMIX_PROBE_MEAN = 1, XMIX_PROBE_LAST = 2 };

/* Device error-word bits set by xmix_route_build. */
enum {
    XMIX_ERR_REQUEST_RANGE = 1u,  /* a live token named a request id >= R_max */
    XMIX_ERR_T_VALID = 2u         /* *T_valid was outside [0, T_max]; clamped */
};

#define XMIX_MAX_APPS 32
#define XMIX_MAX_TOPK 64
#define XMIX_MAX_CLAMP 16
#define XMIX_MAX_SEGMENTS 4

/* Routing table of one hook step (device arrays, caller-owned):
 *   tok_mask  [T_max]          app bitmask of each token slot (0: none)
 *   app_count [n_apps]         number of tokens subscribed to app a
 *   app_tokens[n_apps][T_max]  ascending token slots of app a, then -1
 * n_apps <= 32: bit a of a mask is app a. */
typedef struct {
    uint32_t *tok_mask;
    int32_t *app_count;
    int32_t *app_tokens;
    int32_t T_max;
    int32_t n_apps;
} xmix_route;

/* Readback ring (device memory, caller-owned):
 *   slots [capacity][row_bytes]  row = 16-byte header {int32 token,
 *                                int32 request, int32 layer_id, int32 app_id}
 *                                followed by the payload bytes
 *   head  [2]                    head[0]: monotonic count of rows ever
 *                                written; slot of row i is i mod capacity.
 *                                head[1]: internal, must be zero when the
 *                                ring is created; every call leaves it zero.
 * A reader that consumed up to row r can read rows [r, head[0]); if
 * head[0] - r > capacity, the oldest rows were overwritten.  A call's rows
 * and its head update are visible to work ordered after the call (later
 * work on its stream, or after a synchronisation with it); a reader running
 * concurrently with the call must not rely on head[0]. */
typedef struct {
    uint8_t *slots;
    uint64_t *head;
    int32_t capacity;
    int32_t row_bytes;
} xmix_ring;

/* Encoder dictionary of one SAE app in the library's tiled HBM layout
 * (host struct; `pieces` is caller-owned device memory of m * d bf16).
 * Only xmix_sae_pack_encoder fills it: it permutes a row-major [m, d]
 * matrix into `pieces` and sets m, d and layout = XMIX_SAE_DICT_TILED.
 * Every call that reads a dictionary takes this struct, never a bare
 * pointer, and rejects (XMIX_E_INVAL) a struct whose layout tag is not
 * XMIX_SAE_DICT_TILED or whose d differs from the activation width, so a
 * row-major matrix cannot be passed by mistake. */
#define XMIX_SAE_DICT_TILED 0x31504D58u  /* "XMP1" */
typedef struct {
    const uint16_t *pieces;
    int32_t m;
    int32_t d;
    uint32_t layout;
} xmix_sae_dict;

const char *xmix_status_string(xmix_status s);
const char *xmix_version(void);

/* ---------------------------------------------------------------- routing
 * Token -> request -> app-bitmask table (Sec. 4.2 "Toggling semantics",
 * "Composition model"; Sec. 4.3 "Graph-level toggling and continuous
 * batching": per-request activation inside one batch, without CPU work).
 *   tok_mask[t] = sub_mask[req_of_token[t]] & (2^n_apps - 1) for
 *                 t < *T_valid and 0 <= req_of_token[t] < R_max, else 0.
 *   app_tokens[a][0..app_count[a]) lists, ascending, the tokens with bit a;
 *   the rest of the row is -1.
 * req_of_token [T_max] int32: request id per token slot; negative = padding.
 * T_valid      [1] int32: live tokens; out of [0, T_max] sets
 *              XMIX_ERR_T_VALID and is clamped.
 * sub_mask     [R_max] uint32: app subscription bitmask per request.
 * err_word     [1] uint32: error bits are ORed in (never cleared here).
 * rt           host struct with device arrays; rt->T_max >= 1,
 *              1 <= rt->n_apps <= 32.
 * Errors: XMIX_E_INVAL for a null pointer or a size out of range. */
xmix_status xmix_route_build(const int32_t *req_of_token, const int32_t *T_valid,
                             const uint32_t *sub_mask, int32_t R_max,
                             const xmix_route *rt, uint32_t *err_word, void *stream);

/* ------------------------------------------------------ conditional writes
 * A conditional write applies only where a condition evaluated on the
 * device holds (Sec. 4.1, `.cond(...)`; Sec. 4.2, "Condition classes": an
 * activation-driven condition such as a probe from an earlier layer against
 * a threshold, or a token-driven one such as the token being in a trigger
 * list; Sec. 4.3, device-side control flow).  Both calls narrow the routing
 * entry of one app, in place, after xmix_route_build and before the
 * write calls that use that app:
 *   a token keeps bit app_bit only if the condition holds for it; the app's
 *   count and ascending token list are rebuilt (then -1 up to the old count).
 * Other apps are untouched; the next xmix_route_build starts afresh.
 *
 * xmix_route_gate (activation-driven): the condition is  s >= *threshold
 * with s = signal[t] (req_of_token NULL; signal [T_max], e.g. a token-mode
 * probe's logit row) or s = signal[req_of_token[t]] (signal [n_signal] per
 * request, e.g. a pooled or last-token probe's row); when signal_bit >= 0
 * the token must also carry that bit (the probe ran on it).  NaN and an
 * index outside [0, n_signal) fail.  threshold is a device scalar (fp32).
 *
 * xmix_route_trigger (token-driven): the condition is that token_ids[t]
 * (device [T_max] int32) lies in [0, vocab_size) and bit token_ids[t] of the
 * trigger bitmap vocab_bits (device, (vocab_size + 31) / 32 words) is set.
 *
 * Errors: XMIX_E_INVAL for a null pointer or app_bit / signal_bit outside
 * the route's apps. */
xmix_status xmix_route_gate(const xmix_route *rt, int32_t app_bit, const float *signal,
                            const int32_t *req_of_token, int32_t n_signal, int32_t signal_bit,
                            const float *threshold, void *stream);
xmix_status xmix_route_trigger(const xmix_route *rt, int32_t app_bit, const int32_t *token_ids,
                               const uint32_t *vocab_bits, int32_t vocab_size, void *stream);

/* --------------------------------------------------------------- steering
 * Additive steering, the Write primitive (Sec. 3: add or subtract a vector
 * on the activation; Fig. 2b's steering_vector write).  For each token t with
 * at least one steering bit:
 *   h[t,:] <- round( h[t,:] + sum_{s: bit app_bits[s] in tok_mask[t]}
 *                                alpha[req[t]][s] * vecs[s,:] )
 * accumulated in fp64 and rounded once to the storage type (RNE).  Other
 * rows are not touched.
 * h        [T_max, d] of dtype `dt`, updated in place.
 * vecs     [n_steer, d] of dtype `dt`.
 * app_bits host [n_steer]: the route bit that gates vector s (static per
 *          deployment, baked into the launch).
 * alpha    [R_max][n_steer] fp32 per (request, vector); a negative value
 *          subtracts.
 * Requires 1 <= n_steer <= 32, d % 8 == 0 (bf16) or d % 4 == 0 (fp32). */
xmix_status xmix_steer_apply(void *h, xmix_dtype dt, int32_t d, const xmix_route *rt,
                             const int32_t *req_of_token, const void *vecs,
                             const int32_t *app_bits, const float *alpha,
                             int32_t n_steer, int32_t R_max, void *stream);

/* ------------------------------------------------- probes + steering, fused
 * Reads and writes composed at one hook (Sec. 4.2: several apps on the same
 * layer; reads see the activation as the model produced it, then writes
 * apply): token-mode probes and the steering add in one pass over each row.
 * The result is bit-identical to
 *   xmix_probe_score(h, ..., probe_bits, n_probe, XMIX_PROBE_TOKEN, ...)
 * followed by
 *   xmix_steer_apply(h, ..., steer_bits, alpha, n_steer, R_max, ...)
 * (same arithmetic in the same order): the probes read each row before the
 * steering rewrites it, and each row is read from HBM once instead of twice.
 * Arguments are those of the two calls: h [T_max, d] of dtype `dt`, updated
 * in place; vecs [n_steer, d] and w [n_probe, d] of dtype `dt`; alpha
 * [R_max][n_steer] fp32; b [n_probe] fp32; logit_out and score_out
 * [n_probe][T_max] fp32, written only for tokens with the probe's bit.
 * steer_bits and probe_bits are host arrays.
 * Requires 1 <= n_steer <= 32, 1 <= n_probe <= 32, d % 8 == 0 (bf16) or
 * d % 4 == 0 (fp32).  Errors: XMIX_E_INVAL as for the two calls. */
xmix_status xmix_steer_probe(void *h, xmix_dtype dt, int32_t d, const xmix_route *rt,
                             const int32_t *req_of_token, const void *vecs,
                             const int32_t *steer_bits, const float *alpha, int32_t n_steer,
                             int32_t R_max, const void *w, const float *b,
                             const int32_t *probe_bits, int32_t n_probe, float *logit_out,
                             float *score_out, void *stream);

/* Route build and the pass above in one launch, for a step whose first
 * consumer of the routing is this pass (per-request toggling inside the
 * batch, Sec. 4.2-4.3).  Same effect as
 *   xmix_route_build(req_of_token, T_valid, sub_mask, R_max, rt, err_word)
 * followed by xmix_steer_probe(h, ...): the route holds exactly what the
 * route build writes.  Up to 1024 token slots (and at least one slot per
 * app) the kernel builds the routing itself: each workgroup computes its
 * token's mask, workgroup a publishes app a's list.  Otherwise the two
 * launches are made.  Arguments are those of the two calls. */
xmix_status xmix_route_steer_probe(const int32_t *req_of_token, const int32_t *T_valid,
                                   const uint32_t *sub_mask, int32_t R_max, const xmix_route *rt,
                                   uint32_t *err_word, void *h, xmix_dtype dt, int32_t d,
                                   const void *vecs, const int32_t *steer_bits,
                                   const float *alpha, int32_t n_steer, const void *w,
                                   const float *b, const int32_t *probe_bits, int32_t n_probe,
                                   float *logit_out, float *score_out, void *stream);

/* ------------------------------------------------------ router-logit write
 * Expert (de)activation on a mixture-of-experts router, a write whose locus
 * is the router logits (Table 1, App-7).  For each token t with at least one
 * router bit:
 *   logits[t,e] <- round( logits[t,e] + offsets[s1,e] + offsets[s2,e] + ... )
 * over the token's subscribed router apps s1 < s2 < ... (their index in
 * app_bits), added in that order in fp64 and rounded once (RNE) to the
 * storage type.  An offset of -inf removes expert e for that app's tokens; a
 * large finite offset forces it into the router's selection; other
 * non-finite values follow IEEE arithmetic.  Other rows are not touched.
 * The condition of a conditional app is applied beforehand by narrowing its
 * routing entry (xmix_route_gate / xmix_route_trigger).
 * logits   [T_max, n_experts] of dtype `dt`, updated in place (2-byte
 *          aligned for bf16, 4-byte for fp32).
 * app_bits host [n_router]: the route bit of each router app.
 * offsets  [n_router, n_experts] fp32, device.
 * Requires 1 <= n_router <= 32 and T_max * n_experts < 2^31.
 * Errors: XMIX_E_INVAL (null pointer, bad dtype, alignment, app bit outside
 * the route), XMIX_E_UNSUPPORTED (too many elements). */
xmix_status xmix_router_write(void *logits, xmix_dtype dt, int32_t n_experts,
                              const xmix_route *rt, const int32_t *app_bits,
                              const float *offsets, int32_t n_router, void *stream);

/* ------------------------------------------------------------------ probes
 * Linear probes with a logistic link, the Read primitive (Sec. 3: a linear
 * probe scoring activations; Table 1 App-4).
 * mode XMIX_PROBE_TOKEN: for each token t with bit app_bits[p]:
 *   logit_out[p][t] = b[p] + w[p,:] . h[t,:],  score_out[p][t] = sigmoid(logit)
 *   outputs are [n_probe][T_max] fp32.
 * mode XMIX_PROBE_MEAN: for each request r whose span
 *   [cu_seqlens[r], cu_seqlens[r+1]) is non-empty and whose first token has
 *   bit app_bits[p]:
 *   logit_out[p][r] = b[p] + mean_{t in span} (w[p,:] . h[t,:]) (the probe of
 *   the span's mean activation), score as above; outputs are [n_probe][R_max].
 *   Every token of the span counts, whatever its own mask holds (a
 *   conditional filter may have cleared the bit on later tokens, or the span
 *   may run past T_valid).  The span sums are reduced in a fixed order
 *   (bit-reproducible).
 * mode XMIX_PROBE_LAST: the "last token" condition of a read (Sec. 4.1):
 *   for each request r with a non-empty span whose first token has bit
 *   app_bits[p], logit_out[p][r] = b[p] + w[p,:] . h[cu_seqlens[r+1]-1,:],
 *   score as above; outputs are [n_probe][R_max].
 * h [T_max, d] and w [n_probe, d] of dtype dt; b [n_probe] fp32;
 * app_bits host [n_probe]; cu_seqlens [R_max + 1] int32 (MEAN and LAST:
 * non-decreasing, spans contiguous; a span outside [0, T_max] is not
 * written); the probe reads h as given (call it before any write at the
 * same hook).
 * ws: device workspace of at least xmix_probe_workspace(...) bytes (may be
 * NULL when that is 0).  Requires 1 <= n_probe <= 32. */
size_t xmix_probe_workspace(int32_t T_max, int32_t n_probe, int32_t mode);
xmix_status xmix_probe_score(const void *h, xmix_dtype dt, int32_t d, const xmix_route *rt,
                             const void *w, const float *b, const int32_t *app_bits,
                             int32_t n_probe, int32_t mode, const int32_t *cu_seqlens,
                             int32_t R_max, float *logit_out, float *score_out,
                             void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------- SAE encode + TopK
 * TopK sparse-autoencoder encode of the tokens subscribed to app `app_bit`
 * (sparse autoencoders and feature dictionaries as app artefacts, Sec. 3;
 * feature activations as gate signals, Sec. 4.2):
 *   pre_j = b_enc[j] + W_enc[j,:] . (h[t,:] - b_dec)    for all j < m
 *   the k largest pre_j (equal values: lower j first), ordered by pre
 *   descending;  idx_out[t][q] = j,  val_out[t][q] = bf16(max(pre_j, 0)).
 * Rows t of idx_out/val_out ([T_max, k]) are written only for subscribed t.
 * h [T_max, d] bf16; b_enc [m], b_dec [d] bf16.
 * dict: the encoder dictionary (m latents of width d) as packed once per app
 * by xmix_sae_pack_encoder; dict->d must equal d.
 * c_fold [m] fp32, nullable: b_enc - W_enc . b_dec as produced by
 * xmix_sae_fold_bias.  With c_fold the call never reads b_enc or b_dec and
 * streams the dictionary once; with NULL it folds into the workspace first
 * (one extra read of the dictionary).  The GEMM takes h exactly (bf16 x bf16
 * products, fp32 accumulation), so the fold keeps the subtraction of b_dec
 * exact.
 * Requires d % 256 == 0, m % 256 == 0, 1 <= k <= min(64, m),
 * (m / 256) * k <= 16384.
 * ws: at least xmix_sae_encode_workspace(T_max, d, m, k) bytes.
 * Errors: XMIX_E_INVAL (null pointer, bad size, a dictionary struct not made
 * by xmix_sae_pack_encoder or of another width), XMIX_E_UNSUPPORTED (too
 * many candidates per token), XMIX_E_WORKSPACE. */
size_t xmix_sae_encode_workspace(int32_t T_max, int32_t d, int32_t m, int32_t k);
xmix_status xmix_sae_encode_topk(const uint16_t *h, int32_t d, const xmix_route *rt,
                                 int32_t app_bit, const xmix_sae_dict *dict,
                                 const uint16_t *b_enc, const uint16_t *b_dec,
                                 const float *c_fold, int32_t k,
                                 int32_t *idx_out, uint16_t *val_out,
                                 void *ws, size_t ws_bytes, void *stream);

/* xmix_sae_encode_topk without a workspace argument, for callers that
 * cannot allocate device memory (code under graph capture, tight serving
 * loops, harnesses that forbid allocation).  Same arguments minus ws and
 * ws_bytes, same kernels and results.  The workspace is a device array of
 * XMIX_STATIC_SCRATCH_BYTES inside the library, one per GPU, held until the
 * process ends; the call itself allocates nothing.
 * Limit: xmix_sae_encode_workspace(rt->T_max, d, dict->m, k) must not exceed
 * XMIX_STATIC_SCRATCH_BYTES (16 MiB: e.g. up to 512 token slots at
 * m = 65536, k = 64); larger calls return XMIX_E_UNSUPPORTED and launch
 * nothing.  All calls on one GPU share the array: calls that overlap in
 * time on one GPU (other streams, other threads) race and must be ordered by
 * the caller.  Nothing in the array has to start at zero.
 * Errors: as xmix_sae_encode_topk; XMIX_E_LAUNCH if the array's device
 * address cannot be obtained. */
#define XMIX_STATIC_SCRATCH_BYTES (16 << 20)
xmix_status xmix_sae_encode_topk_noalloc(const uint16_t *h, int32_t d, const xmix_route *rt,
                                         int32_t app_bit, const xmix_sae_dict *dict,
                                         const uint16_t *b_enc, const uint16_t *b_dec,
                                         const float *c_fold, int32_t k, int32_t *idx_out,
                                         uint16_t *val_out, void *stream);

/* The two stages of xmix_sae_encode_topk, callable on their own (same
 * arguments and workspace; run them in this order on one stream):
 *   candidates: the GEMM; for every 256-latent slice of the dictionary and
 *               every subscribed token, a threshold tau is chosen from the
 *               slice's own values and every latent with pre >= tau is kept
 *               in the workspace together with the slice's bound, a value
 *               at most tau that every latent it does not keep lies below
 *               (up to 1024 token slots the next value above the largest
 *               one it does not keep);
 *   merge:      the exact top-k per token, written to idx_out / val_out.
 *               The top-k of the kept latents is the top-k of all m
 *               latents when its k-th value is >= every slice's bound (a
 *               latent left out lies below its slice's bound); otherwise
 *               the merge recomputes slices in descending order of that
 *               bound until no slice left can hide a winner (same result,
 *               slower; it happens only when the winners crowd into a few
 *               slices or tie across whole slices).
 * The same certificate lets a dictionary be split across devices by latent
 * slices: exchange the kept candidates and thresholds, then merge. */
xmix_status xmix_sae_encode_candidates(const uint16_t *h, int32_t d, const xmix_route *rt,
                                       int32_t app_bit, const xmix_sae_dict *dict,
                                       const uint16_t *b_enc, const uint16_t *b_dec,
                                       const float *c_fold, int32_t k,
                                       void *ws, size_t ws_bytes, void *stream);
xmix_status xmix_sae_merge_topk(const uint16_t *h, int32_t d, const xmix_route *rt,
                                int32_t app_bit, const xmix_sae_dict *dict,
                                const float *c_fold, int32_t k,
                                int32_t *idx_out, uint16_t *val_out,
                                void *ws, size_t ws_bytes, void *stream);

/* Route build and the candidates stage in one launch, for a step whose
 * first consumer of the routing is an SAE encode (per-request toggling
 * inside the batch, Sec. 4.2-4.3; the first stage of the encode above).
 * Same effect as
 *   xmix_route_build(req_of_token, T_valid, sub_mask, R_max, rt, err_word)
 * followed by
 *   xmix_sae_encode_candidates(h, d, rt, app_bit, dict, ...):
 * the route's tok_mask, app_count, app_tokens and err_word hold exactly what
 * the route build writes, and the candidates are the same.  Up to 1024
 * token slots the encode kernel builds the routing itself (every workgroup
 * lists its app's tokens in LDS; the separate launch and its kernel
 * boundary are saved); above that the two launches are made.  Arguments are
 * those of the two calls; errors as for them. */
xmix_status xmix_route_sae_encode_candidates(const int32_t *req_of_token, const int32_t *T_valid,
                                             const uint32_t *sub_mask, int32_t R_max,
                                             const xmix_route *rt, uint32_t *err_word,
                                             const uint16_t *h, int32_t d, int32_t app_bit,
                                             const xmix_sae_dict *dict, const uint16_t *b_enc,
                                             const uint16_t *b_dec, const float *c_fold,
                                             int32_t k, void *ws, size_t ws_bytes,
                                             void *stream);

/* Encode + TopK with the readback of each encoded row fused in (the merge
 * writes the ring rows itself, saving the separate compaction pass).  Same
 * arguments and results as xmix_sae_encode_topk / xmix_sae_merge_topk, plus
 * the readback of xmix_readback_compact for segments (idx_out, val_out):
 * rows {t, req_of_token[t], layer_id, app_id} + idx[k] (int32) + val[k]
 * (bf16) in ascending token order at (head + i) mod capacity, only the last
 * `capacity` rows of the call written, head advanced by the count.
 * ring->row_bytes must equal 16 + 6 * k.  Calls that overlap on one ring
 * race, as for xmix_readback_compact. */
xmix_status xmix_sae_encode_topk_ring(const uint16_t *h, int32_t d, const xmix_route *rt,
                                      int32_t app_bit, const xmix_sae_dict *dict,
                                      const uint16_t *b_enc, const uint16_t *b_dec,
                                      const float *c_fold, int32_t k,
                                      int32_t *idx_out, uint16_t *val_out, void *ws,
                                      size_t ws_bytes, const int32_t *req_of_token,
                                      int32_t layer_id, int32_t app_id, const xmix_ring *ring,
                                      void *stream);
xmix_status xmix_sae_merge_topk_ring(const uint16_t *h, int32_t d, const xmix_route *rt,
                                     int32_t app_bit, const xmix_sae_dict *dict,
                                     const float *c_fold, int32_t k,
                                     int32_t *idx_out, uint16_t *val_out, void *ws,
                                     size_t ws_bytes, const int32_t *req_of_token,
                                     int32_t layer_id, int32_t app_id, const xmix_ring *ring,
                                     void *stream);

/* One SAE app of a batched encode: the per-app arguments of
 * xmix_sae_encode_topk (ring == NULL) or xmix_sae_encode_topk_ring (ring
 * set, rows with the given app_id), with the same requirements. */
typedef struct {
    int32_t app_bit;
    const xmix_sae_dict *dict;
    const uint16_t *b_enc;  /* read only when c_fold is NULL */
    const uint16_t *b_dec;
    const float *c_fold;    /* may be NULL: folded into ws first */
    int32_t k;
    int32_t *idx_out;       /* [T_max, k] */
    uint16_t *val_out;      /* [T_max, k] */
    void *ws;               /* this app's own workspace */
    size_t ws_bytes;
    const xmix_ring *ring;  /* NULL: no readback */
    int32_t app_id;
} xmix_sae_app;

/* The SAE apps of one hook (Sec. 4.2, several apps composed at one layer)
 * encoded together: results identical to one xmix_sae_encode_topk (or
 * _ring) call per app, in any order (every app reads h as given).  At
 * decode shapes (T_max <= 1024) the candidates of up to 8 apps come from one
 * launch whose apps' tiles follow each other (a CU that finishes its slice
 * of one app takes a slice of the next) and their merges from one more, so
 * the apps pay two launches together; larger batches run the apps one after
 * the other.  req_of_token [T_max] is required when an app has a ring.
 * Host array `apps` [n_sae], 1 <= n_sae <= 32. */
xmix_status xmix_sae_encode_topk_multi(const uint16_t *h, int32_t d, const xmix_route *rt,
                                       int32_t n_sae, const xmix_sae_app *apps,
                                       const int32_t *req_of_token, int32_t layer_id,
                                       void *stream);
/* The same with the step's routing built by the first launch (as
 * xmix_route_sae_encode_candidates does): results identical to
 * xmix_route_build followed by xmix_sae_encode_topk_multi. */
xmix_status xmix_route_sae_encode_topk_multi(const int32_t *req_of_token,
                                             const int32_t *T_valid, const uint32_t *sub_mask,
                                             int32_t R_max, const xmix_route *rt,
                                             uint32_t *err_word, const uint16_t *h, int32_t d,
                                             int32_t n_sae, const xmix_sae_app *apps,
                                             int32_t layer_id, void *stream);

/* One-time repack of a row-major encoder dictionary W_enc [m, d] (bf16)
 * into the tiled layout the encode kernels stream (same bytes, permuted),
 * written to W_packed (device, m * d bf16, caller-owned, not overlapping
 * W_enc).  *dict (host) is filled to describe W_packed; it stays valid as
 * long as W_packed does.  Requires m % 256 == 0, d % 256 == 0. */
xmix_status xmix_sae_pack_encoder(const uint16_t *W_enc, int32_t m, int32_t d,
                                  uint16_t *W_packed, xmix_sae_dict *dict, void *stream);

/* One-time fold of the encoder biases, run when an SAE app is loaded:
 *   c_fold[j] = b_enc[j] - W_enc[j,:] . b_dec   (fp32), c_fold [dict->m]. */
xmix_status xmix_sae_fold_bias(const xmix_sae_dict *dict, const uint16_t *b_enc,
                               const uint16_t *b_dec, float *c_fold, void *stream);

/* ------------------------------------------------------- SAE clamp-decode
 * Feature clamp with the decoded delta added back (a Write whose payload
 * comes from a Read of the same hook, Sec. 3).  For each token t with bit
 * app_bit:
 *   z_j     = the encoded value of j if j is in idx[t,:], else 0
 *   delta   = sum_q (clamp_vals[q] - z_{clamp_ids[q]}) * W_dec[clamp_ids[q],:]
 *   h[t,:] <- bf16( h[t,:] + delta )        (fp32 accumulation, one RNE)
 * which equals decode(z') - decode(z) with z' = z clamped: the SAE's
 * reconstruction error stays in the residual.  Only n_clamp rows of W_dec
 * are read.
 * h [T_max, d] bf16 in place; idx/val [T_max, k] from xmix_sae_encode_topk;
 * W_dec [m, d] bf16; clamp_ids [n_clamp] int32 in [0, m) and clamp_vals
 * [n_clamp] fp32 (device, may change between replays); delta_out
 * [T_max, d] fp32, nullable, receives delta of every processed token.
 * Requires d % 8 == 0, 1 <= k <= 64, 1 <= n_clamp <= 16. */
xmix_status xmix_sae_clamp_decode(uint16_t *h, int32_t d, const xmix_route *rt,
                                  int32_t app_bit, const int32_t *idx,
                                  const uint16_t *val, int32_t k,
                                  const uint16_t *W_dec, int32_t m,
                                  const int32_t *clamp_ids, const float *clamp_vals,
                                  int32_t n_clamp, float *delta_out, void *stream);

/* One clamp app of a batched clamp-decode: the per-app arguments of
 * xmix_sae_clamp_decode, with the same requirements. */
typedef struct {
    int32_t app_bit;
    const int32_t *idx;
    const uint16_t *val;
    int32_t k;
    const uint16_t *W_dec;
    int32_t m;
    const int32_t *clamp_ids;
    const float *clamp_vals;
    int32_t n_clamp;
    float *delta_out;  /* may be NULL */
} xmix_sae_clamp_app;

/* Several clamp apps of one hook in one launch: h ends identical to one
 * xmix_sae_clamp_decode call per app in the order of `apps` (each app's
 * delta rounded in as that call rounds it; a token's row is read and written
 * once).  Host array `apps` [n], 1 <= n <= 32. */
xmix_status xmix_sae_clamp_decode_multi(uint16_t *h, int32_t d, const xmix_route *rt,
                                        int32_t n, const xmix_sae_clamp_app *apps,
                                        void *stream);

/* ----------------------------------------------------- readback compaction
 * Buffer-mediated readback (Sec. 1; Sec. 4.2 "State and dataflow"): the
 * tokens with bit app_bit, ascending, are appended to `ring`:
 *   slot (head + i) mod capacity <- {t, req_of_token[t], layer_id, app_id}
 *                                   ++ seg[0] row t ++ ... ++ seg[n-1] row t
 *   head += count
 * A later row overwrites an older one in the same slot (only the last
 * `capacity` rows of one call are written).
 * seg_rows  host [n_seg] device pointers; segment s of row t starts at
 *           seg_rows[s] + t * seg_bytes[s].
 * seg_bytes host [n_seg], each a positive even number (rows of any k:
 *           an SAE row is idx[k] int32 then val[k] bf16);
 *           16 + sum(seg_bytes) must equal ring->row_bytes.
 * ring      host struct; slots 4-byte aligned, head 8-byte aligned,
 *           row_bytes even.  Segment rows must be 2-byte aligned.
 * Requires 1 <= n_seg <= 4. */
xmix_status xmix_readback_compact(const void *const *seg_rows, const int32_t *seg_bytes,
                                  int32_t n_seg, const xmix_route *rt, int32_t app_bit,
                                  const int32_t *req_of_token, int32_t layer_id,
                                  int32_t app_id, const xmix_ring *ring, void *stream);

/* ------------------------------------------------------------ step graphs
 * A hook step captured once and replayed, with the kernel-node parameter
 * update of Sec. 4.3 (CUDA-graph-safe kernel design: explicit node handles
 * kept for the dynamic kernels, their arguments updated before launch
 * instead of recapturing; graph-level toggling).
 *
 * xmix_graph_begin starts capturing `stream` (thread-local capture mode);
 * the caller then enqueues library calls on it; xmix_graph_end stops the
 * capture, instantiates the graph and returns it in *out, keeping the handle
 * and the argument values of every kernel node launched by this library.
 * The calls in between are recorded, not run; no call that synchronises may
 * be made on the stream meanwhile.  stream must not be the null stream.
 *
 * xmix_graph_redirect: every pointer argument of those nodes that holds
 * `from` (also a pointer inside the app descriptors of the batched calls:
 * dictionaries, biases, outputs, clamp values, rings) is set to `to` for all
 * later launches; pointers into the middle of `from` (such as parts of a
 * workspace) are not changed (one
 * hipGraphExecKernelNodeSetParams per affected node; the graph is neither
 * recaptured nor re-instantiated).  `to` must be a device buffer of the same
 * size and layout as `from`.  *n_args (optional) receives the number of
 * arguments changed.  The library's own design keeps every per-step value
 * (subscriptions, alpha, thresholds, clamp values, offsets) in device
 * memory, where a captured graph reads the current contents without any
 * update; redirection serves switching between whole parameter buffers.
 *
 * xmix_graph_launch enqueues one replay on `stream`.  xmix_graph_kernel_nodes
 * returns the number of the library's kernel nodes in the graph.
 * xmix_graph_destroy releases the graph (the caller must not destroy it
 * while a launch may still be running).
 *
 * Ownership: the graph (host memory and HIP graph objects) belongs to the
 * caller after xmix_graph_end and is freed by xmix_graph_destroy.
 * Errors: XMIX_E_INVAL for a null argument; XMIX_E_LAUNCH when the runtime
 * rejects the capture, the instantiation, an update or a launch. */
typedef struct xmix_graph xmix_graph;
xmix_status xmix_graph_begin(void *stream);
xmix_status xmix_graph_end(void *stream, xmix_graph **out);
int32_t xmix_graph_kernel_nodes(const xmix_graph *g);
xmix_status xmix_graph_redirect(xmix_graph *g, const void *from, const void *to,
                                int32_t *n_args);
xmix_status xmix_graph_launch(const xmix_graph *g, void *stream);
void xmix_graph_destroy(xmix_graph *g);

#ifdef __cplusplus
}
#endif

#endif /* XMIX_H */
