/*
 * Drives every entry point of the CPU oracle (oracle/oracle.c) and of the
 * input generator (synth/gen.c) on small inputs, edge cases included, for a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer.  Test
 * infrastructure only: it checks memory safety and defined behaviour of the
 * host code, not its values (the pins do that).  Exit status 0 = clean.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint16_t oracle_round_bf16(double x);
void oracle_set_num_threads(int n);
int oracle_num_threads(void);
void oracle_route(const int32_t *req, int32_t T_valid, int32_t T_max, const uint32_t *sub,
                  int32_t R_max, int32_t n_apps, uint32_t *tok_mask, int32_t *count,
                  int32_t *app_tokens, uint32_t *err);
void oracle_route_gate(int32_t T_max, uint32_t *tok_mask, int32_t *app_count,
                       int32_t *app_tokens, int32_t app_bit, const float *signal,
                       int32_t signal_per_request, const int32_t *req_of_token,
                       int32_t n_signal, int32_t signal_bit, float threshold);
void oracle_route_trigger(int32_t T_max, uint32_t *tok_mask, int32_t *app_count,
                          int32_t *app_tokens, int32_t app_bit, const int32_t *token_ids,
                          const uint32_t *vocab_bits, int32_t vocab_size);
void oracle_steer(void *h, int is_bf16, int32_t T_max, int32_t d, const uint32_t *tok_mask,
                  const int32_t *req, const void *v, const int32_t *app_bits,
                  const float *alpha, int32_t n_steer);
void oracle_router_write(void *logits, int is_bf16, int32_t T_max, int32_t n_experts,
                         const uint32_t *tok_mask, const int32_t *app_bits,
                         const float *offsets, int32_t n_router);
void oracle_probe_token(const void *h, int is_bf16, int32_t T_max, int32_t d,
                        const uint32_t *tok_mask, const void *w, const float *b,
                        const int32_t *app_bits, int32_t n_probe, double *logit,
                        double *score);
void oracle_probe_mean(const void *h, int is_bf16, int32_t T_max, int32_t d,
                       const uint32_t *tok_mask, const void *w, const float *b,
                       const int32_t *app_bits, int32_t n_probe, const int32_t *cu_seqlens,
                       int32_t R, double *logit, double *score);
void oracle_probe_last(const void *h, int is_bf16, int32_t T_max, int32_t d,
                       const uint32_t *tok_mask, const void *w, const float *b,
                       const int32_t *app_bits, int32_t n_probe, const int32_t *cu_seqlens,
                       int32_t R, double *logit, double *score);
void oracle_topk(const double *pre, int32_t m, int32_t k, int32_t *idx, double *val_exact,
                 uint16_t *val_bf16);
void oracle_sae_encode(const uint16_t *h, int32_t d, const int32_t *tokens, int32_t n_tok,
                       const uint16_t *W_enc, const uint16_t *b_enc, const uint16_t *b_dec,
                       int32_t m, int32_t k, int32_t *idx_out, uint16_t *val_out,
                       double *val_exact_out, double *pre_out);
void oracle_clamp_decode(uint16_t *h, int32_t T_max, int32_t d, const uint32_t *tok_mask,
                         int32_t app_bit, const int32_t *idx, const uint16_t *val, int32_t k,
                         const uint16_t *W_dec, int32_t m, const int32_t *clamp_ids,
                         const float *clamp_vals, int32_t n_clamp, double *delta_out);
void oracle_compact(const uint8_t *const *seg, const int32_t *seg_bytes, int32_t n_seg,
                    const uint32_t *tok_mask, int32_t T_max, int32_t app_bit,
                    const int32_t *req, int32_t layer_id, int32_t app_id, uint8_t *slots,
                    int32_t capacity, int32_t row_bytes, uint64_t *head);

void synth_normal_bf16(uint64_t key, int64_t n, double mean, double std,
                       const double *chan_scale, int64_t row_len, uint16_t *out);
void synth_normal_f32(uint64_t key, int64_t n, double mean, double std,
                      const double *chan_scale, int64_t row_len, float *out);
void synth_uniform_f32(uint64_t key, int64_t n, double lo, double hi, float *out);
void synth_uniform_f64(uint64_t key, int64_t n, double *out);
void synth_bits(uint64_t key, int64_t n, uint64_t *out);
void synth_rownorm_bf16(const uint16_t *in, int64_t rows, int64_t cols, uint16_t *out);
uint16_t synth_bf16_from_double(double x);

/* exactly-sized heap blocks, so that an overrun is caught at its first byte */
#define NEW(type, n) ((type *)calloc((size_t)(n) > 0 ? (size_t)(n) : 1, sizeof(type)))

int main(void) {
    const int32_t T = 37, d = 24, R = 5, n_apps = 6;
    /* generator */
    uint16_t *hb = NEW(uint16_t, T * d);
    float *hf = NEW(float, T * d);
    double *cs = NEW(double, d);
    for (int i = 0; i < d; ++i) cs[i] = (i % 5 == 0) ? 20.0 : 1.0;
    synth_normal_bf16(11, (int64_t)T * d, 0.0, 1.0, cs, d, hb);
    synth_normal_f32(12, (int64_t)T * d, 0.5, 2.0, NULL, 1, hf);
    float *uf = NEW(float, 9);
    synth_uniform_f32(13, 9, -8.0, 8.0, uf);
    double *ud = NEW(double, 9);
    synth_uniform_f64(14, 9, ud);
    uint64_t *bits = NEW(uint64_t, 9);
    synth_bits(15, 9, bits);
    synth_normal_bf16(16, 0, 0.0, 1.0, NULL, 1, hb);  /* empty draw */
    const double edge[] = {0.0, -0.0, 1e-45, -3e38, 3.4e38, 1e300, -1e300, NAN, INFINITY, 1.0};
    for (int i = 0; i < 10; ++i) {
        (void)synth_bf16_from_double(edge[i]);
        (void)oracle_round_bf16(edge[i]);
    }

    /* routing: padding, bad ids, T_valid beyond T_max */
    int32_t *req = NEW(int32_t, T);
    for (int t = 0; t < T; ++t) req[t] = (t % 7 == 3) ? -1 : (t % 11 == 5) ? R + 2 : t % R;
    uint32_t *sub = NEW(uint32_t, R);
    for (int r = 0; r < R; ++r) sub[r] = 0x3Fu ^ (1u << r);
    uint32_t *tm = NEW(uint32_t, T);
    int32_t *cnt = NEW(int32_t, n_apps), *lists = NEW(int32_t, n_apps * T);
    uint32_t err = 0;
    oracle_route(req, T + 4, T, sub, R, n_apps, tm, cnt, lists, &err);
    oracle_route(req, -1, T, sub, R, n_apps, tm, cnt, lists, &err);
    oracle_route(req, T - 2, T, sub, R, n_apps, tm, cnt, lists, &err);
    float *sig = NEW(float, T);
    for (int t = 0; t < T; ++t) sig[t] = (t % 9 == 0) ? NAN : (float)(t % 4) - 1.5f;
    oracle_route_gate(T, tm, cnt, lists, 2, sig, 0, NULL, T, 1, 0.0f);
    oracle_route_gate(T, tm, cnt, lists, 3, sig, 1, req, R, -1, -0.5f);
    int32_t *ids = NEW(int32_t, T);
    for (int t = 0; t < T; ++t) ids[t] = (t * 13) % 70 - 3;  /* some out of range */
    uint32_t *vocab = NEW(uint32_t, 2);
    vocab[0] = 0xA5A5A5A5u;
    vocab[1] = 0x0000000Fu;
    oracle_route_trigger(T, tm, cnt, lists, 4, ids, vocab, 36);

    /* steering, router write (bf16 and fp32) */
    const int32_t sb[2] = {0, 1};
    uint16_t *vb = NEW(uint16_t, 2 * d);
    float *vf = NEW(float, 2 * d);
    synth_normal_bf16(21, 2 * d, 0.0, 0.2, NULL, 1, vb);
    synth_normal_f32(22, 2 * d, 0.0, 0.2, NULL, 1, vf);
    float *alpha = NEW(float, R * 2);
    synth_uniform_f32(23, R * 2, -8.0, 8.0, alpha);
    oracle_steer(hb, 1, T, d, tm, req, vb, sb, alpha, 2);
    oracle_steer(hf, 0, T, d, tm, req, vf, sb, alpha, 2);
    const int32_t E = 8;
    uint16_t *lgb = NEW(uint16_t, T * E);
    float *lgf = NEW(float, T * E), *off = NEW(float, 2 * E);
    synth_uniform_f32(24, 2 * E, -1.0, 1.0, off);
    off[3] = -INFINITY;
    oracle_router_write(lgb, 1, T, E, tm, sb, off, 2);
    oracle_router_write(lgf, 0, T, E, tm, sb, off, 2);

    /* probes: token, mean (with an empty span), last */
    const int32_t pb[2] = {2, 5};
    float *pbias = NEW(float, 2);
    double *lo = NEW(double, 2 * T), *so = NEW(double, 2 * T);
    oracle_probe_token(hb, 1, T, d, tm, vb, pbias, pb, 2, lo, so);
    oracle_probe_token(hf, 0, T, d, tm, vf, pbias, pb, 2, lo, so);
    int32_t cu[6] = {0, 9, 9, 20, 31, 37};
    double *lm = NEW(double, 2 * R), *sm = NEW(double, 2 * R);
    oracle_probe_mean(hb, 1, T, d, tm, vb, pbias, pb, 2, cu, R, lm, sm);
    oracle_probe_last(hf, 0, T, d, tm, vf, pbias, pb, 2, cu, R, lm, sm);

    /* top-k and SAE encode (k = m included), clamp-decode */
    const int32_t m = 40, k = 40;
    uint16_t *W = NEW(uint16_t, m * d), *be = NEW(uint16_t, m), *bd = NEW(uint16_t, d);
    synth_normal_bf16(31, (int64_t)m * d, 0.0, 0.2, NULL, 1, W);
    synth_normal_bf16(32, m, 0.0, 0.1, NULL, 1, be);
    synth_normal_bf16(33, d, 0.0, 0.1, NULL, 1, bd);
    int32_t toks[3] = {0, 17, 36};
    int32_t *idx = NEW(int32_t, 3 * k);
    uint16_t *val = NEW(uint16_t, 3 * k);
    double *vx = NEW(double, 3 * k), *pre = NEW(double, 3 * m);
    oracle_sae_encode(hb, d, toks, 3, W, be, bd, m, k, idx, val, vx, pre);
    oracle_sae_encode(hb, d, toks, 3, W, be, bd, m, 1, idx, val, NULL, NULL);
    oracle_topk(pre, m, 7, idx, vx, val);
    uint16_t *Wd = NEW(uint16_t, m * d);
    synth_rownorm_bf16(W, m, d, Wd);
    int32_t *idx_t = NEW(int32_t, T * 4);
    uint16_t *val_t = NEW(uint16_t, T * 4);
    for (int i = 0; i < T * 4; ++i) { idx_t[i] = (i * 7) % m; val_t[i] = 0x3F80; }
    const int32_t cid[3] = {0, 5, 39};
    const float cval[3] = {10.0f, 0.0f, -2.0f};
    double *delta = NEW(double, T * d);
    oracle_clamp_decode(hb, T, d, tm, 0, idx_t, val_t, 4, Wd, m, cid, cval, 3, delta);
    oracle_clamp_decode(hb, T, d, tm, 1, idx_t, val_t, 4, Wd, m, cid, cval, 3, NULL);

    /* compaction: odd-sized rows, wrap-around, more rows than slots */
    const int32_t kk = 5, cap = 6, row = 16 + 6 * kk;
    uint8_t *seg0 = NEW(uint8_t, T * 4 * kk), *seg1 = NEW(uint8_t, T * 2 * kk);
    const uint8_t *segs[2] = {seg0, seg1};
    const int32_t seg_bytes[2] = {4 * kk, 2 * kk};
    uint8_t *slots = NEW(uint8_t, cap * row);
    uint64_t head = 3;
    for (int rep = 0; rep < 3; ++rep)
        oracle_compact(segs, seg_bytes, 2, tm, T, 1, req, 7, 1, slots, cap, row, &head);

    oracle_set_num_threads(1);
    oracle_sae_encode(hb, d, toks, 3, W, be, bd, m, k, idx, val, vx, pre);
    oracle_set_num_threads(4);
    printf("sanitized oracle and generator ok (threads %d)\n", oracle_num_threads());
    free(hb); free(hf); free(cs); free(uf); free(ud); free(bits); free(req); free(sub);
    free(tm); free(cnt); free(lists); free(sig); free(ids); free(vocab); free(vb); free(vf);
    free(alpha); free(lgb); free(lgf); free(off); free(pbias); free(lo); free(so); free(lm);
    free(sm); free(W); free(be); free(bd); free(idx); free(val); free(vx); free(pre);
    free(Wd); free(idx_t); free(val_t); free(delta); free(seg0); free(seg1); free(slots);
    return 0;
}
