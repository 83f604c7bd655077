// C ABI of the hook-step library: host-side argument checks, workspace
// sizing and launch.  Nothing here allocates, synchronises or copies; every
// call only enqueues kernels on the caller's stream.
#include <stdint.h>
#include <string.h>

#include "../../include/xmix.h"
#include "launch.hpp"

using namespace xmix;

namespace {

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

xmix_status launched(hipError_t e) { return e == hipSuccess ? XMIX_OK : XMIX_E_LAUNCH; }

bool route_ok(const xmix_route* rt) {
    return rt && rt->tok_mask && rt->app_count && rt->app_tokens && rt->T_max >= 1 &&
           rt->n_apps >= 1 && rt->n_apps <= XMIX_MAX_APPS;
}

bool bits_ok(const int32_t* bits, int32_t n, int32_t n_apps, BitList* out) {
    if (!bits || n < 1 || n > 32) return false;
    memset(out, 0, sizeof(*out));
    for (int i = 0; i < n; ++i) {
        if (bits[i] < 0 || bits[i] >= n_apps) return false;
        out->bit[i] = bits[i];
    }
    return true;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// A dictionary struct made by xmix_sae_pack_encoder, of width d (d < 0:
// any width).
bool dict_ok(const xmix_sae_dict* w, int32_t d) {
    return w && w->layout == XMIX_SAE_DICT_TILED && w->pieces && aligned16(w->pieces) &&
           w->m >= 256 && w->m % 256 == 0 && w->d >= 256 && w->d % 256 == 0 &&
           (d < 0 || w->d == d);
}

const int32_t* app_list(const xmix_route* rt, int32_t a) {
    return rt->app_tokens + static_cast<int64_t>(a) * rt->T_max;
}

}  // namespace

extern "C" {

const char* xmix_status_string(xmix_status s) {
    switch (s) {
        case XMIX_OK: return "ok";
        case XMIX_E_INVAL: return "invalid argument";
        case XMIX_E_UNSUPPORTED: return "unsupported size or combination";
        case XMIX_E_WORKSPACE: return "workspace missing or too small";
        case XMIX_E_LAUNCH: return "kernel launch failed";
    }
    return "unknown status";
}

const char* xmix_version(void) { return "xmix-gfx950 0.1"; }

xmix_status xmix_route_build(const int32_t* req_of_token, const int32_t* T_valid,
                             const uint32_t* sub_mask, int32_t R_max, const xmix_route* rt,
                             uint32_t* err_word, void* stream) {
    if (!req_of_token || !T_valid || !sub_mask || !err_word || R_max < 1 || !route_ok(rt))
        return XMIX_E_INVAL;
    return launched(launch_route_build(req_of_token, T_valid, sub_mask, R_max, rt->T_max,
                                       rt->n_apps, rt->tok_mask, rt->app_count, rt->app_tokens,
                                       err_word, as_stream(stream)));
}

xmix_status xmix_route_gate(const xmix_route* rt, int32_t app_bit, const float* signal,
                            const int32_t* req_of_token, int32_t n_signal, int32_t signal_bit,
                            const float* threshold, void* stream) {
    if (!route_ok(rt) || !signal || !threshold || app_bit < 0 || app_bit >= rt->n_apps ||
        signal_bit >= rt->n_apps || n_signal < 1)
        return XMIX_E_INVAL;
    if (!req_of_token && n_signal < rt->T_max) return XMIX_E_INVAL;  // per-token signal row
    return launched(launch_route_gate(rt->T_max, app_bit, rt->tok_mask, rt->app_count,
                                      rt->app_tokens, signal, req_of_token, n_signal,
                                      signal_bit < 0 ? -1 : signal_bit, threshold,
                                      as_stream(stream)));
}

xmix_status xmix_route_trigger(const xmix_route* rt, int32_t app_bit, const int32_t* token_ids,
                               const uint32_t* vocab_bits, int32_t vocab_size, void* stream) {
    if (!route_ok(rt) || !token_ids || !vocab_bits || vocab_size < 1 || app_bit < 0 ||
        app_bit >= rt->n_apps)
        return XMIX_E_INVAL;
    return launched(launch_route_trigger(rt->T_max, app_bit, rt->tok_mask, rt->app_count,
                                         rt->app_tokens, token_ids, vocab_bits, vocab_size,
                                         as_stream(stream)));
}

xmix_status xmix_steer_apply(void* h, xmix_dtype dt, int32_t d, const xmix_route* rt,
                             const int32_t* req_of_token, const void* vecs,
                             const int32_t* app_bits, const float* alpha, int32_t n_steer,
                             int32_t R_max, void* stream) {
    if (!h || !req_of_token || !vecs || !alpha || !route_ok(rt) || R_max < 1 || d < 1)
        return XMIX_E_INVAL;
    if (dt != XMIX_BF16 && dt != XMIX_F32) return XMIX_E_INVAL;
    if (d % (dt == XMIX_BF16 ? 8 : 4) != 0 || !aligned16(h) || !aligned16(vecs))
        return XMIX_E_INVAL;
    BitList bits;
    if (!bits_ok(app_bits, n_steer, rt->n_apps, &bits)) return XMIX_E_INVAL;
    return launched(launch_steer(h, dt == XMIX_BF16, d, rt->T_max, rt->tok_mask, req_of_token,
                                 vecs, bits, alpha, n_steer, as_stream(stream)));
}

xmix_status xmix_steer_probe(void* h, xmix_dtype dt, int32_t d, const xmix_route* rt,
                             const int32_t* req_of_token, const void* vecs,
                             const int32_t* steer_bits, const float* alpha, int32_t n_steer,
                             int32_t R_max, const void* w, const float* b,
                             const int32_t* probe_bits, int32_t n_probe, float* logit_out,
                             float* score_out, void* stream) {
    if (!h || !req_of_token || !vecs || !alpha || !w || !b || !logit_out || !score_out ||
        !route_ok(rt) || R_max < 1 || d < 1)
        return XMIX_E_INVAL;
    if (dt != XMIX_BF16 && dt != XMIX_F32) return XMIX_E_INVAL;
    if (d % (dt == XMIX_BF16 ? 8 : 4) != 0 || !aligned16(h) || !aligned16(vecs) || !aligned16(w))
        return XMIX_E_INVAL;
    BitList sbits, pbits;
    if (!bits_ok(steer_bits, n_steer, rt->n_apps, &sbits)) return XMIX_E_INVAL;
    if (!bits_ok(probe_bits, n_probe, rt->n_apps, &pbits)) return XMIX_E_INVAL;
    return launched(launch_steer_probe(h, dt == XMIX_BF16, d, rt->T_max, rt->tok_mask,
                                       req_of_token, vecs, sbits, alpha, n_steer, w, b, pbits,
                                       n_probe, logit_out, score_out, as_stream(stream)));
}

xmix_status xmix_route_steer_probe(const int32_t* req_of_token, const int32_t* T_valid,
                                   const uint32_t* sub_mask, int32_t R_max, const xmix_route* rt,
                                   uint32_t* err_word, void* h, xmix_dtype dt, int32_t d,
                                   const void* vecs, const int32_t* steer_bits,
                                   const float* alpha, int32_t n_steer, const void* w,
                                   const float* b, const int32_t* probe_bits, int32_t n_probe,
                                   float* logit_out, float* score_out, void* stream) {
    if (!req_of_token || !T_valid || !sub_mask || !err_word || R_max < 1) return XMIX_E_INVAL;
    if (!h || !vecs || !alpha || !w || !b || !logit_out || !score_out || !route_ok(rt) || d < 1)
        return XMIX_E_INVAL;
    if (dt != XMIX_BF16 && dt != XMIX_F32) return XMIX_E_INVAL;
    if (d % (dt == XMIX_BF16 ? 8 : 4) != 0 || !aligned16(h) || !aligned16(vecs) || !aligned16(w))
        return XMIX_E_INVAL;
    BitList sbits, pbits;
    if (!bits_ok(steer_bits, n_steer, rt->n_apps, &sbits)) return XMIX_E_INVAL;
    if (!bits_ok(probe_bits, n_probe, rt->n_apps, &pbits)) return XMIX_E_INVAL;
    RouteIn r;
    r.req = req_of_token;
    r.T_valid = T_valid;
    r.sub = sub_mask;
    r.R_max = R_max;
    r.n_apps = rt->n_apps;
    r.tok_mask = rt->tok_mask;
    r.app_count = rt->app_count;
    r.app_tokens = rt->app_tokens;
    r.err_word = err_word;
    return launched(launch_steer_probe(h, dt == XMIX_BF16, d, rt->T_max, rt->tok_mask,
                                       req_of_token, vecs, sbits, alpha, n_steer, w, b, pbits,
                                       n_probe, logit_out, score_out, as_stream(stream), &r));
}

xmix_status xmix_router_write(void* logits, xmix_dtype dt, int32_t n_experts,
                              const xmix_route* rt, const int32_t* app_bits,
                              const float* offsets, int32_t n_router, void* stream) {
    if (!logits || !offsets || !route_ok(rt) || n_experts < 1) return XMIX_E_INVAL;
    if (dt != XMIX_BF16 && dt != XMIX_F32) return XMIX_E_INVAL;
    if (reinterpret_cast<uintptr_t>(logits) % (dt == XMIX_BF16 ? 2u : 4u) != 0 ||
        reinterpret_cast<uintptr_t>(offsets) % 4u != 0)
        return XMIX_E_INVAL;
    if (static_cast<int64_t>(rt->T_max) * n_experts > INT32_MAX) return XMIX_E_UNSUPPORTED;
    BitList bits;
    if (!bits_ok(app_bits, n_router, rt->n_apps, &bits)) return XMIX_E_INVAL;
    return launched(launch_router_write(logits, dt == XMIX_BF16, n_experts, rt->T_max,
                                        rt->tok_mask, bits, offsets, n_router,
                                        as_stream(stream)));
}

size_t xmix_probe_workspace(int32_t T_max, int32_t n_probe, int32_t mode) {
    if (mode != XMIX_PROBE_MEAN || T_max < 1 || n_probe < 1) return 0;
    return static_cast<size_t>(T_max) * static_cast<size_t>(n_probe) * sizeof(float);
}

xmix_status xmix_probe_score(const void* h, xmix_dtype dt, int32_t d, const xmix_route* rt,
                             const void* w, const float* b, const int32_t* app_bits,
                             int32_t n_probe, int32_t mode, const int32_t* cu_seqlens,
                             int32_t R_max, float* logit_out, float* score_out, void* ws,
                             size_t ws_bytes, void* stream) {
    if (!h || !w || !b || !logit_out || !score_out || !route_ok(rt) || d < 1) return XMIX_E_INVAL;
    if (dt != XMIX_BF16 && dt != XMIX_F32) return XMIX_E_INVAL;
    if (d % (dt == XMIX_BF16 ? 8 : 4) != 0 || !aligned16(h) || !aligned16(w)) return XMIX_E_INVAL;
    if (mode != XMIX_PROBE_TOKEN && mode != XMIX_PROBE_MEAN && mode != XMIX_PROBE_LAST)
        return XMIX_E_INVAL;
    if (mode != XMIX_PROBE_TOKEN && (!cu_seqlens || R_max < 1)) return XMIX_E_INVAL;
    BitList bits;
    if (!bits_ok(app_bits, n_probe, rt->n_apps, &bits)) return XMIX_E_INVAL;
    const size_t need = xmix_probe_workspace(rt->T_max, n_probe, mode);
    if (need && (!ws || ws_bytes < need)) return XMIX_E_WORKSPACE;
    return launched(launch_probe(h, dt == XMIX_BF16, d, rt->T_max, rt->tok_mask, w, b, bits,
                                 n_probe, mode, cu_seqlens, R_max, logit_out, score_out,
                                 static_cast<float*>(ws), as_stream(stream)));
}

size_t xmix_sae_encode_workspace(int32_t T_max, int32_t d, int32_t m, int32_t k) {
    if (T_max < 1 || d < 1 || m < 256 || k < 1) return 0;
    // folded bias (used when the caller passes none), then the candidates
    // (and, for many token slots, the staged token rows)
    const size_t fold = (static_cast<size_t>(m) * sizeof(float) + 255u) / 256u * 256u;
    return fold + sae_candidate_bytes(T_max, d, m, k);
}

xmix_status xmix_sae_pack_encoder(const uint16_t* W_enc, int32_t m, int32_t d,
                                  uint16_t* W_packed, xmix_sae_dict* dict, void* stream) {
    if (!W_enc || !W_packed || !dict || W_enc == W_packed || m < 256 || m % 256 != 0 ||
        d < 256 || d % 256 != 0 || !aligned16(W_enc) || !aligned16(W_packed))
        return XMIX_E_INVAL;
    const int64_t bytes = static_cast<int64_t>(m) * d * 2;
    const char *a = reinterpret_cast<const char*>(W_enc), *b = reinterpret_cast<char*>(W_packed);
    if (a < b + bytes && b < a + bytes) return XMIX_E_INVAL;  // overlap
    const xmix_status st = launched(launch_sae_pack(W_enc, m, d, W_packed, as_stream(stream)));
    if (st != XMIX_OK) return st;
    dict->pieces = W_packed;
    dict->m = m;
    dict->d = d;
    dict->layout = XMIX_SAE_DICT_TILED;
    return XMIX_OK;
}

xmix_status xmix_sae_fold_bias(const xmix_sae_dict* dict, const uint16_t* b_enc,
                               const uint16_t* b_dec, float* c_fold, void* stream) {
    if (!dict_ok(dict, -1) || !b_enc || !b_dec || !c_fold || !aligned16(b_dec))
        return XMIX_E_INVAL;
    return launched(launch_sae_fold(dict->pieces, b_enc, b_dec, dict->m, dict->d, c_fold,
                                    as_stream(stream)));
}

}  // extern "C"

namespace {

// Checks shared by the encode entry points; returns the folded-bias area
// and the candidate area of the workspace.
xmix_status encode_args(const uint16_t* h, int32_t d, const xmix_route* rt, int32_t app_bit,
                        const xmix_sae_dict* dict, int32_t k, void* ws, size_t ws_bytes,
                        float** fold, void** cand) {
    if (!route_ok(rt) || app_bit < 0 || app_bit >= rt->n_apps) return XMIX_E_INVAL;
    if (!h || !aligned16(h) || d < 256 || d % 256 != 0) return XMIX_E_INVAL;
    if (!dict_ok(dict, d)) return XMIX_E_INVAL;
    const int32_t m = dict->m;
    if (k < 1 || k > XMIX_MAX_TOPK || k > m) return XMIX_E_INVAL;
    // the merge keeps (m / 256) * k candidates per token in registers
    if (static_cast<int64_t>(m / 256) * k > 64 * 256) return XMIX_E_UNSUPPORTED;
    const size_t need = xmix_sae_encode_workspace(rt->T_max, d, m, k);
    if (!ws || ws_bytes < need || !aligned16(ws)) return XMIX_E_WORKSPACE;
    const size_t fold_bytes = (static_cast<size_t>(m) * sizeof(float) + 255u) / 256u * 256u;
    *fold = static_cast<float*>(ws);
    *cand = static_cast<char*>(ws) + fold_bytes;
    return XMIX_OK;
}

}  // namespace

extern "C" {

xmix_status xmix_sae_encode_candidates(const uint16_t* h, int32_t d, const xmix_route* rt,
                                       int32_t app_bit, const xmix_sae_dict* dict,
                                       const uint16_t* b_enc, const uint16_t* b_dec,
                                       const float* c_fold, int32_t k, void* ws,
                                       size_t ws_bytes, void* stream) {
    if (!c_fold && (!b_enc || !b_dec || !aligned16(b_dec))) return XMIX_E_INVAL;
    float* fold;
    void* cand;
    const xmix_status st = encode_args(h, d, rt, app_bit, dict, k, ws, ws_bytes, &fold, &cand);
    if (st != XMIX_OK) return st;
    hipStream_t s = as_stream(stream);
    const int32_t m = dict->m;
    if (!c_fold) {
        if (launch_sae_fold(dict->pieces, b_enc, b_dec, m, d, fold, s) != hipSuccess)
            return XMIX_E_LAUNCH;
        c_fold = fold;
    }
    return launched(launch_sae_candidates(h, d, rt->T_max, rt->app_count + app_bit,
                                          app_list(rt, app_bit), dict->pieces, c_fold, m, k,
                                          cand, s));
}

xmix_status xmix_route_sae_encode_candidates(const int32_t* req_of_token, const int32_t* T_valid,
                                             const uint32_t* sub_mask, int32_t R_max,
                                             const xmix_route* rt, uint32_t* err_word,
                                             const uint16_t* h, int32_t d, int32_t app_bit,
                                             const xmix_sae_dict* dict, const uint16_t* b_enc,
                                             const uint16_t* b_dec, const float* c_fold,
                                             int32_t k, void* ws, size_t ws_bytes,
                                             void* stream) {
    if (!req_of_token || !T_valid || !sub_mask || !err_word || R_max < 1) return XMIX_E_INVAL;
    if (!c_fold && (!b_enc || !b_dec || !aligned16(b_dec))) return XMIX_E_INVAL;
    float* fold;
    void* cand;
    const xmix_status st = encode_args(h, d, rt, app_bit, dict, k, ws, ws_bytes, &fold, &cand);
    if (st != XMIX_OK) return st;
    hipStream_t s = as_stream(stream);
    const int32_t m = dict->m;
    if (!c_fold) {
        if (launch_sae_fold(dict->pieces, b_enc, b_dec, m, d, fold, s) != hipSuccess)
            return XMIX_E_LAUNCH;
        c_fold = fold;
    }
    RouteIn r;
    r.req = req_of_token;
    r.T_valid = T_valid;
    r.sub = sub_mask;
    r.R_max = R_max;
    r.n_apps = rt->n_apps;
    r.app_bit = app_bit;
    r.tok_mask = rt->tok_mask;
    r.app_count = rt->app_count;
    r.app_tokens = rt->app_tokens;
    r.err_word = err_word;
    return launched(launch_sae_candidates(h, d, rt->T_max, rt->app_count + app_bit,
                                          app_list(rt, app_bit), dict->pieces, c_fold, m, k,
                                          cand, s, &r));
}

xmix_status xmix_sae_merge_topk(const uint16_t* h, int32_t d, const xmix_route* rt,
                                int32_t app_bit, const xmix_sae_dict* dict, const float* c_fold,
                                int32_t k, int32_t* idx_out, uint16_t* val_out, void* ws,
                                size_t ws_bytes, void* stream) {
    if (!idx_out || !val_out) return XMIX_E_INVAL;
    float* fold;
    void* cand;
    const xmix_status st = encode_args(h, d, rt, app_bit, dict, k, ws, ws_bytes, &fold, &cand);
    if (st != XMIX_OK) return st;
    return launched(launch_sae_merge(h, d, rt->T_max, rt->app_count + app_bit,
                                     app_list(rt, app_bit), dict->pieces,
                                     c_fold ? c_fold : fold, dict->m, k, idx_out, val_out, cand,
                                     nullptr, as_stream(stream)));
}

xmix_status xmix_sae_merge_topk_ring(const uint16_t* h, int32_t d, const xmix_route* rt,
                                     int32_t app_bit, const xmix_sae_dict* dict,
                                     const float* c_fold, int32_t k, int32_t* idx_out,
                                     uint16_t* val_out, void* ws, size_t ws_bytes,
                                     const int32_t* req_of_token, int32_t layer_id,
                                     int32_t app_id, const xmix_ring* ring, void* stream) {
    if (!idx_out || !val_out || !req_of_token || !ring) return XMIX_E_INVAL;
    if (!ring->slots || !ring->head || ring->capacity < 1 ||
        ring->row_bytes != 16 + 6 * k || (reinterpret_cast<uintptr_t>(ring->slots) & 3u) != 0 ||
        (reinterpret_cast<uintptr_t>(ring->head) & 7u) != 0)
        return XMIX_E_INVAL;
    float* fold;
    void* cand;
    const xmix_status st = encode_args(h, d, rt, app_bit, dict, k, ws, ws_bytes, &fold, &cand);
    if (st != XMIX_OK) return st;
    MergeRing r;
    r.slots = ring->slots;
    r.head = ring->head;
    r.capacity = ring->capacity;
    r.row_bytes = ring->row_bytes;
    r.req = req_of_token;
    r.layer_id = layer_id;
    r.app_id = app_id;
    return launched(launch_sae_merge(h, d, rt->T_max, rt->app_count + app_bit,
                                     app_list(rt, app_bit), dict->pieces,
                                     c_fold ? c_fold : fold, dict->m, k, idx_out, val_out, cand,
                                     &r, as_stream(stream)));
}

xmix_status xmix_sae_encode_topk_ring(const uint16_t* h, int32_t d, const xmix_route* rt,
                                      int32_t app_bit, const xmix_sae_dict* dict,
                                      const uint16_t* b_enc, const uint16_t* b_dec,
                                      const float* c_fold, int32_t k, int32_t* idx_out,
                                      uint16_t* val_out, void* ws, size_t ws_bytes,
                                      const int32_t* req_of_token, int32_t layer_id,
                                      int32_t app_id, const xmix_ring* ring, void* stream) {
    if (!idx_out || !val_out || !req_of_token || !ring || ring->row_bytes != 16 + 6 * k)
        return XMIX_E_INVAL;
    const xmix_status st = xmix_sae_encode_candidates(h, d, rt, app_bit, dict, b_enc, b_dec,
                                                      c_fold, k, ws, ws_bytes, stream);
    if (st != XMIX_OK) return st;
    return xmix_sae_merge_topk_ring(h, d, rt, app_bit, dict, c_fold, k, idx_out, val_out, ws,
                                    ws_bytes, req_of_token, layer_id, app_id, ring, stream);
}

xmix_status xmix_sae_encode_topk(const uint16_t* h, int32_t d, const xmix_route* rt,
                                 int32_t app_bit, const xmix_sae_dict* dict,
                                 const uint16_t* b_enc, const uint16_t* b_dec,
                                 const float* c_fold, int32_t k, int32_t* idx_out,
                                 uint16_t* val_out, void* ws, size_t ws_bytes, void* stream) {
    if (!idx_out || !val_out) return XMIX_E_INVAL;
    const xmix_status st = xmix_sae_encode_candidates(h, d, rt, app_bit, dict, b_enc, b_dec,
                                                      c_fold, k, ws, ws_bytes, stream);
    if (st != XMIX_OK) return st;
    return xmix_sae_merge_topk(h, d, rt, app_bit, dict, c_fold, k, idx_out, val_out, ws,
                               ws_bytes, stream);
}

}  // extern "C"

namespace {

bool ring_ok(const xmix_ring* ring, int32_t k) {
    return ring->slots && ring->head && ring->capacity >= 1 && ring->row_bytes == 16 + 6 * k &&
           (reinterpret_cast<uintptr_t>(ring->slots) & 3u) == 0 &&
           (reinterpret_cast<uintptr_t>(ring->head) & 7u) == 0;
}

// The batched encode: every app is checked before anything is launched;
// apps without a folded bias get it folded into their workspace first.
xmix_status encode_multi(const uint16_t* h, int32_t d, const xmix_route* rt, int32_t n,
                         const xmix_sae_app* apps, const int32_t* req_of_token,
                         int32_t layer_id, hipStream_t s, const RouteIn* route) {
    if (!apps || n < 1 || n > XMIX_MAX_APPS || !route_ok(rt)) return XMIX_E_INVAL;
    SaeAppIn in[XMIX_MAX_APPS];
    MergeRing rings[XMIX_MAX_APPS];
    float* fold[XMIX_MAX_APPS] = {};
    for (int32_t i = 0; i < n; ++i) {
        const xmix_sae_app& a = apps[i];
        if (!a.idx_out || !a.val_out) return XMIX_E_INVAL;
        if (!a.c_fold && (!a.b_enc || !a.b_dec || !aligned16(a.b_dec))) return XMIX_E_INVAL;
        if (a.ring && (!req_of_token || !ring_ok(a.ring, a.k))) return XMIX_E_INVAL;
        void* cand;
        const xmix_status st =
            encode_args(h, d, rt, a.app_bit, a.dict, a.k, a.ws, a.ws_bytes, &fold[i], &cand);
        if (st != XMIX_OK) return st;
        if (a.ring) {
            rings[i] = MergeRing{a.ring->slots, a.ring->head, a.ring->capacity,
                                 a.ring->row_bytes, req_of_token, layer_id, a.app_id};
        }
        in[i] = SaeAppIn{rt->app_count + a.app_bit, app_list(rt, a.app_bit), a.dict->pieces,
                         a.c_fold ? a.c_fold : fold[i], a.dict->m, a.k, a.app_bit, cand,
                         a.idx_out, a.val_out, a.ring ? &rings[i] : nullptr};
    }
    for (int32_t i = 0; i < n; ++i) {
        const xmix_sae_app& a = apps[i];
        if (!a.c_fold && launch_sae_fold(a.dict->pieces, a.b_enc, a.b_dec, a.dict->m, d, fold[i],
                                         s) != hipSuccess)
            return XMIX_E_LAUNCH;
    }
    if (sae_multi_supported(rt->T_max))
        return launched(launch_sae_encode_multi(h, d, rt->T_max, n, in, s, route));
    for (int32_t i = 0; i < n; ++i) {  // many token slots: one app after the other
        const SaeAppIn& a = in[i];
        if (launch_sae_candidates(h, d, rt->T_max, a.app_count, a.tok_list, a.W, a.c_fold, a.m,
                                  a.k, a.cand, s, i == 0 ? route : nullptr) != hipSuccess ||
            launch_sae_merge(h, d, rt->T_max, a.app_count, a.tok_list, a.W, a.c_fold, a.m, a.k,
                             a.idx_out, a.val_out, a.cand, a.ring, s) != hipSuccess)
            return XMIX_E_LAUNCH;
    }
    return XMIX_OK;
}

}  // namespace

extern "C" {

xmix_status xmix_sae_encode_topk_multi(const uint16_t* h, int32_t d, const xmix_route* rt,
                                       int32_t n_sae, const xmix_sae_app* apps,
                                       const int32_t* req_of_token, int32_t layer_id,
                                       void* stream) {
    return encode_multi(h, d, rt, n_sae, apps, req_of_token, layer_id, as_stream(stream),
                        nullptr);
}

xmix_status xmix_route_sae_encode_topk_multi(const int32_t* req_of_token,
                                             const int32_t* T_valid, const uint32_t* sub_mask,
                                             int32_t R_max, const xmix_route* rt,
                                             uint32_t* err_word, const uint16_t* h, int32_t d,
                                             int32_t n_sae, const xmix_sae_app* apps,
                                             int32_t layer_id, void* stream) {
    if (!req_of_token || !T_valid || !sub_mask || !err_word || R_max < 1 || !route_ok(rt))
        return XMIX_E_INVAL;
    RouteIn r;
    r.req = req_of_token;
    r.T_valid = T_valid;
    r.sub = sub_mask;
    r.R_max = R_max;
    r.n_apps = rt->n_apps;
    r.tok_mask = rt->tok_mask;
    r.app_count = rt->app_count;
    r.app_tokens = rt->app_tokens;
    r.err_word = err_word;
    return encode_multi(h, d, rt, n_sae, apps, req_of_token, layer_id, as_stream(stream), &r);
}

xmix_status xmix_sae_clamp_decode(uint16_t* h, int32_t d, const xmix_route* rt,
                                  int32_t app_bit, const int32_t* idx, const uint16_t* val,
                                  int32_t k, const uint16_t* W_dec, int32_t m,
                                  const int32_t* clamp_ids, const float* clamp_vals,
                                  int32_t n_clamp, float* delta_out, void* stream) {
    if (!h || !idx || !val || !W_dec || !clamp_ids || !clamp_vals || !route_ok(rt))
        return XMIX_E_INVAL;
    if (app_bit < 0 || app_bit >= rt->n_apps) return XMIX_E_INVAL;
    if (d < 8 || d % 8 != 0 || m < 1 || k < 1 || k > XMIX_MAX_TOPK) return XMIX_E_INVAL;
    if (n_clamp < 1 || n_clamp > XMIX_MAX_CLAMP) return XMIX_E_INVAL;
    if (!aligned16(h) || !aligned16(W_dec) || (delta_out && !aligned16(delta_out)))
        return XMIX_E_INVAL;
    return launched(launch_clamp_decode(h, d, rt->app_count + app_bit, app_list(rt, app_bit),
                                        rt->T_max, idx, val, k, W_dec, m, clamp_ids, clamp_vals,
                                        n_clamp, delta_out, as_stream(stream)));
}

xmix_status xmix_sae_clamp_decode_multi(uint16_t* h, int32_t d, const xmix_route* rt, int32_t n,
                                        const xmix_sae_clamp_app* apps, void* stream) {
    if (!h || !apps || n < 1 || n > XMIX_MAX_APPS || !route_ok(rt)) return XMIX_E_INVAL;
    if (d < 8 || d % 8 != 0 || !aligned16(h)) return XMIX_E_INVAL;
    ClampAppIn in[XMIX_MAX_APPS];
    for (int32_t i = 0; i < n; ++i) {
        const xmix_sae_clamp_app& a = apps[i];
        if (!a.idx || !a.val || !a.W_dec || !a.clamp_ids || !a.clamp_vals) return XMIX_E_INVAL;
        if (a.app_bit < 0 || a.app_bit >= rt->n_apps) return XMIX_E_INVAL;
        if (a.m < 1 || a.k < 1 || a.k > XMIX_MAX_TOPK) return XMIX_E_INVAL;
        if (a.n_clamp < 1 || a.n_clamp > XMIX_MAX_CLAMP) return XMIX_E_INVAL;
        if (!aligned16(a.W_dec) || (a.delta_out && !aligned16(a.delta_out))) return XMIX_E_INVAL;
        in[i] = ClampAppIn{a.idx, a.val, a.W_dec, a.clamp_ids, a.clamp_vals, a.delta_out,
                           a.k, a.m, a.n_clamp, a.app_bit};
    }
    return launched(launch_clamp_multi(h, d, rt->T_max, rt->tok_mask, n, in,
                                       as_stream(stream)));
}

xmix_status xmix_readback_compact(const void* const* seg_rows, const int32_t* seg_bytes,
                                  int32_t n_seg, const xmix_route* rt, int32_t app_bit,
                                  const int32_t* req_of_token, int32_t layer_id, int32_t app_id,
                                  const xmix_ring* ring, void* stream) {
    if (!seg_rows || !seg_bytes || !req_of_token || !ring || !route_ok(rt)) return XMIX_E_INVAL;
    if (n_seg < 1 || n_seg > XMIX_MAX_SEGMENTS) return XMIX_E_INVAL;
    if (app_bit < 0 || app_bit >= rt->n_apps) return XMIX_E_INVAL;
    if (!ring->slots || !ring->head || ring->capacity < 1 || ring->row_bytes < 16 ||
        ring->row_bytes % 2 != 0 || (reinterpret_cast<uintptr_t>(ring->slots) & 3u) != 0 ||
        (reinterpret_cast<uintptr_t>(ring->head) & 7u) != 0)
        return XMIX_E_INVAL;
    Segments segs;
    memset(&segs, 0, sizeof(segs));
    int64_t total = 16;
    for (int s = 0; s < n_seg; ++s) {
        if (!seg_rows[s] || seg_bytes[s] < 2 || seg_bytes[s] % 2 != 0 ||
            (reinterpret_cast<uintptr_t>(seg_rows[s]) & 1u) != 0)
            return XMIX_E_INVAL;
        segs.ptr[s] = static_cast<const uint8_t*>(seg_rows[s]);
        segs.bytes[s] = seg_bytes[s];
        total += seg_bytes[s];
    }
    segs.n = n_seg;
    if (total != ring->row_bytes) return XMIX_E_INVAL;
    return launched(launch_compact(segs, rt->app_count + app_bit, app_list(rt, app_bit),
                                   rt->T_max, req_of_token, layer_id, app_id, ring->slots,
                                   ring->head, ring->capacity, ring->row_bytes,
                                   as_stream(stream)));
}

}  // extern "C"
