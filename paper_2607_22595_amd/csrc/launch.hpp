// Kernel launchers behind the C ABI (internal; one definition per .hip file).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace xmix {

struct BitList {  // static app bits, passed by value into a launch
    int32_t bit[32];
};

hipError_t launch_route_build(const int32_t* req, const int32_t* T_valid, const uint32_t* sub,
                              int32_t R_max, int32_t T_max, int32_t n_apps, uint32_t* tok_mask,
                              int32_t* app_count, int32_t* app_tokens, uint32_t* err_word,
                              hipStream_t stream);

hipError_t launch_route_gate(int32_t T_max, int32_t app_bit, uint32_t* tok_mask,
                             int32_t* app_count, int32_t* app_tokens, const float* signal,
                             const int32_t* req, int32_t n_signal, int32_t signal_bit,
                             const float* threshold, hipStream_t stream);
hipError_t launch_route_trigger(int32_t T_max, int32_t app_bit, uint32_t* tok_mask,
                                int32_t* app_count, int32_t* app_tokens,
                                const int32_t* token_ids, const uint32_t* vocab_bits,
                                int32_t vocab_size, hipStream_t stream);

hipError_t launch_steer(void* h, bool bf16, int32_t d, int32_t T_max, const uint32_t* tok_mask,
                        const int32_t* req, const void* vecs, const BitList& bits,
                        const float* alpha, int32_t n_steer, hipStream_t stream);


hipError_t launch_router_write(void* logits, bool bf16, int32_t n_experts, int32_t T_max,
                               const uint32_t* tok_mask, const BitList& bits,
                               const float* offsets, int32_t n_router, hipStream_t stream);

hipError_t launch_probe(const void* h, bool bf16, int32_t d, int32_t T_max,
                        const uint32_t* tok_mask, const void* w, const float* b,
                        const BitList& bits, int32_t n_probe, int32_t mode,
                        const int32_t* cu_seqlens, int32_t R_max, float* logit, float* score,
                        float* ws, hipStream_t stream);

size_t sae_candidate_bytes(int32_t T_max, int32_t d, int32_t m, int32_t k);
hipError_t launch_sae_pack(const uint16_t* W_enc, int32_t m, int32_t d, uint16_t* W_packed,
                           hipStream_t stream);
hipError_t launch_sae_fold(const uint16_t* W_enc, const uint16_t* b_enc, const uint16_t* b_dec,
                           int32_t m, int32_t d, float* c_fold, hipStream_t stream);
constexpr int kMultiMax = 8;  // SAE apps per batched launch

// Routing inputs and outputs for an encode launch that also builds the
// step's routing (see xmix_route_sae_encode_candidates).
struct RouteIn {
    const int32_t* req = nullptr;
    const int32_t* T_valid = nullptr;
    const uint32_t* sub = nullptr;
    int32_t R_max = 0, n_apps = 0, app_bit = 0;
    uint32_t* tok_mask = nullptr;
    int32_t* app_count = nullptr;
    int32_t* app_tokens = nullptr;
    uint32_t* err_word = nullptr;
};

hipError_t launch_steer_probe(void* h, bool bf16, int32_t d, int32_t T_max,
                              const uint32_t* tok_mask, const int32_t* req, const void* vecs,
                              const BitList& sbits, const float* alpha, int32_t n_steer,
                              const void* w, const float* b, const BitList& pbits,
                              int32_t n_probe, float* logit, float* score, hipStream_t stream,
                              const RouteIn* route = nullptr);

hipError_t launch_sae_candidates(const uint16_t* h, int32_t d, int32_t T_max,
                                 const int32_t* app_count, const int32_t* tok_list,
                                 const uint16_t* W_enc, const float* c_fold, int32_t m,
                                 int32_t k, void* cand, hipStream_t stream,
                                 const RouteIn* route = nullptr);
struct MergeRing {  // readback of the merged rows into a ring
    uint8_t* slots;
    uint64_t* head;
    int32_t capacity, row_bytes;
    const int32_t* req;
    int32_t layer_id, app_id;
};
hipError_t launch_sae_merge(const uint16_t* h, int32_t d, int32_t T_max,
                            const int32_t* app_count, const int32_t* tok_list,
                            const uint16_t* W_enc, const float* c_fold, int32_t m, int32_t k,
                            int32_t* idx_out, uint16_t* val_out, void* cand,
                            const MergeRing* ring, hipStream_t stream);
// One SAE app of a batched encode: its list, dictionary, folded bias,
// candidate area, outputs and optional ring.
struct SaeAppIn {
    const int32_t* app_count;
    const int32_t* tok_list;
    const uint16_t* W;
    const float* c_fold;
    int32_t m, k, bit;
    void* cand;
    int32_t* idx_out;
    uint16_t* val_out;
    const MergeRing* ring;
};
// The candidates of up to kMultiMax apps in one launch, then their merges in
// one launch (decode shapes: T_max < the prefill threshold).
hipError_t launch_sae_encode_multi(const uint16_t* h, int32_t d, int32_t T_max, int32_t n,
                                   const SaeAppIn* apps, hipStream_t stream,
                                   const RouteIn* route = nullptr);
bool sae_multi_supported(int32_t T_max);

hipError_t launch_clamp_decode(uint16_t* h, int32_t d, const int32_t* app_count,
                               const int32_t* tok_list, int32_t T_max, const int32_t* idx,
                               const uint16_t* val, int32_t k, const uint16_t* W_dec, int32_t m,
                               const int32_t* clamp_ids, const float* clamp_vals,
                               int32_t n_clamp, float* delta_out, hipStream_t stream);
// One clamp app of a batched clamp-decode.
struct ClampAppIn {
    const int32_t* idx;
    const uint16_t* val;
    const uint16_t* W_dec;
    const int32_t* clamp_ids;
    const float* clamp_vals;
    float* delta_out;
    int32_t k, m, n_clamp, bit;
};
// Up to kMultiMax clamp apps in one launch, one workgroup per token slot,
// the apps applied to each row in the given order.
hipError_t launch_clamp_multi(uint16_t* h, int32_t d, int32_t T_max, const uint32_t* tok_mask,
                              int32_t n, const ClampAppIn* apps, hipStream_t stream);

struct Segments {
    const uint8_t* ptr[4];
    int32_t bytes[4];  // bytes per row of each segment (even)
    int32_t n;
};
hipError_t launch_compact(const Segments& segs, const int32_t* app_count,
                          const int32_t* tok_list, int32_t T_max, const int32_t* req,
                          int32_t layer_id, int32_t app_id, uint8_t* slots, uint64_t* head,
                          int32_t capacity, int32_t row_bytes, hipStream_t stream);

}  // namespace xmix
