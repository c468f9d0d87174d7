// Internal launchers of librevisit. Each takes already-validated arguments
// (see capi.cpp) and queues its kernel on `stream`; the return value is the
// hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace revisit {

struct RetrieveArgs {
    const float* bank_c2w;
    int32_t n_bank;
    const float* query_c2w;
    const int32_t* query_chunk;
    int32_t n_query;
    double E, w_v, tau_c, cos_tau_v;
    int32_t delta, first_candidate, k;
    int32_t* out_idx;
    float* out_score;
    int32_t* out_count;
    int32_t frames_per_chunk;
    int32_t* out_frame_sel;
};
hipError_t launch_retrieve(const RetrieveArgs& a, hipStream_t stream);

struct ReprojectArgs {
    const float* tgt_depth;
    const float* tgt_c2w;
    const float* tgt_K;
    const float* src_depth;
    const float* src_c2w;
    const float* src_K;
    const int32_t* src_sel;  // nullable
    int32_t n_src;
    int32_t B, Tq, S, h, w, p;
    double eps;
    float* out_uv;
    int32_t* out_idx;
};
hipError_t launch_reproject(const ReprojectArgs& a, hipStream_t stream);

struct AttentionArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    float* lse;  // nullable
    int32_t Lq, Lk, H, D, h, w;
    const int32_t* slot;  // [Lk / (h w)]
    const float* corr_uv;  // [S][Lq][2]
    const int32_t* corr_idx;  // [S][Lq]
    int32_t S;  // 0 = bias off
    float softmax_scale, lambda, sigma;
};
hipError_t launch_attention_bf16(const AttentionArgs& a, hipStream_t stream);
hipError_t launch_attention_f32(const AttentionArgs& a, hipStream_t stream);

}  // namespace revisit
