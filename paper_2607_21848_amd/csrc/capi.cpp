// C entry points of librevisit: argument validation on the host, then the
// kernel launches on the caller's stream. The only state is a per-thread
// last-error string; scratch memory comes from the caller (workspace
// arguments sized by the rc_*_workspace_size queries). The streaming driver's
// entry points are in stream.cpp.

#include <math.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <hip/hip_runtime.h>

#include "../../include/revisit.h"
#include "internal.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}

int launched(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(REVISIT_ERR_LAUNCH, "%s: launch failed: %s", what, hipGetErrorString(e));
    return REVISIT_OK;
}

bool finite(float x) { return isfinite(x); }

bool aligned(const void* ptr, uintptr_t bytes) { return ((uintptr_t)ptr % bytes) == 0; }

constexpr int64_t kMaxElems = (int64_t)1 << 40;
constexpr int kMaxFrames = 1024;
constexpr int kMaxGridSide = 256;  // token-grid rows / columns of the bf16 kernel's bias tables
constexpr int kMaxKeyParts = 64;
constexpr uintptr_t kWorkspaceAlign = 16;

// Checks a caller's workspace against the bytes a call needs.
int check_workspace(const char* fn, size_t need, const void* ws, size_t ws_bytes) {
    if (need == 0) return REVISIT_OK;
    if (ws_bytes < need)
        return fail(REVISIT_ERR_SHAPE, "%s: workspace of %zu bytes given, %zu needed", fn, ws_bytes, need);
    if (!ws) return fail(REVISIT_ERR_NULL, "%s: workspace is NULL (%zu bytes needed)", fn, need);
    if (!aligned(ws, kWorkspaceAlign)) return fail(REVISIT_ERR_SHAPE, "%s: workspace must be 16-byte aligned", fn);
    return REVISIT_OK;
}

// Compute units of the current device.
hipError_t device_compute_units(int* cus) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    return hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
}

// Shape, dtype and key-part checks shared by biased_chunk_attention and
// rc_attention_workspace_size.
int check_attention_shape(const char* fn, int32_t dtype, int32_t Lq, int32_t Lk, int32_t H, int32_t D,
                          int32_t key_parts) {
    if (dtype != REVISIT_BF16 && dtype != REVISIT_F32 && dtype != REVISIT_FP8_QK)
        return fail(REVISIT_ERR_UNSUPPORTED, "%s: dtype %d not supported", fn, dtype);
    if ((dtype == REVISIT_BF16 || dtype == REVISIT_FP8_QK) && D != 128)
        return fail(REVISIT_ERR_UNSUPPORTED, "%s: bf16 / fp8 needs D = 128 (got %d)", fn, D);
    if (dtype == REVISIT_F32 && D != 64 && D != 128)
        return fail(REVISIT_ERR_UNSUPPORTED, "%s: fp32 needs D = 64 or 128 (got %d)", fn, D);
    if (Lq < 0 || Lk < 1 || H < 1) return fail(REVISIT_ERR_SHAPE, "%s: need Lq >= 0, Lk >= 1, H >= 1", fn);
    if (H > 65535) return fail(REVISIT_ERR_SHAPE, "%s: H > 65535", fn);
    if ((int64_t)Lk * H * D > kMaxElems || (int64_t)Lq * H * D > kMaxElems)
        return fail(REVISIT_ERR_SHAPE, "%s: problem too large", fn);
    // (head, key part, 128-query tile) workgroups of the bf16 kernel: a 32-bit count
    if (((int64_t)Lq + 127) / 128 * H * kMaxKeyParts > ((int64_t)1 << 31))
        return fail(REVISIT_ERR_SHAPE, "%s: problem too large", fn);
    if (key_parts < 0 || key_parts > kMaxKeyParts)
        return fail(REVISIT_ERR_PARAM, "%s: key_parts=%d outside [0, %d]", fn, key_parts, kMaxKeyParts);
    return REVISIT_OK;
}

// Key parts of the bf16 / fp8 kernel for this call (0 = automatic), and the
// workspace bytes they need. AttentionArgs needs only Lq, Lk and H here.
int attention_parts(const char* fn, const revisit::AttentionArgs& a, int32_t key_parts, int32_t* parts,
                    size_t* bytes) {
    int32_t P = key_parts;
    if (P == 0) {
        int cus = 0;
        const hipError_t e = device_compute_units(&cus);
        if (e != hipSuccess) return fail(REVISIT_ERR_LAUNCH, "%s: device query failed: %s", fn, hipGetErrorString(e));
        P = revisit::attention_bf16_key_parts(a, 2 * cus);  // two resident workgroups per compute unit
    }
    const int32_t tiles = (a.Lk + 31) / 32;
    P = P < tiles ? P : tiles;  // at least one key tile per part
    *parts = P;
    *bytes = revisit::attention_bf16_workspace_bytes(a, P);
    return REVISIT_OK;
}

}  // namespace

namespace revisit {
int fail_status(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}
}  // namespace revisit

extern "C" {

const char* rc_status_string(int status) {
    switch (status) {
        case REVISIT_OK: return "ok";
        case REVISIT_ERR_NULL: return "null pointer";
        case REVISIT_ERR_SHAPE: return "bad shape";
        case REVISIT_ERR_UNSUPPORTED: return "unsupported";
        case REVISIT_ERR_PARAM: return "bad parameter";
        case REVISIT_ERR_LAUNCH: return "launch error";
        case REVISIT_ERR_MEMORY: return "out of memory";
        default: return "unknown status";
    }
}

const char* rc_last_error(void) { return g_last_error; }

int retrieve_chunks(const float* bank_c2w, int32_t n_bank, const float* query_c2w, const int32_t* query_chunk,
                    int32_t n_query, float E, float w_v, float tau_c, float tau_v, int32_t delta,
                    int32_t first_candidate, int32_t k, int32_t* out_idx, float* out_score, int32_t* out_count,
                    int32_t frames_per_chunk, int32_t* out_frame_sel, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
    size_t need = 0;
    int st = rc_retrieve_workspace_size(n_bank, n_query, k, &need);
    if (st != REVISIT_OK) return st;
    if (!(finite(E) && E > 0.0f)) return fail(REVISIT_ERR_PARAM, "retrieve_chunks: E must be finite and > 0");
    if (!finite(w_v) || !finite(tau_c) || !finite(tau_v))
        return fail(REVISIT_ERR_PARAM, "retrieve_chunks: w_v, tau_c and tau_v must be finite");
    if (out_frame_sel && (frames_per_chunk < 1 || (int64_t)k * frames_per_chunk > (1 << 20)))
        return fail(REVISIT_ERR_PARAM, "retrieve_chunks: frames_per_chunk=%d invalid", frames_per_chunk);
    if (n_query == 0) return REVISIT_OK;
    if (!query_c2w || !query_chunk || !out_idx || !out_count || (n_bank > 0 && !bank_c2w))
        return fail(REVISIT_ERR_NULL, "retrieve_chunks: required pointer is NULL");
    // the scan reads the pose columns it needs as 8-byte pairs
    if (!aligned(bank_c2w, 8)) return fail(REVISIT_ERR_SHAPE, "retrieve_chunks: bank_c2w must be 8-byte aligned");
    revisit::RetrieveArgs a;
    a.bank_c2w = bank_c2w;
    a.n_bank = n_bank;
    a.query_c2w = query_c2w;
    a.query_chunk = query_chunk;
    a.n_query = n_query;
    a.E = (double)E;
    a.w_v = (double)w_v;
    a.tau_c = (double)tau_c;
    a.cos_tau_v = cos((double)tau_v);
    a.delta = delta;
    a.first_candidate = first_candidate;
    a.k = k;
    a.out_idx = out_idx;
    a.out_score = out_score;
    a.out_count = out_count;
    a.frames_per_chunk = frames_per_chunk;
    a.out_frame_sel = out_frame_sel;
    a.n_seg = revisit::retrieve_segments(n_bank);
    a.seg_s = nullptr;
    a.seg_j = nullptr;
    st = check_workspace("retrieve_chunks", need, workspace, workspace_bytes);
    if (st != REVISIT_OK) return st;
    if (a.n_seg > 0) {
        a.seg_s = static_cast<double*>(workspace);
        a.seg_j = reinterpret_cast<int32_t*>(a.seg_s + (size_t)a.n_seg * n_query * k);
    }
    return launched(revisit::launch_retrieve(a, stream), "retrieve_chunks");
}

int rc_retrieve_workspace_size(int32_t n_bank, int32_t n_query, int32_t k, size_t* bytes) {
    if (!bytes) return fail(REVISIT_ERR_NULL, "rc_retrieve_workspace_size: bytes is NULL");
    *bytes = 0;
    if (n_bank < 0 || n_query < 0) return fail(REVISIT_ERR_SHAPE, "retrieve_chunks: negative n_bank or n_query");
    if (n_bank > (1 << 30)) return fail(REVISIT_ERR_SHAPE, "retrieve_chunks: n_bank=%d above 2^30", n_bank);
    if (k < 1 || k > REVISIT_MAX_K) return fail(REVISIT_ERR_PARAM, "retrieve_chunks: k=%d outside [1, %d]", k, REVISIT_MAX_K);
    const int32_t n_seg = revisit::retrieve_segments(n_bank);
    if (n_seg > 0 && (int64_t)n_seg * n_query * k > ((int64_t)1 << 31))
        return fail(REVISIT_ERR_SHAPE, "retrieve_chunks: n_bank * n_query too large");
    *bytes = n_seg > 0 ? revisit::retrieve_workspace_bytes(n_bank, n_query, k) : 0;
    return REVISIT_OK;
}

int reproject_correspondence(const float* tgt_depth, const float* tgt_c2w, const float* tgt_K,
                             const float* src_depth, const float* src_c2w, const float* src_K,
                             const int32_t* src_sel, int32_t n_src, int32_t B, int32_t Tq, int32_t S, int32_t h,
                             int32_t w, int32_t p, float eps, float* out_uv, int32_t* out_idx, hipStream_t stream) {
    if (B < 0 || Tq < 0 || S < 0 || h < 1 || w < 1 || p < 1)
        return fail(REVISIT_ERR_SHAPE, "reproject_correspondence: need B, Tq, S >= 0 and h, w, p >= 1");
    if ((int64_t)h * w * p * p > ((int64_t)1 << 28) || (int64_t)h * p > (1 << 20) || (int64_t)w * p > (1 << 20))
        return fail(REVISIT_ERR_SHAPE, "reproject_correspondence: frame too large");
    if ((int64_t)B * Tq * h * w > ((int64_t)1 << 31) - 1 || (int64_t)B * S * Tq * h * w > kMaxElems)
        return fail(REVISIT_ERR_SHAPE, "reproject_correspondence: problem too large");
    if (src_sel && n_src < 0) return fail(REVISIT_ERR_SHAPE, "reproject_correspondence: n_src < 0");
    if (S > 64) return fail(REVISIT_ERR_SHAPE, "reproject_correspondence: more than 64 source frames per problem");
    if (!(finite(eps) && eps >= 0.0f)) return fail(REVISIT_ERR_PARAM, "reproject_correspondence: eps must be finite and >= 0");
    if (B == 0 || Tq == 0 || S == 0) return REVISIT_OK;
    if (!tgt_depth || !tgt_c2w || !tgt_K || !out_uv || !out_idx)
        return fail(REVISIT_ERR_NULL, "reproject_correspondence: required pointer is NULL");
    if ((!src_sel || n_src > 0) && (!src_depth || !src_c2w || !src_K))
        return fail(REVISIT_ERR_NULL, "reproject_correspondence: source pointer is NULL");
    if (!aligned(out_uv, 8) || !aligned(out_idx, 4) || !aligned(tgt_depth, 4) || !aligned(src_depth, 4) ||
        !aligned(src_sel, 4))
        return fail(REVISIT_ERR_SHAPE, "reproject_correspondence: out_uv must be 8-byte aligned, arrays 4-byte");
    revisit::ReprojectArgs a;
    a.tgt_depth = tgt_depth;
    a.tgt_c2w = tgt_c2w;
    a.tgt_K = tgt_K;
    a.src_depth = src_depth;
    a.src_c2w = src_c2w;
    a.src_K = src_K;
    a.src_sel = src_sel;
    a.n_src = src_sel ? n_src : 0;
    a.B = B;
    a.Tq = Tq;
    a.S = S;
    a.h = h;
    a.w = w;
    a.p = p;
    a.eps = (double)eps;
    a.out_uv = out_uv;
    a.out_idx = out_idx;
    a.paired = 0;
    return launched(revisit::launch_reproject(a, stream), "reproject_correspondence");
}

int reproject_rotation(const float* tgt_c2w, const float* tgt_K, const float* src_c2w, const float* src_K,
                       const int32_t* src_sel, int32_t n_src, int32_t B, int32_t Tq, int32_t S, int32_t h, int32_t w,
                       int32_t p, float* out_uv, int32_t* out_idx, hipStream_t stream) {
    if (B < 0 || Tq < 0 || S < 0 || h < 1 || w < 1 || p < 1)
        return fail(REVISIT_ERR_SHAPE, "reproject_rotation: need B, Tq, S >= 0 and h, w, p >= 1");
    if ((int64_t)h * w > ((int64_t)1 << 28))
        return fail(REVISIT_ERR_SHAPE, "reproject_rotation: frame too large");
    if ((int64_t)B * Tq * h * w > ((int64_t)1 << 31) - 1 || (int64_t)B * S * Tq * h * w > kMaxElems)
        return fail(REVISIT_ERR_SHAPE, "reproject_rotation: problem too large");
    if (src_sel && n_src < 0) return fail(REVISIT_ERR_SHAPE, "reproject_rotation: n_src < 0");
    if (S > 64) return fail(REVISIT_ERR_SHAPE, "reproject_rotation: more than 64 source frames per problem");
    if (B == 0 || Tq == 0 || S == 0) return REVISIT_OK;
    if (!tgt_c2w || !tgt_K || !out_uv || !out_idx)
        return fail(REVISIT_ERR_NULL, "reproject_rotation: required pointer is NULL");
    if ((!src_sel || n_src > 0) && (!src_c2w || !src_K))
        return fail(REVISIT_ERR_NULL, "reproject_rotation: source pointer is NULL");
    if (!aligned(out_uv, 8) || !aligned(out_idx, 4) || !aligned(src_sel, 4))
        return fail(REVISIT_ERR_SHAPE, "reproject_rotation: out_uv must be 8-byte aligned, arrays 4-byte");
    revisit::ReprojectArgs a;
    a.tgt_depth = nullptr;
    a.tgt_c2w = tgt_c2w;
    a.tgt_K = tgt_K;
    a.src_depth = nullptr;
    a.src_c2w = src_c2w;
    a.src_K = src_K;
    a.src_sel = src_sel;
    a.n_src = src_sel ? n_src : 0;
    a.B = B;
    a.Tq = Tq;
    a.S = S;
    a.h = h;
    a.w = w;
    a.p = p;
    a.eps = 0.0;
    a.out_uv = out_uv;
    a.out_idx = out_idx;
    a.paired = aligned(out_uv, 16) && aligned(out_idx, 8);
    return launched(revisit::launch_rotation(a, stream), "reproject_rotation");
}

}  // extern "C"

namespace {

// Validation shared by both attention entry points: fills `a` for a launch,
// or returns a non-zero status. *nothing = true when there is nothing to do.
int prepare_attention(const char* fn, const void* q, const void* k, const void* v, void* o, float* lse, int32_t dtype,
                      int32_t Lq, int32_t Lk, int32_t H, int32_t D, int32_t h, int32_t w,
                      const int32_t* kv_frame_slot, const float* corr_uv, const int32_t* corr_idx, int32_t S,
                      float softmax_scale, float lambda, float sigma, int32_t key_parts, revisit::AttentionArgs& a,
                      bool* nothing) {
    *nothing = false;
    int st = check_attention_shape(fn, dtype, Lq, Lk, H, D, key_parts);
    if (st != REVISIT_OK) return st;
    if (h < 1 || w < 1 || S < 0) return fail(REVISIT_ERR_SHAPE, "%s: need h, w >= 1, S >= 0", fn);
    const int64_t hw = (int64_t)h * w;
    if (Lk % hw != 0) return fail(REVISIT_ERR_SHAPE, "%s: Lk=%d not a multiple of h*w=%lld", fn, Lk, (long long)hw);
    if (Lk / hw > kMaxFrames) return fail(REVISIT_ERR_SHAPE, "%s: more than %d KV frames", fn, kMaxFrames);
    if ((int64_t)S * Lq > kMaxElems) return fail(REVISIT_ERR_SHAPE, "%s: problem too large", fn);
    if (!(finite(softmax_scale) && softmax_scale > 0.0f))
        return fail(REVISIT_ERR_PARAM, "%s: softmax_scale must be finite and > 0", fn);
    if (!(finite(sigma) && sigma > 0.0f)) return fail(REVISIT_ERR_PARAM, "%s: sigma must be finite and > 0", fn);
    if (!finite(lambda)) return fail(REVISIT_ERR_PARAM, "%s: lambda must be finite", fn);
    const float gamma = lambda / (2.0f * sigma * sigma * softmax_scale);
    if (!finite(gamma)) return fail(REVISIT_ERR_PARAM, "%s: lambda / (2 sigma^2 scale) overflows", fn);
    if (Lq == 0) {
        *nothing = true;
        return REVISIT_OK;
    }
    const bool bias = S > 0 && lambda != 0.0f;
    // the bf16 / fp8 kernel keeps per-column and per-row bias operands of the token grid in LDS
    if (bias && dtype != REVISIT_F32 && (h > kMaxGridSide || w > kMaxGridSide))
        return fail(REVISIT_ERR_SHAPE, "%s: bf16 / fp8 with bias needs h, w <= %d (got %d x %d)", fn, kMaxGridSide, h, w);
    if (!q || !k || !v || !o) return fail(REVISIT_ERR_NULL, "%s: q, k, v and o are required", fn);
    if (bias && (!kv_frame_slot || !corr_uv || !corr_idx))
        return fail(REVISIT_ERR_NULL, "%s: slot table and correspondence map are required when S > 0", fn);
    // the kernels move q/k/v/o rows in 16-byte vectors and u^ pairs in 8-byte ones
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) || !aligned(lse, 4) ||
        (bias && (!aligned(corr_uv, 8) || !aligned(corr_idx, 4) || !aligned(kv_frame_slot, 4))))
        return fail(REVISIT_ERR_SHAPE, "%s: q, k, v, o must be 16-byte aligned, corr_uv 8-byte", fn);
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.lse = lse;
    a.Lq = Lq;
    a.Lk = Lk;
    a.H = H;
    a.D = D;
    a.h = h;
    a.w = w;
    a.slot = kv_frame_slot;
    a.corr_uv = corr_uv;
    a.corr_idx = corr_idx;
    a.S = bias ? S : 0;
    a.softmax_scale = softmax_scale;
    a.lambda = lambda;
    a.sigma = sigma;
    a.fp8_qk = dtype == REVISIT_FP8_QK;
    return REVISIT_OK;
}

}  // namespace

extern "C" {

int biased_chunk_attention(const void* q, const void* k, const void* v, void* o, float* lse, int32_t dtype,
                           int32_t Lq, int32_t Lk, int32_t H, int32_t D, int32_t h, int32_t w,
                           const int32_t* kv_frame_slot, const float* corr_uv, const int32_t* corr_idx, int32_t S,
                           float softmax_scale, float lambda, float sigma, int32_t key_parts, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
    revisit::AttentionArgs a{};
    bool nothing = false;
    int st = prepare_attention("biased_chunk_attention", q, k, v, o, lse, dtype, Lq, Lk, H, D, h, w, kv_frame_slot,
                               corr_uv, corr_idx, S, softmax_scale, lambda, sigma, key_parts, a, &nothing);
    if (st != REVISIT_OK || nothing) return st;
    if (dtype == REVISIT_F32) return launched(revisit::launch_attention_f32(a, stream), "biased_chunk_attention");
    int32_t parts = 1;
    size_t need = 0;
    st = attention_parts("biased_chunk_attention", a, key_parts, &parts, &need);
    if (st != REVISIT_OK) return st;
    st = check_workspace("biased_chunk_attention", need, workspace, workspace_bytes);
    if (st != REVISIT_OK) return st;
    return launched(revisit::launch_attention_bf16(a, parts, static_cast<float*>(workspace), stream),
                    "biased_chunk_attention");
}

int biased_chunk_attention_noalloc(const void* q, const void* k, const void* v, void* o, float* lse, int32_t dtype,
                                   int32_t Lq, int32_t Lk, int32_t H, int32_t D, int32_t h, int32_t w,
                                   const int32_t* kv_frame_slot, const float* corr_uv, const int32_t* corr_idx,
                                   int32_t S, float softmax_scale, float lambda, float sigma, int32_t key_parts,
                                   hipStream_t stream) {
    const char* fn = "biased_chunk_attention_noalloc";
    revisit::AttentionArgs a{};
    bool nothing = false;
    int st = prepare_attention(fn, q, k, v, o, lse, dtype, Lq, Lk, H, D, h, w, kv_frame_slot, corr_uv, corr_idx, S,
                               softmax_scale, lambda, sigma, key_parts, a, &nothing);
    if (st != REVISIT_OK || nothing) return st;
    if (dtype == REVISIT_F32) return launched(revisit::launch_attention_f32(a, stream), fn);
    int32_t parts = 1;
    size_t need = 0;
    st = attention_parts(fn, a, key_parts, &parts, &need);
    if (st != REVISIT_OK) return st;
    if (need > revisit::kAttentionScratchBytes) {
        if (key_parts != 0)
            return fail(REVISIT_ERR_SHAPE, "%s: %d key parts need %zu bytes of scratch, more than the %zu bytes it holds "
                                           "(use fewer parts, or biased_chunk_attention with a workspace)",
                        fn, parts, need, revisit::kAttentionScratchBytes);
        // the automatic split, cut to the most parts whose partial results fit
        while (parts > 1 && revisit::attention_bf16_workspace_bytes(a, parts) > revisit::kAttentionScratchBytes)
            --parts;
        need = revisit::attention_bf16_workspace_bytes(a, parts);
    }
    float* scratch = nullptr;
    if (need > 0) {
        const hipError_t e = revisit::attention_scratch(&scratch);
        if (e != hipSuccess)
            return fail(REVISIT_ERR_LAUNCH, "%s: device address of the scratch array: %s", fn, hipGetErrorString(e));
    }
    return launched(revisit::launch_attention_bf16(a, parts, scratch, stream), fn);
}

int rc_attention_workspace_size(int32_t dtype, int32_t Lq, int32_t Lk, int32_t H, int32_t D, int32_t key_parts,
                                size_t* bytes) {
    if (!bytes) return fail(REVISIT_ERR_NULL, "rc_attention_workspace_size: bytes is NULL");
    *bytes = 0;
    const int st = check_attention_shape("rc_attention_workspace_size", dtype, Lq, Lk, H, D, key_parts);
    if (st != REVISIT_OK || dtype == REVISIT_F32 || Lq == 0) return st;
    revisit::AttentionArgs a{};
    a.Lq = Lq;
    a.Lk = Lk;
    a.H = H;
    int32_t parts = 1;
    return attention_parts("rc_attention_workspace_size", a, key_parts, &parts, bytes);
}

int pack_retrieved_kv(const void* store_k, const void* store_v, const int32_t* store_pos, int32_t n_store,
                      const int32_t* sel, int32_t n_sel, int32_t dst_pos, void* cache_k, void* cache_v,
                      int32_t dst_row0, int32_t cache_rows, int32_t n_layers, int32_t dtype, int32_t F, int32_t h,
                      int32_t w, int32_t H, int32_t D, int32_t rope_t_pairs, float rope_theta, hipStream_t stream) {
    if (dtype != REVISIT_BF16 && dtype != REVISIT_F32)
        return fail(REVISIT_ERR_UNSUPPORTED, "pack_retrieved_kv: dtype %d not supported", dtype);
    if (D < 8 || D > 512 || D % 8 != 0)
        return fail(REVISIT_ERR_UNSUPPORTED, "pack_retrieved_kv: D=%d (need a multiple of 8 in [8, 512])", D);
    if (n_store < 0 || n_sel < 0 || n_layers < 0 || F < 1 || h < 1 || w < 1 || H < 1 || dst_row0 < 0 || cache_rows < 0)
        return fail(REVISIT_ERR_SHAPE, "pack_retrieved_kv: need n_store, n_sel, n_layers, dst_row0, cache_rows >= 0 "
                                       "and F, h, w, H >= 1");
    const int64_t T = (int64_t)F * h * w;
    if (T > INT32_MAX) return fail(REVISIT_ERR_SHAPE, "pack_retrieved_kv: F*h*w too large");
    if ((int64_t)dst_row0 + (int64_t)n_sel * T > cache_rows)
        return fail(REVISIT_ERR_SHAPE, "pack_retrieved_kv: %d slots of %lld rows from row %d exceed cache_rows=%d", n_sel,
                    (long long)T, dst_row0, cache_rows);
    const int64_t row = (int64_t)H * D;
    if ((double)n_layers * n_store * T * row > (double)kMaxElems || (double)n_layers * cache_rows * row > (double)kMaxElems)
        return fail(REVISIT_ERR_SHAPE, "pack_retrieved_kv: store or cache too large");
    if (rope_t_pairs < 0 || rope_t_pairs > D / 2)
        return fail(REVISIT_ERR_PARAM, "pack_retrieved_kv: rope_t_pairs=%d outside [0, D/2]", rope_t_pairs);
    if (rope_t_pairs > 0 && !(finite(rope_theta) && rope_theta > 0.0f))
        return fail(REVISIT_ERR_PARAM, "pack_retrieved_kv: rope_theta must be finite and > 0");
    if (n_layers == 0 || n_sel == 0) return REVISIT_OK;
    if (!sel || !cache_k || !cache_v || (n_store > 0 && (!store_k || !store_v)))
        return fail(REVISIT_ERR_NULL, "pack_retrieved_kv: required pointer is NULL");
    // the kernel moves 16-byte vectors
    if (!aligned(store_k, 16) || !aligned(store_v, 16) || !aligned(cache_k, 16) || !aligned(cache_v, 16) ||
        !aligned(sel, 4) || !aligned(store_pos, 4))
        return fail(REVISIT_ERR_SHAPE, "pack_retrieved_kv: store and cache must be 16-byte aligned, sel and store_pos 4-byte");
    revisit::KvPackArgs a;
    a.store_k = store_k;
    a.store_v = store_v;
    a.store_pos = store_pos;
    a.n_store = n_store;
    a.sel = sel;
    a.n_sel = n_sel;
    a.dst_pos = dst_pos;
    a.cache_k = cache_k;
    a.cache_v = cache_v;
    a.dst_row0 = dst_row0;
    a.cache_rows = cache_rows;
    a.n_layers = n_layers;
    a.esize = dtype == REVISIT_BF16 ? 2 : 4;
    a.F = F;
    a.T = (int32_t)T;
    a.H = H;
    a.D = D;
    a.n_t = rope_t_pairs;
    a.theta = (double)rope_theta;
    if (revisit::kvpack_blocks(a) > INT32_MAX) return fail(REVISIT_ERR_SHAPE, "pack_retrieved_kv: problem too large");
    return launched(revisit::launch_kvpack(a, stream), "pack_retrieved_kv");
}

int pool_token_depth(const float* depth, int32_t n_frames, int32_t h, int32_t w, int32_t p, float* out,
                     hipStream_t stream) {
    if (n_frames < 0 || h < 1 || w < 1 || p < 1)
        return fail(REVISIT_ERR_SHAPE, "pool_token_depth: need n_frames >= 0 and h, w, p >= 1");
    if ((int64_t)h * p > (1 << 20) || (int64_t)w * p > (1 << 20) ||
        (double)n_frames * h * w * p * p > (double)kMaxElems)
        return fail(REVISIT_ERR_SHAPE, "pool_token_depth: depth maps too large");
    if (n_frames == 0) return REVISIT_OK;
    if (!depth || !out) return fail(REVISIT_ERR_NULL, "pool_token_depth: depth and out are required");
    if (!aligned(depth, 4) || !aligned(out, 4)) return fail(REVISIT_ERR_SHAPE, "pool_token_depth: arrays must be 4-byte aligned");
    return launched(revisit::launch_pool_depth(depth, (int64_t)n_frames * h * w, h, w, p, out, stream), "pool_token_depth");
}

}  // extern "C"
