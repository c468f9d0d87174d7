// Internal launchers of librevisit. Each takes already-validated arguments
// (see capi.cpp) and queues its kernel on `stream`; the return value is the
// hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace revisit {

// Workgroups of a 1-D grid are dealt to the 8 XCDs round-robin (workgroup L
// runs on XCD L % 8). xcd_item() turns that into "each XCD takes one
// contiguous range of work items", so the work items that share data (one
// head's K/V, one problem's source depth) meet in the same L2. The grid is
// padded to a multiple of 8; the returned item may be >= n_items (nothing to do).
constexpr int kXcds = 8;
__host__ __device__ inline unsigned xcd_grid(unsigned n_items) { return (n_items + kXcds - 1) / kXcds * kXcds; }
__device__ inline unsigned xcd_item(unsigned block, unsigned n_items) {
    const unsigned per_xcd = (n_items + kXcds - 1) / kXcds;
    return (block % kXcds) * per_xcd + block / kXcds;
}

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
    // segmented path for large banks (retrieve_segments(n_bank) > 0): per
    // (query, segment) the k best (score, j), from a workspace of
    // retrieve_workspace_bytes
    int32_t n_seg;
    double* seg_s;
    int32_t* seg_j;
};
int32_t retrieve_segments(int32_t n_bank);
size_t retrieve_workspace_bytes(int32_t n_bank, int32_t n_query, int32_t k);
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
    // rotation path: out_uv is 16-byte and out_idx 8-byte aligned, so an
    // even token index starts an aligned pair of both
    int32_t paired;
};
hipError_t launch_reproject(const ReprojectArgs& a, hipStream_t stream);
// rotation-only correspondence: ReprojectArgs with the depth maps and eps unused
hipError_t launch_rotation(const ReprojectArgs& a, hipStream_t stream);

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
    int32_t fp8_qk;  // bf16 kernel: q and k are fp8 e4m3 (v, o bf16)
};
hipError_t launch_attention_f32(const AttentionArgs& a, hipStream_t stream);

// bf16 attention: the key tiles of each (head, 128-query tile) item are cut
// into `parts` equal ranges, one workgroup each; with parts > 1 a second
// kernel merges the partial results kept in `workspace`
// (attention_bf16_workspace_bytes). attention_bf16_key_parts picks the
// number of parts that fills `slots` resident workgroups best.
int32_t attention_bf16_key_parts(const AttentionArgs& a, int32_t slots);
size_t attention_bf16_workspace_bytes(const AttentionArgs& a, int32_t parts);
hipError_t launch_attention_bf16(const AttentionArgs& a, int32_t parts, float* workspace, hipStream_t stream);

// Scratch of biased_chunk_attention_noalloc: a file-scope device array in
// attention.hip of kAttentionScratchBytes, one per device for the life of the
// process. attention_scratch() returns its device address on the current
// device (looked up once per device).
constexpr size_t kAttentionScratchBytes = (size_t)128 << 20;
hipError_t attention_scratch(float** ptr);

// Cache packing of retrieved chunks (kvpack.hip). Element size 2 (bf16) or
// 4 (fp32); T = tokens per chunk; store [L][n_store][T][H][D], cache
// [L][cache_rows][H][D].
struct KvPackArgs {
    const void* store_k;
    const void* store_v;
    const int32_t* store_pos;  // nullable: chunk j at frame position F j
    int32_t n_store;
    const int32_t* sel;
    int32_t n_sel;
    int32_t dst_pos;
    void* cache_k;
    void* cache_v;
    int32_t dst_row0;
    int32_t cache_rows;
    int32_t n_layers;
    int32_t esize;
    int32_t F;
    int32_t T;
    int32_t H;
    int32_t D;
    int32_t n_t;
    double theta;
};
int64_t kvpack_blocks(const KvPackArgs& a);
hipError_t launch_kvpack(const KvPackArgs& a, hipStream_t stream);

// Streaming driver device steps (stream_kernels.hip).
struct StreamCommitArgs {
    const float* depth;  // [F][h p][w p]
    const float* c2w;    // [F][4][4]
    const float* K;      // [F][4] depth-pixel intrinsics
    int32_t F, h, w, p;
    int32_t n;     // chunk id
    int32_t slot;  // its ring slot
    float* ring_depth;  // [C][F][h][w]
    float* ring_c2w;    // [C][F][4][4]
    float* ring_K;      // [C][F][4] token-grid intrinsics
    float* bank;        // [max_chunks][4][4] representative poses
    int32_t* query_chunk;
};
hipError_t launch_stream_commit(const StreamCommitArgs& a, hipStream_t stream);

constexpr int kStreamMaxParts = 5;
struct StreamSlotsArgs {
    int32_t n, F, capacity;
    int32_t n_parts;
    int32_t ret_part;  // index of the retrieved / extension part, -1 if absent
    int32_t has_ret;
    int32_t part_chunk[kStreamMaxParts];  // chunk of every other part
    const int32_t* ret_idx;
    const int32_t* ret_count;
    int32_t* part_slot;  // [n_parts] ring slots in layout order
    int32_t* kv_slot;    // [n_parts * F]
    int32_t* src_sel;    // [F]
};
hipError_t launch_stream_slots(const StreamSlotsArgs& a, hipStream_t stream);
hipError_t launch_pool_depth(const float* depth, int64_t n_tokens, int32_t h, int32_t w, int32_t p, float* out,
                             hipStream_t stream);

// Sets the calling thread's last-error string and returns status (capi.cpp).
int fail_status(int status, const char* fmt, ...);

}  // namespace revisit
