// Streaming driver: the paper's cache layout run chunk by chunk (Sec. 4.2,
// cache layout, loop-closure retrieval and cache packing; Sec. 4.3).
//
// A stream object owns the device memory of one generated sequence: the pose
// bank, the history ring (pre-pooled token depth, frame poses, token-grid
// intrinsics and every layer's keys and values of the anchor and the
// capacity - 1 newest chunks), the packed attention cache and the per-chunk
// tables. rc_stream_step() enqueues one chunk on the caller's stream with no
// host synchronisation: the retrieval result stays on the device and the
// layout tables are built there from it. Only the shape of the layout (which
// parts exist) depends on the chunk index, which the host knows.
//
// Layout of chunk n's attention range, positions fixed per role so that the
// cache stays in a fixed position range: anchor (chunk 0, frames 0..F-1),
// retrieved (F..2F-1; when nothing is admissible, chunk n-3, the extension of
// the recent window, unbiased), recent n-2 (2F..3F-1) and n-1 (3F..4F-1), and
// the current chunk (4F..5F-1). Parts that do not exist yet are left out
// (chunk 0 attends to itself; the anchor is never also a recent chunk; the
// retrieved slot exists from n = 4 on). Keys enter the ring as the network
// produced them, at the current positions 4F + f, and are re-rotated by
// the packing kernel when they are placed in another role.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <new>

#include "../../include/revisit.h"
#include "internal.h"

struct rc_stream {
    rc_stream_config cfg;
    int32_t T;         // tokens per chunk
    int32_t max_rows;  // cache rows per layer: 5 parts
    size_t esize;
    int32_t n;  // next chunk id
    int device;
    // device memory
    float* bank;
    float* ring_depth;
    float* ring_c2w;
    float* ring_K;
    void* ring_k;
    void* ring_v;
    void* cache_k;
    void* cache_v;
    float* corr_uv;
    int32_t* corr_idx;
    int32_t* ret_idx;
    float* ret_score;
    int32_t* ret_count;
    int32_t* query_chunk;
    int32_t* part_slot;
    int32_t* kv_slot;
    int32_t* src_sel;
    int32_t* store_pos;
    int32_t* zero;
    void* workspace;  // attention key split and retrieval scratch of the largest step
    size_t workspace_bytes;
    // the last step's layout
    int32_t last_n, last_parts, last_ret_part;
};

namespace {

struct Part {
    int32_t chunk;  // -1: resolved on the device (retrieved or extension)
    int32_t pos;    // first frame position
    bool current;
};

int ring_slot(int32_t m, int32_t capacity) { return m == 0 ? 0 : 1 + (m - 1) % (capacity - 1); }

int layout(int32_t n, int32_t F, Part* parts, int32_t* ret_part) {
    int k = 0;
    *ret_part = -1;
    if (n >= 1) parts[k++] = Part{0, 0, false};
    if (n >= 4) {
        *ret_part = k;
        parts[k++] = Part{-1, F, false};
    }
    if (n - 2 >= 1) parts[k++] = Part{n - 2, 2 * F, false};
    if (n - 1 >= 1) parts[k++] = Part{n - 1, 3 * F, false};
    parts[k++] = Part{n, 4 * F, true};
    return k;
}

void release(rc_stream* s) {
    void* bufs[] = {s->bank,      s->ring_depth, s->ring_c2w,   s->ring_K,      s->ring_k,    s->ring_v,
                    s->cache_k,   s->cache_v,    s->corr_uv,    s->corr_idx,    s->ret_idx,   s->ret_score,
                    s->ret_count, s->query_chunk, s->part_slot, s->kv_slot,     s->src_sel,   s->store_pos,
                    s->zero,      s->workspace};
    for (void* b : bufs)
        if (b) (void)hipFree(b);
}

template <typename Ptr>
bool alloc(Ptr** p, size_t bytes) {
    void* v = nullptr;
    if (hipMalloc(&v, bytes > 0 ? bytes : 16) != hipSuccess) return false;
    *p = static_cast<Ptr*>(v);
    return true;
}

bool is_finite(float x) { return isfinite(x); }

bool aligned(const void* ptr, uintptr_t bytes) { return ((uintptr_t)ptr % bytes) == 0; }

}  // namespace

extern "C" {

int rc_stream_create(const rc_stream_config* cfg, rc_stream** out) {
    if (!cfg || !out) return revisit::fail_status(REVISIT_ERR_NULL, "rc_stream_create: cfg and out are required");
    *out = nullptr;
    const rc_stream_config& c = *cfg;
    if (c.dtype != REVISIT_BF16 && c.dtype != REVISIT_F32)
        return revisit::fail_status(REVISIT_ERR_UNSUPPORTED, "rc_stream_create: dtype %d not supported", c.dtype);
    if ((c.dtype == REVISIT_BF16 && c.D != 128) || (c.dtype == REVISIT_F32 && c.D != 64 && c.D != 128))
        return revisit::fail_status(REVISIT_ERR_UNSUPPORTED, "rc_stream_create: head dim %d not supported for this dtype", c.D);
    if (c.F < 1 || c.F > 64 || c.h < 1 || c.w < 1 || c.p < 1 || c.H < 1 || c.layers < 1 || c.max_chunks < 1)
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_create: need 1 <= F <= 64 and h, w, p, H, layers, max_chunks >= 1");
    if (c.dtype == REVISIT_BF16 && (c.h > 256 || c.w > 256))
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_create: bf16 attention with bias needs h, w <= 256");
    if (c.capacity < 5 || c.capacity > (1 << 20))
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_create: capacity %d outside [5, 2^20]", c.capacity);
    const int64_t T = (int64_t)c.F * c.h * c.w;
    if (T * 5 > (1 << 30) || (int64_t)c.h * c.p > (1 << 20) || (int64_t)c.w * c.p > (1 << 20) ||
        (int64_t)c.max_chunks > (1 << 30))
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_create: chunk too large");
    if (c.H > 65535 || c.layers > (1 << 16))
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_create: need H <= 65535 and layers <= 65536");
    // the ring's rows of one layer are addressed with 32-bit row indices
    if ((int64_t)c.capacity * T > INT32_MAX)
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_create: capacity x tokens per chunk above 2^31 - 1");
    // keys and values of the ring and the cache: at most 2^50 bytes each (no size_t overflow below)
    const double kv_ring_bytes = (double)c.layers * c.capacity * (double)T * c.H * c.D * 4.0;
    const double kv_cache_bytes = (double)c.layers * 5.0 * (double)T * c.H * c.D * 4.0;
    if (kv_ring_bytes > 1125899906842624.0 || kv_cache_bytes > 1125899906842624.0)
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_create: ring or cache above 2^50 bytes");
    if (!(is_finite(c.E) && c.E > 0.0f) || !is_finite(c.w_v) || !is_finite(c.tau_c) || !is_finite(c.tau_v) ||
        !(is_finite(c.eps) && c.eps >= 0.0f) || !is_finite(c.lambda) || !(is_finite(c.sigma) && c.sigma > 0.0f) ||
        !(is_finite(c.softmax_scale) && c.softmax_scale > 0.0f))
        return revisit::fail_status(REVISIT_ERR_PARAM, "rc_stream_create: a method parameter is out of its domain");
    if (c.rope_t_pairs < 0 || c.rope_t_pairs > c.D / 2 || (c.rope_t_pairs > 0 && !(is_finite(c.rope_theta) && c.rope_theta > 0.0f)))
        return revisit::fail_status(REVISIT_ERR_PARAM, "rc_stream_create: rope_t_pairs / rope_theta out of range");

    rc_stream* s = new (std::nothrow) rc_stream();
    if (!s) return revisit::fail_status(REVISIT_ERR_MEMORY, "rc_stream_create: out of host memory");
    s->cfg = c;
    s->T = (int32_t)T;
    s->max_rows = (int32_t)(5 * T);
    s->esize = c.dtype == REVISIT_BF16 ? 2 : 4;
    s->n = 0;
    s->last_n = -1;
    s->last_parts = 0;
    s->last_ret_part = -1;
    if (hipGetDevice(&s->device) != hipSuccess) {
        delete s;
        return revisit::fail_status(REVISIT_ERR_LAUNCH, "rc_stream_create: no current device");
    }
    // workspace of the largest step on this device: attention over 1..5 parts of
    // T keys (the automatic key split), retrieval over up to max_chunks entries
    size_t ws = 0;
    for (int32_t np = 1; np <= revisit::kStreamMaxParts; ++np) {
        size_t b = 0;
        const int st = rc_attention_workspace_size(c.dtype, (int32_t)T, np * (int32_t)T, c.H, c.D, 0, &b);
        if (st != REVISIT_OK) {
            delete s;
            return st;
        }
        ws = b > ws ? b : ws;
    }
    {
        size_t b = 0;
        const int st = rc_retrieve_workspace_size(c.max_chunks, 1, 1, &b);
        if (st != REVISIT_OK) {
            delete s;
            return st;
        }
        ws = b > ws ? b : ws;
    }
    s->workspace_bytes = ws;
    const size_t C = (size_t)c.capacity, F = (size_t)c.F, hw = (size_t)c.h * c.w;
    const size_t kv_ring = (size_t)c.layers * C * T * c.H * c.D * s->esize;
    const size_t kv_cache = (size_t)c.layers * s->max_rows * c.H * c.D * s->esize;
    const bool ok = alloc(&s->bank, (size_t)c.max_chunks * 16 * 4) && alloc(&s->ring_depth, C * F * hw * 4) &&
                    alloc(&s->ring_c2w, C * F * 16 * 4) && alloc(&s->ring_K, C * F * 4 * 4) &&
                    alloc(&s->ring_k, kv_ring) && alloc(&s->ring_v, kv_ring) && alloc(&s->cache_k, kv_cache) &&
                    alloc(&s->cache_v, kv_cache) && alloc(&s->corr_uv, F * T * 2 * 4) &&
                    alloc(&s->corr_idx, F * T * 4) && alloc(&s->ret_idx, 16) && alloc(&s->ret_score, 16) &&
                    alloc(&s->ret_count, 16) && alloc(&s->query_chunk, 16) &&
                    alloc(&s->part_slot, revisit::kStreamMaxParts * 4) &&
                    alloc(&s->kv_slot, revisit::kStreamMaxParts * F * 4) && alloc(&s->src_sel, F * 4) &&
                    alloc(&s->store_pos, C * 4) && alloc(&s->zero, 16) && alloc(&s->workspace, ws);
    if (!ok) {
        release(s);
        delete s;
        return revisit::fail_status(REVISIT_ERR_MEMORY, "rc_stream_create: device allocation failed");
    }
    // every chunk's keys carry the rotary embedding of the current role (frame 4F + f)
    int32_t* pos = static_cast<int32_t*>(malloc(C * 4));
    if (!pos) {
        release(s);
        delete s;
        return revisit::fail_status(REVISIT_ERR_MEMORY, "rc_stream_create: out of host memory");
    }
    for (size_t i = 0; i < C; ++i) pos[i] = 4 * c.F;
    const int32_t zero[4] = {0, 0, 0, 0};
    const bool copied = hipMemcpy(s->store_pos, pos, C * 4, hipMemcpyHostToDevice) == hipSuccess &&
                        hipMemcpy(s->zero, zero, 16, hipMemcpyHostToDevice) == hipSuccess;
    free(pos);
    if (!copied) {
        release(s);
        delete s;
        return revisit::fail_status(REVISIT_ERR_LAUNCH, "rc_stream_create: device copy failed");
    }
    *out = s;
    return REVISIT_OK;
}

int rc_stream_destroy(rc_stream* s) {
    if (!s) return REVISIT_OK;
    int cur = 0;
    const bool switch_dev = hipGetDevice(&cur) == hipSuccess && cur != s->device;
    if (switch_dev) (void)hipSetDevice(s->device);
    (void)hipDeviceSynchronize();
    release(s);
    if (switch_dev) (void)hipSetDevice(cur);
    delete s;
    return REVISIT_OK;
}

int rc_stream_step(rc_stream* s, const float* depth, const float* c2w, const float* K, const void* q, const void* k,
                   const void* v, void* o, float* lse, hipStream_t stream) {
    if (!s || !depth || !c2w || !K || !q || !k || !v || !o)
        return revisit::fail_status(REVISIT_ERR_NULL, "rc_stream_step: required pointer is NULL");
    const rc_stream_config& c = s->cfg;
    if (s->n >= c.max_chunks)
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_step: the pose bank holds %d chunks", c.max_chunks);
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess || cur != s->device)
        return revisit::fail_status(REVISIT_ERR_PARAM, "rc_stream_step: the stream's device is not current");
    // the configuration was validated at creation; with these alignments every
    // stage call below passes its own validation, so only a launch can fail
    if (!aligned(depth, 4) || !aligned(c2w, 4) || !aligned(K, 4) || !aligned(q, 16) || !aligned(k, 16) ||
        !aligned(v, 16) || !aligned(o, 16) || !aligned(lse, 4))
        return revisit::fail_status(REVISIT_ERR_SHAPE, "rc_stream_step: q, k, v, o must be 16-byte aligned, "
                                                       "depth, c2w, K and lse 4-byte");
    const int32_t n = s->n, F = c.F, T = s->T, C = c.capacity, hw = c.h * c.w;
    const size_t row = (size_t)c.H * c.D * s->esize;
    const int32_t slot_n = ring_slot(n, C);
    int st;

    // the chunk enters the history ring and the pose bank
    revisit::StreamCommitArgs ca{depth, c2w, K, F, c.h, c.w, c.p, n, slot_n, s->ring_depth, s->ring_c2w, s->ring_K,
                                 s->bank, s->query_chunk};
    hipError_t e = revisit::launch_stream_commit(ca, stream);
    if (e != hipSuccess) return revisit::fail_status(REVISIT_ERR_LAUNCH, "rc_stream_step: commit: %s", hipGetErrorString(e));
    st = pack_retrieved_kv(k, v, nullptr, 1, s->zero, 1, 0, s->ring_k, s->ring_v, slot_n * T, C * T, c.layers, c.dtype,
                           F, c.h, c.w, c.H, c.D, 0, 1.0f, stream);
    if (st != REVISIT_OK) return st;

    // retrieval (k = 1) over the resident history
    if (n >= 1) {
        const int32_t first = n - C + 2 > 1 ? n - C + 2 : 1;
        st = retrieve_chunks(s->bank, n, s->bank + (size_t)n * 16, s->query_chunk, 1, c.E, c.w_v, c.tau_c, c.tau_v,
                             c.delta, first, 1, s->ret_idx, s->ret_score, s->ret_count, 0, nullptr, s->workspace,
                             s->workspace_bytes, stream);
        if (st != REVISIT_OK) return st;
    }

    // the layout and its tables
    Part parts[revisit::kStreamMaxParts];
    int32_t ret_part = -1;
    const int n_parts = layout(n, F, parts, &ret_part);
    revisit::StreamSlotsArgs sa{};
    sa.n = n;
    sa.F = F;
    sa.capacity = C;
    sa.n_parts = n_parts;
    sa.ret_part = ret_part;
    sa.has_ret = ret_part >= 0;
    for (int i = 0; i < n_parts; ++i) sa.part_chunk[i] = parts[i].chunk;
    sa.ret_idx = s->ret_idx;
    sa.ret_count = s->ret_count;
    sa.part_slot = s->part_slot;
    sa.kv_slot = s->kv_slot;
    sa.src_sel = s->src_sel;
    e = revisit::launch_stream_slots(sa, stream);
    if (e != hipSuccess) return revisit::fail_status(REVISIT_ERR_LAUNCH, "rc_stream_step: slots: %s", hipGetErrorString(e));

    // correspondence of the current tokens into the retrieved chunk's frames, on the pooled maps
    const float* tgt_d = s->ring_depth + (size_t)slot_n * F * hw;
    if (ret_part >= 0) {
        st = reproject_correspondence(tgt_d, s->ring_c2w + (size_t)slot_n * F * 16, s->ring_K + (size_t)slot_n * F * 4,
                                      s->ring_depth, s->ring_c2w, s->ring_K, s->src_sel, C * F, 1, F, F, c.h, c.w, 1,
                                      c.eps, s->corr_uv, s->corr_idx, stream);
        if (st != REVISIT_OK) return st;
    }

    // the packed cache: runs of consecutive positions in one call each; the current chunk unrotated.
    // From chunk 2 on, part 0 is the anchor at rows 0..T-1 and positions 0..F-1, exactly as the
    // previous step packed it (chunk 0 never leaves ring slot 0 and nothing else writes those rows),
    // so it is not packed again.
    for (int i0 = n >= 2 ? 1 : 0; i0 < n_parts;) {
        int i1 = i0 + 1;
        while (i1 < n_parts && !parts[i1].current && !parts[i0].current && parts[i1].pos == parts[i1 - 1].pos + F) ++i1;
        st = pack_retrieved_kv(s->ring_k, s->ring_v, s->store_pos, C, s->part_slot + i0, i1 - i0, parts[i0].pos,
                               s->cache_k, s->cache_v, i0 * T, s->max_rows, c.layers, c.dtype, F, c.h, c.w, c.H, c.D,
                               parts[i0].current ? 0 : c.rope_t_pairs, c.rope_theta, stream);
        if (st != REVISIT_OK) return st;
        i0 = i1;
    }

    // biased attention of every layer over its packed cache
    const int32_t Lk = n_parts * T;
    for (int32_t l = 0; l < c.layers; ++l) {
        const size_t qo = (size_t)l * T * row, co = (size_t)l * s->max_rows * row;
        st = biased_chunk_attention(static_cast<const uint8_t*>(q) + qo, static_cast<const uint8_t*>(s->cache_k) + co,
                                    static_cast<const uint8_t*>(s->cache_v) + co, static_cast<uint8_t*>(o) + qo,
                                    lse ? lse + (size_t)l * c.H * T : nullptr, c.dtype, T, Lk, c.H, c.D, c.h, c.w,
                                    s->kv_slot, s->corr_uv, s->corr_idx, ret_part >= 0 ? F : 0, c.softmax_scale,
                                    c.lambda, c.sigma, 0, s->workspace, s->workspace_bytes, stream);
        if (st != REVISIT_OK) return st;
    }
    s->last_n = n;
    s->last_parts = n_parts;
    s->last_ret_part = ret_part;
    s->n = n + 1;
    return REVISIT_OK;
}

int rc_stream_view(const rc_stream* s, rc_stream_state* out) {
    if (!s || !out) return revisit::fail_status(REVISIT_ERR_NULL, "rc_stream_view: stream and out are required");
    out->n = s->last_n;
    out->n_parts = s->last_parts;
    out->ret_part = s->last_ret_part;
    out->Lk = s->last_parts * s->T;
    out->cache_rows = s->max_rows;
    out->ret_idx = s->ret_idx;
    out->ret_count = s->ret_count;
    out->part_slot = s->part_slot;
    out->kv_slot = s->kv_slot;
    out->src_sel = s->src_sel;
    out->corr_uv = s->corr_uv;
    out->corr_idx = s->corr_idx;
    out->cache_k = s->cache_k;
    out->cache_v = s->cache_v;
    return REVISIT_OK;
}

}  // extern "C"
