// Token-depth pooling (pool_token_depth: the depth of Sec. 4.3 at token
// resolution, kept per stored frame), and the device steps of the streaming
// driver (stream.cpp) that are not one of the method's stages: putting a new
// chunk into the history ring, and turning the retrieval result into the
// cache layout's tables (Sec. 4.2, cache layout and loop-closure retrieval).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

#pragma clang fp contract(off)

namespace revisit {
namespace {

constexpr int kBlock = 256;

// Token depth: mean of the p x p block of depth pixels of token (r, c),
// summed row-major in double and rounded to fp32 once.
__device__ __forceinline__ float pooled_token(const float* __restrict__ frame, int Wd, int r, int c, int p) {
    const float* d = frame + (size_t)(r * p) * Wd + (size_t)c * p;
    double acc = 0.0;
    bool first = true;
    for (int y = 0; y < p; ++y) {
        for (int x = 0; x < p; ++x) {
            const double v = d[(size_t)y * Wd + x];
            acc = first ? v : acc + v;
            first = false;
        }
    }
    return (float)(acc / (double)(p * p));
}

__global__ __launch_bounds__(kBlock) void pool_depth_kernel(const float* __restrict__ depth, int64_t n_tokens, int h,
                                                            int w, int p, float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n_tokens) return;
    const int64_t hw = (int64_t)h * w;
    const int64_t f = i / hw;
    const int t = (int)(i - f * hw);
    const int r = t / w;
    out[i] = pooled_token(depth + f * hw * p * p, w * p, r, t - r * w, p);
}

// Chunk n enters the ring at slot `slot`: every frame's depth pooled to the
// token grid, frame poses copied, intrinsics divided by p (double, rounded to
// fp32); the middle frame's pose becomes bank entry n, and n is written for
// the retrieval's query index.
__global__ __launch_bounds__(kBlock) void stream_commit_kernel(StreamCommitArgs a) {
    const int hw = a.h * a.w;
    const int total = a.F * hw;
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i < total) {
        const int f = i / hw;
        const int t = i - f * hw;
        const int r = t / a.w;
        a.ring_depth[((size_t)a.slot * a.F + f) * hw + t] =
            pooled_token(a.depth + (size_t)f * hw * a.p * a.p, a.w * a.p, r, t - r * a.w, a.p);
    }
    if (blockIdx.x == 0) {
        const int tid = threadIdx.x;
        for (int e = tid; e < a.F * 16; e += kBlock) a.ring_c2w[(size_t)a.slot * a.F * 16 + e] = a.c2w[e];
        for (int e = tid; e < a.F * 4; e += kBlock)
            a.ring_K[(size_t)a.slot * a.F * 4 + e] = (float)((double)a.K[e] / (double)a.p);
        if (tid < 16) a.bank[(size_t)a.n * 16 + tid] = a.c2w[(a.F / 2) * 16 + tid];
        if (tid == 0) *a.query_chunk = a.n;
    }
}

__device__ __forceinline__ int ring_slot_of(int m, int capacity) { return m == 0 ? 0 : 1 + (m - 1) % (capacity - 1); }

// The layout's tables from the retrieval result, one thread: the ring slot of
// every part (in layout order), the KV frame slot table (retrieved frames
// 0..F-1 when a chunk was retrieved, -1 elsewhere) and the reprojection's
// source frames (the retrieved chunk's frames in the ring, or -1).
__global__ void stream_slots_kernel(StreamSlotsArgs a) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const bool retrieved = a.has_ret && *a.ret_count > 0;
    const int j = retrieved ? a.ret_idx[0] : a.n - 3;
    for (int i = 0; i < a.n_parts; ++i) {
        int m = a.part_chunk[i];
        if (i == a.ret_part) m = j;
        a.part_slot[i] = ring_slot_of(m, a.capacity);
        for (int f = 0; f < a.F; ++f) a.kv_slot[i * a.F + f] = (retrieved && i == a.ret_part) ? f : -1;
    }
    for (int f = 0; f < a.F; ++f) a.src_sel[f] = retrieved ? ring_slot_of(j, a.capacity) * a.F + f : -1;
}

}  // namespace

hipError_t launch_stream_commit(const StreamCommitArgs& a, hipStream_t stream) {
    const int total = a.F * a.h * a.w;
    const unsigned blocks = (unsigned)((total + kBlock - 1) / kBlock);
    hipLaunchKernelGGL(stream_commit_kernel, dim3(blocks > 0 ? blocks : 1), dim3(kBlock), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_pool_depth(const float* depth, int64_t n_tokens, int32_t h, int32_t w, int32_t p, float* out,
                             hipStream_t stream) {
    if (n_tokens == 0) return hipSuccess;
    hipLaunchKernelGGL(pool_depth_kernel, dim3((unsigned)((n_tokens + kBlock - 1) / kBlock)), dim3(kBlock), 0, stream,
                       depth, n_tokens, h, w, p, out);
    return hipGetLastError();
}

hipError_t launch_stream_slots(const StreamSlotsArgs& a, hipStream_t stream) {
    hipLaunchKernelGGL(stream_slots_kernel, dim3(1), dim3(64), 0, stream, a);
    return hipGetLastError();
}

}  // namespace revisit
