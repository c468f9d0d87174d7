// Pose retrieval over the history bank (Sec. 4.2, Eq. retrieval).
//
// One wave64 per query chunk. Each lane streams the bank entries
// j = lane, lane + 64, ... (one 64-byte pose row each, coalesced across the
// wave), evaluates the score and the three admissibility gates in double
// precision and keeps its own KMAX best (score, j) pairs sorted in registers.
// The wave then merges the 64 sorted lists with k rounds of a butterfly
// argmin over the lanes' heads; the winning lane pops its head. Scores are
// computed with exactly the IEEE double operations of the definition, in the
// order written, with contraction disabled, so that the choice of chunks is
// reproducible bit for bit on the host.
//
// Large banks (more than kDirectMax entries) are cut into segments of
// kSegEntries, one workgroup of kSegWaves waves per (query, segment), so that
// enough waves stream the bank to keep HBM busy; each workgroup merges its
// waves' lists in LDS and leaves the segment's k best (score, j) pairs in a
// workspace, and one workgroup per query merges those in the same order. The
// result is the same as the single-wave scan.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

#pragma clang fp contract(off)

namespace revisit {
namespace {

constexpr int kWave = 64;
constexpr int kWaveEntries = 16 * kWave;                // bank entries per scanning wave (64 KiB of poses)
constexpr int kSegWaves = 16;                           // scanning waves per segment workgroup
constexpr int kSegEntries = kSegWaves * kWaveEntries;   // bank entries per segment
constexpr int kDirectMax = 8192;                        // larger banks take the segmented path

// (s1, j1) strictly before (s2, j2): smaller score, then smaller index.
__device__ __forceinline__ bool before(double s1, int j1, double s2, int j2) {
    return s1 < s2 || (s1 == s2 && j1 < j2);
}

// A lane's KMAX best (score, j) pairs, sorted; (INFINITY, INT32_MAX) = empty.
template <int KMAX>
struct LaneTop {
    double s[KMAX];
    int j[KMAX];

    __device__ __forceinline__ void clear() {
#pragma unroll
        for (int i = 0; i < KMAX; ++i) {
            s[i] = INFINITY;
            j[i] = INT32_MAX;
        }
    }
    // sorted insertion, top down: slot i takes the new pair if it belongs
    // exactly there, or the pair above it if the new one goes higher up
    __device__ __forceinline__ void offer(double ns, int nj) {
        if (!before(ns, nj, s[KMAX - 1], j[KMAX - 1])) return;
#pragma unroll
        for (int i = KMAX - 1; i >= 0; --i) {
            if (before(ns, nj, s[i], j[i])) {
                const bool here = (i == 0) || before(s[i > 0 ? i - 1 : 0], j[i > 0 ? i - 1 : 0], ns, nj);
                if (here) {
                    s[i] = ns;
                    j[i] = nj;
                } else {
                    s[i] = s[i - 1];
                    j[i] = j[i - 1];
                }
            }
        }
    }
    // round r of the wave merge: the wave's best remaining pair (all lanes
    // agree); the lane that holds it pops it
    __device__ __forceinline__ void wave_best(double& bs, int& bj) {
        bs = s[0];
        bj = j[0];
#pragma unroll
        for (int off = kWave / 2; off >= 1; off >>= 1) {
            const double os = __shfl_xor(bs, off);
            const int oj = __shfl_xor(bj, off);
            if (before(os, oj, bs, bj)) {
                bs = os;
                bj = oj;
            }
        }
        if (bj != INT32_MAX && j[0] == bj) {
#pragma unroll
            for (int i = 0; i < KMAX - 1; ++i) {
                s[i] = s[i + 1];
                j[i] = j[i + 1];
            }
            s[KMAX - 1] = INFINITY;
            j[KMAX - 1] = INT32_MAX;
        }
    }
};

// A query chunk: its centre (last column of c2w), viewing direction R e_z
// (third column) and chunk index.
struct QueryPose {
    double cx, cy, cz, vx, vy, vz;
    int64_t n;
};

__device__ __forceinline__ QueryPose query_pose(const RetrieveArgs& a, int qi) {
    const float* qm = a.query_c2w + (size_t)qi * 16;
    return QueryPose{qm[3], qm[7], qm[11], qm[2], qm[6], qm[10], a.query_chunk[qi]};
}

// The part of bank entry j that retrieval reads: columns 2 (viewing
// direction) and 3 (centre) of the first three rows.
struct PoseCols {
    float2 r0, r1, r2;  // (R_i2, c_i) for i = 0, 1, 2
};

__device__ __forceinline__ PoseCols load_cols(const RetrieveArgs& a, int j) {
    const float* m = a.bank_c2w + (size_t)j * 16;
    return PoseCols{*reinterpret_cast<const float2*>(m + 2), *reinterpret_cast<const float2*>(m + 6),
                    *reinterpret_cast<const float2*>(m + 10)};
}

// Score and gates of bank entry j for query qp (Eq. retrieval); offers the
// pair to `top` when admissible.
template <int KMAX>
__device__ __forceinline__ void score_entry(const RetrieveArgs& a, int j, const PoseCols& m, const QueryPose& qp,
                                            LaneTop<KMAX>& top) {
    const double dx = (double)m.r0.y - qp.cx;
    const double dy = (double)m.r1.y - qp.cy;
    const double dz = (double)m.r2.y - qp.cz;
    const double d = sqrt(dx * dx + dy * dy + dz * dz) / a.E;
    const double al = (double)m.r0.x * qp.vx + (double)m.r1.x * qp.vy + (double)m.r2.x * qp.vz;
    const double s = d + a.w_v * (1.0 - al);
    const bool ok = j >= a.first_candidate && qp.n - j >= a.delta && d <= a.tau_c && al >= a.cos_tau_v;
    if (ok) top.offer(s, j);
}

// Entries j = first + lane, + 64, ... below end, kUnroll per lane at a time:
// all their loads are issued before any is scored (an index past `end` is
// clamped to end - 1 for the load and not scored).
constexpr int kUnroll = 4;

template <int KMAX>
__device__ __forceinline__ void scan_range(const RetrieveArgs& a, int first, int end, int lane, const QueryPose& qp,
                                           LaneTop<KMAX>& top) {
    for (int j0 = first + lane; j0 < end; j0 += kUnroll * kWave) {
        PoseCols m[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) m[u] = load_cols(a, min(j0 + u * kWave, end - 1));
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if (j0 + u * kWave < end) score_entry(a, j0 + u * kWave, m[u], qp, top);
        }
    }
}

// The k results of query qi from the lanes' sorted lists: out_idx,
// out_score, out_count and the frame selection.
template <int KMAX>
__device__ __forceinline__ void emit(const RetrieveArgs& a, int qi, int lane, LaneTop<KMAX>& top) {
    int mine = -1;  // lane r keeps the r-th result
    int count = 0;
    for (int r = 0; r < a.k; ++r) {
        double bs;
        int bj;
        top.wave_best(bs, bj);
        const bool found = bj != INT32_MAX;
        if (lane == 0) {
            a.out_idx[(size_t)qi * a.k + r] = found ? bj : -1;
            if (a.out_score) a.out_score[(size_t)qi * a.k + r] = found ? (float)bs : INFINITY;
        }
        if (lane == r) mine = found ? bj : -1;
        count += found ? 1 : 0;
    }
    if (lane == 0) a.out_count[qi] = count;

    if (a.out_frame_sel) {
        const int F = a.frames_per_chunk;
        const int total = a.k * F;
        for (int t0 = 0; t0 < total; t0 += kWave) {
            const int t = t0 + lane;
            const int src_lane = (t < total ? t : 0) / F;
            const int c = __shfl(mine, src_lane);
            if (t < total) {
                a.out_frame_sel[(size_t)qi * total + t] = (t / F < count) ? c * F + (t % F) : -1;
            }
        }
    }
}

template <int KMAX>
__global__ __launch_bounds__(kWave) void retrieve_kernel(RetrieveArgs a) {
    const int qi = blockIdx.x;
    const int lane = threadIdx.x;
    const QueryPose qp = query_pose(a, qi);
    LaneTop<KMAX> top;
    top.clear();
    scan_range(a, 0, a.n_bank, lane, qp, top);
    emit(a, qi, lane, top);
}

// Segment `seg` of the bank for query qi, one workgroup of kSegWaves waves:
// each wave scans kWaveEntries entries and reduces its lanes' lists to its k
// best pairs in LDS; the first wave merges those and writes the segment's k
// best to seg_s / seg_j [qi][seg][0 .. k), (INFINITY, INT32_MAX) past the
// admissible ones.
template <int KMAX>
__global__ __launch_bounds__(kSegWaves * kWave) void retrieve_segment_kernel(RetrieveArgs a) {
    __shared__ double lds_s[kSegWaves][KMAX];
    __shared__ int lds_j[kSegWaves][KMAX];
    const int qi = blockIdx.x / a.n_seg;
    const int seg = blockIdx.x - qi * a.n_seg;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const QueryPose qp = query_pose(a, qi);
    LaneTop<KMAX> top;
    top.clear();
    const int64_t j0 = (int64_t)seg * kSegEntries + (int64_t)wave * kWaveEntries;
    const int j_begin = (int)min((int64_t)a.n_bank, j0);
    const int j_end = (int)min((int64_t)a.n_bank, j0 + kWaveEntries);
    scan_range(a, j_begin, j_end, lane, qp, top);
    for (int r = 0; r < a.k; ++r) {
        double bs;
        int bj;
        top.wave_best(bs, bj);
        if (lane == 0) {
            lds_s[wave][r] = bs;
            lds_j[wave][r] = bj;
        }
    }
    __syncthreads();
    if (wave == 0) {
        LaneTop<KMAX> top2;
        top2.clear();
        for (int c = lane; c < kSegWaves * a.k; c += kWave) {
            const int w = c / a.k, r = c - w * a.k;
            if (lds_j[w][r] != INT32_MAX) top2.offer(lds_s[w][r], lds_j[w][r]);
        }
        const size_t base = ((size_t)qi * a.n_seg + seg) * a.k;
        for (int r = 0; r < a.k; ++r) {
            double bs;
            int bj;
            top2.wave_best(bs, bj);
            if (lane == 0) {
                a.seg_s[base + r] = bs;
                a.seg_j[base + r] = bj;
            }
        }
    }
}

// One workgroup of kMergeThreads per query over its n_seg * k segment
// results: every lane keeps its KMAX best, each wave reduces its lanes' lists
// to its k best in LDS, and the first wave merges those and emits.
constexpr int kMergeThreads = 1024;
constexpr int kMergeWaves = kMergeThreads / kWave;

template <int KMAX>
__global__ __launch_bounds__(kMergeThreads) void retrieve_merge_kernel(RetrieveArgs a) {
    __shared__ double lds_s[kMergeWaves][KMAX];
    __shared__ int lds_j[kMergeWaves][KMAX];
    const int qi = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    LaneTop<KMAX> top;
    top.clear();
    const size_t base = (size_t)qi * a.n_seg * a.k;
    const int n_cand = a.n_seg * a.k;
    for (int c = tid; c < n_cand; c += kMergeThreads) {
        const int j = a.seg_j[base + c];
        if (j != INT32_MAX) top.offer(a.seg_s[base + c], j);
    }
    for (int r = 0; r < a.k; ++r) {
        double bs;
        int bj;
        top.wave_best(bs, bj);
        if (lane == 0) {
            lds_s[wave][r] = bs;
            lds_j[wave][r] = bj;
        }
    }
    __syncthreads();
    if (wave == 0) {
        LaneTop<KMAX> top2;
        top2.clear();
        for (int c = lane; c < kMergeWaves * a.k; c += kWave) {
            const int w = c / a.k, r = c - (c / a.k) * a.k;
            if (lds_j[w][r] != INT32_MAX) top2.offer(lds_s[w][r], lds_j[w][r]);
        }
        emit(a, qi, lane, top2);
    }
}

}  // namespace

int32_t retrieve_segments(int32_t n_bank) {
    return n_bank > kDirectMax ? (n_bank + kSegEntries - 1) / kSegEntries : 0;
}

size_t retrieve_workspace_bytes(int32_t n_bank, int32_t n_query, int32_t k) {
    const int32_t n_seg = retrieve_segments(n_bank);
    return (size_t)n_seg * n_query * k * (sizeof(double) + sizeof(int32_t));
}

template <int KMAX>
static hipError_t launch_k(const RetrieveArgs& a, hipStream_t stream) {
    const dim3 block(kWave);
    if (a.n_seg == 0) {
        hipLaunchKernelGGL(retrieve_kernel<KMAX>, dim3(a.n_query), block, 0, stream, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(retrieve_segment_kernel<KMAX>, dim3((unsigned)a.n_query * a.n_seg), dim3(kSegWaves * kWave), 0,
                       stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(retrieve_merge_kernel<KMAX>, dim3(a.n_query), dim3(kMergeThreads), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_retrieve(const RetrieveArgs& a, hipStream_t stream) {
    if (a.n_query == 0) return hipSuccess;
    if (a.k <= 4) return launch_k<4>(a, stream);
    if (a.k <= 8) return launch_k<8>(a, stream);
    if (a.k <= 16) return launch_k<16>(a, stream);
    return launch_k<32>(a, stream);
}

}  // namespace revisit
