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

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

#pragma clang fp contract(off)

namespace revisit {
namespace {

constexpr int kWave = 64;

// (s1, j1) strictly before (s2, j2): smaller score, then smaller index.
__device__ __forceinline__ bool before(double s1, int j1, double s2, int j2) {
    return s1 < s2 || (s1 == s2 && j1 < j2);
}

template <int KMAX>
__global__ __launch_bounds__(kWave) void retrieve_kernel(RetrieveArgs a) {
    const int qi = blockIdx.x;
    const int lane = threadIdx.x;
    const float* qm = a.query_c2w + (size_t)qi * 16;
    // query centre (last column) and viewing direction R e_z (third column)
    const double cnx = qm[3], cny = qm[7], cnz = qm[11];
    const double vnx = qm[2], vny = qm[6], vnz = qm[10];
    const int64_t n = a.query_chunk[qi];

    double ls[KMAX];
    int lj[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
        ls[i] = INFINITY;
        lj[i] = INT32_MAX;
    }

    for (int j = lane; j < a.n_bank; j += kWave) {
        const float* m = a.bank_c2w + (size_t)j * 16;
        const double dx = (double)m[3] - cnx;
        const double dy = (double)m[7] - cny;
        const double dz = (double)m[11] - cnz;
        const double d = sqrt(dx * dx + dy * dy + dz * dz) / a.E;
        const double al = (double)m[2] * vnx + (double)m[6] * vny + (double)m[10] * vnz;
        const double s = d + a.w_v * (1.0 - al);
        const bool ok = j >= a.first_candidate && n - j >= a.delta && d <= a.tau_c && al >= a.cos_tau_v;
        if (ok && before(s, j, ls[KMAX - 1], lj[KMAX - 1])) {
            // sorted insertion, top down: slot i takes the new pair if it
            // belongs exactly there, or the pair above it if the new one
            // goes higher up
#pragma unroll
            for (int i = KMAX - 1; i >= 0; --i) {
                if (before(s, j, ls[i], lj[i])) {
                    const bool here = (i == 0) || before(ls[i > 0 ? i - 1 : 0], lj[i > 0 ? i - 1 : 0], s, j);
                    if (here) {
                        ls[i] = s;
                        lj[i] = j;
                    } else {
                        ls[i] = ls[i - 1];
                        lj[i] = lj[i - 1];
                    }
                }
            }
        }
    }

    // k rounds of wave argmin over the lanes' list heads
    int mine = -1;  // lane r keeps the r-th result
    int count = 0;
    for (int r = 0; r < a.k; ++r) {
        double bs = ls[0];
        int bj = lj[0];
#pragma unroll
        for (int off = kWave / 2; off >= 1; off >>= 1) {
            const double os = __shfl_xor(bs, off);
            const int oj = __shfl_xor(bj, off);
            if (before(os, oj, bs, bj)) {
                bs = os;
                bj = oj;
            }
        }
        const bool found = bj != INT32_MAX;
        if (found && lj[0] == bj) {  // the winner pops its head
#pragma unroll
            for (int i = 0; i < KMAX - 1; ++i) {
                ls[i] = ls[i + 1];
                lj[i] = lj[i + 1];
            }
            ls[KMAX - 1] = INFINITY;
            lj[KMAX - 1] = INT32_MAX;
        }
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

}  // namespace

hipError_t launch_retrieve(const RetrieveArgs& a, hipStream_t stream) {
    if (a.n_query == 0) return hipSuccess;
    const dim3 grid(a.n_query), block(kWave);
    if (a.k <= 4) {
        hipLaunchKernelGGL(retrieve_kernel<4>, grid, block, 0, stream, a);
    } else if (a.k <= 8) {
        hipLaunchKernelGGL(retrieve_kernel<8>, grid, block, 0, stream, a);
    } else if (a.k <= 16) {
        hipLaunchKernelGGL(retrieve_kernel<16>, grid, block, 0, stream, a);
    } else {
        hipLaunchKernelGGL(retrieve_kernel<32>, grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace revisit
