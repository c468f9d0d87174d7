// Per-token depth/pose reprojection with the occlusion-aware visibility test
// (Sec. 4.3, Eq. reprojection and Eq. visibility; rejection causes of
// design choice (iii)).
//
// Launch: one thread per query token; a 256-thread block covers 256 tokens
// of one (problem b, target frame t) pair. The pose and
// intrinsics of (b, t) and of each source frame are wave-uniform, so they
// arrive through scalar loads; the thread pools its token's p x p depth
// block once, lifts it to the world once, then loops over the S source
// frames: relative transform, projection, grid test, a p x p gather of the
// source depth around u^ (cache-resident: a source frame is at most a few
// hundred KB) and the visibility test. Outputs are structure-of-arrays
// [B][S][Tq*h*w] so that for every s consecutive threads store consecutive
// tokens (8-byte u^ pairs and 4-byte codes, fully coalesced).
//
// Arithmetic is IEEE double in the order of the definition with
// contraction disabled; the code and u^ (rounded to fp32 once) are
// therefore bit-identical to any IEEE evaluation of the same expressions.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

#pragma clang fp contract(off)

namespace revisit {
namespace {

constexpr int kBlock = 256;

// Mean of the p x p depth block of token (i, j): rows outer, columns inner.
__device__ __forceinline__ double pooled(const float* __restrict__ d, int Wd, int i, int j, int p) {
    const float* base = d + (size_t)(i * p) * Wd + (size_t)j * p;
    double acc = 0.0;
    bool first = true;
    for (int a = 0; a < p; ++a) {
        for (int b = 0; b < p; ++b) {
            const double x = base[(size_t)a * Wd + b];
            acc = first ? x : acc + x;
            first = false;
        }
    }
    return acc / (double)(p * p);
}

__global__ __launch_bounds__(kBlock) void reproject_kernel(ReprojectArgs a) {
    const int hw = a.h * a.w;
    const int blocks_per_frame = (hw + kBlock - 1) / kBlock;
    const int bt = blockIdx.x / blocks_per_frame;  // b * Tq + t
    const int b = bt / a.Tq;
    const int t = bt - b * a.Tq;
    const int tok = (blockIdx.x - bt * blocks_per_frame) * kBlock + threadIdx.x;
    if (tok >= hw) return;
    const int i = tok / a.w;
    const int j = tok - i * a.w;
    const int p = a.p;
    const int Wd = a.w * p;
    const size_t frame_px = (size_t)hw * p * p;
    const int Lq = a.Tq * hw;
    const double pd = (double)p;

    const float* Mt = a.tgt_c2w + (size_t)bt * 16;
    const float* Kt = a.tgt_K + (size_t)bt * 4;
    const double fxt = (double)Kt[0] / pd, fyt = (double)Kt[1] / pd;
    const double cxt = (double)Kt[2] / pd, cyt = (double)Kt[3] / pd;

    const double z = pooled(a.tgt_depth + (size_t)bt * frame_px, Wd, i, j, p);
    const bool defined = isfinite(z) && z > 0.0;

    // X_t = z K_t^-1 u~, then R_t X_t + c_t (the source centre comes later)
    const double ux = (double)j + 0.5, uy = (double)i + 0.5;
    const double Xt = ((ux - cxt) / fxt) * z;
    const double Yt = ((uy - cyt) / fyt) * z;
    const double Zt = z;
    double Wt[3];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        Wt[r] = (((double)Mt[4 * r + 0] * Xt + (double)Mt[4 * r + 1] * Yt) + (double)Mt[4 * r + 2] * Zt) +
                (double)Mt[4 * r + 3];
    }
    const double tol = 1.0 + a.eps;

    for (int s = 0; s < a.S; ++s) {
        const size_t o = ((size_t)b * a.S + s) * Lq + (size_t)t * hw + tok;
        float2* uv_out = reinterpret_cast<float2*>(a.out_uv) + o;
        int f;  // source frame index into the src arrays
        if (a.src_sel) {
            f = a.src_sel[(size_t)b * a.S + s];
            if (f < 0 || f >= a.n_src) {
                *uv_out = make_float2(NAN, NAN);
                a.out_idx[o] = -5;
                continue;
            }
        } else {
            f = b * a.S + s;
        }
        if (!defined) {
            *uv_out = make_float2(NAN, NAN);
            a.out_idx[o] = -1;
            continue;
        }
        const float* Ms = a.src_c2w + (size_t)f * 16;
        const float* Ks = a.src_K + (size_t)f * 4;
        // R_t X_t + c_t - c_s
        const double W0 = Wt[0] - (double)Ms[3];
        const double W1 = Wt[1] - (double)Ms[7];
        const double W2 = Wt[2] - (double)Ms[11];
        // X_s = R_s^T (...): component r is column r of R_s dotted with W
        const double Xs = ((double)Ms[0] * W0 + (double)Ms[4] * W1) + (double)Ms[8] * W2;
        const double Ys = ((double)Ms[1] * W0 + (double)Ms[5] * W1) + (double)Ms[9] * W2;
        const double Zs = ((double)Ms[2] * W0 + (double)Ms[6] * W1) + (double)Ms[10] * W2;
        if (!(Zs > 0.0)) {
            *uv_out = make_float2(NAN, NAN);
            a.out_idx[o] = -2;
            continue;
        }
        const double fxs = (double)Ks[0] / pd, fys = (double)Ks[1] / pd;
        const double cxs = (double)Ks[2] / pd, cys = (double)Ks[3] / pd;
        const double uhx = (fxs * Xs + cxs * Zs) / Zs;
        const double uhy = (fys * Ys + cys * Zs) / Zs;
        *uv_out = make_float2((float)uhx, (float)uhy);
        if (!(uhx >= 0.0 && uhx < (double)a.w && uhy >= 0.0 && uhy < (double)a.h)) {
            a.out_idx[o] = -3;
            continue;
        }
        const int kx = (int)floor(uhx);
        const int ky = (int)floor(uhy);
        const double Ds = pooled(a.src_depth + (size_t)f * frame_px, Wd, ky, kx, p);
        a.out_idx[o] = (Zs <= tol * Ds) ? ky * a.w + kx : -4;
    }
}

}  // namespace

hipError_t launch_reproject(const ReprojectArgs& a, hipStream_t stream) {
    const int hw = a.h * a.w;
    if (a.B == 0 || a.Tq == 0 || a.S == 0 || hw == 0) return hipSuccess;
    const int64_t blocks = (int64_t)((hw + kBlock - 1) / kBlock) * a.B * a.Tq;
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks), block(kBlock);
    hipLaunchKernelGGL(reproject_kernel, grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace revisit
