// Per-token depth/pose reprojection with the occlusion-aware visibility test
// (Sec. 4.3, Eq. reprojection and Eq. visibility; rejection causes of
// design choice (iii)).
//
// Launch: one thread per query token; a 128-thread block covers 128 tokens
// of one (problem b, target frame t) pair. The pose and
// intrinsics of (b, t) and of each source frame are wave-uniform, so they
// arrive through scalar loads; the thread pools its token's p x p depth
// block once, lifts it to the world once, then loops over the S source
// frames: relative transform, projection, grid test, a p x p gather of the
// source depth around u^ (cache-resident: a source frame is at most a few
// hundred KB) and the visibility test. Outputs are structure-of-arrays
// [B][S][Tq*h*w] so that for every s consecutive threads store consecutive
// tokens (u^ pairs and codes, fully coalesced, non-temporal).
//
// Arithmetic is IEEE double in the order of the definition with
// contraction disabled; the code and u^ (rounded to fp32 once) are
// therefore bit-identical to any IEEE evaluation of the same expressions.
// The quotients are the IEEE ones: where every input lies in a range that
// keeps all intermediates normal (checked per block and per wave), the two
// coordinates of u^ share one correctly rounded reciprocal of [X_s]_z and
// take one Markstein correction each (quotient.h), which equals the IEEE
// quotient there; elsewhere the kernel divides.
// For the usual p = 2 the kernel is specialised: dividing by 2 or by 4 is
// the same IEEE result as multiplying by 0.5 or 0.25, so the token-grid
// intrinsics and the pooling mean cost a multiply instead of a division,
// and each 2x2 depth block is read as two 8-byte loads. p = 1 (maps pooled
// beforehand, intrinsics already on the token grid) reads one value per token.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "internal.h"
#include "quotient.h"

#pragma clang fp contract(off)

namespace revisit {
namespace {

constexpr int kBlock = 128;  // measured 1-2% faster than 256 (and than 64, 512, 1024)
constexpr int kMaxSrcLds = 64;  // source frames per problem
constexpr int64_t kSmallLaunch = 512;  // token blocks below which a block takes one source

// Mean of the p x p depth block of token (i, j): rows outer, columns inner.
// P = 1 or 2: compile-time block; P = 0: runtime p.
template <int P>
__device__ __forceinline__ double pooled(const float* __restrict__ d, int Wd, int i, int j, int p) {
    if constexpr (P == 1) {
        return (double)d[(size_t)i * Wd + j];  // pre-pooled map: one value per token
    } else if constexpr (P == 2) {
        const float2 r0 = *reinterpret_cast<const float2*>(d + (size_t)(2 * i) * Wd + 2 * j);
        const float2 r1 = *reinterpret_cast<const float2*>(d + (size_t)(2 * i + 1) * Wd + 2 * j);
        return ((((double)r0.x + (double)r0.y) + (double)r1.x) + (double)r1.y) * 0.25;  // == / 4
    } else {
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
}

// K / p on the token grid (exact multiply by 0.5 when P = 2).
template <int P>
__device__ __forceinline__ double per_token(float k, double pd) {
    if constexpr (P == 1) return (double)k;  // == k / 1
    else if constexpr (P == 2) return (double)k * 0.5;
    else return (double)k / pd;
}

// Outputs are written once and never read back by this kernel: non-temporal
// stores keep them from displacing the depth maps in the caches.
__device__ __forceinline__ void st_uv(float2* p, float2 v) {
    __builtin_nontemporal_store(v.x, &p->x);
    __builtin_nontemporal_store(v.y, &p->y);
}
__device__ __forceinline__ void st_code(int32_t* p, int v) { __builtin_nontemporal_store(v, p); }

// A target token lifted to the world: R_t X_t + c_t, or undefined depth.
struct Lifted {
    double W[3];
    bool defined;
};

// Result for one (token, source): u^ (NaN when not computed) and the code.
struct Corr {
    float2 uv;
    int code;
};

// Frames of the block's problem converted to doubles in LDS: per source s,
// R (row-major), c, token-grid (fx, fy, cx, cy), and its frame index (-1 = no
// source); the same 16 values of the block's target frame in tc, and the
// correctly rounded reciprocals of its fx and fy in trcp.
struct SrcFrames {
    double c[kMaxSrcLds][16];
    int f[kMaxSrcLds];
    double tc[16];
    double trcp[2];
    int out_of_range[kBlock / 64];  // per wave: a frame value outside the shared-reciprocal range
};

// The 16 doubles of a frame: R row-major, c, then K / p on the token grid.
template <int P>
__device__ __forceinline__ double frame_value(const float* M, const float* K, int v, double pd) {
    if (v < 9) return (double)M[4 * (v / 3) + v % 3];
    if (v < 12) return (double)M[4 * (v - 9) + 3];
    return per_token<P>(K[v - 12], pd);
}

// Range condition of the shared-reciprocal quotients (quotient.h) on a frame
// value: zero or of magnitude in [2^-64, 2^64]; fx and fy (v = 12, 13)
// nonzero; cx and cy (v = 14, 15) not -0. With every frame value of a problem
// in range and the target depth z in [2^-40, 2^40], every quantity the
// correspondence computes is zero or of magnitude in [2^-850, 2^800]: the
// operands are products of a few in-range factors (numerators at least
// 2^-540, denominators in [2^-423, 2^302]), every nonzero sum is a multiple
// of the smallest unit of its terms, and the quotients' residuals are
// multiples of 2^-644. The quotients' intermediates therefore stay normal and
// no numerator is -0, so the shared-reciprocal quotient is the IEEE one.
__device__ __forceinline__ bool frame_value_in_range(double x, int v) {
    const double m = fabs(x);
    const bool mag = m >= 0x1p-64 && m <= 0x1p64;
    if (v == 12 || v == 13) return mag;
    if (v >= 14 && x == 0.0 && signbit(x)) return false;
    return x == 0.0 || mag;
}

// X_t = z K_t^-1 u~ lifted to the world: R_t X_t + c_t (the source centre
// comes later). T holds the target frame's 16 doubles, Trcp 1 / fx, 1 / fy;
// kShared selects the shared-reciprocal quotients.
template <bool kShared>
__device__ __forceinline__ Lifted lift(double z, int i, int j, const double* T, const double* Trcp) {
    Lifted L;
    L.defined = isfinite(z) && z > 0.0;
    const double ux = (double)j + 0.5, uy = (double)i + 0.5;
    double qx, qy;
    if constexpr (kShared) {
        qx = quotient_from_reciprocal(ux - T[14], T[12], Trcp[0]);
        qy = quotient_from_reciprocal(uy - T[15], T[13], Trcp[1]);
    } else {
        qx = (ux - T[14]) / T[12];
        qy = (uy - T[15]) / T[13];
    }
    const double Xt = qx * z;
    const double Yt = qy * z;
    const double Zt = z;
#pragma unroll
    for (int r = 0; r < 3; ++r) L.W[r] = ((T[3 * r + 0] * Xt + T[3 * r + 1] * Yt) + T[3 * r + 2] * Zt) + T[9 + r];
    return L;
}

// Pooled depth of cell (i, j) of a source frame whose base is uniform across
// the wave; the in-frame byte offset fits in 32 bits (a frame holds at most
// 2^28 pixels).
template <int P>
__device__ __forceinline__ double pooled_at(const uint8_t* frame, int Wd, int i, int j, int p) {
    if constexpr (P == 1) {
        const uint32_t off = ((uint32_t)i * (uint32_t)Wd + (uint32_t)j) * 4u;
        return (double)*reinterpret_cast<const float*>(frame + off);
    } else if constexpr (P == 2) {
        const uint32_t off = ((uint32_t)(2 * i) * (uint32_t)Wd + (uint32_t)(2 * j)) * 4u;
        const float2 r0 = *reinterpret_cast<const float2*>(frame + off);
        const float2 r1 = *reinterpret_cast<const float2*>(frame + (off + (uint32_t)Wd * 4u));
        return ((((double)r0.x + (double)r0.y) + (double)r1.x) + (double)r1.y) * 0.25;  // == / 4
    } else {
        return pooled<0>(reinterpret_cast<const float*>(frame), Wd, i, j, p);
    }
}

// Eq. reprojection and Eq. visibility for one (lifted token, source frame).
// Every lane evaluates the whole expression and the rejection causes pick
// the result by selects, so a wave that mixes accepted and rejected tokens
// takes no divergent branch; a rejected lane's values are discarded. Both
// coordinates of u^ share one reciprocal of [X_s]_z when kShared.
// floor(u^) is a truncation on the grid (u^ >= 0).
template <int P, bool kShared>
__device__ __forceinline__ Corr correspond(const ReprojectArgs& a, const Lifted& L, const double* C,
                                           const uint8_t* frame, int Wd, int p, double tol) {
    // R_t X_t + c_t - c_s
    const double W0 = L.W[0] - C[9];
    const double W1 = L.W[1] - C[10];
    const double W2 = L.W[2] - C[11];
    // X_s = R_s^T (...): component r is column r of R_s dotted with W
    const double Xs = (C[0] * W0 + C[3] * W1) + C[6] * W2;
    const double Ys = (C[1] * W0 + C[4] * W1) + C[7] * W2;
    const double Zs = (C[2] * W0 + C[5] * W1) + C[8] * W2;
    const double hx = C[12] * Xs + C[14] * Zs;
    const double hy = C[13] * Ys + C[15] * Zs;
    double uhx, uhy;
    if constexpr (kShared) {
        const double y = 1.0 / Zs;
        uhx = quotient_from_reciprocal(hx, Zs, y);
        uhy = quotient_from_reciprocal(hy, Zs, y);
    } else {
        uhx = hx / Zs;
        uhy = hy / Zs;
    }
    const bool front = L.defined && Zs > 0.0;
    const bool on_grid = front && uhx >= 0.0 && uhx < (double)a.w && uhy >= 0.0 && uhy < (double)a.h;
    const int kx = on_grid ? (int)uhx : 0;
    const int ky = on_grid ? (int)uhy : 0;
    const double Ds = pooled_at<P>(frame, Wd, ky, kx, p);
    int code = on_grid ? ((Zs <= tol * Ds) ? ky * a.w + kx : -4) : -3;
    code = front ? code : (L.defined ? -2 : -1);
    const float2 uv = front ? make_float2((float)uhx, (float)uhy) : make_float2(NAN, NAN);
    return Corr{uv, code};
}

// One token against sources s_begin .. s_end - 1: lift, then correspond and
// store per source.
template <int P, bool kShared>
__device__ __forceinline__ void token_sources(const ReprojectArgs& a, const SrcFrames& sf, double z, int i, int j,
                                              int b, int t, int tok, int s_begin, int s_end, int Lq, int hw, int Wd,
                                              size_t frame_px, int p, double tol) {
    const Lifted L = lift<kShared>(z, i, j, sf.tc, sf.trcp);
    for (int s = s_begin; s < s_end; ++s) {
        const size_t o = ((size_t)b * a.S + s) * Lq + (size_t)t * hw + tok;
        const int f = __builtin_amdgcn_readfirstlane(sf.f[s]);
        Corr c{make_float2(NAN, NAN), -5};
        if (f >= 0) {
            const uint8_t* frame = reinterpret_cast<const uint8_t*>(a.src_depth) + (size_t)f * frame_px * 4;
            c = correspond<P, kShared>(a, L, sf.c[s], frame, Wd, p, tol);
        }
        st_uv(reinterpret_cast<float2*>(a.out_uv) + o, c.uv);
        st_code(a.out_idx + o, c.code);
    }
}

// kPerSource = false: a thread handles one token and loops over the S
// source frames (the lift is done once). kPerSource = true: a thread handles
// one (token, source) pair, for launches too small to fill the GPU with one
// thread per token; the arithmetic and its order are the same.
template <int P, bool kPerSource>
__global__ __launch_bounds__(kBlock) void reproject_kernel(ReprojectArgs a) {
    const int hw = a.h * a.w;
    const int blocks_per_frame = (hw + kBlock - 1) / kBlock;
    // work item = (problem, target frame, token block[, source]), problem-major,
    // each XCD a contiguous range so one problem's source depth stays in one L2
    const int per_item_src = kPerSource ? a.S : 1;
    const unsigned n_items = (unsigned)(blocks_per_frame * a.B * a.Tq * per_item_src);
    const int item_all = (int)__builtin_amdgcn_readfirstlane(xcd_item(blockIdx.x, n_items));
    if (item_all >= (int)n_items) return;  // grid padding (uniform, before the barrier)
    const int s_item = kPerSource ? item_all % a.S : 0;
    const int item = kPerSource ? item_all / a.S : item_all;
    const int s_begin = kPerSource ? s_item : 0;
    const int s_end = kPerSource ? s_item + 1 : a.S;
    // (problem, target frame) of this block; uniform, kept in scalar registers
    const int bt = __builtin_amdgcn_readfirstlane(item / blocks_per_frame);  // b * Tq + t
    const int b = __builtin_amdgcn_readfirstlane(bt / a.Tq);
    const int t = bt - b * a.Tq;
    const int tok = (item - bt * blocks_per_frame) * kBlock + threadIdx.x;
    const int tok_c = tok < hw ? tok : hw - 1;  // threads past the frame compute a valid token, store nothing
    const int i = tok_c / a.w;
    const int j = tok_c - i * a.w;
    const int p = P > 0 ? P : a.p;
    const int Wd = a.w * p;
    const size_t frame_px = (size_t)hw * p * p;
    const int Lq = a.Tq * hw;
    const double pd = (double)p;
    const double z = pooled<P>(a.tgt_depth + (size_t)bt * frame_px, Wd, i, j, p);
    const double tol = 1.0 + a.eps;

    // the target frame and the problem's source frames (this block's one with
    // kPerSource), converted to doubles once per block, with the range check
    // of the shared-reciprocal quotients
    __shared__ SrcFrames sf;
    const float* Mt = a.tgt_c2w + (size_t)bt * 16;
    const float* Kt = a.tgt_K + (size_t)bt * 4;
    int out_of_range = 0;
    if (threadIdx.x < 16) {
        const double x = frame_value<P>(Mt, Kt, threadIdx.x, pd);
        sf.tc[threadIdx.x] = x;
        out_of_range |= !frame_value_in_range(x, threadIdx.x);
    } else if (threadIdx.x < 18) {
        sf.trcp[threadIdx.x - 16] = 1.0 / frame_value<P>(Mt, Kt, threadIdx.x - 4, pd);
    }
    // one thread per (source, value)
    for (int e = threadIdx.x; e < (s_end - s_begin) * 16; e += kBlock) {
        const int s = s_begin + (e >> 4), v = e & 15;
        int f = b * a.S + s;
        if (a.src_sel) {
            f = a.src_sel[(size_t)b * a.S + s];
            if (f < 0 || f >= a.n_src) f = -1;
        }
        if (v == 0) sf.f[s] = f;
        if (f >= 0) {
            const double x = frame_value<P>(a.src_c2w + (size_t)f * 16, a.src_K + (size_t)f * 4, v, pd);
            sf.c[s][v] = x;
            out_of_range |= !frame_value_in_range(x, v);
        }
    }
    // one flag per wave (a ballot), read by every wave after the barrier
    const int any_out = __any(out_of_range);
    if ((threadIdx.x & 63) == 0) sf.out_of_range[threadIdx.x >> 6] = any_out;
    __syncthreads();
    bool frames_in_range = true;
#pragma unroll
    for (int wv = 0; wv < kBlock / 64; ++wv) frames_in_range = frames_in_range && !sf.out_of_range[wv];
    if (tok >= hw) return;
    // a depth outside [2^-40, 2^40] sends its wave to the division path
    // (undefined depths are rejected whatever the path computes for them)
    const bool z_in_range = !(isfinite(z) && z > 0.0) || (z >= 0x1p-40 && z <= 0x1p40);
    if (frames_in_range && __all(z_in_range))
        token_sources<P, true>(a, sf, z, i, j, b, t, tok, s_begin, s_end, Lq, hw, Wd, frame_px, p, tol);
    else
        token_sources<P, false>(a, sf, z, i, j, b, t, tok, s_begin, s_end, Lq, hw, Wd, frame_px, p, tol);
}

// Rotation-only path (Sec. 4.3: with c_s = c_t the depth cancels in Eq.
// reprojection, leaving the homography u^ = pi(K_s R_s^T R_t K_t^-1 u~)).
// No depth is read and no visibility test applies. The block forms, per
// source frame, H = (K_s (R_s^T R_t)) K_t^-1 in double in LDS, in the order
//     A[r][c] = (Rs[0][r] Rt[0][c] + Rs[1][r] Rt[1][c]) + Rs[2][r] Rt[2][c]
//     M = rows (fx_s A0 + cx_s A2, fy_s A1 + cy_s A2, A2)
//     H[r] = (M[r][0] / fx_t, M[r][1] / fy_t, (M[r][2] - H[r][0] cx_t) - H[r][1] cy_t)
// and each thread evaluates v = H u~ for two adjacent tokens, so the launch
// is a pure write stream of 12 bytes per (token, source). Where H is in the
// shared-reciprocal range (homography_in_range), u^ = (v_0 / v_2, v_1 / v_2)
// share one reciprocal of v_2 (quotient.h): the IEEE quotients there. The pair's u^ go
// out as one 16-byte store and its codes as one 8-byte store where the pair
// is aligned (an even element index in outputs whose base addresses are 16-
// and 8-byte aligned: the common case), else one token at a time.
struct SrcHomographies {
    double H[kMaxSrcLds][9];
    int status[kMaxSrcLds];  // 0 = use H, else the code of every token (-5, -6)
    int shared[kMaxSrcLds];  // 1: H is in the shared-reciprocal range
};

// Range condition of the shared-reciprocal quotients (quotient.h) for a
// homography: every entry zero or of magnitude in [2^-200, 2^200], and
// neither numerator row (0, 1) all -0. Token centres are multiples of 1/2 in
// [1/2, 2^28) (a frame holds at most 2^28 tokens), so every nonzero v_r is
// a multiple of 2^-253 of magnitude below 2^230, the quotients lie in
// [2^-483, 2^483] and their residuals are multiples of 2^-840: every
// intermediate stays normal. A numerator is -0 only when its whole row is
// -0 (the token centres are positive), which the condition excludes, so the
// shared-reciprocal quotient is the IEEE one.
__device__ __forceinline__ bool homography_in_range(const double* H) {
    bool ok = true;
#pragma unroll
    for (int e = 0; e < 9; ++e) {
        const double m = fabs(H[e]);
        ok = ok && (H[e] == 0.0 || (m >= 0x1p-200 && m <= 0x1p200));
    }
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const bool neg_zero_row = H[3 * r] == 0.0 && signbit(H[3 * r]) && H[3 * r + 1] == 0.0 &&
                                  signbit(H[3 * r + 1]) && H[3 * r + 2] == 0.0 && signbit(H[3 * r + 2]);
        ok = ok && !neg_zero_row;
    }
    return ok;
}

template <int P>
__global__ __launch_bounds__(kBlock) void rotation_kernel(ReprojectArgs a) {
    const int hw = a.h * a.w;
    const int blocks_per_frame = (hw + 2 * kBlock - 1) / (2 * kBlock);
    const unsigned n_items = (unsigned)(blocks_per_frame * a.B * a.Tq);
    const int item = (int)__builtin_amdgcn_readfirstlane(xcd_item(blockIdx.x, n_items));
    if (item >= (int)n_items) return;  // grid padding (uniform, before the barrier)
    const int bt = __builtin_amdgcn_readfirstlane(item / blocks_per_frame);  // b * Tq + t
    const int b = __builtin_amdgcn_readfirstlane(bt / a.Tq);
    const int t = bt - b * a.Tq;
    const int tok = 2 * ((item - bt * blocks_per_frame) * kBlock + threadIdx.x);
    const int Lq = a.Tq * hw;
    const double pd = (double)(P > 0 ? P : a.p);

    __shared__ SrcHomographies sh;
    for (int s = threadIdx.x; s < a.S; s += kBlock) {
        int f = b * a.S + s;
        if (a.src_sel) {
            f = a.src_sel[(size_t)b * a.S + s];
            if (f < 0 || f >= a.n_src) f = -1;
        }
        int status = 0, shared = 0;
        if (f < 0) {
            status = -5;
        } else {
            const float* Mt = a.tgt_c2w + (size_t)bt * 16;
            const float* Ms = a.src_c2w + (size_t)f * 16;
            if (!(Mt[3] == Ms[3] && Mt[7] == Ms[7] && Mt[11] == Ms[11])) {
                status = -6;
            } else {
                const float* Kt = a.tgt_K + (size_t)bt * 4;
                const float* Ks = a.src_K + (size_t)f * 4;
                const double fxt = per_token<P>(Kt[0], pd), fyt = per_token<P>(Kt[1], pd);
                const double cxt = per_token<P>(Kt[2], pd), cyt = per_token<P>(Kt[3], pd);
                const double fxs = per_token<P>(Ks[0], pd), fys = per_token<P>(Ks[1], pd);
                const double cxs = per_token<P>(Ks[2], pd), cys = per_token<P>(Ks[3], pd);
                double A[3][3];
                for (int r = 0; r < 3; ++r)
                    for (int c = 0; c < 3; ++c)
                        A[r][c] = ((double)Ms[r] * (double)Mt[c] + (double)Ms[4 + r] * (double)Mt[4 + c]) +
                                  (double)Ms[8 + r] * (double)Mt[8 + c];
                for (int c = 0; c < 3; ++c) {
                    const double m0 = fxs * A[0][c] + cxs * A[2][c];
                    const double m1 = fys * A[1][c] + cys * A[2][c];
                    const double m2 = A[2][c];
                    A[0][c] = m0;
                    A[1][c] = m1;
                    A[2][c] = m2;
                }
                double Hs[9];
                for (int r = 0; r < 3; ++r) {
                    const double h0 = A[r][0] / fxt;
                    const double h1 = A[r][1] / fyt;
                    Hs[3 * r + 0] = h0;
                    Hs[3 * r + 1] = h1;
                    Hs[3 * r + 2] = (A[r][2] - h0 * cxt) - h1 * cyt;
                }
                for (int e = 0; e < 9; ++e) sh.H[s][e] = Hs[e];
                shared = homography_in_range(Hs);
            }
        }
        sh.status[s] = status;
        sh.shared[s] = shared;
    }
    __syncthreads();
    if (tok >= hw) return;
    const bool two = tok + 1 < hw;
    int i0 = tok / a.w;
    int j0 = tok - i0 * a.w;
    int i1 = i0, j1 = j0 + 1;
    if (j1 == a.w) { j1 = 0; i1 = i0 + 1; }
    const double ux0 = (double)j0 + 0.5, uy0 = (double)i0 + 0.5;
    const double ux1 = (double)j1 + 0.5, uy1 = (double)i1 + 0.5;
    typedef float f4 __attribute__((ext_vector_type(4)));
    typedef int i2 __attribute__((ext_vector_type(2)));
    // the pair's second token (past the frame when tok + 1 == hw: computed, not stored)
    for (int s = 0; s < a.S; ++s) {
        const size_t o = ((size_t)b * a.S + s) * Lq + (size_t)t * hw + tok;
        float2 uv[2] = {make_float2(NAN, NAN), make_float2(NAN, NAN)};
        int code[2] = {sh.status[s], sh.status[s]};
        // both tokens of the pair, with one reciprocal of v_2 per token in the
        // shared-reciprocal range (kShared), else two divisions
        auto evaluate = [&](auto shared_tag) {
            constexpr bool kShared = decltype(shared_tag)::value;
            const double* H = sh.H[s];
#pragma unroll
            for (int g = 0; g < 2; ++g) {
                const double ux = g ? ux1 : ux0, uy = g ? uy1 : uy0;
                const double v0 = (H[0] * ux + H[1] * uy) + H[2];
                const double v1 = (H[3] * ux + H[4] * uy) + H[5];
                const double v2 = (H[6] * ux + H[7] * uy) + H[8];
                if (!(v2 > 0.0)) {
                    code[g] = -2;
                } else {
                    double uhx, uhy;
                    if constexpr (kShared) {
                        const double y = 1.0 / v2;
                        uhx = quotient_from_reciprocal(v0, v2, y);
                        uhy = quotient_from_reciprocal(v1, v2, y);
                    } else {
                        uhx = v0 / v2;
                        uhy = v1 / v2;
                    }
                    uv[g] = make_float2((float)uhx, (float)uhy);
                    code[g] = (uhx >= 0.0 && uhx < (double)a.w && uhy >= 0.0 && uhy < (double)a.h)
                                  ? (int)floor(uhy) * a.w + (int)floor(uhx)
                                  : -3;
                }
            }
        };
        if (code[0] == 0) {
            if (sh.shared[s]) evaluate(std::true_type{});
            else evaluate(std::false_type{});
        }
        if (two && a.paired && (o & 1) == 0) {
            f4 v = {uv[0].x, uv[0].y, uv[1].x, uv[1].y};
            __builtin_nontemporal_store(v, reinterpret_cast<f4*>(a.out_uv + 2 * o));
            i2 c = {code[0], code[1]};
            __builtin_nontemporal_store(c, reinterpret_cast<i2*>(a.out_idx + o));
        } else {
            st_uv(reinterpret_cast<float2*>(a.out_uv) + o, uv[0]);
            st_code(a.out_idx + o, code[0]);
            if (two) {
                st_uv(reinterpret_cast<float2*>(a.out_uv) + o + 1, uv[1]);
                st_code(a.out_idx + o + 1, code[1]);
            }
        }
    }
}

}  // namespace

template <bool kPerSource>
static void launch_p(const ReprojectArgs& a, dim3 grid, hipStream_t stream) {
    const dim3 block(kBlock);
    if (a.p == 2) {
        hipLaunchKernelGGL((reproject_kernel<2, kPerSource>), grid, block, 0, stream, a);
    } else if (a.p == 1) {
        hipLaunchKernelGGL((reproject_kernel<1, kPerSource>), grid, block, 0, stream, a);
    } else {
        hipLaunchKernelGGL((reproject_kernel<0, kPerSource>), grid, block, 0, stream, a);
    }
}

hipError_t launch_reproject(const ReprojectArgs& a, hipStream_t stream) {
    const int hw = a.h * a.w;
    if (a.B == 0 || a.Tq == 0 || a.S == 0 || hw == 0) return hipSuccess;
    const int64_t blocks = (int64_t)((hw + kBlock - 1) / kBlock) * a.B * a.Tq;
    // fewer token blocks than two per compute unit: one block per (token block, source)
    const bool per_source = a.S > 1 && blocks < kSmallLaunch;
    const int64_t grid_blocks = per_source ? blocks * a.S : blocks;
    if (grid_blocks > INT32_MAX - kXcds) return hipErrorInvalidValue;
    const dim3 grid(xcd_grid((unsigned)grid_blocks));
    if (per_source) launch_p<true>(a, grid, stream);
    else launch_p<false>(a, grid, stream);
    return hipGetLastError();
}

hipError_t launch_rotation(const ReprojectArgs& a, hipStream_t stream) {
    const int hw = a.h * a.w;
    if (a.B == 0 || a.Tq == 0 || a.S == 0 || hw == 0) return hipSuccess;
    const int64_t blocks = (int64_t)((hw + 2 * kBlock - 1) / (2 * kBlock)) * a.B * a.Tq;
    if (blocks > INT32_MAX - kXcds) return hipErrorInvalidValue;
    const dim3 grid(xcd_grid((unsigned)blocks)), block(kBlock);
    if (a.p == 2) hipLaunchKernelGGL((rotation_kernel<2>), grid, block, 0, stream, a);
    else if (a.p == 1) hipLaunchKernelGGL((rotation_kernel<1>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((rotation_kernel<0>), grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace revisit
