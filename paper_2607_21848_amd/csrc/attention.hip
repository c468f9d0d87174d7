// Chunk attention with the Gaussian correspondence bias fused in
// (Sec. 4.3, Eq. bias; design choices (ii) and (iii)).
//
// Both kernels compute, per head, O = softmax(scale Q K^T + lambda B) V with
// an online (flash-style) softmax over key tiles, never materialising the
// Lq x Lk logits or the bias.
//
// Layout on the matrix cores. Each wave owns 32 queries and computes the
// TRANSPOSED logit tile S^T = K Q^T with 32x32 MFMAs: keys are the M
// dimension (A operand, streamed from LDS), queries the N dimension (B
// operand, resident in registers). In the 32x32 accumulator a lane holds one
// column (one query) and 16 rows (keys), so the softmax row max and row sum
// are in-lane reductions plus one exchange between the two wave halves. The
// probabilities then feed O^T = V^T P^T directly as the B operand without
// any shuffle: the bf16 kernel loads the K rows in a permuted order (bits 2
// and 3 of the row index swapped) so that each half-wave's 8 consecutive
// accumulator registers are 8 consecutive keys, which is the register
// layout the bf16 B operand wants.
//
// The bias on the matrix cores. With centred token coordinates
// a = u_k - c and u' = u^ - c (c = grid centre) and gamma =
// lambda / (2 sigma^2 scale),
//     (lambda / scale) B = 2 gamma a.u' - gamma |a|^2 - gamma |u'|^2,
// a sum of four products of a per-key factor and a per-query factor. Both
// kernels add it into the logit accumulator with one extra short MFMA per
// 32-key block that touches a retrieved frame: key side
// [2 a_x, 2 a_y, -gamma |a|^2, 1], query side [gamma u'_x, gamma u'_y, 1,
// -gamma |u'|^2], zeroed for keys outside the frame and for rejected
// queries (so unbiased logits are bit-identical to plain attention). In the
// bf16 kernel every fp32 factor is split into three bf16 pieces whose sum
// is the fp32 value exactly; the half-integer a's are exact in bf16. The
// softmax loop therefore pays nothing for the bias: it is one MFMA per
// biased 32x32 block next to the eight of the QK^T product.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace revisit {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Accumulator row held by register i of a lane in wave half `hh` (32x32 MFMA).
__device__ __forceinline__ int acc_row(int hh, int i) { return 8 * (i >> 2) + 4 * hh + (i & 3); }

struct BiasGeom {
    float gamma;  // lambda / (2 sigma^2 softmax_scale)
    float cx, cy;  // grid centre (w / 2, h / 2)
    int hw, w;
};

// Frame of `key` and its centred token coordinates.
__device__ __forceinline__ void key_coords(int key, const BiasGeom& g, int& frame, float& ax, float& ay) {
    frame = key / g.hw;
    const int t = key - frame * g.hw;
    const int ky = t / g.w;
    const int kx = t - ky * g.w;
    ax = ((float)kx + 0.5f) - g.cx;
    ay = ((float)ky + 0.5f) - g.cy;
}

// Per-query bias factors for source frame s: gamma u'_x, gamma u'_y,
// -gamma |u'|^2; valid = the correspondence was accepted.
__device__ __forceinline__ void query_factors(const float* corr_uv, const int32_t* corr_idx, int Lq, int s, int q,
                                              const BiasGeom& g, bool& valid, float& gx, float& gy, float& q0) {
    valid = false;
    gx = gy = q0 = 0.0f;
    if (q < Lq) {
        const size_t o = (size_t)s * Lq + q;
        if (corr_idx[o] >= 0) {
            const float2 u = reinterpret_cast<const float2*>(corr_uv)[o];
            const float ux = u.x - g.cx, uy = u.y - g.cy;
            valid = true;
            gx = g.gamma * ux;
            gy = g.gamma * uy;
            q0 = -g.gamma * (ux * ux + uy * uy);
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 kernel: v_mfma_f32_32x32x2_f32. 4 waves x 32 queries per workgroup,
// 32-key tiles staged in LDS.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(AttentionArgs a, BiasGeom g, float c_log2, bool bias_on) {
    constexpr int TK = 32;
    __shared__ float Ks[TK][D + 1];
    __shared__ float Vs[TK][D];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int hh = lane >> 5;
    const int n = lane & 31;
    const int hd = blockIdx.y;
    const int H = a.H;
    const int q = blockIdx.x * 128 + wave * 32 + n;
    const bool q_ok = q < a.Lq;
    const float* Qg = static_cast<const float*>(a.q);
    const float* Kg = static_cast<const float*>(a.k);
    const float* Vg = static_cast<const float*>(a.v);

    float qf[D / 2];
#pragma unroll
    for (int kk = 0; kk < D / 2; ++kk) qf[kk] = q_ok ? Qg[((size_t)q * H + hd) * D + 2 * kk + hh] : 0.0f;

    floatx16 O[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) O[db] = floatx16{0};
    float m_run = -INFINITY, l_run = 0.0f;
    const int n_frames = a.Lk / g.hw;

    for (int tile0 = 0; tile0 < a.Lk; tile0 += TK) {
        __syncthreads();
        for (int e = tid; e < TK * D; e += 256) {
            const int r = e / D, c = e - (e / D) * D;
            const int key = tile0 + r;
            const bool in = key < a.Lk;
            Ks[r][c] = in ? Kg[((size_t)key * H + hd) * D + c] : 0.0f;
            Vs[r][c] = in ? Vg[((size_t)key * H + hd) * D + c] : 0.0f;
        }
        __syncthreads();

        floatx16 acc = floatx16{0};
        if (bias_on) {
            const int k_last = min(tile0 + TK, a.Lk) - 1;
            const int f0 = tile0 / g.hw, f1 = k_last / g.hw;
            for (int f = f0; f <= f1 && f < n_frames; ++f) {
                const int s = a.slot[f];
                if (s < 0 || s >= a.S) continue;
                int kf;
                float ax, ay;
                const int key = tile0 + n;  // this lane's A-operand row
                key_coords(key, g, kf, ax, ay);
                const bool in_f = key <= k_last && kf == f;
                bool valid;
                float gx, gy, q0;
                query_factors(a.corr_uv, a.corr_idx, a.Lq, s, q, g, valid, gx, gy, q0);
                const float k0 = -g.gamma * (ax * ax + ay * ay);
                const float a0 = in_f ? (hh ? 2.0f * ay : 2.0f * ax) : 0.0f;
                const float a1 = in_f ? (hh ? 1.0f : k0) : 0.0f;
                const float b0 = valid ? (hh ? gy : gx) : 0.0f;
                const float b1 = valid ? (hh ? q0 : 1.0f) : 0.0f;
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc, 0, 0, 0);
            }
        }
#pragma unroll
        for (int kk = 0; kk < D / 2; ++kk) {
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(Ks[n][2 * kk + hh], qf[kk], acc, 0, 0, 0);
        }

        // online softmax over this tile (column n = this lane's query)
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            if (tile0 + acc_row(hh, i) >= a.Lk) acc[i] = -INFINITY;
            mx = fmaxf(mx, acc[i]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx * c_log2);
        const float alpha = exp2f(m_run - m_new);
        float lsum = 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            acc[i] = exp2f(acc[i] * c_log2 - m_new);
            lsum += acc[i];
        }
        l_run = l_run * alpha + lsum;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) O[db] *= alpha;

        // O^T += V^T P^T: contraction step kk pairs accumulator register kk
        // (key acc_row(hh, kk)) in both operands
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            const int kr = acc_row(hh, kk);
#pragma unroll
            for (int db = 0; db < D / 32; ++db) {
                O[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(Vs[kr][32 * db + n], acc[kk], O[db], 0, 0, 0);
            }
        }
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.0f / l_tot;
    if (q_ok) {
        float* Og = static_cast<float*>(a.o) + ((size_t)q * H + hd) * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
#pragma unroll
            for (int i = 0; i < 16; ++i) Og[32 * db + acc_row(hh, i)] = O[db][i] * inv;
        }
        if (a.lse && hh == 0) a.lse[(size_t)hd * a.Lq + q] = (m_run + log2f(l_tot)) * kLn2;
    }
}

// ---------------------------------------------------------------------------
// bf16 kernel: v_mfma_f32_32x32x16_bf16, D = 128. 4 waves x 32 queries per
// workgroup; 64-key tiles (two 32-row MFMA blocks); K staged row-major and V
// staged transposed in LDS; the next tile is prefetched into registers while
// the current one is consumed.
// ---------------------------------------------------------------------------
constexpr int kD = 128;
constexpr int kTK = 64;
constexpr int kKPitch = kD + 8;    // bf16 elements per K row in LDS (272 B)
constexpr int kVPitch = kTK + 8;   // bf16 elements per V^T row in LDS (144 B)
constexpr float kRescaleSlack = 8.0f;  // lazy rescale: tolerate p up to 2^8

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Row swap that makes a half-wave's accumulator registers 8t..8t+7 hold 8
// consecutive keys: exchanges bits 2 and 3 of the row index.
__device__ __forceinline__ int perm_row(int m) { return (m & ~12) | ((m & 8) >> 1) | ((m & 4) << 1); }

__device__ __forceinline__ uint32_t bf16_bits_rne(float x) {
    const __bf16 b = (__bf16)x;
    return (uint32_t)__builtin_bit_cast(unsigned short, b);
}
__device__ __forceinline__ float bf16_value(uint32_t bits) { return __uint_as_float(bits << 16); }

// x = hi + mid + lo exactly (three bf16 pieces of an fp32 value).
__device__ __forceinline__ void split3(float x, uint32_t& hi, uint32_t& mid, uint32_t& lo) {
    hi = bf16_bits_rne(x);
    const float r1 = x - bf16_value(hi);
    mid = bf16_bits_rne(r1);
    const float r2 = r1 - bf16_value(mid);
    lo = bf16_bits_rne(r2);
}

__device__ __forceinline__ uint32_t pack2(uint32_t lo16, uint32_t hi16) { return lo16 | (hi16 << 16); }

__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(AttentionArgs a, BiasGeom g, float c_log2, bool bias_on) {
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kTK * kKPitch];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[kD * kVPitch];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int hh = lane >> 5;
    const int n = lane & 31;
    const int hd = blockIdx.y;
    const int H = a.H;
    const int Lk = a.Lk;
    const int q = blockIdx.x * 128 + wave * 32 + n;
    const bool q_ok = q < a.Lq;
    const uint16_t* Qg = static_cast<const uint16_t*>(a.q);
    const uint16_t* Kg = static_cast<const uint16_t*>(a.k);
    const uint16_t* Vg = static_cast<const uint16_t*>(a.v);
    const size_t row_stride = (size_t)H * kD;  // elements between consecutive tokens

    // Q fragments: lane (hh, n) holds Q[q][16 kk + 8 hh .. +8)
    bf16x8 qf[8];
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
        u32x4 v = u32x4{0, 0, 0, 0};
        if (q_ok) v = *reinterpret_cast<const u32x4*>(Qg + (size_t)q * row_stride + (size_t)hd * kD + 16 * kk + 8 * hh);
        qf[kk] = as_bf16x8(v);
    }

    // staging assignment: K chunk c = tid + 256 r -> row c / 16, col (c % 16) * 8;
    // V: key pair pi = tid % 32 (keys 2pi, 2pi+1), d-chunks dc and dc + 8
    const int v_pi = tid & 31;
    const int v_dc = tid >> 5;
    u32x4 kreg[4], vreg[4];
    auto load_tile = [&](int tile0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int c = tid + 256 * r;
            const int row = c >> 4;
            const int col = (c & 15) * 8;
            const int key = tile0 + row;
            kreg[r] = key < Lk ? *reinterpret_cast<const u32x4*>(Kg + (size_t)key * row_stride + (size_t)hd * kD + col)
                               : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int key = tile0 + 2 * v_pi + (r & 1);
            const int col = (v_dc + 8 * (r >> 1)) * 8;
            vreg[r] = key < Lk ? *reinterpret_cast<const u32x4*>(Vg + (size_t)key * row_stride + (size_t)hd * kD + col)
                               : u32x4{0, 0, 0, 0};
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int c = tid + 256 * r;
            *reinterpret_cast<u32x4*>(Ks + (c >> 4) * kKPitch + (c & 15) * 8) = kreg[r];
        }
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const u32x4 k0 = vreg[2 * half], k1 = vreg[2 * half + 1];
            const int d0 = (v_dc + 8 * half) * 8;
#pragma unroll
            for (int wd = 0; wd < 4; ++wd) {
                // elements 2wd (low halves) and 2wd+1 (high halves) of both keys
                const uint32_t lo = (k0[wd] & 0xffffu) | (k1[wd] << 16);
                const uint32_t hi = (k0[wd] >> 16) | (k1[wd] & 0xffff0000u);
                *reinterpret_cast<uint32_t*>(Vt + (d0 + 2 * wd) * kVPitch + 2 * v_pi) = lo;
                *reinterpret_cast<uint32_t*>(Vt + (d0 + 2 * wd + 1) * kVPitch + 2 * v_pi) = hi;
            }
        }
    };

    floatx16 O[4];
#pragma unroll
    for (int db = 0; db < 4; ++db) O[db] = floatx16{0};
    float m_run = -INFINITY, l_run = 0.0f;
    const int n_frames = Lk / g.hw;

    // query-side bias operand, rebuilt when the retrieved frame changes
    int cached_s = -1;
    bf16x8 qb = as_bf16x8(u32x4{0, 0, 0, 0});

    const int n_tiles = (Lk + kTK - 1) / kTK;
    load_tile(0);
    for (int it = 0; it < n_tiles; ++it) {
        const int tile0 = it * kTK;
        __syncthreads();
        store_tile();
        __syncthreads();
        if (it + 1 < n_tiles) load_tile(tile0 + kTK);

        floatx16 acc[2];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
            acc[rb] = floatx16{0};
            const int k0 = tile0 + 32 * rb;
            if (bias_on && k0 < Lk) {
                const int k_last = min(k0 + 31, Lk - 1);
                const int f0 = k0 / g.hw, f1 = k_last / g.hw;
                for (int f = f0; f <= f1 && f < n_frames; ++f) {
                    const int s = a.slot[f];
                    if (s < 0 || s >= a.S) continue;
                    if (s != cached_s) {
                        bool valid;
                        float gx, gy, q0;
                        query_factors(a.corr_uv, a.corr_idx, a.Lq, s, q, g, valid, gx, gy, q0);
                        uint32_t xh, xm, xl, yh, ym, yl, zh, zm, zl;
                        split3(gx, xh, xm, xl);
                        split3(gy, yh, ym, yl);
                        split3(q0, zh, zm, zl);
                        const uint32_t one = 0x3f80u;
                        u32x4 v;
                        if (hh == 0) v = u32x4{pack2(xh, xm), pack2(xl, yh), pack2(ym, yl), pack2(one, one)};
                        else v = u32x4{pack2(one, zh), pack2(zm, zl), 0u, 0u};
                        if (!valid) v = u32x4{0, 0, 0, 0};
                        qb = as_bf16x8(v);
                        cached_s = s;
                    }
                    int kf;
                    float ax, ay;
                    const int key = k0 + perm_row(n);
                    key_coords(key, g, kf, ax, ay);
                    const bool in_f = key <= k_last && kf == f;
                    u32x4 kv = u32x4{0, 0, 0, 0};
                    if (in_f) {
                        const uint32_t x2 = bf16_bits_rne(2.0f * ax), y2 = bf16_bits_rne(2.0f * ay);
                        uint32_t kh, km, kl;
                        split3(-g.gamma * (ax * ax + ay * ay), kh, km, kl);
                        const uint32_t one = 0x3f80u;
                        if (hh == 0) kv = u32x4{pack2(x2, x2), pack2(x2, y2), pack2(y2, y2), pack2(kh, km)};
                        else kv = u32x4{pack2(kl, one), pack2(one, one), 0u, 0u};
                    }
                    acc[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv), qb, acc[rb], 0, 0, 0);
                }
            }
            const uint16_t* krow = Ks + (32 * rb + perm_row(n)) * kKPitch + 8 * hh;
#pragma unroll
            for (int kk = 0; kk < 8; ++kk) {
                const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4*>(krow + 16 * kk));
                acc[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], acc[rb], 0, 0, 0);
            }
        }

        // online softmax; register i of block rb holds key
        // tile0 + 32 rb + 16 (i / 8) + 8 hh + (i % 8)
        float mx = -INFINITY;
        if (tile0 + kTK > Lk) {
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    if (tile0 + 32 * rb + 16 * (i >> 3) + 8 * hh + (i & 7) >= Lk) acc[rb][i] = -INFINITY;
                }
            }
        }
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, acc[rb][i]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32)) * c_log2;
        if (__any(mx > m_run + kRescaleSlack)) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = exp2f(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < 4; ++db) O[db] *= alpha;
            m_run = m_new;
        }
        bf16x8 pf[2][2];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                uint32_t w4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = exp2f(fmaf(acc[rb][8 * t + 2 * e], c_log2, -m_run));
                    const float p1 = exp2f(fmaf(acc[rb][8 * t + 2 * e + 1], c_log2, -m_run));
                    l_run += p0 + p1;
                    w4[e] = pack2(bf16_bits_rne(p0), bf16_bits_rne(p1));
                }
                pf[rb][t] = as_bf16x8(u32x4{w4[0], w4[1], w4[2], w4[3]});
            }
        }

        // O^T += V^T P^T
#pragma unroll
        for (int db = 0; db < 4; ++db) {
            const uint16_t* vrow = Vt + (32 * db + n) * kVPitch + 8 * hh;
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const bf16x8 vf = as_bf16x8(*reinterpret_cast<const u32x4*>(vrow + 32 * rb + 16 * t));
                    O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[rb][t], O[db], 0, 0, 0);
                }
            }
        }
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.0f / l_tot;
    if (q_ok) {
        uint16_t* Og = static_cast<uint16_t*>(a.o) + (size_t)q * row_stride + (size_t)hd * kD;
#pragma unroll
        for (int db = 0; db < 4; ++db) {
#pragma unroll
            for (int gi = 0; gi < 4; ++gi) {
                const int d = 32 * db + 8 * gi + 4 * hh;
                const uint32_t w0 = pack2(bf16_bits_rne(O[db][4 * gi] * inv), bf16_bits_rne(O[db][4 * gi + 1] * inv));
                const uint32_t w1 = pack2(bf16_bits_rne(O[db][4 * gi + 2] * inv), bf16_bits_rne(O[db][4 * gi + 3] * inv));
                *reinterpret_cast<uint2*>(Og + d) = make_uint2(w0, w1);
            }
        }
        if (a.lse && hh == 0) a.lse[(size_t)hd * a.Lq + q] = (m_run + log2f(l_tot)) * kLn2;
    }
}

BiasGeom make_geom(const AttentionArgs& a) {
    BiasGeom g;
    g.gamma = a.lambda / (2.0f * a.sigma * a.sigma * a.softmax_scale);
    g.cx = 0.5f * (float)a.w;
    g.cy = 0.5f * (float)a.h;
    g.hw = a.h * a.w;
    g.w = a.w;
    return g;
}

}  // namespace

hipError_t launch_attention_f32(const AttentionArgs& a, hipStream_t stream) {
    if (a.Lq == 0) return hipSuccess;
    const BiasGeom g = make_geom(a);
    const bool bias_on = a.S > 0 && a.lambda != 0.0f;
    const dim3 grid((a.Lq + 127) / 128, a.H), block(256);
    const float c = a.softmax_scale * kLog2e;
    if (a.D == 64) {
        hipLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, stream, a, g, c, bias_on);
    } else {
        hipLaunchKernelGGL(attn_f32_kernel<128>, grid, block, 0, stream, a, g, c, bias_on);
    }
    return hipGetLastError();
}

hipError_t launch_attention_bf16(const AttentionArgs& a, hipStream_t stream) {
    if (a.Lq == 0) return hipSuccess;
    const BiasGeom g = make_geom(a);
    const bool bias_on = a.S > 0 && a.lambda != 0.0f;
    const dim3 grid((a.Lq + 127) / 128, a.H), block(256);
    hipLaunchKernelGGL(attn_bf16_kernel, grid, block, 0, stream, a, g, a.softmax_scale * kLog2e, bias_on);
    return hipGetLastError();
}

}  // namespace revisit
