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
// The bias. With gamma = lambda / (2 sigma^2 scale) the biased logit is
// scale (q.k + (lambda / scale) B), so both kernels put (lambda / scale) B
// into the logit accumulator before the QK^T MFMAs. The fp32 kernel
// evaluates it per logit, -gamma |u_k - u^|^2 with the differences taken
// first. The bf16 kernel uses the separable form: with centred token
// coordinates a = u_k - c and u' = u^ - c (c = grid centre),
//     (lambda / scale) B = 2 gamma a.u' - gamma |a|^2 - gamma |u'|^2,
// a sum of four products of a per-key factor and a per-query factor, added
// with one extra MFMA per 32-key block that touches a retrieved frame: key
// side [2 a_x, 2 a_y, -gamma |a|^2, 1], query side [gamma u'_x, gamma u'_y,
// 1, -gamma |u'|^2], zeroed for keys outside the frame and for rejected
// queries (so unbiased logits are bit-identical to plain attention). Every
// fp32 factor is split into three bf16 pieces whose sum is the fp32 value
// exactly; the half-integer a's are exact in bf16. The softmax loop
// therefore pays one MFMA per biased 32x32 block next to the eight of the
// QK^T product.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <type_traits>

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
    int hw, w, h;
};

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

        // the bias of this lane's 16 logits (query q, keys of rows acc_row(hh, i)),
        // evaluated directly as -gamma ((u_k,x - u^_x)^2 + (u_k,y - u^_y)^2),
        // differences first; it is the accumulator's start value
        floatx16 acc = floatx16{0};
        if (bias_on && q_ok) {
            int cf = -1;  // frame whose query factors are loaded
            bool valid = false;
            float2 u = make_float2(0.0f, 0.0f);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = tile0 + acc_row(hh, i);
                if (key >= a.Lk) continue;
                const int f = key / g.hw;
                if (f != cf) {
                    cf = f;
                    const int s = a.slot[f];
                    valid = false;
                    if (s >= 0 && s < a.S) {
                        const size_t o = (size_t)s * a.Lq + q;
                        if (a.corr_idx[o] >= 0) {
                            valid = true;
                            u = reinterpret_cast<const float2*>(a.corr_uv)[o];
                        }
                    }
                }
                if (valid) {
                    const int t = key - f * g.hw;
                    const int ky = t / g.w;
                    const int kx = t - ky * g.w;
                    const float dx = ((float)kx + 0.5f) - u.x;
                    const float dy = ((float)ky + 0.5f) - u.y;
                    acc[i] = -g.gamma * (dx * dx + dy * dy);
                }
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
// workgroup, 32-key tiles (one 32-row MFMA block each), two workgroups per CU.
//
// Memory path. K and V tiles travel global -> LDS with direct 16-byte loads
// (no register staging, no VALU). Both stay in their natural [key][d]
// layout (256-byte rows) with the 16-byte chunks of row r stored at chunk
// position c ^ swz(r). K rows are read with 16-byte LDS loads (the A operand
// of S^T = K Q^T); V is read with the LDS transpose load (ds_read_b64_tr_b16),
// which hands each lane 4 keys of one column d, so the A operand of
// O^T = V^T P^T needs no transposed copy. swz makes both access patterns hit
// 16 distinct chunk positions per 256 bytes.
//
// Pipeline. K runs one tile ahead of V: in step j a wave computes
// S_{j+1} = K_{j+1} Q^T on the matrix cores while its VALU turns S_j into
// probabilities, then accumulates O += P_j V_j while the VALU reduces the
// row maxima of S_{j+1}. The LDS holds a ring of three slots; slot t mod 3
// carries K_t and V_{t-1}. Right after its one barrier, step j refills slot
// j mod 3 (no wave reads K_j or V_{j-1} any more) with K_{j+3} and V_{j+2},
// so a direct load has two steps to land and each lane waits only for its
// loads of two steps back. The steady loop is unrolled over a period of six
// (ring slot and current logit registers are then compile-time). Inside a
// step the instruction order is fixed by hand with scheduling fences: the
// QK MFMAs run back to back with the K reads three MFMAs ahead, then the
// bias MFMA and most of the softmax, then the PV MFMAs carrying the V
// transpose reads, the last softmax units and the row maxima. The two waves
// of a SIMD fill each other's gaps: one wave's softmax runs beside the
// other's MFMA chain, which measured faster than one wave pairing every QK
// MFMA with a softmax unit of its own. Work units are mapped XCD-aware so
// the workgroups of one head (and key range) share an L2.
//
// Softmax. exp2 on the raw hardware instruction with scale * log2(e) folded
// into one FMA, probabilities packed to bf16 pairwise and summed with bf16
// dot products (the row sum then matches the rounded P fed to the PV
// product), and a lazy rescale that only touches O when a row maximum grows
// by more than 2^8.
//
// Bias. The four key/query factor pairs are laid out separably over the
// two halves of the MFMA contraction: lanes of the first half carry the
// column terms [2 a_x (x3), -gamma a_x^2 (3 pieces), 1, 1], lanes of the
// second half the row terms [2 a_y (x3), -gamma a_y^2 (3 pieces), 1, 0]; the
// query side is [gamma u'_x (3 pieces), 1, 1, 1, q0_hi, q0_mid] and
// [gamma u'_y (3 pieces), 1, 1, 1, q0_lo, 0] with q0 = -gamma |u'|^2. A key
// operand is then one 16-byte read from a per-workgroup table indexed by the
// key's column (first half) or row (second half).
// ---------------------------------------------------------------------------
constexpr int kD = 128;
constexpr int kTK = 32;
constexpr int kRowBytes = kD * 2;             // 256
constexpr int kTileBytes = kTK * kRowBytes;   // 8 KB per K or V tile
constexpr int kStages = 3;                    // K / V tiles in flight or resident per ring
constexpr int kWaitVm0 = 0x0f70;              // s_waitcnt immediate: vmcnt(0), other counters unconstrained
constexpr float kRescaleSlack = 8.0f;         // lazy rescale: tolerate p up to 2^8
constexpr int kMaxFramesLds = 1024;           // KV frames (slot table entries) of the bf16 kernel
constexpr int kMaxGridSide = 256;             // token-grid rows / columns of the bf16 bias tables
constexpr int kCorrLds = 16;                  // retrieved frames whose correspondences are staged in LDS

// Key split: the key tiles of every item (head, 128-query tile) are cut into
// `parts` equal ranges, part p = tiles [p n / parts, (p + 1) n / parts). One
// workgroup per (item, part); with parts > 1 each leaves its unnormalised
// result in partial slot item * parts + p for attn_merge_kernel.
struct KeySplit {
    int32_t parts;
    float* part;
};
constexpr int kPartFloats = 128 * kD + 2 * 128;  // O [128 queries][kD], then m [128], l [128]

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef int int8v __attribute__((ext_vector_type(8)));

// 32 fp8 operand bytes from two 16-byte reads
__device__ __forceinline__ int8v join8(u32x4 a, u32x4 b) {
    return int8v{(int)a[0], (int)a[1], (int)a[2], (int)a[3], (int)b[0], (int)b[1], (int)b[2], (int)b[3]};
}
// D += A B on the fp8 matrix cores, A and B e4m3 (format code 0), no block
// scaling: lane l supplies row / column l % 32 and contraction indices
// 32 (l / 32) .. + 32, and D comes back in the same 32 x 32 accumulator layout
// as v_mfma_f32_32x32x16_bf16 (both checked on the device)
__device__ __forceinline__ floatx16 mfma_fp8(int8v a, int8v b, floatx16 c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Row swap that makes a half-wave's accumulator registers 8t..8t+7 hold 8
// consecutive keys: exchanges bits 2 and 3 of the row index.
__device__ __forceinline__ int perm_row(int m) { return (m & ~12) | ((m & 8) >> 1) | ((m & 4) << 1); }

// Chunk swizzle of LDS row r (16 chunks of 16 bytes per row).
__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

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

__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2){lo, hi}, bf16x2));
}

// max(a, b, c) in one instruction (the logits are finite or -inf, never NaN)
__device__ __forceinline__ float max3(float a, float b, float c) {
    float r;
    asm volatile("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// max / sum of x over the lane and its partner in the other wave half
__device__ __forceinline__ float half_swap_max(float x) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

// Direct global -> LDS loads of one K or V tile of 32 rows. Wave `wave`
// fills its quarter of the tile with 1 KB instructions (64 lanes x 16
// bytes). Lane byte offsets relative to the tile's first row are fixed for
// the whole kernel (`off`); only the uniform base moves. On the last tile,
// rows past Lk are redirected to the last valid row (their logits are
// masked), so no load leaves the tensor. Rows are 256 bytes (bf16) or 128
// bytes (fp8 keys); the 16-byte chunks of row r sit at chunk position
// c ^ swz(r), a swizzle under which every operand read pattern of the kernel
// touches distinct bank groups.
template <int ROW_BYTES>
struct TileFmt {
    static constexpr int kChunks = ROW_BYTES / 16;
    static constexpr int kLoads = kTK * ROW_BYTES / (256 * 16);  // 16-byte direct loads per lane per tile
    static __device__ __forceinline__ int swizzle(int r) { return ROW_BYTES == 256 ? swz(r) : ((r >> 1) & 7); }
};
using RowsBf16 = TileFmt<256>;
using RowsFp8 = TileFmt<128>;
constexpr int kLoadsPerLane = RowsBf16::kLoads;  // V tiles (and bf16 K tiles)

template <class Fmt>
struct TileLoad {
    uint32_t off[Fmt::kLoads];  // byte offset of this lane's chunk from the tile's first row
};

template <class Fmt>
__device__ __forceinline__ void tile_chunk(int wave, int lane, int i, int& r, int& lc) {
    const int pos = (wave * Fmt::kLoads + i) * 64 + lane;  // 16-byte chunk position in the tile
    r = pos / Fmt::kChunks;
    lc = (pos % Fmt::kChunks) ^ Fmt::swizzle(r);  // logical chunk stored at this position
}

// row_bytes: bytes between consecutive tokens in global memory; head hd's
// row starts hd * ROW_BYTES into it
template <class Fmt>
__device__ __forceinline__ TileLoad<Fmt> make_tile_load(size_t row_bytes, int hd, int wave, int lane) {
    TileLoad<Fmt> t;
#pragma unroll
    for (int i = 0; i < Fmt::kLoads; ++i) {
        int r, lc;
        tile_chunk<Fmt>(wave, lane, i, r, lc);
        t.off[i] = (uint32_t)(r * (int)row_bytes + hd * (Fmt::kChunks * 16) + lc * 16);
    }
    return t;
}

// One direct load of 16 bytes per lane: global (base + voff) -> LDS
// (lds + 16 * lane). Written as inline asm so that the compiler's own
// wait-count bookkeeping, which cannot tell the ring slots apart and would
// drain every load in flight before reading any slot, does not see it; the
// pipeline orders these loads with explicit vmcnt waits (extra loads the
// compiler issues can only make those waits stricter: loads retire in order).
// M0 carries the LDS address and needs one wait state before the load. M0 is
// a reserved register that the compiler never allocates, and nothing else in
// these kernels reads it (it feeds only LDS-DMA, GWS and message
// instructions), so the asm need not preserve it.
__device__ __forceinline__ void dma_b128(const uint8_t* base, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(lds), "v"(voff), "s"(base)
                 : "memory");
}

// LDS byte address of a pointer into __shared__ memory
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const lds_void*)p;
}

// lds_wave: LDS byte address of this wave's quarter of the destination tile
// (uniform); base: the tile's first row (tile0 of the key range). kFull: the
// caller knows the tile lies inside Lk (every tile but the range's last).
template <class Fmt, bool kFull = false>
__device__ __forceinline__ void load_tile_at(const uint8_t* __restrict__ base, uint32_t lds_wave, int tile0, int Lk,
                                             size_t row_bytes, const TileLoad<Fmt>& tl, int hd, int wave, int lane) {
    if (kFull || tile0 + kTK <= Lk) {
#pragma unroll
        for (int i = 0; i < Fmt::kLoads; ++i) dma_b128(base, tl.off[i], lds_wave + i * 1024);
    } else {
        const int last = Lk - 1 - tile0;
#pragma unroll
        for (int i = 0; i < Fmt::kLoads; ++i) {
            int r, lc;
            tile_chunk<Fmt>(wave, lane, i, r, lc);
            const uint32_t off = (uint32_t)(min(r, last) * (int)row_bytes + hd * (Fmt::kChunks * 16) + lc * 16);
            dma_b128(base, off, lds_wave + i * 1024);
        }
    }
}
template <class Fmt>
__device__ __forceinline__ void load_tile_lds(const uint8_t* __restrict__ src, uint32_t lds_wave, int tile0, int Lk,
                                              size_t row_bytes, const TileLoad<Fmt>& tl, int hd, int wave, int lane) {
    load_tile_at<Fmt>(src + (size_t)tile0 * row_bytes, lds_wave, tile0, Lk, row_bytes, tl, hd, wave, lane);
}

// Workgroup barrier with no memory fence. __syncthreads() would also drain
// every direct global -> LDS load still in flight (they count as LDS writes);
// the pipeline orders those itself with per-lane vmcnt waits before the
// barrier. The empty asm statements keep the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void wg_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}


// kFp8: q and k hold fp8 e4m3 values and Q K^T runs on the fp8 matrix cores
// (v_mfma_f32_32x32x64_f8f6f4, two per 32-key tile); v, o and P V stay bf16.
template <bool kBias, bool kFp8>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(AttentionArgs a, BiasGeom g, float c_log2, KeySplit ks) {
    // Three-slot ring: slot t mod 3 holds K_t in its first half and V_{t-1}
    // in its second. Step j refills slot j mod 3 (K_{j+3}, V_{j+2}) while it
    // reads slot j + 1 mod 3 (K_{j+1}, V_j); separate arrays let the compiler
    // see that those reads never touch the loads still landing.
    __shared__ __attribute__((aligned(1024))) uint8_t lds_r0[2 * kTileBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_r1[2 * kTileBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_r2[2 * kTileBytes];
    auto ring = [&](auto slot_tag) -> uint8_t* {
        constexpr int i = decltype(slot_tag)::value % kStages;
        if constexpr (i == 0) return lds_r0;
        else if constexpr (i == 1) return lds_r1;
        else return lds_r2;
    };
    __shared__ int lds_slot[kBias ? kMaxFramesLds : 1];        // KV frame -> retrieved frame (or -1)
    // key operands by column (first contraction half, [0]) and by row (second half, [1])
    __shared__ u32x4 lds_tab[2][kBias ? kMaxGridSide : 1];
    __shared__ float2 lds_corr[kBias ? kCorrLds : 1][128];      // centred u^ per (retrieved frame, query)

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int hh = lane >> 5;
    const int n = lane & 31;
    // Work unit = (head, key part, 128-query tile), in that order of
    // significance, so that the workgroups running together on one XCD read
    // the same keys and values; each XCD takes a contiguous range of units.
    const int n_qt = (a.Lq + 127) / 128;
    const int Lk = a.Lk;
    const int n_tiles = (Lk + kTK - 1) / kTK;
    const unsigned n_units = (unsigned)(n_qt * a.H * ks.parts);
    const unsigned unit = xcd_item(blockIdx.x, n_units);
    if (unit >= n_units) return;  // grid padding (uniform, before any barrier)
    const int qt = (int)(unit % (unsigned)n_qt);
    const int hp = (int)(unit / (unsigned)n_qt);
    const int hd = hp / ks.parts;
    const int kp = hp - hd * ks.parts;
    const int t0 = (int)((int64_t)kp * n_tiles / ks.parts);
    const int nt = (int)((int64_t)(kp + 1) * n_tiles / ks.parts) - t0;
    const int H = a.H;
    using KFmt = std::conditional_t<kFp8, RowsFp8, RowsBf16>;
    const uint8_t* Qg = static_cast<const uint8_t*>(a.q);
    const uint8_t* Kg = static_cast<const uint8_t*>(a.k);
    const uint8_t* Vg = static_cast<const uint8_t*>(a.v);
    const size_t row_stride = (size_t)H * kD;              // elements between consecutive tokens (o)
    const size_t qk_row_bytes = row_stride * (kFp8 ? 1 : 2);
    const size_t v_row_bytes = row_stride * 2;
    using R0 = std::integral_constant<int, 0>;
    using R1 = std::integral_constant<int, 1>;
    using R2 = std::integral_constant<int, 2>;
    // this wave's quarter of the K tile of a ring slot, and of its V tile (kTileBytes further)
    const uint32_t wave_off_k = (uint32_t)__builtin_amdgcn_readfirstlane(wave * KFmt::kLoads * 1024);
    const uint32_t wave_off_v = (uint32_t)__builtin_amdgcn_readfirstlane(wave * kLoadsPerLane * 1024);
    auto kdst = [&](auto slot_tag) -> uint32_t { return lds_addr(ring(slot_tag)) + wave_off_k; };
    auto vdst = [&](auto slot_tag) -> uint32_t { return lds_addr(ring(slot_tag)) + kTileBytes + wave_off_v; };

    // LDS byte offsets (within a tile) of this lane's operand reads
    const int krow = perm_row(n);
    // bf16: eight 16-byte reads per tile, kk -> d 16 kk + 8 hh ..; fp8: two 32-byte
    // operands per tile, kk -> d 64 kk + 32 hh .., each two 16-byte reads
    constexpr int kKReads = kFp8 ? 4 : 8;
    int koff[kKReads];
#pragma unroll
    for (int i = 0; i < kKReads; ++i) {
        if constexpr (kFp8) koff[i] = krow * 128 + (((4 * (i >> 1) + 2 * hh + (i & 1)) ^ RowsFp8::swizzle(krow)) << 4);
        else koff[i] = krow * kRowBytes + (((2 * i + hh) ^ swz(krow)) << 4);
    }
    // V transpose reads: lane t of 16-lane group G reads row 8 hh + t / 4 (+4 for the
    // second half) at columns 32 db + 16 (G % 2) + 4 (t % 4) .. +3
    const int t16 = lane & 15;
    const int grp = lane >> 4;
    const int vrow0 = 8 * hh + (t16 >> 2);
    const int vcc = 2 * (grp & 1) + ((t16 >> 1) & 1);
    const int vbyte = 8 * (t16 & 1);
    int voff[2][4];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
        for (int db = 0; db < 4; ++db) {
            const int r = vrow0 + 4 * half;
            voff[half][db] = r * kRowBytes + (((4 * db + vcc) ^ swz(r)) << 4) + vbyte;
        }
    }

    // ---- bias state -------------------------------------------------------
    const int n_frames = Lk / g.hw;
    const uint32_t one_bf = 0x3f80u;
    // the slot table's loads are issued here and stored to LDS after the
    // query and correspondence loads have been issued too
    constexpr int kSlotsPerThread = kBias ? kMaxFramesLds / 256 : 1;
    int slot_v[kSlotsPerThread];
    if (kBias) {
#pragma unroll
        for (int i = 0; i < kSlotsPerThread; ++i) {
            const int f = tid + 256 * i;
            slot_v[i] = f < n_frames ? a.slot[f] : -1;
        }
        for (int i = tid; i < g.w + g.h; i += 256) {
            const bool col = i < g.w;
            const int k = col ? i : i - g.w;
            const float ac = ((float)k + 0.5f) - (col ? g.cx : g.cy);
            const uint32_t a2 = bf16_bits_rne(2.0f * ac);
            uint32_t ph, pm, pl;
            split3(-g.gamma * (ac * ac), ph, pm, pl);
            const u32x4 v = u32x4{pack2(a2, a2), pack2(a2, ph), pack2(pm, pl), col ? pack2(one_bf, one_bf) : one_bf};
            lds_tab[col ? 0 : 1][k] = v;
        }
    }
    const float inv_w = 1.0f / (float)g.w;

    const int q = qt * 128 + wave * 32 + n;
    const bool q_ok = q < a.Lq;

    // start streaming the first tiles: K_0, V_0, K_1, V_1, K_2 of the key
    // part, everything its first step expects in place. With fewer tiles the missing
    // ones repeat the last tile (never read; loading them anyway keeps these
    // loads free of branches).
    const TileLoad<KFmt> tlk = make_tile_load<KFmt>(qk_row_bytes, hd, wave, lane);
    const TileLoad<RowsBf16> tlv = make_tile_load<RowsBf16>(v_row_bytes, hd, wave, lane);
    const int tile0 = t0 * kTK, tile1 = (t0 + min(1, nt - 1)) * kTK, tile2 = (t0 + min(2, nt - 1)) * kTK;
    load_tile_lds(Kg, kdst(R0{}), tile0, Lk, qk_row_bytes, tlk, hd, wave, lane);
    load_tile_lds(Vg, vdst(R1{}), tile0, Lk, v_row_bytes, tlv, hd, wave, lane);
    load_tile_lds(Kg, kdst(R1{}), tile1, Lk, qk_row_bytes, tlk, hd, wave, lane);
    load_tile_lds(Vg, vdst(R2{}), tile1, Lk, v_row_bytes, tlv, hd, wave, lane);
    load_tile_lds(Kg, kdst(R2{}), tile2, Lk, qk_row_bytes, tlk, hd, wave, lane);
    // the loads of the steps: K_{j+3} and V_{j+2} at step j, through pointers
    // that advance one tile per step (no per-step 64-bit multiply)
    const size_t k_stride = (size_t)kTK * qk_row_bytes, v_stride = (size_t)kTK * v_row_bytes;
    const uint8_t* k_load = Kg + (size_t)(t0 + 3) * k_stride;
    const uint8_t* v_load = Vg + (size_t)(t0 + 2) * v_stride;

    // Q fragments: lane (hh, n) holds Q[q][16 kk + 8 hh .. +8)
    // (fp8: lane (hh, n) holds Q[q][64 kk + 32 hh .. +32), kk = 0, 1)
    constexpr int kQFrags = kFp8 ? 2 : 8;
    using QFrag = std::conditional_t<kFp8, int8v, bf16x8>;
    QFrag qf[kQFrags];
#pragma unroll
    for (int kk = 0; kk < kQFrags; ++kk) {
        if constexpr (kFp8) {
            u32x4 v0 = u32x4{0, 0, 0, 0}, v1 = u32x4{0, 0, 0, 0};
            if (q_ok) {
                const uint8_t* qp = Qg + (size_t)q * qk_row_bytes + (size_t)hd * kD + 64 * kk + 32 * hh;
                v0 = *reinterpret_cast<const u32x4*>(qp);
                v1 = *reinterpret_cast<const u32x4*>(qp + 16);
            }
            qf[kk] = int8v{(int)v0[0], (int)v0[1], (int)v0[2], (int)v0[3], (int)v1[0], (int)v1[1], (int)v1[2], (int)v1[3]};
        } else {
            u32x4 v = u32x4{0, 0, 0, 0};
            if (q_ok) v = *reinterpret_cast<const u32x4*>(Qg + ((size_t)q * row_stride + (size_t)hd * kD + 16 * kk + 8 * hh) * 2);
            qf[kk] = as_bf16x8(v);
        }
    }

    // Correspondences of the 128 queries for the first kCorrLds
    // retrieved frames, staged into LDS (centred u^, NaN = rejected), so that
    // no global load sits in the key loop; frames beyond load on demand.
    // Every load is issued before any is used, so the staging waits for one
    // memory latency rather than two per entry.
    if (kBias) {
        const int n_s = min(a.S, kCorrLds);
        constexpr int kPerThread = kCorrLds * 128 / 256;
        int cidx[kPerThread];
        float2 cuv[kPerThread];
#pragma unroll
        for (int i = 0; i < kPerThread; ++i) {
            const int e = tid + 256 * i;
            const int s = e >> 7, qq = qt * 128 + (e & 127);
            cidx[i] = -1;
            cuv[i] = make_float2(0.0f, 0.0f);
            if (s < n_s && qq < a.Lq) {
                const size_t o = (size_t)s * a.Lq + qq;
                cidx[i] = a.corr_idx[o];
                cuv[i] = reinterpret_cast<const float2*>(a.corr_uv)[o];
            }
        }
#pragma unroll
        for (int i = 0; i < kSlotsPerThread; ++i) {
            const int f = tid + 256 * i;
            if (f < n_frames) lds_slot[f] = (slot_v[i] >= 0 && slot_v[i] < a.S) ? slot_v[i] : -1;
        }
#pragma unroll
        for (int i = 0; i < kPerThread; ++i) {
            const int e = tid + 256 * i;
            const int s = e >> 7;
            if (s < n_s)
                lds_corr[s][e & 127] = cidx[i] >= 0 ? make_float2(cuv[i].x - g.cx, cuv[i].y - g.cy) : make_float2(NAN, NAN);
        }
    }
    // query-side bias operand of retrieved frame s for this lane's query
    auto query_operand = [&](int s) -> bf16x8 {
        float ux = NAN, uy = NAN;
        if (s < kCorrLds) {
            const float2 v = lds_corr[s][wave * 32 + n];
            ux = v.x;
            uy = v.y;
        } else if (q_ok) {
            const size_t o = (size_t)s * a.Lq + q;
            if (a.corr_idx[o] >= 0) {
                const float2 u = reinterpret_cast<const float2*>(a.corr_uv)[o];
                ux = u.x - g.cx;
                uy = u.y - g.cy;
            }
        }
        u32x4 v = u32x4{0, 0, 0, 0};
        if (!__builtin_isnan(ux)) {
            uint32_t xh, xm, xl, yh, ym, yl, zh, zm, zl;
            split3(g.gamma * ux, xh, xm, xl);
            split3(g.gamma * uy, yh, ym, yl);
            split3(-g.gamma * (ux * ux + uy * uy), zh, zm, zl);
            if (hh == 0) v = u32x4{pack2(xh, xm), pack2(xl, one_bf), pack2(one_bf, one_bf), pack2(zh, zm)};
            else v = u32x4{pack2(yh, ym), pack2(yl, one_bf), pack2(one_bf, one_bf), zl};
        }
        return as_bf16x8(v);
    };
    // query operand of the frame the last fast-path tile lay in (zeros for an unbiased frame)
    bf16x8 qcur = as_bf16x8(u32x4{0, 0, 0, 0});
    // slot of the frame the last fast-path tile lay in (uniform): looked up again only when the frame changes
    int scur_f = -1, scur = -1;
    // frame and in-frame offset of the next QK tile's first key (uniform)
    int blk_f = tile0 / g.hw, blk_t = tile0 - blk_f * g.hw;
    // this lane's key operand for in-frame key position t (< hw)
    auto key_operand = [&](int t) -> u32x4 {
        const int ky = (int)(((float)t + 0.5f) * inv_w);
        const int kx = t - ky * g.w;
        return lds_tab[hh][hh ? ky : kx];
    };

    // Bias of the QK tile starting at key k0, added to its logits after the
    // QK MFMAs, in two parts. bias_classify runs at the start of a step, so
    // that the key operand read from LDS lands while the QK MFMAs run: it
    // returns 1 for a tile inside one retrieved frame (the fast path; kop then
    // holds the lane's key operand), 0 for a tile inside a frame that is not
    // retrieved (no bias) and -1 for a tile that crosses a frame boundary or
    // Lk. bias_add then issues one MFMA for a fast-path tile and none for an
    // unbiased one: a uniform branch costs less than an MFMA of zeros, whose
    // energy counts, as the chip runs this kernel at its power limit. The
    // frame's slot and query operand are looked up again only when the frame
    // changes. A crossing tile adds one masked MFMA per retrieved frame it
    // touches.
    auto bias_classify = [&](auto inside_tag, int k0, u32x4& kop) -> int {
        constexpr bool kInside = decltype(inside_tag)::value;  // the tile is known to lie inside Lk
        const bool inside = kInside || k0 + 31 < Lk;
        if (__builtin_expect(inside && blk_t + 31 < g.hw, 1)) {
            if (__builtin_expect(scur_f != blk_f, 0)) {
                scur = __builtin_amdgcn_readfirstlane(lds_slot[blk_f]);
                scur_f = blk_f;
                qcur = scur >= 0 ? query_operand(scur) : as_bf16x8(u32x4{0, 0, 0, 0});
            }
            if (scur < 0) return 0;  // frame not retrieved: no bias
            kop = key_operand(blk_t + krow);
            return 1;
        }
        return -1;
    };
    // Adds the bias of the QK tile starting at key k0 to acc, its logits.
    auto bias_add = [&](floatx16 init, int k0, int cls, const u32x4& kop) -> floatx16 {
        // the fast path's MFMA; a crossing tile adds its frames instead
        if (cls > 0) init = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kop), qcur, init, 0, 0, 0);
        if (__builtin_expect(cls < 0, 0)) {
            const int span = min(31, Lk - 1 - k0);
            int lane_t = blk_t + krow, lane_f = blk_f;
            while (lane_t >= g.hw) {
                lane_t -= g.hw;
                ++lane_f;
            }
            const bool row_live = krow <= span;
            for (int f = blk_f, fs = -blk_t; fs <= span && f < n_frames; ++f, fs += g.hw) {
                const int s = __builtin_amdgcn_readfirstlane(lds_slot[f]);
                if (s < 0) continue;
                const bf16x8 qv = query_operand(s);
                u32x4 kv = u32x4{0, 0, 0, 0};
                if (row_live && lane_f == f) kv = key_operand(lane_t);
                init = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv), qv, init, 0, 0, 0);
            }
        }
        blk_t += 32;
        if (__builtin_expect(blk_t >= g.hw, 0)) {
            do {
                blk_t -= g.hw;
                ++blk_f;
            } while (blk_t >= g.hw);
        }
        return init;
    };

    // QK^T of one 32-key tile from LDS (buffer kt) into S, then its bias
    auto qk_tile = [&](const uint8_t* kt, int k0, floatx16& S) {
        u32x4 kop = u32x4{0, 0, 0, 0};
        int cls = 0;
        if constexpr (kBias) cls = bias_classify(std::false_type{}, k0, kop);
        S = floatx16{0};
#pragma unroll
        for (int kk = 0; kk < kQFrags; ++kk) {
            if constexpr (kFp8) {
                const u32x4 k0 = *reinterpret_cast<const u32x4*>(kt + koff[2 * kk]);
                const u32x4 k1 = *reinterpret_cast<const u32x4*>(kt + koff[2 * kk + 1]);
                S = mfma_fp8(join8(k0, k1), qf[kk], S);
            } else {
                const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4*>(kt + koff[kk]));
                S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], S, 0, 0, 0);
            }
        }
        if constexpr (kBias) S = bias_add(S, k0, cls, kop);
    };
    // mask keys past Lk (only the last tile can hold any) and reduce this lane's maximum
    auto tile_max = [&](auto mask_tag, floatx16& S, int k0) -> float {
        if constexpr (decltype(mask_tag)::value) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                if (k0 + 16 * (i >> 3) + 8 * hh + (i & 7) >= Lk) S[i] = -INFINITY;
            }
        }
        float m = fmaxf(S[0], S[1]);
#pragma unroll
        for (int i = 2; i < 16; i += 2) m = max3(m, S[i], S[i + 1]);
        return m;
    };

    floatx16 O[4];
#pragma unroll
    for (int db = 0; db < 4; ++db) O[db] = floatx16{0};
    float m_run = -INFINITY, l_run0 = 0.0f, l_run1 = 0.0f;
    // a raw logit above this calls for a rescale: (m_run + kRescaleSlack) / c_log2,
    // so the check needs neither the row's other half nor the scale
    float m_thr = -INFINITY;
    const uint32_t ones2 = 0x3f803f80u;  // bf16 (1, 1)
    using True = std::integral_constant<bool, true>;
    using False = std::integral_constant<bool, false>;

    floatx16 Sa, Sb;
    float mx_cur;

    // One pipeline step for tile j. After the barrier, K_{j+3} and V_{j+2} are
    // loaded into ring slot j mod 3, which held K_j and V_{j-1} (no wave reads
    // those any more), then softmax + PV of tile j (logits in S_cur) run while
    // the logits of tile j + 1 are computed into S_next.
    // P = j mod 6 fixes the ring slots and which of Sa / Sb is current at
    // compile time. Kinds by the tiles left (d = n_tiles - j): 0 = d >= 4,
    // 1 = d = 3, 2 = d = 2 (tile j + 1 is the last), 3 = d = 1 (tile j is the last).
    // Loads issued in step j - 1 may stay in flight: each lane waits only for
    // those of step j - 2, which carried K_{j+1} and V_j.
    // The body takes the ring slots (knext: the slot holding K_{j+1} and V_j;
    // refill: the LDS address of slot j mod 3) and the logit buffers as
    // arguments: compile-time in the steady loop, chosen at run time in the
    // last few steps.
    auto step_core = [&](auto kind_tag, int j, floatx16& S_cur, floatx16& S_next, const uint8_t* knext,
                         const uint32_t refill) __attribute__((always_inline)) {
        // kind 4: a step of the steady loop (kind 0 whose tiles j + 1 .. j + 3
        // all lie inside Lk and are not the range's last)
        constexpr bool kSteady = decltype(kind_tag)::value == 4;
        constexpr int kind = kSteady ? 0 : decltype(kind_tag)::value;
        constexpr bool has_next = kind != 3;
        const uint8_t* vcur = knext + kTileBytes;
        // this lane's loads issued in step j - 1: K_{j+2} if it exists, V_{j+1} if it exists
        if constexpr (kind <= 1) {
            __builtin_amdgcn_s_waitcnt(kWaitVm0 + KFmt::kLoads + kLoadsPerLane);
        } else if constexpr (kind == 2) {
            __builtin_amdgcn_s_waitcnt(kWaitVm0 + kLoadsPerLane);
        } else {
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
        }
        wg_barrier();
        // the K_{j+1} operands of the first QK MFMAs first (the chain waits on them),
        // then the refill of slot j mod 3 (it has two steps to land)
        const int nk0 = (t0 + j + 1) * kTK;
        auto kread = [&](int i) -> u32x4 { return *reinterpret_cast<const u32x4*>(knext + koff[i]); };
        u32x4 kf[kKReads];
        if constexpr (has_next) {
            kf[0] = kread(0);
            kf[1] = kread(1);
            kf[2] = kread(2);
        }
        if constexpr (kind == 0) {
            load_tile_at<KFmt, kSteady>(k_load, refill + wave_off_k, (t0 + j + 3) * kTK, Lk, qk_row_bytes, tlk, hd, wave,
                                        lane);
            k_load += k_stride;
        }
        if constexpr (kind <= 1) {
            load_tile_at<RowsBf16, kSteady>(v_load, refill + kTileBytes + wave_off_v, (t0 + j + 2) * kTK, Lk, v_row_bytes,
                                            tlv, hd, wave, lane);
            v_load += v_stride;
        }

        // the bias of tile j + 1 is added after its QK MFMAs, so its key
        // operand read has the whole QK chain to land
        u32x4 bias_kop = u32x4{0, 0, 0, 0};
        int bias_cls = 0;
        if constexpr (kBias && has_next) bias_cls = bias_classify(std::integral_constant<bool, kSteady>{}, nk0, bias_kop);

        // lazy rescale: tested on each lane's half of the row maximum of tile j
        // (reduced during the previous step); the whole row's maximum only when needed
        if (__builtin_expect(__any(mx_cur > m_thr), 0)) {
            const float mx = half_swap_max(mx_cur) * c_log2;
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            l_run0 *= alpha;
            l_run1 *= alpha;
#pragma unroll
            for (int db = 0; db < 4; ++db) O[db] *= alpha;
            m_run = m_new;
            m_thr = (m_run + kRescaleSlack) / c_log2;
        }
        if constexpr (has_next) S_next = floatx16{0};

        // The rest of the step is scheduled by hand: every chunk below ends in
        // a scheduling fence. Matrix-core and VALU work are grouped rather
        // than paired within a wave, so that the other wave of the SIMD can
        // run its VALU work beside this wave's MFMAs and the other way round.
        // softmax unit (t, e): probabilities of logits 8 t + 2 e and 8 t + 2 e + 1
        // of tile j, packed to bf16 and added to the running sums
        uint32_t w4[2][4];
        auto unit = [&](int t, int e) {
            const float p0 = __builtin_amdgcn_exp2f(fmaf(S_cur[8 * t + 2 * e], c_log2, -m_run));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(S_cur[8 * t + 2 * e + 1], c_log2, -m_run));
            w4[t][e] = cvt_pk_bf16(p0, p1);
            float& l = (e & 1) ? l_run1 : l_run0;
            l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w4[t][e]), __builtin_bit_cast(bf16x2, ones2),
                                                l, false);
        };
        // V_j operand of the PV MFMA (key half t, head dims 32 db ..): two transposing reads
        shortx4 vlo[2][4], vhi[2][4];
        auto vread = [&](int t, int db) {
            const uint8_t* vt = vcur + 16 * t * kRowBytes;
            vlo[t][db] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(vt + voff[0][db]));
            vhi[t][db] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_shortx4*)(vt + voff[1][db]));
        };
        auto voperand = [&](int t, int db) -> bf16x8 {
            const shortx4 lo = vlo[t][db], hi = vhi[t][db];
            u32x4 w;
            w[0] = __builtin_bit_cast(uint32_t, (short __attribute__((ext_vector_type(2)))){lo[0], lo[1]});
            w[1] = __builtin_bit_cast(uint32_t, (short __attribute__((ext_vector_type(2)))){lo[2], lo[3]});
            w[2] = __builtin_bit_cast(uint32_t, (short __attribute__((ext_vector_type(2)))){hi[0], hi[1]});
            w[3] = __builtin_bit_cast(uint32_t, (short __attribute__((ext_vector_type(2)))){hi[2], hi[3]});
            return as_bf16x8(w);
        };
        __builtin_amdgcn_sched_barrier(0);

        float mx_next = -INFINITY;
        if constexpr (kBias) {
            // Region A: the QK MFMAs of tile j + 1 (K operands read ahead) and the
            // V reads of key half 0, then the bias of tile j + 1, then softmax
            // units (0, 0..3) and (1, 0..1) of tile j. No softmax work sits
            // between the QK MFMAs: with two waves on each SIMD the other wave's
            // VALU work runs beside this wave's MFMA chain, and this order
            // measured faster than pairing each QK MFMA with a softmax unit.
            if constexpr (kFp8) {
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    if constexpr (has_next) {
                        if (kk == 0) kf[3] = kread(3);
                        S_next = mfma_fp8(join8(kf[2 * kk], kf[2 * kk + 1]), qf[kk], S_next);
                    }
                    if (kk == 1) {
#pragma unroll
                        for (int db = 0; db < 4; ++db) vread(0, db);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else {
#pragma unroll
                for (int kk = 0; kk < 8; ++kk) {
                    if constexpr (has_next) {
                        if (kk + 3 < 8) kf[kk + 3] = kread(kk + 3);
                        S_next = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[kk]), qf[kk], S_next, 0, 0, 0);
                    }
                    if (kk >= 4) vread(0, kk - 4);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            if constexpr (has_next) {
                S_next = bias_add(S_next, nk0, bias_cls, bias_kop);
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int u = 0; u < 6; ++u) unit(u >> 2, u & 3);
            __builtin_amdgcn_sched_barrier(0);
            // keep the row sums of these units here (otherwise they sink to the
            // start of the next step, where they serialise behind the bias MFMA)
            asm volatile("" ::"v"(l_run0), "v"(l_run1));
            const bf16x8 pf0 = as_bf16x8(u32x4{w4[0][0], w4[0][1], w4[0][2], w4[0][3]});

            // region B1: PV of key half 0, softmax units (1, 2..3), V reads of key half 1
#pragma unroll
            for (int db = 0; db < 4; ++db) {
                O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(voperand(0, db), pf0, O[db], 0, 0, 0);
                if (db < 2) unit(1, 2 + db);
                vread(1, db);
                __builtin_amdgcn_sched_barrier(0);
            }
            asm volatile("" ::"v"(l_run0), "v"(l_run1));
            const bf16x8 pf1 = as_bf16x8(u32x4{w4[1][0], w4[1][1], w4[1][2], w4[1][3]});

            // region B2: PV of key half 1, row maximum of tile j + 1 (keys past Lk
            // masked when tile j + 1 is the last)
#pragma unroll
            for (int db = 0; db < 4; ++db) {
                O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(voperand(1, db), pf1, O[db], 0, 0, 0);
                if constexpr (has_next) {
#pragma unroll
                    for (int i = 4 * db; i < 4 * db + 4; ++i) {
                        if constexpr (kind == 2) {
                            if (nk0 + 16 * (i >> 3) + 8 * hh + (i & 7) >= Lk) S_next[i] = -INFINITY;
                        }
                    }
                    // v_max3 only (fmaxf would add canonicalising maxes of its operands)
                    if (db == 0) mx_next = max3(max3(S_next[0], S_next[1], S_next[2]), S_next[3], S_next[3]);
                    else mx_next = max3(mx_next, max3(S_next[4 * db], S_next[4 * db + 1], S_next[4 * db + 2]), S_next[4 * db + 3]);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        } else {
            // Without the bias each step is one VALU block and one matrix-core
            // block: the V reads of key half 0 and all softmax units of tile
            // j, then P V of tile j (V reads of key half 1 under key half 0)
            // and Q K^T of tile j + 1 (K operands read ahead), then its row
            // maximum. The two waves of a SIMD then alternate between the
            // blocks; this measured faster without the bias (+0.1-2.8% bf16,
            // +4% fp8) and slower with it, whose step keeps the order above.
#pragma unroll
            for (int db = 0; db < 4; ++db) vread(0, db);
#pragma unroll
            for (int u = 0; u < 8; ++u) unit(u >> 2, u & 3);
            __builtin_amdgcn_sched_barrier(0);
            const bf16x8 pf0 = as_bf16x8(u32x4{w4[0][0], w4[0][1], w4[0][2], w4[0][3]});
            const bf16x8 pf1 = as_bf16x8(u32x4{w4[1][0], w4[1][1], w4[1][2], w4[1][3]});
#pragma unroll
            for (int db = 0; db < 4; ++db) {
                O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(voperand(0, db), pf0, O[db], 0, 0, 0);
                vread(1, db);
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int db = 0; db < 4; ++db) {
                O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(voperand(1, db), pf1, O[db], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (kFp8) {
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    if constexpr (has_next) {
                        if (kk == 0) kf[3] = kread(3);
                        S_next = mfma_fp8(join8(kf[2 * kk], kf[2 * kk + 1]), qf[kk], S_next);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else {
#pragma unroll
                for (int kk = 0; kk < 8; ++kk) {
                    if constexpr (has_next) {
                        if (kk + 3 < 8) kf[kk + 3] = kread(kk + 3);
                        S_next = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[kk]), qf[kk], S_next, 0, 0, 0);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            // row maximum of tile j + 1 (keys past Lk masked when it is the last)
            if constexpr (has_next) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    if constexpr (kind == 2) {
                        if (nk0 + 16 * (i >> 3) + 8 * hh + (i & 7) >= Lk) S_next[i] = -INFINITY;
                    }
                }
                mx_next = max3(max3(S_next[0], S_next[1], S_next[2]), S_next[3], S_next[3]);
#pragma unroll
                for (int db = 1; db < 4; ++db)
                    mx_next = max3(mx_next, max3(S_next[4 * db], S_next[4 * db + 1], S_next[4 * db + 2]), S_next[4 * db + 3]);
            }
        }
        mx_cur = mx_next;
    };
    auto step = [&](auto phase_tag, auto kind_tag, int j) __attribute__((always_inline)) {
        constexpr int P = decltype(phase_tag)::value;
        step_core(kind_tag, j, (P & 1) ? Sb : Sa, (P & 1) ? Sa : Sb, ring(std::integral_constant<int, P + 1>{}),
                  lds_addr(ring(std::integral_constant<int, P>{})));
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    using I4 = std::integral_constant<int, 4>;
    using I5 = std::integral_constant<int, 5>;

    // prologue: logits of tile 0
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
    qk_tile(ring(R0{}), tile0, Sa);
    mx_cur = t0 + 1 == n_tiles ? tile_max(True{}, Sa, tile0) : tile_max(False{}, Sa, tile0);

    // steady state in periods of six tiles, while each of them has at least
    // three more after it
    int j = 0;
    for (; j + 9 <= nt; j += 6) {
        step(I0{}, I4{}, j);
        step(I1{}, I4{}, j + 1);
        step(I2{}, I4{}, j + 2);
        step(I3{}, I4{}, j + 3);
        step(I4{}, I4{}, j + 4);
        step(I5{}, I4{}, j + 5);
    }
    // the last 1 .. 8 tiles: one copy of the step body per kind, ring slot
    // chosen at run time. The steady loop leaves off at a multiple of six, so
    // step j refills slot 0 and the logits of tile j are in Sa; after each
    // step the logits of tile j + 1 move from Sb to Sa.
    auto slot_base = [&](int slot) -> const uint8_t* { return slot == 0 ? lds_r0 : (slot == 1 ? lds_r1 : lds_r2); };
    int slot = 0;
    auto tail_step = [&](auto kind_tag) __attribute__((always_inline)) {
        const int nxt = slot == 2 ? 0 : slot + 1;
        step_core(kind_tag, j, Sa, Sb, slot_base(nxt), lds_addr(slot_base(slot)));
        if constexpr (decltype(kind_tag)::value != 3) Sa = Sb;
        slot = nxt;
        ++j;
    };
    while (nt - j > 3) tail_step(I0{});
    if (nt - j == 3) tail_step(I1{});
    if (nt - j == 2) tail_step(I2{});
    tail_step(I3{});

    const float l_tot = half_swap_sum(l_run0 + l_run1);
    if (t0 == 0 && nt == n_tiles) {
        // the whole key range: normalise and store
        const float inv = 1.0f / l_tot;
        if (q_ok) {
            uint16_t* Og = static_cast<uint16_t*>(a.o) + (size_t)q * row_stride + (size_t)hd * kD;
#pragma unroll
            for (int db = 0; db < 4; ++db) {
#pragma unroll
                for (int gi = 0; gi < 4; ++gi) {
                    const int d = 32 * db + 8 * gi + 4 * hh;
                    const uint32_t w0 = cvt_pk_bf16(O[db][4 * gi] * inv, O[db][4 * gi + 1] * inv);
                    const uint32_t w1 = cvt_pk_bf16(O[db][4 * gi + 2] * inv, O[db][4 * gi + 3] * inv);
                    *reinterpret_cast<uint2*>(Og + d) = make_uint2(w0, w1);
                }
            }
            if (a.lse && hh == 0) a.lse[(size_t)hd * a.Lq + q] = (m_run + log2f(l_tot)) * kLn2;
        }
    } else {
        // one part of the key range: unnormalised O with its running max and
        // sum, merged by attn_merge_kernel
        float* part = ks.part + ((size_t)(hd * n_qt + qt) * ks.parts + kp) * kPartFloats;
        const int qi = wave * 32 + n;
#pragma unroll
        for (int db = 0; db < 4; ++db) {
#pragma unroll
            for (int gi = 0; gi < 4; ++gi) {
                const int d = 32 * db + 8 * gi + 4 * hh;
                *reinterpret_cast<float4*>(part + qi * kD + d) =
                    make_float4(O[db][4 * gi], O[db][4 * gi + 1], O[db][4 * gi + 2], O[db][4 * gi + 3]);
            }
        }
        if (hh == 0) {
            part[128 * kD + qi] = m_run;
            part[128 * kD + 128 + qi] = l_tot;
        }
    }
}

BiasGeom make_geom(const AttentionArgs& a) {
    BiasGeom g;
    g.gamma = a.lambda / (2.0f * a.sigma * a.sigma * a.softmax_scale);
    g.cx = 0.5f * (float)a.w;
    g.cy = 0.5f * (float)a.h;
    g.hw = a.h * a.w;
    g.w = a.w;
    g.h = a.h;
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

namespace {

// O = sum_p 2^(m_p - M) O_p / sum_p 2^(m_p - M) l_p over the key parts p of
// an item, M = max_p m_p (logits in log2 units). A workgroup merges 8 queries
// of one item: thread t takes query t / 32 and head dims 4 (t % 32) .. +3, so
// that each wave reads two whole 512-byte partial rows per load.
constexpr int kMergeQueries = 8;
constexpr int kMergeBatch = 8;  // parts merged from registers loaded up front

__global__ __launch_bounds__(256) void attn_merge_kernel(AttentionArgs a, KeySplit ks) {
    const int n_qt = (a.Lq + 127) / 128;
    const int item = blockIdx.x / (128 / kMergeQueries);
    const int qi = (blockIdx.x % (128 / kMergeQueries)) * kMergeQueries + (threadIdx.x >> 5);
    const int d = 4 * (threadIdx.x & 31);
    const int hd = item / n_qt;
    const int q = (item - hd * n_qt) * 128 + qi;
    if (q >= a.Lq) return;
    const float* base = ks.part + (size_t)item * ks.parts * kPartFloats;
    float M = -INFINITY;
    float L = 0.0f;
    float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    auto add = [&](float m, float l, float4 v) {
        const float c = __builtin_amdgcn_exp2f(m - M);
        L = fmaf(c, l, L);
        acc = make_float4(fmaf(c, v.x, acc.x), fmaf(c, v.y, acc.y), fmaf(c, v.z, acc.z), fmaf(c, v.w, acc.w));
    };
    if (ks.parts <= kMergeBatch) {
        // every part's loads issued before any is used: one memory latency,
        // not two per part
        float m[kMergeBatch], l[kMergeBatch];
        float4 v[kMergeBatch];
#pragma unroll
        for (int p = 0; p < kMergeBatch; ++p) {
            if (p < ks.parts) {
                const float* P = base + (size_t)p * kPartFloats;
                m[p] = P[128 * kD + qi];
                l[p] = P[128 * kD + 128 + qi];
                v[p] = *reinterpret_cast<const float4*>(P + qi * kD + d);
            }
        }
#pragma unroll
        for (int p = 0; p < kMergeBatch; ++p) {
            if (p < ks.parts) M = fmaxf(M, m[p]);
        }
#pragma unroll
        for (int p = 0; p < kMergeBatch; ++p) {
            if (p < ks.parts) add(m[p], l[p], v[p]);
        }
    } else {
        for (int p = 0; p < ks.parts; ++p) M = fmaxf(M, base[(size_t)p * kPartFloats + 128 * kD + qi]);
        for (int p = 0; p < ks.parts; ++p) {
            const float* P = base + (size_t)p * kPartFloats;
            add(P[128 * kD + qi], P[128 * kD + 128 + qi], *reinterpret_cast<const float4*>(P + qi * kD + d));
        }
    }
    const float inv = 1.0f / L;
    uint16_t* Og = static_cast<uint16_t*>(a.o) + (size_t)q * a.H * kD + (size_t)hd * kD + d;
    *reinterpret_cast<uint2*>(Og) = make_uint2(cvt_pk_bf16(acc.x * inv, acc.y * inv), cvt_pk_bf16(acc.z * inv, acc.w * inv));
    if (a.lse && d == 0) a.lse[(size_t)hd * a.Lq + q] = (M + log2f(L)) * kLn2;
}

}  // namespace

int32_t attention_bf16_key_parts(const AttentionArgs& a, int32_t slots) {
    // Smallest number of key parts (at most kMaxParts, each of at least
    // kMinTiles key tiles) whose workgroups fill the last round of `slots`
    // resident workgroups to 97 % or more. When none does: one part if the
    // items alone make four rounds or more (the tail is then short), else the
    // most parts allowed. Every part costs a prologue, a 66 KB partial write
    // and its share of the merge, so past four parts the better-filled last
    // round no longer pays: with 444 items on 512 slots, 4 parts measured
    // 2-5 % faster than 8 (filled) and than 1.
    constexpr int kMinTiles = 128, kMaxParts = 4;
    const int64_t items = (int64_t)((a.Lq + 127) / 128) * a.H;
    const int n_tiles = (a.Lk + kTK - 1) / kTK;
    int largest = 1;
    for (int p = 1; p <= kMaxParts && (p == 1 || n_tiles / p >= kMinTiles); ++p) {
        const int64_t units = items * p;
        const int64_t rounds = (units + slots - 1) / slots;
        if ((double)units >= 0.97 * (double)(rounds * slots)) return p;
        largest = p;
    }
    return items >= 4 * (int64_t)slots ? 1 : largest;
}

size_t attention_bf16_workspace_bytes(const AttentionArgs& a, int32_t parts) {
    if (parts <= 1) return 0;
    const int64_t items = (int64_t)((a.Lq + 127) / 128) * a.H;
    return (size_t)items * parts * kPartFloats * sizeof(float);
}

// The key split's partial results for biased_chunk_attention_noalloc. Each
// device holds its own copy of this array; host code never passes the name
// itself to a kernel (on the host it is only a stand-in): it passes the
// device address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) float scratch[kAttentionScratchBytes / sizeof(float)];

namespace {
// The device address of the array on each device, looked up on the first call
// there and kept in a fixed table, so that the lookup allocates nothing. Two
// threads that look it up at once store the same address.
constexpr int kScratchDevices = 64;
std::atomic<float*> g_scratch_ptr[kScratchDevices];  // by device; nullptr = not looked up yet
}  // namespace

hipError_t attention_scratch(float** ptr) {
    *ptr = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
    float* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        void* addr = nullptr;
        e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        p = static_cast<float*>(addr);
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return hipSuccess;
}

hipError_t launch_attention_bf16(const AttentionArgs& a, int32_t parts, float* workspace, hipStream_t stream) {
    if (a.Lq == 0) return hipSuccess;
    const BiasGeom g = make_geom(a);
    const bool bias_on = a.S > 0 && a.lambda != 0.0f;
    const unsigned items = (unsigned)(((a.Lq + 127) / 128) * a.H);
    const KeySplit ks{parts, workspace};
    const dim3 grid(xcd_grid(items * (unsigned)parts)), block(256);
    const float c_log2 = a.softmax_scale * kLog2e;
    if (a.fp8_qk) {
        if (bias_on) hipLaunchKernelGGL((attn_bf16_kernel<true, true>), grid, block, 0, stream, a, g, c_log2, ks);
        else hipLaunchKernelGGL((attn_bf16_kernel<false, true>), grid, block, 0, stream, a, g, c_log2, ks);
    } else {
        if (bias_on) hipLaunchKernelGGL((attn_bf16_kernel<true, false>), grid, block, 0, stream, a, g, c_log2, ks);
        else hipLaunchKernelGGL((attn_bf16_kernel<false, false>), grid, block, 0, stream, a, g, c_log2, ks);
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && parts > 1) {
        hipLaunchKernelGGL(attn_merge_kernel, dim3(items * (128 / kMergeQueries)), block, 0, stream, a, ks);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace revisit
