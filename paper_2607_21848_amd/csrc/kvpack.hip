// Cache packing of retrieved chunks (Sec. 4.2, cache layout and cache
// packing): the keys and values of each selected historical chunk are copied
// from the history store into its slot of the attention cache, and the keys'
// temporal rotary embedding is turned from the chunk's stored frame position
// to the packed one, next to the recent window.
//
// The work is a stream: every byte is read once and written once, so the
// kernel is bound by HBM and is laid out for it. One 256-thread block moves
// 16 KiB of one (layer, slot, K or V) chunk image: four 16-byte vectors per
// thread, block-strided so that every load and store instruction covers 4 KiB
// of consecutive bytes, all four loads in flight before the first use (more
// per thread, or larger blocks, measured slower).
// Loads and stores are non-temporal: neither side is reused by this kernel,
// and the store is far larger than the caches.
//
// Keys: a 16-byte vector never straddles a head row (D % 8 == 0), so its
// position in the row tells which of its element pairs belong to the temporal
// band (pair index < n_t). Those pairs are rotated by delta * omega_i,
// omega_i = theta^(-i / n_t), delta = packed frame position minus stored one
// (the same for the whole chunk), in double precision in the order
// x c - y s, x s + y c with contraction off, then rounded once to the storage
// type. For bf16 the single rounding is done as round-to-odd into fp32
// followed by round-to-nearest-even into bf16, which equals rounding the
// double directly (fp32 keeps 16 more bits than bf16, in the normal and the
// subnormal range). cos and sin of the slot's angles come from a table in
// LDS that the block computes while its loads are in flight. All other key
// elements and every value are copied bit for bit.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

#pragma clang fp contract(off)

namespace revisit {
namespace {

constexpr int kBlock = 256;
constexpr int kVecsPerThread = 4;
constexpr int kSpan = kBlock * kVecsPerThread;  // 16-byte vectors per block
constexpr int kMaxPairs = 256;                  // D <= 512

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// double -> bf16 bits, one rounding to nearest even (see the header comment)
__device__ __forceinline__ uint32_t bf16_rne(double x) {
    const float t = __double2float_rz(x);
    uint32_t u = __float_as_uint(t);
    if ((double)t != x) u |= 1u;  // round to odd: inexact truncations get a set last bit (NaN stays NaN)
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;  // quiet NaN
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ double bf16_val(uint32_t bits16) { return (double)__uint_as_float(bits16 << 16); }

struct Rot {
    double c, s;
};

// rotate the (x, y) pair
__device__ __forceinline__ void turn(double x, double y, const Rot r, double& xo, double& yo) {
    xo = x * r.c - y * r.s;
    yo = x * r.s + y * r.c;
}

template <int ESIZE>
__global__ __launch_bounds__(kBlock) void kvpack_kernel(KvPackArgs a, int32_t parts) {
    __shared__ Rot table[kMaxPairs];
    const int tid = threadIdx.x;
    const int part = blockIdx.x % parts;
    const int unit = blockIdx.x / parts;  // ((layer * n_sel + slot) * 2 + kv)
    const int kv = unit & 1;
    const int ls = unit >> 1;
    const int slot = ls % a.n_sel;
    const int layer = ls / a.n_sel;
    const int j = a.sel[slot];
    if (j < 0 || j >= a.n_store) return;  // empty slot: left as it is (uniform exit)

    const int64_t row_elems = (int64_t)a.H * a.D;
    const int64_t chunk_elems = (int64_t)a.T * row_elems;
    const int64_t chunk_vecs = chunk_elems * ESIZE / 16;
    const uint8_t* src = static_cast<const uint8_t*>(kv ? a.store_v : a.store_k) +
                         ((int64_t)layer * a.n_store + j) * chunk_elems * ESIZE;
    uint8_t* dst = static_cast<uint8_t*>(kv ? a.cache_v : a.cache_k) +
                   ((int64_t)layer * a.cache_rows + a.dst_row0 + (int64_t)slot * a.T) * row_elems * ESIZE;
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    u32x4* d4 = reinterpret_cast<u32x4*>(dst);

    const int64_t v0 = (int64_t)part * kSpan + tid;
    u32x4 buf[kVecsPerThread];
#pragma unroll
    for (int i = 0; i < kVecsPerThread; ++i) {
        const int64_t v = v0 + (int64_t)i * kBlock;
        buf[i] = v < chunk_vecs ? __builtin_nontemporal_load(s4 + v) : u32x4{0, 0, 0, 0};
    }

    const bool rotate = kv == 0 && a.n_t > 0;
    if (rotate) {  // uniform per block
        if (tid < a.n_t) {
            const int64_t pos_j = a.store_pos ? (int64_t)a.store_pos[j] : (int64_t)a.F * j;
            const int64_t delta = (int64_t)a.dst_pos + (int64_t)slot * a.F - pos_j;
            const double omega = pow(a.theta, -((double)tid / (double)a.n_t));
            const double phi = (double)delta * omega;
            table[tid] = Rot{cos(phi), sin(phi)};
        }
        __syncthreads();
        // vectors per head row, and the first pair index of this thread's first vector
        constexpr int kPairsPerVec = 8 / ESIZE;
        const int row_vecs = a.D * ESIZE / 16;
        int m = (int)(v0 % row_vecs);
        const int m_step = kBlock % row_vecs;
#pragma unroll
        for (int i = 0; i < kVecsPerThread; ++i) {
            const int p0 = m * kPairsPerVec;
            if (p0 < a.n_t) {
                u32x4& w = buf[i];
                if constexpr (ESIZE == 2) {
                    // four bf16 pairs, one per 32-bit word: (low half, high half) = (x, y)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        if (p0 + q < a.n_t) {
                            double xo, yo;
                            turn(bf16_val(w[q] & 0xffffu), bf16_val(w[q] >> 16), table[p0 + q], xo, yo);
                            w[q] = bf16_rne(xo) | (bf16_rne(yo) << 16);
                        }
                    }
                } else {
                    // two fp32 pairs: words (0, 1) and (2, 3)
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        if (p0 + q < a.n_t) {
                            double xo, yo;
                            turn((double)__uint_as_float(w[2 * q]), (double)__uint_as_float(w[2 * q + 1]),
                                 table[p0 + q], xo, yo);
                            w[2 * q] = __float_as_uint(__double2float_rn(xo));
                            w[2 * q + 1] = __float_as_uint(__double2float_rn(yo));
                        }
                    }
                }
            }
            m += m_step;
            if (m >= row_vecs) m -= row_vecs;
        }
    }

#pragma unroll
    for (int i = 0; i < kVecsPerThread; ++i) {
        const int64_t v = v0 + (int64_t)i * kBlock;
        if (v < chunk_vecs) __builtin_nontemporal_store(buf[i], d4 + v);
    }
}

int64_t parts_per_chunk(const KvPackArgs& a) {
    const int64_t chunk_vecs = (int64_t)a.T * a.H * a.D * a.esize / 16;
    return (chunk_vecs + kSpan - 1) / kSpan;
}

}  // namespace

int64_t kvpack_blocks(const KvPackArgs& a) { return (int64_t)a.n_layers * a.n_sel * 2 * parts_per_chunk(a); }

hipError_t launch_kvpack(const KvPackArgs& a, hipStream_t stream) {
    if (a.n_layers == 0 || a.n_sel == 0 || a.T == 0) return hipSuccess;
    const int32_t parts = (int32_t)parts_per_chunk(a);  // the caller keeps kvpack_blocks(a) below 2^31
    const dim3 grid((unsigned)kvpack_blocks(a)), block(kBlock);
    if (a.esize == 2) {
        hipLaunchKernelGGL(kvpack_kernel<2>, grid, block, 0, stream, a, parts);
    } else {
        hipLaunchKernelGGL(kvpack_kernel<4>, grid, block, 0, stream, a, parts);
    }
    return hipGetLastError();
}

}  // namespace revisit
