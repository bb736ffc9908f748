// Device-side helpers shared by the HIP kernels (gfx950).
#pragma once

#include <cfloat>
#include <cmath>
#include <cstdint>

#include "kernels.h"

namespace mgi {
namespace kern {

typedef float f4 __attribute__((ext_vector_type(4)));

// Activation as one clamp (v_med3_f32): [lo, hi] = (-inf, inf) for none,
// (0, inf) for ReLU, (0, 6) for ReLU6; act is uniform, so lo and hi are
// computed once per kernel.
__device__ __forceinline__ float act_apply(float v, int act) {
    const float lo = act == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = act == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    return __builtin_amdgcn_fmed3f(v, lo, hi);
}

__device__ __forceinline__ h8 zero_h8() {
    h8 z;
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = (_Float16)0.0f;
    return z;
}

// q = x / d, r = x % d for 0 <= x < 2^31, 1 <= d, from a host-computed
// reciprocal inv = 1.0 / d: the double product is within one of the
// quotient, and one correction step makes it exact.
__device__ __forceinline__ void divmod_fast(int x, int d, double inv, int &q, int &r) {
    q = (int)((double)x * inv);
    r = x - q * d;
    if (r < 0) {
        --q;
        r += d;
    } else if (r >= d) {
        ++q;
        r -= d;
    }
}

// Workgroups are dispatched to the 8 XCDs round-robin (block b -> XCD b % 8).
// Give every XCD a contiguous range of tiles so that tiles sharing input rows
// (same pixel block, neighbouring channel blocks) meet in the same L2.
__device__ __forceinline__ int xcd_tile(int bid, int nblocks) {
    const int xcd = bid & 7, idx = bid >> 3;
    const int per = nblocks >> 3, rem = nblocks & 7;
    return xcd * per + min(xcd, rem) + idx;
}

// v_fma_mix_f32: fp32 acc += fp16 a * fp16 b, both halves taken from the same
// position (low or high) of a packed pair; the product of two fp16 values is
// exact in fp32, so this equals fmaf((float)a, (float)b, acc) with no
// conversion instructions.
template <int HI>
__device__ __forceinline__ void fma_mix(float &acc, uint32_t a, uint32_t b) {
    if (HI)
        asm volatile("v_fma_mix_f32 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,1,0]"
                     : "+v"(acc) : "v"(a), "v"(b));
    else
        asm volatile("v_fma_mix_f32 %0, %1, %2, %0 op_sel:[0,0,0] op_sel_hi:[1,1,0]"
                     : "+v"(acc) : "v"(a), "v"(b));
}

// the same with a separate addend: out = a * b + c (the first tap of an
// output takes its bias this way, so no register copy initialises it)
template <int HI>
__device__ __forceinline__ float fma_mix_from(uint32_t a, uint32_t b, float c) {
    float out;
    if (HI)
        asm volatile("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[1,1,0] op_sel_hi:[1,1,0]"
                     : "=v"(out) : "v"(a), "v"(b), "v"(c));
    else
        asm volatile("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[0,0,0] op_sel_hi:[1,1,0]"
                     : "=v"(out) : "v"(a), "v"(b), "v"(c));
    return out;
}

typedef uint32_t u4x __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u4x as_u4(h8 v) { return __builtin_bit_cast(u4x, v); }

// whole-wave lane shift of a 16-byte value: kWaveShr1 gives lane l the value
// of lane l-1, kWaveShl1 that of lane l+1; the lane with no source gets zero
// (DPP bound control)
constexpr int kWaveShl1 = 0x130, kWaveShr1 = 0x138;
template <int CTRL>
__device__ __forceinline__ h8 wave_shift(h8 v) {
    const u4x u = as_u4(v);
    u4x r;
#pragma unroll
    for (int d = 0; d < 4; ++d) r[d] = (uint32_t)__builtin_amdgcn_mov_dpp((int)u[d], CTRL, 0xf, 0xf, true);
    return __builtin_bit_cast(h8, r);
}

// acc[0..7] += w * v channel-wise, w and v fp16 x 8
__device__ __forceinline__ void fma8(float *acc, u4x w, u4x v) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        fma_mix<0>(acc[2 * d], w[d], v[d]);
        fma_mix<1>(acc[2 * d + 1], w[d], v[d]);
    }
}

// acc[0..7] = w * v + c0 channel-wise
__device__ __forceinline__ void fma8_from(float *acc, const float *c0, u4x w, u4x v) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        acc[2 * d] = fma_mix_from<0>(w[d], v[d], c0[2 * d]);
        acc[2 * d + 1] = fma_mix_from<1>(w[d], v[d], c0[2 * d + 1]);
    }
}

// Storage element traits.  Activations and weights are stored as 16-bit
// floats, 8 per 16-byte element, either fp16 or bf16 (mgi_options.dtype);
// kernels move elements as raw 16-byte values and only convert at these
// points.  Products of two 16-bit values are exact in fp32 for both types.
typedef __bf16 bh8 __attribute__((ext_vector_type(8)));
typedef __bf16 bh4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

struct F16 {
    static constexpr bool bf = false;
    __device__ static float get(h8 v, int i) { return (float)v[i]; }
    __device__ static h8 pack(const float *v) {
        h8 o;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = (_Float16)v[i];
        return o;
    }
    __device__ static f4 mma(h8 a, h8 b, f4 c) { return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0); }
    __device__ static void fma8(float *acc, h8 w, h8 v) { kern::fma8(acc, as_u4(w), as_u4(v)); }
    __device__ static void fma8_from(float *acc, const float *c0, h8 w, h8 v) {
        kern::fma8_from(acc, c0, as_u4(w), as_u4(v));
    }
    __device__ static float get4(h4 v, int i) { return (float)v[i]; }
    __device__ static h4 pack4(const float *v) {
        h4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (_Float16)v[i];
        return o;
    }
    __device__ static uint16_t bits(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
};

struct BF16 {
    static constexpr bool bf = true;
    __device__ static float get(h8 v, int i) {
        return __uint_as_float((uint32_t)__builtin_bit_cast(u16x8, v)[i] << 16);
    }
    __device__ static h8 pack(const float *v) {
        bh8 o;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = (__bf16)v[i];
        return __builtin_bit_cast(h8, o);
    }
    __device__ static f4 mma(h8 a, h8 b, f4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bh8, a), __builtin_bit_cast(bh8, b), c,
                                                      0, 0, 0);
    }
    __device__ static void fma8(float *acc, h8 w, h8 v) {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(get(w, i), get(v, i), acc[i]);
    }
    __device__ static void fma8_from(float *acc, const float *c0, h8 w, h8 v) {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(get(w, i), get(v, i), c0[i]);
    }
    __device__ static float get4(h4 v, int i) {
        return __uint_as_float((uint32_t)__builtin_bit_cast(u16x4, v)[i] << 16);
    }
    __device__ static h4 pack4(const float *v) {
        bh4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (__bf16)v[i];
        return __builtin_bit_cast(h4, o);
    }
    __device__ static uint16_t bits(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
};

// 16 bytes per lane from global memory straight into LDS: lane l writes
// lds + 16*l, so the LDS side is one contiguous KiB per wave.  Issued as
// inline asm so that the compiler does not track it: it would otherwise
// conservatively wait for every such load before any LDS read it cannot
// prove independent (at loop heads it cannot), serialising the ring.  The
// loads are ordered by explicit s_waitcnt + s_barrier instead.
__device__ __forceinline__ void load_lds16(const h8 *src, const h8 *lds) {
    const unsigned la = (unsigned)(size_t)(__attribute__((address_space(3))) const void *)lds;
    asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(la) : "memory");
}

// wait until at most N vector-memory instructions of this wave are in flight
// and all of its LDS reads have returned (expcnt left at its maximum)
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4));
}

// ---------------------------------------------------------------------------
// Input band of a convolution over an NHWC graph input: rows [iy0, iy0 +
// nrows) of image n, row r of the band at band + r * rs (16-bit storage
// values, the data from column lead on).  The padding cells (rows outside
// the image, columns before and after the data) are zeroed, then the rows
// are copied with each thread loading NV units (16-byte vectors, or single
// elements when rows are not 16-byte aligned) before storing any, so that a
// workgroup's loads are in flight together.  A thread's place in a row is
// found with one division; rows shorter than the workgroup are copied
// several per pass.  The caller synchronises before reading the band.
// ---------------------------------------------------------------------------
template <typename E, typename TIN, int NT, int NV>
__device__ __forceinline__ void stage_input_band(_Float16 *band, const TIN *x, int n, int H, int W, int C,
                                                 int iy0, int nrows, int rs, int lead, int tid) {
    constexpr int VEC = 16 / sizeof(TIN);
    typedef TIN tv __attribute__((ext_vector_type(VEC)));
    const int rowlen = W * C;
    const int r_lo = max(0, -iy0), r_hi = min(nrows, H - iy0);   // band rows inside the image
    const TIN *src0 = x + ((size_t)n * H + iy0) * rowlen;
    const bool vec = (rowlen % 8) == 0 && (lead % 8) == 0 && (rs % 8) == 0;
    const int upr = vec ? rowlen / VEC : rowlen;                  // load units per row
    uint16_t *b16 = (uint16_t *)band;
    const int tail = rs - lead - rowlen;                         // zero columns after the data
    for (int r = 0; r < nrows; ++r) {
        if (r >= r_lo && r < r_hi) {
            for (int c = tid; c < lead + tail; c += NT) b16[r * rs + (c < lead ? c : rowlen + c)] = 0;
        } else {
            for (int c = tid; c < rs; c += NT) b16[r * rs + c] = 0;
        }
    }
    auto copy_unit = [&](int r, int c, const tv &v, TIN e) {
        if (vec) {
            _Float16 *dst = band + r * rs + lead + c * VEC;
            float f[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) f[i] = (float)v[i];
            if (VEC == 8 && !E::bf) *(tv *)dst = v;                  // fp16 input, fp16 storage
            else if (VEC == 8) *(h8 *)dst = E::pack(f);
            else *(h4 *)dst = E::pack4(f);
        } else {
            b16[r * rs + lead + c] = E::bits((float)e);
        }
    };
    tv bv[NV];
    TIN bs[NV];
    if (upr <= NT) {
        const int P = NT / upr;                                   // rows per pass
        const int rq = tid / upr, cq = tid - rq * upr;
        const int npass = (r_hi - r_lo + P - 1) / P;
        for (int p0 = 0; p0 < npass; p0 += NV) {
#pragma unroll
            for (int u = 0; u < NV; ++u) {
                const int r = r_lo + (p0 + u) * P + rq;
                if (rq < P && r < r_hi) {
                    if (vec) bv[u] = *(const tv *)(src0 + (size_t)r * rowlen + cq * VEC);
                    else bs[u] = src0[(size_t)r * rowlen + cq];
                }
            }
#pragma unroll
            for (int u = 0; u < NV; ++u) {
                const int r = r_lo + (p0 + u) * P + rq;
                if (rq < P && r < r_hi) copy_unit(r, cq, bv[u], bs[u]);
            }
        }
    } else {
        for (int r = r_lo; r < r_hi; ++r) {                       // rows longer than the workgroup
            for (int c0 = 0; c0 < upr; c0 += NT * NV) {
#pragma unroll
                for (int u = 0; u < NV; ++u) {
                    const int c = c0 + u * NT + tid;
                    if (c < upr) {
                        if (vec) bv[u] = *(const tv *)(src0 + (size_t)r * rowlen + c * VEC);
                        else bs[u] = src0[(size_t)r * rowlen + c];
                    }
                }
#pragma unroll
                for (int u = 0; u < NV; ++u) {
                    const int c = c0 + u * NT + tid;
                    if (c < upr) copy_unit(r, c, bv[u], bs[u]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Coalesced epilogue.  An MFMA accumulator gives a lane 4 channels of one
// pixel (half of a 16-byte sliced element, the other half in lane l+16);
// storing that directly makes every quarter-wave write half-masked 64-byte
// pieces, which costs several times the bandwidth of whole lines.  Instead
// each wave parks act1(acc) (the accumulators include the bias) in its own LDS tile
// [2*FN slices][16*FM pixels][8] fp32, then re-reads it so that consecutive
// lanes own consecutive pixels of one slice: residual reads and output writes
// are whole 16-byte elements, 1 KiB per wave instruction.  No barrier: a wave
// reads back only what it wrote.
// ---------------------------------------------------------------------------
// mlim: pixels at or past it are not stored (default: p.M).
// Bias of the four channels a lane holds in a 16x16 accumulator tile of
// output block nb (blocks past the last are clamped: never stored).  Every
// pointwise GEMM kernel starts its accumulators from this value, so the bias
// enters the sum first, in the same place in every kernel.
__device__ __forceinline__ f4 bias_frag(const float *bias, int nb, int nb16, int lane) {
    const float *b = bias + min(nb, nb16 - 1) * 16 + 4 * (lane >> 4);
    return f4{b[0], b[1], b[2], b[3]};
}

// accumulators (bias included) -> act1 -> (+ residual -> act2) -> sliced store
template <typename E, int FM, int FN>
__device__ __forceinline__ void store_tile_c8(const GemmParams &p, const f4 (&acc)[FN][FM], int m0,
                                              int nb0, float *stage, int lane, int mlim = -1) {
    constexpr int NPIX = 16 * FM, NSL = 2 * FN;
    const int lim = mlim < 0 ? p.M : mlim;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const int sl = 2 * i + ((lane >> 4) >> 1), half = 4 * ((lane >> 4) & 1);
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            f4 v;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r], p.act1);
            *(f4 *)(stage + ((sl * NPIX) + j * 16 + (lane & 15)) * 8 + half) = v;
        }
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int t = 0; t < (NSL * NPIX + 63) / 64; ++t) {
        const int e = lane + 64 * t;
        if ((NSL * NPIX) % 64 != 0 && e >= NSL * NPIX) break;   // a single 16x16 block: half a wave
        const int sl = e / NPIX, px = e - sl * NPIX;
        const int os = nb0 * 2 + sl, m = m0 + px;
        if (os >= p.ns || m >= lim) continue;
        const f4 lo = *(const f4 *)(stage + e * 8), hi = *(const f4 *)(stage + e * 8 + 4);
        float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        const size_t off = (size_t)os * p.M + m;
        if (p.res) {
            const h8 rv = p.res[off];
#pragma unroll
            for (int r = 0; r < 8; ++r) v[r] = act_apply(v[r] + E::get(rv, r), p.act2);
        }
        ((h8 *)p.y)[off] = E::pack(v);
    }
}

// Softmax of one fp32 row of `cols` values by one wave: up to 1024 columns
// are held in registers (16 per lane, all loads issued at once; columns past
// the end repeat the last one, which leaves the max unchanged and is kept out
// of the sum), longer rows take a looped path; max and sum reduce by a fixed
// butterfly.  The standalone softmax kernel and the FC kernel's fused softmax
// both use it, so the two forms round alike.  softmax_load / softmax_finish
// are its two halves for rows of at most kSoftmaxRegCols columns (a caller
// may load several rows before finishing any).
constexpr int kSoftmaxPer = 16, kSoftmaxRegCols = 64 * kSoftmaxPer;
__device__ inline void softmax_load(const float *zr, int cols, int lane, float (&v)[kSoftmaxPer]) {
#pragma unroll
    for (int i = 0; i < kSoftmaxPer; ++i) v[i] = zr[min(lane + 64 * i, cols - 1)];
}
__device__ inline void softmax_finish(float (&v)[kSoftmaxPer], float *yr, int cols, int lane) {
    constexpr int PER = kSoftmaxPer;
    float m = -FLT_MAX;
#pragma unroll
    for (int i = 0; i < PER; ++i) m = fmaxf(m, v[i]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        v[i] = expf(v[i] - m);
        s += lane + 64 * i < cols ? v[i] : 0.0f;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    const float inv = 1.0f / s;
#pragma unroll
    for (int i = 0; i < PER; ++i)
        if (lane + 64 * i < cols) yr[lane + 64 * i] = v[i] * inv;
}
__device__ inline void softmax_row(const float *zr, float *yr, int cols, int lane) {
    if (cols <= kSoftmaxRegCols) {
        float v[kSoftmaxPer];
        softmax_load(zr, cols, lane, v);
        softmax_finish(v, yr, cols, lane);
        return;
    }
    float m = -FLT_MAX;
    for (int j = lane; j < cols; j += 64) m = fmaxf(m, zr[j]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
    float s = 0.0f;
    for (int j = lane; j < cols; j += 64) {
        const float e = expf(zr[j] - m);
        yr[j] = e;
        s += e;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    const float inv = 1.0f / s;
    for (int j = lane; j < cols; j += 64) yr[j] *= inv;
}

}  // namespace kern
}  // namespace mgi
