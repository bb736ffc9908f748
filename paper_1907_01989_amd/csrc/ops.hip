// Bandwidth-bound kernels on the sliced (C8) layout: depthwise convolution,
// element-wise add / activation, global average pool, softmax, concat,
// bilinear resize (optionally fused with the per-pixel argmax), argmax, and
// the conversions between NHWC graph I/O and the sliced layout.
//
// Thread order follows the paper's observation (Sec. 4.1) that neighbouring
// threads should read neighbouring cache lines: consecutive lanes take
// consecutive pixels of one 8-channel slice, so a wave's 16-byte loads cover
// 1 KiB of contiguous memory.
#include <cfloat>
#include <cmath>
#include <cstdint>

#include "device.h"

namespace mgi {
namespace kern {

static inline unsigned blocks_for(size_t n, int per) { return (unsigned)((n + per - 1) / per); }

LaunchEvents &launch_events() {
    static thread_local LaunchEvents ev;
    return ev;
}

// ---------------------------------------------------------------------------
// Depthwise 3x3 convolution, column strips.  A thread owns one output column
// of one 8-channel slice of one image and R consecutive output rows: it reads
// the (R-1)*S + 2*D + 1 input rows of its three input columns once (16 bytes
// each), and every input value feeds all the outputs whose window covers it,
// accumulating in fp32 with fp16 taps (exact products).  Consecutive lanes
// take consecutive columns, so each load instruction of a wave covers a
// contiguous run of one row.  Taps outside the input read a zeroed 16-byte
// element instead of branching, so all loads are issued unconditionally.
// Launch: 1-D, thread g -> column g % OW, strip (g / OW) % nstrips, plane
// g / (OW * nstrips) (plane = slice * N + image); the divisions are
// reciprocal products with one correction step (divmod_fast), a few
// instructions instead of an integer division sequence each.
// ---------------------------------------------------------------------------
template <typename E, int S_, int D_, int R>
__global__ __launch_bounds__(256) void dw3_kernel(DwParams p, int nstrips, DivConsts dc) {
    constexpr int NR = (R - 1) * S_ + 2 * D_ + 1;
    const int g = blockIdx.x * 256 + threadIdx.x;
    int rest, ox, plane, strip, s, img;
    divmod_fast(g, p.OW, dc.inv_ow, rest, ox);
    divmod_fast(rest, nstrips, dc.inv_nstrips, plane, strip);
    if (plane >= p.S * p.N) return;
    divmod_fast(plane, p.N, dc.inv_n, s, img);
    (void)img;
    const int oy0 = strip * R;
    const h8 *xin = p.x + (size_t)plane * p.H * p.W;
    const h8 *wp = p.w + (size_t)s * 9;
    h8 w[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) w[t] = wp[t];
    const int iy0 = oy0 * S_ - p.pt, ix0 = ox * S_ - p.pl;
    int cx[3];
    bool cv[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        cx[k] = ix0 + k * D_;
        cv[k] = cx[k] >= 0 && cx[k] < p.W;
    }
    h8 v[NR][3];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int iy = iy0 + r;
        const bool rv = iy >= 0 && iy < p.H;
#pragma unroll
        for (int k = 0; k < 3; ++k)
            v[r][k] = *((rv && cv[k]) ? xin + (size_t)iy * p.W + cx[k] : p.zero);
    }
    // accumulation per output: bias, then taps ky = 0..2, kx = 0..2 (the
    // first tap takes the bias as its addend)
    float bias[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) bias[c] = p.bias[s * 8 + c];
    float acc[R][8];
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int ky = 0; ky < 3; ++ky) {
            const int t = r - ky * D_;
            if (t >= 0 && t % S_ == 0 && t / S_ < R) {
#pragma unroll
                for (int k = 0; k < 3; ++k) {
                    if (ky == 0 && k == 0) E::fma8_from(acc[t / S_], bias, w[0], v[r][0]);
                    else E::fma8(acc[t / S_], w[ky * 3 + k], v[r][k]);
                }
            }
        }
    // activation as one clamp: [lo, hi] = (-inf, inf), (0, inf) or (0, 6)
    const float lo = p.act == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    h8 *yout = p.y + (size_t)plane * p.OH * p.OW + ox;
#pragma unroll
    for (int o = 0; o < R; ++o) {
        if (oy0 + o >= p.OH) break;
        float q[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) q[c] = __builtin_amdgcn_fmed3f(acc[o][c], lo, hi);
        yout[(size_t)(oy0 + o) * p.OW] = E::pack(q);
    }
}

// Any window size: one thread per output pixel of one slice, fp32
// accumulation over the kh x kw window.
template <typename E>
__global__ __launch_bounds__(256) void dw_kernel(DwParams p, int tpp) {
    const int plane = blockIdx.x / tpp;
    const int pix = (blockIdx.x - plane * tpp) * 256 + threadIdx.x;
    const int ohw = p.OH * p.OW;
    if (pix >= ohw) return;
    const int s = plane / p.N;
    const int oy = pix / p.OW, ox = pix - oy * p.OW;
    const h8 *xin = p.x + (size_t)plane * p.H * p.W;
    const h8 *wt = p.w + (size_t)s * p.KH * p.KW;
    float acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = p.bias[s * 8 + c];
    for (int ky = 0; ky < p.KH; ++ky) {
        const int iy = oy * p.sh + ky * p.dh - p.pt;
        if (iy < 0 || iy >= p.H) continue;
        for (int kx = 0; kx < p.KW; ++kx) {
            const int ix = ox * p.sw + kx * p.dw - p.pl;
            if (ix < 0 || ix >= p.W) continue;
            const h8 v = xin[(size_t)iy * p.W + ix];
            const h8 wk = wt[ky * p.KW + kx];
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[c] = fmaf(E::get(wk, c), E::get(v, c), acc[c]);
        }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = act_apply(acc[c], p.act);
    p.y[(size_t)plane * ohw + pix] = E::pack(acc);
}

template <typename E, int S_, int D_, int R>
static hipError_t launch_dw3(const DwParams &p, hipStream_t st) {
    const int nstrips = (p.OH + R - 1) / R;
    const size_t threads = (size_t)p.OW * nstrips * p.S * p.N;
    if (threads > 0x7fffffffull) return hipErrorInvalidValue;
    const DivConsts dc{1.0 / p.OW, 1.0 / nstrips, 1.0 / p.N};
    launch((dw3_kernel<E, S_, D_, R>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st,
           p, nstrips, dc);
    return hipGetLastError();
}

hipError_t launch_depthwise(const DwParams &p, int rows, hipStream_t st) {
    const int ohw = p.OH * p.OW;
    if (ohw <= 0 || p.N <= 0 || p.S <= 0) return hipSuccess;
    if (p.KH == 3 && p.KW == 3 && p.sh == p.sw && p.dh == p.dw) {
        // output rows per thread: 4 at stride 1, 2 at stride 2 unless chosen
        const int R = rows > 0 ? rows : (p.sh == 1 ? 4 : 2);
#define MGI_DW_CASE(S_, D_, R_) \
        if (p.sh == S_ && p.dh == D_ && R == R_) \
            return p.bf16 ? launch_dw3<BF16, S_, D_, R_>(p, st) : launch_dw3<F16, S_, D_, R_>(p, st);
        MGI_DW_CASE(1, 1, 2) MGI_DW_CASE(1, 1, 4) MGI_DW_CASE(1, 1, 8)
        MGI_DW_CASE(2, 1, 1) MGI_DW_CASE(2, 1, 2) MGI_DW_CASE(2, 1, 4)
        MGI_DW_CASE(1, 2, 2) MGI_DW_CASE(1, 2, 4) MGI_DW_CASE(1, 2, 8)
        MGI_DW_CASE(2, 2, 1) MGI_DW_CASE(2, 2, 2) MGI_DW_CASE(2, 2, 4)
#undef MGI_DW_CASE
        if (rows > 0) return hipErrorInvalidValue;
    }
    const int tpp = (ohw + 255) / 256;
    const size_t nblk = (size_t)tpp * p.S * p.N;
    if (nblk > 0x7fffffffu) return hipErrorInvalidValue;
    if (p.bf16) launch(dw_kernel<BF16>, dim3((unsigned)nblk), dim3(256), 0, st, p, tpp);
    else launch(dw_kernel<F16>, dim3((unsigned)nblk), dim3(256), 0, st, p, tpp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Spatial zero padding of a sliced tensor (a PAD that could not be merged into
// a convolution): one thread per output element of 16 bytes.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pad_kernel(const h8 *x, h8 *y, int N, int H, int W, int OH,
                                                  int OW, int pt, int pl, size_t total) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const size_t plane = i / ((size_t)OH * OW);
    const int r = (int)(i - plane * OH * OW);
    const int oy = r / OW, ox = r - oy * OW;
    const int iy = oy - pt, ix = ox - pl;
    h8 v;
    if (iy >= 0 && iy < H && ix >= 0 && ix < W) {
        v = x[(plane * H + iy) * W + ix];
    } else {
#pragma unroll
        for (int c = 0; c < 8; ++c) v[c] = (_Float16)0.0f;
    }
    y[i] = v;
}

hipError_t launch_pad(const h8 *x, h8 *y, int N, int S, int H, int W, int OH, int OW, int pt, int pl,
                      hipStream_t st) {
    const size_t total = (size_t)S * N * OH * OW;
    if (!total) return hipSuccess;
    launch(pad_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, st, x, y, N, H, W, OH, OW, pt, pl,
           total);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// element-wise
// ---------------------------------------------------------------------------
template <typename E>
__global__ __launch_bounds__(256) void add_kernel(const h8 *a, const h8 *b, h8 *y, size_t n, int act) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const h8 u = a[i], v = b[i];
    float o[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) o[c] = act_apply(E::get(u, c) + E::get(v, c), act);
    y[i] = E::pack(o);
}

hipError_t launch_add(const h8 *a, const h8 *b, h8 *y, size_t count, int act, bool bf16, hipStream_t st) {
    if (!count) return hipSuccess;
    if (bf16) launch(add_kernel<BF16>, dim3(blocks_for(count, 256)), dim3(256), 0, st, a, b, y, count, act);
    else launch(add_kernel<F16>, dim3(blocks_for(count, 256)), dim3(256), 0, st, a, b, y, count, act);
    return hipGetLastError();
}

template <typename E>
__global__ __launch_bounds__(256) void act_kernel(const h8 *x, h8 *y, size_t n, int act) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const h8 u = x[i];
    float o[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) o[c] = act_apply(E::get(u, c), act);
    y[i] = E::pack(o);
}

hipError_t launch_act(const h8 *x, h8 *y, size_t count, int act, bool bf16, hipStream_t st) {
    if (!count) return hipSuccess;
    if (bf16) launch(act_kernel<BF16>, dim3(blocks_for(count, 256)), dim3(256), 0, st, x, y, count, act);
    else launch(act_kernel<F16>, dim3(blocks_for(count, 256)), dim3(256), 0, st, x, y, count, act);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void zero_words_kernel(unsigned *p, size_t n) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = 0u;
}

hipError_t launch_zero_words(unsigned *dst, size_t words, hipStream_t st) {
    if (!words) return hipSuccess;
    launch(zero_words_kernel, dim3(blocks_for(words, 256)), dim3(256), 0, st, dst, words);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// global average pool: one 256-thread workgroup per (slice, image); thread t
// sums pixels t, t + 256, ... four loads at a time (all issued before any
// add; pixels past the end read the zero element), then a fixed butterfly in
// each wave and the four wave sums in a fixed order (deterministic).  Output
// is the sliced (n, 1, 1, c) tensor in the storage type.
// ---------------------------------------------------------------------------
template <typename E>
__global__ __launch_bounds__(256) void gap_kernel(const h8 *x, h8 *y, const h8 *zero, int HW) {
    __shared__ float part[4][8];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const h8 *xin = x + (size_t)blockIdx.x * HW;
    float acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = 0.0f;
    for (int p0 = 0; p0 < HW; p0 += 4 * 256) {
        h8 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int px = p0 + u * 256 + tid;
            v[u] = *(px < HW ? xin + px : zero);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[c] += E::get(v[u], c);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[c] += __shfl_xor(acc[c], off, 64);
    if (lane == 0)
#pragma unroll
        for (int c = 0; c < 8; ++c) part[wave][c] = acc[c];
    __syncthreads();
    if (tid == 0) {
        const float inv = 1.0f / (float)HW;
        float m[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) m[c] = ((part[0][c] + part[1][c]) + (part[2][c] + part[3][c])) * inv;
        y[blockIdx.x] = E::pack(m);
    }
}

// Small planes (up to 64 pixels): 8 lanes per (slice, image); lane j sums
// pixels j, j+8, ... with all loads issued at once (pixels past the end read
// the zero element instead of branching), then a 3-step butterfly inside the
// 8-lane group.  Fixed order, so deterministic.
template <typename E>
__global__ __launch_bounds__(256) void gap_small_kernel(const h8 *x, h8 *y, const h8 *zero,
                                                        int planes, int HW) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    const int idx = t >> 3, j = t & 7;
    const bool live = idx < planes;
    const h8 *xin = x + (size_t)(live ? idx : 0) * HW;
    h8 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int px = j + 8 * i;
        v[i] = *((live && px < HW) ? xin + px : zero);
    }
    float acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        float a = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) a += E::get(v[i], c);
        acc[c] = a;
    }
#pragma unroll
    for (int off = 4; off >= 1; off >>= 1)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[c] += __shfl_xor(acc[c], off, 8);
    if (live && j == 0) {
        const float inv = 1.0f / (float)HW;
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[c] *= inv;
        y[idx] = E::pack(acc);
    }
}

hipError_t launch_gap(const h8 *x, h8 *y, const h8 *zero, int N, int HW, int S, bool bf16,
                      hipStream_t st) {
    const size_t planes = (size_t)S * N;
    if (!planes) return hipSuccess;
    if (HW <= 64) {
        if (bf16)
            launch(gap_small_kernel<BF16>, dim3(blocks_for(planes * 8, 256)), dim3(256), 0, st, x, y, zero,
                   (int)planes, HW);
        else
            launch(gap_small_kernel<F16>, dim3(blocks_for(planes * 8, 256)), dim3(256), 0, st, x, y, zero,
                   (int)planes, HW);
    } else {
        if (bf16) launch(gap_kernel<BF16>, dim3((unsigned)planes), dim3(256), 0, st, x, y, zero, HW);
        else launch(gap_kernel<F16>, dim3((unsigned)planes), dim3(256), 0, st, x, y, zero, HW);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// softmax over rows of an fp32 (rows x cols) array; one wave per row
// (softmax_row)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void softmax_kernel(const float *z, float *y, int rows, int cols) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;  // whole wave
    softmax_row(z + (size_t)row * cols, y + (size_t)row * cols, cols, threadIdx.x & 63);
}

hipError_t launch_softmax(const float *z, float *y, int rows, int cols, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    launch(softmax_kernel, dim3(blocks_for(rows, 4)), dim3(256), 0, st, z, y, rows, cols);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// channel concat: one thread per output (slice, pixel)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void concat_kernel(ConcatParams p) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (size_t)p.S * p.M) return;
    const int s = (int)(i / p.M);
    const int m = (int)(i - (size_t)s * p.M);
    // 16-bit values are moved as raw bits (the same for fp16 and bf16 storage)
    u16x8 o = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int c = s * 8 + j;
        if (c >= p.C) break;
        int k = 0;
        while (k + 1 < p.nin && c >= p.coff[k + 1]) ++k;
        const int cc = c - p.coff[k];
        o[j] = ((const uint16_t *)p.src[k])[((size_t)(cc >> 3) * p.M + m) * 8 + (cc & 7)];
    }
    p.y[i] = __builtin_bit_cast(h8, o);
}

hipError_t launch_concat(const ConcatParams &p, hipStream_t st) {
    const size_t n = (size_t)p.S * p.M;
    if (!n) return hipSuccess;
    launch(concat_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, p);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// bilinear resize (optionally followed by argmax over the real channels)
// ---------------------------------------------------------------------------
struct Lerp {
    int i0, i1;
    float f;
};

__device__ __forceinline__ Lerp lerp_coord(int d, int in, int out, int align_corners) {
    float src;
    if (align_corners) src = out > 1 ? (float)d * ((float)(in - 1) / (float)(out - 1)) : 0.0f;
    else src = (float)d * ((float)in / (float)out);
    int i0 = (int)floorf(src);
    if (i0 > in - 1) i0 = in - 1;
    const int i1 = i0 + 1 < in ? i0 + 1 : in - 1;
    return Lerp{i0, i1, src - (float)i0};
}

template <typename E>
__global__ __launch_bounds__(256) void resize_kernel(ResizeParams p) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t opix = (size_t)p.N * p.OH * p.OW;
    if (i >= opix * p.S) return;
    const int s = (int)(i / opix);
    const size_t r = i - (size_t)s * opix;
    const int n = (int)(r / ((size_t)p.OH * p.OW));
    const int q = (int)(r - (size_t)n * p.OH * p.OW);
    const int oy = q / p.OW, ox = q - oy * p.OW;
    const Lerp ly = lerp_coord(oy, p.H, p.OH, p.align_corners);
    const Lerp lx = lerp_coord(ox, p.W, p.OW, p.align_corners);
    const h8 *plane = p.x + ((size_t)s * p.N + n) * p.H * p.W;
    const h8 v00 = plane[(size_t)ly.i0 * p.W + lx.i0], v01 = plane[(size_t)ly.i0 * p.W + lx.i1];
    const h8 v10 = plane[(size_t)ly.i1 * p.W + lx.i0], v11 = plane[(size_t)ly.i1 * p.W + lx.i1];
    float o[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const float top = (1.0f - lx.f) * E::get(v00, c) + lx.f * E::get(v01, c);
        const float bot = (1.0f - lx.f) * E::get(v10, c) + lx.f * E::get(v11, c);
        o[c] = (1.0f - ly.f) * top + ly.f * bot;
    }
    ((h8 *)p.y)[i] = E::pack(o);
}

template <typename E>
__global__ __launch_bounds__(256) void resize_argmax_kernel(ResizeParams p) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t opix = (size_t)p.N * p.OH * p.OW;
    if (i >= opix) return;
    const int n = (int)(i / ((size_t)p.OH * p.OW));
    const int q = (int)(i - (size_t)n * p.OH * p.OW);
    const int oy = q / p.OW, ox = q - oy * p.OW;
    const Lerp ly = lerp_coord(oy, p.H, p.OH, p.align_corners);
    const Lerp lx = lerp_coord(ox, p.W, p.OW, p.align_corners);
    float best = -FLT_MAX;
    int arg = 0;
    for (int s = 0; s < p.S; ++s) {
        const h8 *plane = p.x + ((size_t)s * p.N + n) * p.H * p.W;
        const h8 v00 = plane[(size_t)ly.i0 * p.W + lx.i0], v01 = plane[(size_t)ly.i0 * p.W + lx.i1];
        const h8 v10 = plane[(size_t)ly.i1 * p.W + lx.i0], v11 = plane[(size_t)ly.i1 * p.W + lx.i1];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int ch = s * 8 + c;
            if (ch >= p.C) break;
            const float top = (1.0f - lx.f) * E::get(v00, c) + lx.f * E::get(v01, c);
            const float bot = (1.0f - lx.f) * E::get(v10, c) + lx.f * E::get(v11, c);
            const float v = (1.0f - ly.f) * top + ly.f * bot;
            if (ch == 0 || v > best) {
                best = v;
                arg = ch;
            }
        }
    }
    ((int *)p.y)[i] = arg;
}

hipError_t launch_resize(const ResizeParams &p, bool argmax, hipStream_t st) {
    const size_t opix = (size_t)p.N * p.OH * p.OW;
    if (!opix) return hipSuccess;
    if (argmax) {
        if (p.bf16) launch(resize_argmax_kernel<BF16>, dim3(blocks_for(opix, 256)), dim3(256), 0, st, p);
        else launch(resize_argmax_kernel<F16>, dim3(blocks_for(opix, 256)), dim3(256), 0, st, p);
    } else {
        if (p.bf16) launch(resize_kernel<BF16>, dim3(blocks_for(opix * p.S, 256)), dim3(256), 0, st, p);
        else launch(resize_kernel<F16>, dim3(blocks_for(opix * p.S, 256)), dim3(256), 0, st, p);
    }
    return hipGetLastError();
}

template <typename E>
__global__ __launch_bounds__(256) void argmax_kernel(const h8 *x, int *y, int M, int S, int C) {
    const int m = blockIdx.x * 256 + threadIdx.x;
    if (m >= M) return;
    float best = -FLT_MAX;
    int arg = 0;
    for (int s = 0; s < S; ++s) {
        const h8 v = x[(size_t)s * M + m];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int ch = s * 8 + c;
            if (ch >= C) break;
            const float f = E::get(v, c);
            if (ch == 0 || f > best) {
                best = f;
                arg = ch;
            }
        }
    }
    y[m] = arg;
}

hipError_t launch_argmax(const h8 *x, int *y, int M, int S, int C, bool bf16, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    if (bf16) launch(argmax_kernel<BF16>, dim3(blocks_for(M, 256)), dim3(256), 0, st, x, y, M, S, C);
    else launch(argmax_kernel<F16>, dim3(blocks_for(M, 256)), dim3(256), 0, st, x, y, M, S, C);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// NHWC graph input -> sliced fp16, and sliced -> NHWC fp32 output.  One thread
// per (pixel, slice) with the slice index fastest, so a wave reads one
// contiguous run of NHWC memory.
// ---------------------------------------------------------------------------
template <typename E, typename TIN>
__global__ __launch_bounds__(256) void ingest_kernel(const TIN *x, h8 *y, int M, int C, int S) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (size_t)M * S) return;
    const int m = (int)(i / S), s = (int)(i - (size_t)m * S);
    const TIN *src = x + (size_t)m * C + s * 8;
    float o[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) o[c] = s * 8 + c < C ? (float)src[c] : 0.0f;
    y[(size_t)s * M + m] = E::pack(o);
}

template <typename E>
static hipError_t launch_ingest_e(const void *x, bool fp16_in, h8 *y, int M, int C, hipStream_t st) {
    const int S = (C + 7) / 8;
    const size_t n = (size_t)M * S;
    if (!n) return hipSuccess;
    if (fp16_in)
        launch((ingest_kernel<E, _Float16>), dim3(blocks_for(n, 256)), dim3(256), 0, st,
                           (const _Float16 *)x, y, M, C, S);
    else
        launch((ingest_kernel<E, float>), dim3(blocks_for(n, 256)), dim3(256), 0, st,
                           (const float *)x, y, M, C, S);
    return hipGetLastError();
}

hipError_t launch_ingest(const void *x, bool fp16_in, h8 *y, int M, int C, bool bf16, hipStream_t st) {
    return bf16 ? launch_ingest_e<BF16>(x, fp16_in, y, M, C, st) : launch_ingest_e<F16>(x, fp16_in, y, M, C, st);
}

template <typename E>
__global__ __launch_bounds__(256) void export_kernel(const h8 *x, float *y, int M, int C, int S) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (size_t)M * S) return;
    const int m = (int)(i / S), s = (int)(i - (size_t)m * S);
    const h8 v = x[(size_t)s * M + m];
    float *dst = y + (size_t)m * C + s * 8;
#pragma unroll
    for (int c = 0; c < 8; ++c)
        if (s * 8 + c < C) dst[c] = E::get(v, c);
}

hipError_t launch_export(const h8 *x, float *y, int M, int C, bool bf16, hipStream_t st) {
    const int S = (C + 7) / 8;
    const size_t n = (size_t)M * S;
    if (!n) return hipSuccess;
    if (bf16) launch(export_kernel<BF16>, dim3(blocks_for(n, 256)), dim3(256), 0, st, x, y, M, C, S);
    else launch(export_kernel<F16>, dim3(blocks_for(n, 256)), dim3(256), 0, st, x, y, M, C, S);
    return hipGetLastError();
}

}  // namespace kern
}  // namespace mgi
