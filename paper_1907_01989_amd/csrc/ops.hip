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

#include "kernels.h"

namespace mgi {
namespace kern {

__device__ __forceinline__ float act_apply(float v, int act) {
    if (act == MGI_ACT_RELU) return fmaxf(v, 0.0f);
    if (act == MGI_ACT_RELU6) return fminf(fmaxf(v, 0.0f), 6.0f);
    return v;
}

__device__ __forceinline__ h8 zero_h8() {
    h8 z;
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = (_Float16)0.0f;
    return z;
}

static inline unsigned blocks_for(size_t n, int per) { return (unsigned)((n + per - 1) / per); }

// ---------------------------------------------------------------------------
// depthwise convolution: one thread per output pixel of one slice (8
// channels), fp32 accumulation over the kh x kw window, bias + activation
// epilogue.  The launch is 1-D: block b covers pixels [256*(b % tpp), +256) of
// plane b / tpp, a plane being one (slice, image) pair.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void dw_kernel(DwParams p, int tpp) {
    const int plane = blockIdx.x / tpp;
    const int pix = (blockIdx.x - plane * tpp) * 256 + threadIdx.x;
    const int ohw = p.OH * p.OW;
    if (pix >= ohw) return;
    const int s = plane / p.N;
    const int oy = pix / p.OW, ox = pix - oy * p.OW;
    const h8 *xin = p.x + (size_t)plane * p.H * p.W;
    const float *wt = p.w + (size_t)s * p.KH * p.KW * 8;
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
            const float *wk = wt + (ky * p.KW + kx) * 8;
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[c] = fmaf(wk[c], (float)v[c], acc[c]);
        }
    }
    h8 o;
#pragma unroll
    for (int c = 0; c < 8; ++c) o[c] = (_Float16)act_apply(acc[c], p.act);
    p.y[(size_t)plane * ohw + pix] = o;
}

hipError_t launch_depthwise(const DwParams &p, hipStream_t st) {
    const int ohw = p.OH * p.OW;
    if (ohw <= 0 || p.N <= 0 || p.S <= 0) return hipSuccess;
    const int tpp = (ohw + 255) / 256;
    const size_t nblk = (size_t)tpp * p.S * p.N;
    if (nblk > 0x7fffffffu) return hipErrorInvalidValue;
    hipLaunchKernelGGL(dw_kernel, dim3((unsigned)nblk), dim3(256), 0, st, p, tpp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// element-wise
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void add_kernel(const h8 *a, const h8 *b, h8 *y, size_t n, int act) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const h8 u = a[i], v = b[i];
    h8 o;
#pragma unroll
    for (int c = 0; c < 8; ++c) o[c] = (_Float16)act_apply((float)u[c] + (float)v[c], act);
    y[i] = o;
}

hipError_t launch_add(const h8 *a, const h8 *b, h8 *y, size_t count, int act, hipStream_t st) {
    if (!count) return hipSuccess;
    hipLaunchKernelGGL(add_kernel, dim3(blocks_for(count, 256)), dim3(256), 0, st, a, b, y, count, act);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void act_kernel(const h8 *x, h8 *y, size_t n, int act) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const h8 u = x[i];
    h8 o;
#pragma unroll
    for (int c = 0; c < 8; ++c) o[c] = (_Float16)act_apply((float)u[c], act);
    y[i] = o;
}

hipError_t launch_act(const h8 *x, h8 *y, size_t count, int act, hipStream_t st) {
    if (!count) return hipSuccess;
    hipLaunchKernelGGL(act_kernel, dim3(blocks_for(count, 256)), dim3(256), 0, st, x, y, count, act);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// global average pool: one wave per (slice, image); lanes stride over the
// pixels, then a fixed butterfly reduction (deterministic).  Output is the
// sliced (n, 1, 1, c) tensor in fp16.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gap_kernel(const h8 *x, h8 *y, int N, int HW, int S) {
    const int lane = threadIdx.x & 63;
    const int idx = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (idx >= S * N) return;  // whole wave exits together
    const h8 *xin = x + (size_t)idx * HW;
    float acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = 0.0f;
    for (int p = lane; p < HW; p += 64) {
        const h8 v = xin[p];
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[c] += (float)v[c];
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[c] += __shfl_xor(acc[c], off, 64);
    if (lane == 0) {
        const float inv = 1.0f / (float)HW;
        h8 o;
#pragma unroll
        for (int c = 0; c < 8; ++c) o[c] = (_Float16)(acc[c] * inv);
        y[idx] = o;
    }
}

hipError_t launch_gap(const h8 *x, h8 *y, int N, int HW, int S, hipStream_t st) {
    const size_t waves = (size_t)S * N;
    if (!waves) return hipSuccess;
    hipLaunchKernelGGL(gap_kernel, dim3(blocks_for(waves, 4)), dim3(256), 0, st, x, y, N, HW, S);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// softmax over rows of an fp32 (rows x cols) array; one workgroup per row.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float block_reduce(float v, bool is_max, float *red) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float o = __shfl_xor(v, off, 64);
        v = is_max ? fmaxf(v, o) : v + o;
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float r = red[0];
#pragma unroll
    for (int w = 1; w < 4; ++w) r = is_max ? fmaxf(r, red[w]) : r + red[w];
    return r;
}

__global__ __launch_bounds__(256) void softmax_kernel(const float *z, float *y, int cols) {
    __shared__ float red[4];
    const float *zr = z + (size_t)blockIdx.x * cols;
    float *yr = y + (size_t)blockIdx.x * cols;
    float m = -FLT_MAX;
    for (int j = threadIdx.x; j < cols; j += 256) m = fmaxf(m, zr[j]);
    m = block_reduce(m, true, red);
    float s = 0.0f;
    for (int j = threadIdx.x; j < cols; j += 256) {
        const float e = expf(zr[j] - m);
        yr[j] = e;
        s += e;
    }
    s = block_reduce(s, false, red);
    const float inv = 1.0f / s;
    for (int j = threadIdx.x; j < cols; j += 256) yr[j] *= inv;
}

hipError_t launch_softmax(const float *z, float *y, int rows, int cols, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    hipLaunchKernelGGL(softmax_kernel, dim3(rows), dim3(256), 0, st, z, y, cols);
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
    h8 o = zero_h8();
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int c = s * 8 + j;
        if (c >= p.C) break;
        int k = 0;
        while (k + 1 < p.nin && c >= p.coff[k + 1]) ++k;
        const int cc = c - p.coff[k];
        o[j] = ((const _Float16 *)p.src[k])[((size_t)(cc >> 3) * p.M + m) * 8 + (cc & 7)];
    }
    p.y[i] = o;
}

hipError_t launch_concat(const ConcatParams &p, hipStream_t st) {
    const size_t n = (size_t)p.S * p.M;
    if (!n) return hipSuccess;
    hipLaunchKernelGGL(concat_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, p);
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
    h8 o;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const float top = (1.0f - lx.f) * (float)v00[c] + lx.f * (float)v01[c];
        const float bot = (1.0f - lx.f) * (float)v10[c] + lx.f * (float)v11[c];
        o[c] = (_Float16)((1.0f - ly.f) * top + ly.f * bot);
    }
    ((h8 *)p.y)[i] = o;
}

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
            const float top = (1.0f - lx.f) * (float)v00[c] + lx.f * (float)v01[c];
            const float bot = (1.0f - lx.f) * (float)v10[c] + lx.f * (float)v11[c];
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
        hipLaunchKernelGGL(resize_argmax_kernel, dim3(blocks_for(opix, 256)), dim3(256), 0, st, p);
    } else {
        hipLaunchKernelGGL(resize_kernel, dim3(blocks_for(opix * p.S, 256)), dim3(256), 0, st, p);
    }
    return hipGetLastError();
}

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
            const float f = (float)v[c];
            if (ch == 0 || f > best) {
                best = f;
                arg = ch;
            }
        }
    }
    y[m] = arg;
}

hipError_t launch_argmax(const h8 *x, int *y, int M, int S, int C, hipStream_t st) {
    if (M <= 0) return hipSuccess;
    hipLaunchKernelGGL(argmax_kernel, dim3(blocks_for(M, 256)), dim3(256), 0, st, x, y, M, S, C);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// NHWC graph input -> sliced fp16, and sliced -> NHWC fp32 output.  One thread
// per (pixel, slice) with the slice index fastest, so a wave reads one
// contiguous run of NHWC memory.
// ---------------------------------------------------------------------------
template <typename TIN>
__global__ __launch_bounds__(256) void ingest_kernel(const TIN *x, h8 *y, int M, int C, int S) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (size_t)M * S) return;
    const int m = (int)(i / S), s = (int)(i - (size_t)m * S);
    const TIN *src = x + (size_t)m * C + s * 8;
    h8 o = zero_h8();
#pragma unroll
    for (int c = 0; c < 8; ++c)
        if (s * 8 + c < C) o[c] = (_Float16)(float)src[c];
    y[(size_t)s * M + m] = o;
}

hipError_t launch_ingest(const void *x, bool fp16_in, h8 *y, int M, int C, hipStream_t st) {
    const int S = (C + 7) / 8;
    const size_t n = (size_t)M * S;
    if (!n) return hipSuccess;
    if (fp16_in)
        hipLaunchKernelGGL((ingest_kernel<_Float16>), dim3(blocks_for(n, 256)), dim3(256), 0, st,
                           (const _Float16 *)x, y, M, C, S);
    else
        hipLaunchKernelGGL((ingest_kernel<float>), dim3(blocks_for(n, 256)), dim3(256), 0, st,
                           (const float *)x, y, M, C, S);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void export_kernel(const h8 *x, float *y, int M, int C, int S) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (size_t)M * S) return;
    const int m = (int)(i / S), s = (int)(i - (size_t)m * S);
    const h8 v = x[(size_t)s * M + m];
    float *dst = y + (size_t)m * C + s * 8;
#pragma unroll
    for (int c = 0; c < 8; ++c)
        if (s * 8 + c < C) dst[c] = (float)v[c];
}

hipError_t launch_export(const h8 *x, float *y, int M, int C, hipStream_t st) {
    const int S = (C + 7) / 8;
    const size_t n = (size_t)M * S;
    if (!n) return hipSuccess;
    hipLaunchKernelGGL(export_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, x, y, M, C, S);
    return hipGetLastError();
}

}  // namespace kern
}  // namespace mgi
