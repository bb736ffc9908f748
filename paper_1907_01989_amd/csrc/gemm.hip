// MFMA GEMM kernels for gfx950: pointwise (1x1) convolution, implicit-GEMM
// convolution over a window, fully-connected layers, and the network stem.
//
// The paper specialises the 1x1 convolution as its own program (Sec. 3.2) and
// fuses bias and activation into it.  On CDNA4 a 1x1 convolution over the
// sliced layout is a GEMM   D[cout][pixel] = W[cout][cin] * X[cin][pixel]
// and runs on v_mfma_f32_16x16x32_f16 with fp32 accumulation:
//   - the A operand is a 16 (output channels) x 32 (K) weight fragment: lane l
//     holds row l%16, K group l/16 (8 halves); packed weights make the 64
//     lanes' fragment one contiguous KiB;
//   - the B operand is a 32 (K) x 16 (pixels) activation fragment: lane l holds
//     pixel l%16 and channel slice l/16, i.e. exactly one 16-byte sliced
//     element, so fragments are read straight from the sliced layout;
//   - the accumulator gives lane l four consecutive output channels
//     4*(l/16)+r of pixel l%16, half a sliced element: the epilogue adds bias,
//     applies the activation(s) and the residual and writes 8 bytes per lane.
// Weight and activation tiles for four K slices (32 channels) per step are
// staged through LDS, double-buffered with one barrier per step, the next
// step's global loads issued before the current step's MFMAs.
#include "kernels.h"

namespace mgi {
namespace kern {

typedef float f4 __attribute__((ext_vector_type(4)));

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

// Workgroups are dispatched to the 8 XCDs round-robin (block b -> XCD b % 8).
// Give every XCD a contiguous range of tiles so that tiles sharing input rows
// (same pixel block, neighbouring channel blocks) meet in the same L2.
__device__ __forceinline__ int xcd_tile(int bid, int nblocks) {
    const int xcd = bid & 7, idx = bid >> 3;
    const int per = nblocks >> 3, rem = nblocks & 7;
    return xcd * per + min(xcd, rem) + idx;
}

template <int BM, int BN, bool TAPS, bool F32OUT>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
    constexpr int WM = BM / 2, WN = BN / 2;      // 2 x 2 waves
    constexpr int FM = WM / 16, FN = WN / 16;    // fragments per wave
    constexpr int XCH = 4 * BM;                  // 16-byte activation chunks per K step
    constexpr int WCH = (BN / 16) * 64;          // 16-byte weight chunks per K step
    constexpr int XPT = (XCH + 255) / 256, WPT = (WCH + 255) / 256;
    __shared__ h8 xs[2][XCH];
    __shared__ h8 ws[2][WCH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int mt = tile / p.ntiles, nt = tile - mt * p.ntiles;
    const int m0 = mt * BM, nb0 = nt * (BN / 16);

    // per-thread loader coordinates (fixed over the K loop)
    int xsl[XPT], xm[XPT];
    bool xon[XPT];
    int xn[XPT], xiy[XPT], xix[XPT];
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
        const int c = tid + 256 * i;
        xsl[i] = c / BM;
        xm[i] = m0 + (c % BM);
        xon[i] = (c < XCH) && (xm[i] < p.M);
        xn[i] = xiy[i] = xix[i] = 0;
        if (TAPS && xon[i]) {
            const int hw = p.OH * p.OW;
            const int n = xm[i] / hw, r = xm[i] - n * hw;
            const int oy = r / p.OW, ox = r - oy * p.OW;
            xn[i] = n;
            xiy[i] = oy * p.sh - p.pt;
            xix[i] = ox * p.sw - p.pl;
        }
    }
    const int ksteps = p.ksp >> 2;
    h8 xr[XPT], wr[WPT];

    auto gload = [&](int kk) {
#pragma unroll
        for (int i = 0; i < XPT; ++i) {
            h8 v = zero_h8();
            const int ks = kk * 4 + xsl[i];
            if (xon[i] && ks < p.ksl) {
                if (!TAPS) {
                    v = p.x[(size_t)ks * p.M + xm[i]];
                } else {
                    const int tap = ks / p.sin, s = ks - tap * p.sin;
                    const int ky = tap / p.kw, kx = tap - ky * p.kw;
                    const int iy = xiy[i] + ky * p.dh, ix = xix[i] + kx * p.dw;
                    if (iy >= 0 && iy < p.H && ix >= 0 && ix < p.W)
                        v = p.x[(size_t)s * p.Min + ((size_t)xn[i] * p.H + iy) * p.W + ix];
                }
            }
            xr[i] = v;
        }
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int c = tid + 256 * i;
            h8 v = zero_h8();
            if (c < WCH) {
                const int nb = nb0 + (c >> 6);
                if (nb < p.nb16) v = p.w[((size_t)nb * p.ksp + kk * 4) * 16 + (c & 63)];
            }
            wr[i] = v;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < XPT; ++i) {
            const int c = tid + 256 * i;
            if (c < XCH) xs[buf][c] = xr[i];
        }
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int c = tid + 256 * i;
            if (c < WCH) ws[buf][c] = wr[i];
        }
    };

    f4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    gload(0);
    lstore(0);
    __syncthreads();
    for (int kk = 0; kk < ksteps; ++kk) {
        const int cur = kk & 1;
        const bool more = kk + 1 < ksteps;
        if (more) gload(kk + 1);
        h8 a[FN], b[FM];
#pragma unroll
        for (int i = 0; i < FN; ++i) a[i] = ws[cur][(wn * FN + i) * 64 + lane];
#pragma unroll
        for (int j = 0; j < FM; ++j) b[j] = xs[cur][(lane >> 4) * BM + wm * WM + j * 16 + (lane & 15)];
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int j = 0; j < FM; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], b[j], acc[i][j], 0, 0, 0);
        if (more) lstore(cur ^ 1);
        __syncthreads();
    }

    // epilogue
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const int nb = nb0 + wn * FN + i;
        if (nb >= p.nb16) continue;
        const int nbase = nb * 16 + 4 * (lane >> 4);
        float bv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) bv[r] = p.bias[nbase + r];
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int m = m0 + wm * WM + j * 16 + (lane & 15);
            if (m >= p.M) continue;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r] + bv[r], p.act1);
            if (F32OUT) {
                float *y = (float *)p.y + (size_t)m * p.cout;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (nbase + r < p.cout) y[nbase + r] = v[r];
            } else {
                const int os = nbase >> 3, hoff = nbase & 7;
                if (os >= p.ns) continue;
                const size_t off = ((size_t)os * p.M + m) * 8 + hoff;
                if (p.res) {
                    const h4 rv = *(const h4 *)((const _Float16 *)p.res + off);
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] = act_apply(v[r] + (float)rv[r], p.act2);
                }
                h4 o;
#pragma unroll
                for (int r = 0; r < 4; ++r) o[r] = (_Float16)v[r];
                *(h4 *)((_Float16 *)p.y + off) = o;
            }
        }
    }
}

template <int BM, int BN>
static hipError_t launch_bm_bn(const GemmParams &p, bool taps, bool f32out, hipStream_t st) {
    GemmParams q = p;
    q.mtiles = (p.M + BM - 1) / BM;
    q.ntiles = (p.nb16 * 16 + BN - 1) / BN;
    const dim3 grid(q.mtiles * q.ntiles), block(256);
    if (f32out) {
        if (taps) return hipErrorInvalidValue;
        hipLaunchKernelGGL((gemm_kernel<BM, BN, false, true>), grid, block, 0, st, q);
    } else if (taps) {
        hipLaunchKernelGGL((gemm_kernel<BM, BN, true, false>), grid, block, 0, st, q);
    } else {
        hipLaunchKernelGGL((gemm_kernel<BM, BN, false, false>), grid, block, 0, st, q);
    }
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmParams &p, int bm, int bn, bool taps, bool f32out,
                       hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
#define MGI_GEMM_CASE(BM_, BN_) \
    if (bm == BM_ && bn == BN_) return launch_bm_bn<BM_, BN_>(p, taps, f32out, st);
    MGI_GEMM_CASE(32, 32)
    MGI_GEMM_CASE(32, 64)
    MGI_GEMM_CASE(32, 128)
    MGI_GEMM_CASE(64, 32)
    MGI_GEMM_CASE(64, 64)
    MGI_GEMM_CASE(64, 128)
    MGI_GEMM_CASE(128, 32)
    MGI_GEMM_CASE(128, 64)
    MGI_GEMM_CASE(128, 128)
#undef MGI_GEMM_CASE
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Stem: a convolution that reads the NHWC graph input directly.  The whole
// window (kh*kw*c <= 32 values) is one K step: lane l gathers im2col entries
// k = 8*(l/16) .. +7 of pixel l%16, converted to fp16, as its B fragment.
// Each wave covers 4 x 16 pixels and all output blocks (NB <= 4).
// ---------------------------------------------------------------------------
template <typename TIN, int NB>
__global__ __launch_bounds__(256) void stem_kernel(StemParams p) {
    constexpr int FM = 4;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int mbase = (blockIdx.x * 4 + wave) * (FM * 16);
    const TIN *x = (const TIN *)p.x;

    int dy[8], dx[8], ci[8];
    bool kv[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int k = 8 * (lane >> 4) + t;
        kv[t] = k < p.K;
        const int kk = kv[t] ? k : 0;
        const int tap = kk / p.C;
        ci[t] = kk - tap * p.C;
        const int ky = tap / p.KW, kx = tap - ky * p.KW;
        dy[t] = ky * p.dh - p.pt;
        dx[t] = kx * p.dw - p.pl;
    }
    h8 a[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) a[i] = p.w[(size_t)i * 64 + lane];
    const int hw = p.OH * p.OW;
    f4 acc[NB][FM];
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        const int m = mbase + j * 16 + (lane & 15);
        h8 b = zero_h8();
        if (m < p.M) {
            const int n = m / hw, r = m - n * hw;
            const int oy = r / p.OW, ox = r - oy * p.OW;
            const int iy0 = oy * p.sh, ix0 = ox * p.sw;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int iy = iy0 + dy[t], ix = ix0 + dx[t];
                if (kv[t] && iy >= 0 && iy < p.H && ix >= 0 && ix < p.W)
                    b[t] = (_Float16)(float)x[(((size_t)n * p.H + iy) * p.W + ix) * p.C + ci[t]];
            }
        }
#pragma unroll
        for (int i = 0; i < NB; ++i)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], b, f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int nbase = i * 16 + 4 * (lane >> 4);
        const int os = nbase >> 3, hoff = nbase & 7;
        if (os >= p.ns) continue;
        float bv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) bv[r] = p.bias[nbase + r];
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int m = mbase + j * 16 + (lane & 15);
            if (m >= p.M) continue;
            const size_t off = ((size_t)os * p.M + m) * 8 + hoff;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r] + bv[r], p.act1);
            if (p.res) {
                const h4 rv = *(const h4 *)((const _Float16 *)p.res + off);
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = act_apply(v[r] + (float)rv[r], p.act2);
            }
            h4 o;
#pragma unroll
            for (int r = 0; r < 4; ++r) o[r] = (_Float16)v[r];
            *(h4 *)((_Float16 *)p.y + off) = o;
        }
    }
}

template <typename TIN>
static hipError_t launch_stem_t(const StemParams &p, hipStream_t st) {
    const dim3 grid((p.M + 255) / 256), block(256);
    switch (p.nb16) {
        case 1: hipLaunchKernelGGL((stem_kernel<TIN, 1>), grid, block, 0, st, p); break;
        case 2: hipLaunchKernelGGL((stem_kernel<TIN, 2>), grid, block, 0, st, p); break;
        case 3: hipLaunchKernelGGL((stem_kernel<TIN, 3>), grid, block, 0, st, p); break;
        case 4: hipLaunchKernelGGL((stem_kernel<TIN, 4>), grid, block, 0, st, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_stem(const StemParams &p, bool fp16_in, hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
    return fp16_in ? launch_stem_t<_Float16>(p, st) : launch_stem_t<float>(p, st);
}

}  // namespace kern
}  // namespace mgi
