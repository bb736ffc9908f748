// Depthwise 3x3 convolution fused into the pointwise convolution that
// consumes it (an extension of the paper's fusion of element-wise operators
// into the expensive operator, Sec. 3.2, to the depthwise-separable pair).
//
// The unfused pair writes the depthwise output to HBM and reads it straight
// back; in the early MobileNet layers that round trip is a third of the
// layer's bytes.  Here a workgroup owns BM consecutive output pixels and all
// FN*16 output channels of the pointwise convolution, and walks K (the
// depthwise channels) in chunks of four slices: for each chunk it computes
// the depthwise outputs of its pixels (same tap order, fp32 accumulation,
// activation and fp16 rounding as the standalone depthwise kernel) straight
// into an LDS B tile, stages the chunk's packed weights next to it, and runs
// the MFMAs (v_mfma_f32_16x16x32_f16, K ascending as in the GEMM kernels).
// The result is therefore bit-identical to the unfused pair.  Loads for
// chunk k+1 are issued before the MFMAs of chunk k; LDS is double-buffered
// with one barrier per chunk.  The four waves split the pixels (BM/64
// fragments of 16 each) and each holds all FN channel blocks.
#include "device.h"

namespace mgi {
namespace kern {

template <int BM, int FN, int S_>
__global__ __launch_bounds__(256) void dwpw_kernel(DwPwParams p) {
    constexpr int FMW = BM / 64;                 // pixel fragments per wave
    constexpr int PPT = BM / 64;                 // (pixel, slice) pairs per thread and chunk
    constexpr int BT = 4 * BM, AT = FN * 64;     // B tile and A chunk, in 16-byte elements
    constexpr int BUF = BT + AT;
    constexpr int WPT = (AT + 255) / 256;        // weight elements per thread and chunk
    constexpr int STAGE = 4 * 4 * FMW * 256;     // epilogue floats (4 waves, 4 blocks per pass)
    constexpr int LDS_H8 = 2 * BUF > STAGE / 4 ? 2 * BUF : STAGE / 4;
    __shared__ h8 lds[LDS_H8];
    const GemmParams &g = p.g;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m0 = blockIdx.x * BM;
    const int nk = g.ksp >> 2;

    // this thread's pixel (fixed over K) and the element offsets of its taps
    const int px = tid % BM;
    const int ohw = p.OH * p.OW;
    const int mc = min(m0 + px, g.M - 1);        // pixels past M are computed, never stored
    const int n = mc / ohw, r = mc - n * ohw;
    const int oy = r / p.OW, ox = r - oy * p.OW;
    int off[9];
#pragma unroll
    for (int ky = 0; ky < 3; ++ky)
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) {
            const int iy = oy * S_ - p.pt + ky, ix = ox * S_ - p.pl + kx;
            off[ky * 3 + kx] = (iy >= 0 && iy < p.H && ix >= 0 && ix < p.W) ? (n * p.H + iy) * p.W + ix : -1;
        }
    const int min_px = p.N * p.H * p.W;          // pixels per slice of the depthwise input

    h8 v[PPT][9], wr[WPT];
    auto gload = [&](int kc) {
#pragma unroll
        for (int j = 0; j < PPT; ++j) {
            const int s = min(kc * 4 + tid / BM + j * (256 / BM), g.ksl - 1);   // K tail: zero weights
            const h8 *base = p.x + (size_t)s * min_px;
#pragma unroll
            for (int t = 0; t < 9; ++t) v[j][t] = *(off[t] >= 0 ? base + off[t] : p.zero);
        }
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int e = tid + 256 * i;
            const int blk = min(e >> 6, g.nb16 - 1);  // blocks past nb16 are never stored
            if (AT % 256 == 0 || e < AT) wr[i] = g.w[((size_t)blk * g.ksp + kc * 4) * 16 + (e & 63)];
        }
    };
    const float lo = p.act == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    auto lstore = [&](int kc, h8 *buf) {
#pragma unroll
        for (int j = 0; j < PPT; ++j) {
            const int sl = tid / BM + j * (256 / BM);
            const int s = min(kc * 4 + sl, g.ksl - 1);
            const h8 *wt = p.dww + (size_t)s * 9;
            float acc[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[c] = p.dwb[s * 8 + c];
#pragma unroll
            for (int t = 0; t < 9; ++t) fma8(acc, as_u4(wt[t]), as_u4(v[j][t]));
            h8 o;
#pragma unroll
            for (int c = 0; c < 8; ++c) o[c] = (_Float16)__builtin_amdgcn_fmed3f(acc[c], lo, hi);
            buf[sl * BM + px] = o;
        }
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int e = tid + 256 * i;
            if (AT % 256 == 0 || e < AT) buf[BT + e] = wr[i];
        }
    };

    f4 acc[FN][FMW];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FMW; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};

    gload(0);
    lstore(0, lds);
    __syncthreads();
    for (int kc = 0; kc < nk; ++kc) {
        const h8 *cur = lds + (kc & 1) * BUF;
        if (kc + 1 < nk) gload(kc + 1);
        h8 b[FMW];
#pragma unroll
        for (int j = 0; j < FMW; ++j) b[j] = cur[(lane >> 4) * BM + (wave * FMW + j) * 16 + (lane & 15)];
#pragma unroll
        for (int i = 0; i < FN; ++i) {
            const h8 a = cur[BT + i * 64 + lane];
#pragma unroll
            for (int j = 0; j < FMW; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b[j], acc[i][j], 0, 0, 0);
        }
        if (kc + 1 < nk) lstore(kc + 1, lds + ((kc + 1) & 1) * BUF);
        __syncthreads();
    }

    // epilogue in passes of four channel blocks through a per-wave stage
    float *stage = (float *)lds + wave * (4 * FMW * 256);
    const int mw = m0 + wave * FMW * 16;
#pragma unroll
    for (int g4 = 0; g4 < FN; g4 += 4) {
        constexpr int REM = FN % 4 == 0 ? 4 : FN % 4;
        if (g4 + 4 <= FN) {
            store_tile_c8<FMW, 4>(g, *reinterpret_cast<const f4(*)[4][FMW]>(&acc[g4]), mw, g4, stage, lane);
        } else {
            store_tile_c8<FMW, REM>(g, *reinterpret_cast<const f4(*)[REM][FMW]>(&acc[g4]), mw, g4, stage,
                                    lane);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

template <int BM, int FN>
static hipError_t launch_dwpw_fn(const DwPwParams &p, hipStream_t st) {
    const unsigned blocks = (unsigned)((p.g.M + BM - 1) / BM);
    if (p.sh == 1) launch((dwpw_kernel<BM, FN, 1>), dim3(blocks), dim3(256), 0, st, p);
    else launch((dwpw_kernel<BM, FN, 2>), dim3(blocks), dim3(256), 0, st, p);
    return hipGetLastError();
}

int dwpw_blocks(int nb16) {
    const int fns[7] = {1, 2, 4, 8, 12, 16, 20};
    for (int f : fns)
        if (nb16 <= f) return f;
    return 0;
}

hipError_t launch_dwpw(const DwPwParams &p, int bm, hipStream_t st) {
    if (p.g.M <= 0) return hipSuccess;
    if (p.sh != p.sw || (p.sh != 1 && p.sh != 2)) return hipErrorInvalidValue;
    const int fn = dwpw_blocks(p.g.nb16);
#define MGI_DWPW_CASE(BM_, FN_) \
    if (bm == BM_ && fn == FN_) return launch_dwpw_fn<BM_, FN_>(p, st);
    MGI_DWPW_CASE(64, 1) MGI_DWPW_CASE(64, 2) MGI_DWPW_CASE(64, 4) MGI_DWPW_CASE(64, 8)
    MGI_DWPW_CASE(64, 12) MGI_DWPW_CASE(64, 16) MGI_DWPW_CASE(64, 20)
    MGI_DWPW_CASE(128, 1) MGI_DWPW_CASE(128, 2) MGI_DWPW_CASE(128, 4) MGI_DWPW_CASE(128, 8)
    MGI_DWPW_CASE(128, 12) MGI_DWPW_CASE(128, 16) MGI_DWPW_CASE(128, 20)
#undef MGI_DWPW_CASE
    return hipErrorInvalidValue;
}

}  // namespace kern
}  // namespace mgi
