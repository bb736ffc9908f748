// Depthwise 3x3 convolution fused into the pointwise convolution that
// consumes it (an extension of the paper's fusion of element-wise operators
// into the expensive operator, Sec. 3.2, to the depthwise-separable pair).
//
// The unfused pair writes the depthwise output to HBM and reads it straight
// back; in the early MobileNet layers that round trip is a third of the
// layer's bytes.  Here a workgroup owns RB whole output rows of one image
// (RB * OW <= 64 * FMW pixels) and all FN*16 output channels of the
// pointwise convolution, and walks K (the depthwise channels) in chunks of
// four slices.  For each chunk it
//   1. stages the input rows its outputs need (with the zero padding written
//      out as zeros) in LDS, each element loaded once;
//   2. computes the depthwise outputs from LDS (same tap order, fp32
//      accumulation, activation and fp16 rounding as the standalone kernel)
//      into an LDS B tile;
//   3. runs the MFMAs (v_mfma_f32_16x16x32_f16, K ascending as in the GEMM
//      kernels) against the chunk's packed weights, staged next to it.
// The result is bit-identical to the unfused pair.  The next chunk's band
// and weights are loaded into registers while the current chunk computes.
// The four waves split the pixel fragments; each holds all FN channel blocks.
#include "device.h"

namespace mgi {
namespace kern {

__device__ __forceinline__ int fdiv_exact(int a, float inv) { return (int)(((float)a + 0.5f) * inv); }

template <typename E, int FMW, int FN, int S_>
__global__ __launch_bounds__(256) void dwpw_kernel(DwPwParams p, DwPwTile t) {
    constexpr int BM = 64 * FMW;                 // pixels computed per workgroup
    constexpr int BT = 4 * BM, AT = FN * 64;     // B tile and A chunk, 16-byte elements
    constexpr int EPT = (kDwPwBandMax + 255) / 256;
    constexpr int WPT = (AT + 255) / 256;
    constexpr int PPT = (4 * BM + 255) / 256;    // depthwise (pixel, slice) pairs per thread
    constexpr int STAGE_H8 = 4 * 4 * FMW * 256 / 4;
    constexpr int MAIN_H8 = kDwPwBandMax + BT + AT;
    __shared__ h8 lds[MAIN_H8 > STAGE_H8 ? MAIN_H8 : STAGE_H8];
    h8 *band = lds, *btile = lds + kDwPwBandMax, *atile = lds + kDwPwBandMax + BT;
    const GemmParams &g = p.g;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = blockIdx.x / t.nbands, oy0 = (blockIdx.x - n * t.nbands) * t.RB;
    const int m0 = (n * p.OH + oy0) * p.OW;
    const int valid = t.RB * p.OW;
    const int nk = g.ksp >> 2;
    const int per = t.NRB * t.WP, band_n = 4 * per;
    const int min_px = p.N * p.H * p.W;

    // band element e of this thread: slice-in-chunk and spatial offset (fixed over K)
    int bsl[EPT], boff[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int e = tid + 256 * i;
        const int sl = fdiv_exact(e, t.inv_per), rem = e - sl * per;
        const int r = fdiv_exact(rem, t.inv_wp), c = rem - r * t.WP;
        const int iy = oy0 * S_ - p.pt + r, ix = c - p.pl;
        bsl[i] = sl;
        boff[i] = (e < band_n && iy >= 0 && iy < p.H && ix >= 0 && ix < p.W) ? (n * p.H + iy) * p.W + ix : -1;
    }
    // depthwise outputs of this thread: slice-in-chunk, pixel, LDS base of its window
    int dsl[PPT], dpx[PPT], dbase[PPT];
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
        const int q = tid + 256 * j;
        dsl[j] = q / BM;
        dpx[j] = q - dsl[j] * BM;
        const int r = fdiv_exact(dpx[j], t.inv_ow), x = dpx[j] - r * p.OW;
        dbase[j] = (dsl[j] * t.NRB + r * S_) * t.WP + x * S_;
    }

    h8 bv[EPT], wr[WPT];
    auto gload = [&](int kc) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const int s = min(kc * 4 + bsl[i], g.ksl - 1);   // K tail: its weights are zero
            bv[i] = *(boff[i] >= 0 ? p.x + (size_t)s * min_px + boff[i] : p.zero);
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

    f4 acc[FN][FMW];
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const f4 b0 = bias_frag(g.bias, i, g.nb16, lane);
#pragma unroll
        for (int j = 0; j < FMW; ++j) acc[i][j] = b0;
    }

    gload(0);
    for (int kc = 0; kc < nk; ++kc) {
        __syncthreads();                         // the previous chunk is done with LDS
#pragma unroll
        for (int i = 0; i < EPT; ++i)
            if (tid + 256 * i < band_n) band[tid + 256 * i] = bv[i];
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int e = tid + 256 * i;
            if (AT % 256 == 0 || e < AT) atile[e] = wr[i];
        }
        __syncthreads();
        if (kc + 1 < nk) gload(kc + 1);
#pragma unroll
        for (int j = 0; j < PPT; ++j) {
            if (dpx[j] >= valid || dsl[j] >= 4) continue;   // padding pixels: never stored
            const int s = min(kc * 4 + dsl[j], g.ksl - 1);
            const h8 *wt = p.dww + (size_t)s * 9;
            float a8[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) a8[c] = p.dwb[s * 8 + c];
#pragma unroll
            for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                for (int kx = 0; kx < 3; ++kx)
                    E::fma8(a8, wt[ky * 3 + kx], band[dbase[j] + ky * t.WP + kx]);
#pragma unroll
            for (int c = 0; c < 8; ++c) a8[c] = __builtin_amdgcn_fmed3f(a8[c], lo, hi);
            btile[dsl[j] * BM + dpx[j]] = E::pack(a8);
        }
        __syncthreads();
        h8 b[FMW];
#pragma unroll
        for (int j = 0; j < FMW; ++j) b[j] = btile[(lane >> 4) * BM + (wave * FMW + j) * 16 + (lane & 15)];
#pragma unroll
        for (int i = 0; i < FN; ++i) {
            const h8 a = atile[i * 64 + lane];
#pragma unroll
            for (int j = 0; j < FMW; ++j)
                acc[i][j] = E::mma(a, b[j], acc[i][j]);
        }
    }
    __syncthreads();

    // epilogue in passes of four channel blocks through a per-wave stage;
    // pixels past this band's rows belong to the next band and are not stored
    float *stage = (float *)lds + wave * (4 * FMW * 256);
    const int mw = m0 + wave * FMW * 16, mlim = m0 + valid;
#pragma unroll
    for (int g4 = 0; g4 < FN; g4 += 4) {
        constexpr int REM = FN % 4 == 0 ? 4 : FN % 4;
        if (g4 + 4 <= FN) {
            store_tile_c8<E, FMW, 4>(g, *reinterpret_cast<const f4(*)[4][FMW]>(&acc[g4]), mw, g4, stage, lane,
                                  mlim);
        } else {
            store_tile_c8<E, FMW, REM>(g, *reinterpret_cast<const f4(*)[REM][FMW]>(&acc[g4]), mw, g4, stage,
                                    lane, mlim);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

template <int FMW, int FN>
static hipError_t launch_dwpw_fn(const DwPwParams &p, const DwPwTile &t, hipStream_t st) {
    const unsigned blocks = (unsigned)(p.N * t.nbands);
    if (p.g.bf16) {
        if (p.sh == 1) launch((dwpw_kernel<BF16, FMW, FN, 1>), dim3(blocks), dim3(256), 0, st, p, t);
        else launch((dwpw_kernel<BF16, FMW, FN, 2>), dim3(blocks), dim3(256), 0, st, p, t);
    } else {
        if (p.sh == 1) launch((dwpw_kernel<F16, FMW, FN, 1>), dim3(blocks), dim3(256), 0, st, p, t);
        else launch((dwpw_kernel<F16, FMW, FN, 2>), dim3(blocks), dim3(256), 0, st, p, t);
    }
    return hipGetLastError();
}

int dwpw_blocks(int nb16) {
    const int fns[7] = {1, 2, 4, 8, 12, 16, 20};
    for (int f : fns)
        if (nb16 <= f) return f;
    return 0;
}

bool dwpw_tile(int OH, int OW, int S, int N, DwPwTile &t, int max_px) {
    int rb = 0;
    for (int r = 1; r <= OH; ++r)
        if (OH % r == 0 && r * OW <= max_px) rb = r;
    if (!rb) return false;
    t.RB = rb;
    t.nbands = OH / rb;
    t.NRB = (rb - 1) * S + 3;
    t.WP = (OW - 1) * S + 3;
    if (4 * t.NRB * t.WP > kDwPwBandMax) return false;
    t.fmw = rb * OW <= 64 ? 1 : 2;
    t.inv_per = 1.0f / (float)(t.NRB * t.WP);
    t.inv_wp = 1.0f / (float)t.WP;
    t.inv_ow = 1.0f / (float)OW;
    (void)N;
    return true;
}

hipError_t launch_dwpw(const DwPwParams &p, const DwPwTile &t, hipStream_t st) {
    if (p.g.M <= 0) return hipSuccess;
    if (p.sh != p.sw || (p.sh != 1 && p.sh != 2)) return hipErrorInvalidValue;
    if (t.RB <= 0 || p.OH % t.RB != 0 || t.RB * p.OW > 64 * t.fmw || 4 * t.NRB * t.WP > kDwPwBandMax)
        return hipErrorInvalidValue;
    const int fn = dwpw_blocks(p.g.nb16);
#define MGI_DWPW_CASE(FMW_, FN_) \
    if (t.fmw == FMW_ && fn == FN_) return launch_dwpw_fn<FMW_, FN_>(p, t, st);
    MGI_DWPW_CASE(1, 1) MGI_DWPW_CASE(1, 2) MGI_DWPW_CASE(1, 4) MGI_DWPW_CASE(1, 8)
    MGI_DWPW_CASE(1, 12) MGI_DWPW_CASE(1, 16) MGI_DWPW_CASE(1, 20)
    MGI_DWPW_CASE(2, 1) MGI_DWPW_CASE(2, 2) MGI_DWPW_CASE(2, 4) MGI_DWPW_CASE(2, 8)
    MGI_DWPW_CASE(2, 12) MGI_DWPW_CASE(2, 16) MGI_DWPW_CASE(2, 20)
#undef MGI_DWPW_CASE
    return hipErrorInvalidValue;
}

}  // namespace kern
}  // namespace mgi
