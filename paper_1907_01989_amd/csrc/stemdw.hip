// Network stem fused with the depthwise 3x3 convolution that reads its output.
//
// In the MobileNet-family networks (Sec. 6, Table 3's v1 and v2) the first
// convolution over the image is followed by a depthwise 3x3 at stride 1 whose
// only input is that convolution's output, the largest tensor of both
// networks after the first pointwise layer (n x 112 x 112 x 32 at 224x224).
// One kernel here computes both: a workgroup owns R output rows of one image;
// it stages the NHWC input rows those rows need in LDS (as the stem kernel
// does), computes the stem outputs of the R + 2 rows the depthwise step reads
// with one MFMA per 16 pixels x 16 channels into fp16 channel planes in LDS,
// and then runs the depthwise taps from those planes.  The stem rows next to
// a band boundary are computed by both neighbouring bands.
//
// Arithmetic: the stem's MFMA, bias and activation are the stem kernel's, the
// planes hold the values the stem kernel would store, and the depthwise step
// accumulates each output in the depthwise kernel's order (bias, then rows
// ky = 0..2, columns kx = 0..2, fp16 x fp16 + fp32 products), so the fused
// node is bit-identical to the two kernels run separately.
#include <cmath>

#include "device.h"

namespace mgi {
namespace kern {

namespace {

constexpr int NT = 512;                           // threads per workgroup

template <typename E, typename TIN, int NB, int R>
__global__ __launch_bounds__(NT) void stemdw_kernel(StemDwParams p) {
    constexpr int NSL = 2 * NB;                   // channel planes (8 channels each)
    constexpr int NWV = NT / 64;                  // waves
    extern __shared__ h8 lds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int n = tile / p.nbands, bnd = tile - n * p.nbands;
    const int oy_lo = bnd * R, oy_hi = min(p.OH, oy_lo + R);
    // stem rows [sr0, sr1) read by the band's depthwise outputs, and the
    // input rows [iy0, iy0 + nrows) those stem rows read
    const int sr0 = max(0, oy_lo - p.dpt), sr1 = min(p.SH, oy_hi - 1 - p.dpt + 3);
    const int nsr = sr1 - sr0;
    const int iy0 = sr0 * p.sh - p.pt;
    const int nrows = (nsr - 1) * p.sh + (p.KH - 1) * p.dh + 1;
    const int rs = p.rs;
    // LDS: planes [NSL][pstride] | input band [nrows][rs] halves | taps
    // [NSL][9] | depthwise bias [NSL * 8] fp32 | one zero element
    h8 *planes = lds;
    _Float16 *band = (_Float16 *)(lds + NSL * p.pstride);
    h8 *taps = lds + NSL * p.pstride + p.band_h8;
    float *dwb = (float *)(taps + NSL * 9);
    h8 *zslot = (h8 *)(dwb + NSL * 8);

    // 1. taps, biases and stem weights (loads issued first), then the input
    // rows of the band (all of the workgroup's loads in flight together)
    h8 tq = p.dw_w[min(tid, NSL * 9 - 1)];
    float bq = p.dw_b[min(tid, NSL * 8 - 1)];
    h8 a[NB];
    f4 c0[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        a[i] = p.w[(size_t)i * 64 + lane];
        c0[i] = bias_frag(p.bias, i, p.nb16, lane);
    }
    stage_input_band<E, TIN, NT, 4>(band, (const TIN *)p.x, n, p.H, p.W, p.C, iy0, nrows, rs, p.pl * p.C, tid);
    if (tid < NSL * 9) taps[tid] = tq;
    if (tid < NSL * 8) dwb[tid] = bq;
    if (tid == 0) *zslot = zero_h8();
    // offsets of the lane's 8 im2col entries inside a window
    int koff[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) koff[t] = p.koff[8 * (lane >> 4) + t];
    __syncthreads();

    // 2. stem outputs of rows [sr0, sr1) into the planes: one 16-pixel
    // fragment per wave step, NB MFMAs over K <= 32 (accumulator = bias)
    const int fpr = (p.SW + 15) >> 4;
    const int nfr = nsr * fpr;
    const int sub = 4 * ((lane >> 4) & 1);        // half of a sliced element
    int syl = wave / fpr, fx = wave - syl * fpr;  // fragment f = syl * fpr + fx, stepped below
    for (int f = wave; f < nfr; f += NWV, fx += NWV) {
        while (fx >= fpr) {
            fx -= fpr;
            ++syl;
        }
        const int sx = fx * 16 + (lane & 15);
        const int base = syl * p.sh * rs + min(sx, p.SW - 1) * p.sw * p.C;
        h8 b;
#pragma unroll
        for (int t = 0; t < 8; ++t) b[t] = band[base + koff[t]];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const f4 acc = E::mma(a[i], b, c0[i]);
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[r], p.act1);
            if (sx < p.SW)
                *(h4 *)((_Float16 *)(planes + (2 * i + (lane >> 5)) * p.pstride + syl * p.SW + sx) + sub) =
                    E::pack4(v);
        }
    }
    __syncthreads();

    // 3. depthwise 3x3 (stride 1) from the planes: a thread owns one output
    // column of one plane and the band's R rows
    const float lo = p.act2 == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act2 == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    const int ntask = p.ns * p.OW;
    for (int t = tid; t < ntask; t += NT) {
        const int sl = t / p.OW, ox = t - sl * p.OW;
        const h8 *plane = planes + sl * p.pstride;
        h8 w[9];
#pragma unroll
        for (int k = 0; k < 9; ++k) w[k] = taps[sl * 9 + k];
        int cx[3];
        bool cv[3];
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            cx[k] = ox - p.dpl + k;
            cv[k] = cx[k] >= 0 && cx[k] < p.SW;
        }
        float acc[R][8];
#pragma unroll
        for (int o = 0; o < R; ++o)
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[o][c] = dwb[sl * 8 + c];
#pragma unroll
        for (int r = 0; r < R + 2; ++r) {
            const int sy = oy_lo - p.dpt + r;
            const bool rv = sy >= sr0 && sy < sr1;
            h8 v[3];
#pragma unroll
            for (int k = 0; k < 3; ++k) v[k] = *((rv && cv[k]) ? plane + (sy - sr0) * p.SW + cx[k] : zslot);
#pragma unroll
            for (int ky = 0; ky < 3; ++ky) {
                const int o = r - ky;
                if (o >= 0 && o < R) {
#pragma unroll
                    for (int k = 0; k < 3; ++k) E::fma8(acc[o], w[ky * 3 + k], v[k]);
                }
            }
        }
        h8 *yout = p.y + ((size_t)sl * p.N + n) * p.OH * p.OW + ox;
#pragma unroll
        for (int o = 0; o < R; ++o) {
            if (oy_lo + o >= oy_hi) break;
            float q[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) q[c] = __builtin_amdgcn_fmed3f(acc[o][c], lo, hi);
            yout[(size_t)(oy_lo + o) * p.OW] = E::pack(q);
        }
    }
}

constexpr int kRows[2] = {4, 2};                  // band heights, one configuration each

int stem_rs(const StemDwParams &p) {
    int rs = ((p.SW - 1) * p.sw + (p.KW - 1) * p.dw + 1) * p.C;
    rs = rs > (p.W + p.pl) * p.C ? rs : (p.W + p.pl) * p.C;
    return (rs + 7) & ~7;
}

bool geometry(const StemDwParams &p, int cfg, StemDwGeom &g) {
    if (cfg < 0 || cfg >= 2) return false;
    const int R = kRows[cfg];
    const int nsl = 2 * p.nb16;
    const int rs = stem_rs(p);
    const int nsr = R + 2 < p.SH ? R + 2 : p.SH;                      // stem rows at most
    const int nrows = (nsr - 1) * p.sh + (p.KH - 1) * p.dh + 1;
    g.rows = R;
    g.nbands = (p.OH + R - 1) / R;
    g.rs = rs;
    g.pstride = nsr * p.SW;
    g.band_h8 = (nrows * rs + 7) / 8;
    g.lds = ((size_t)nsl * g.pstride + g.band_h8 + nsl * 9) * 16 + (size_t)nsl * 8 * 4 + 16;
    return g.lds <= 160 * 1024;
}

template <typename E, typename TIN>
hipError_t launch_t(const StemDwParams &p, int R, size_t lds, hipStream_t st) {
    const dim3 grid(p.N * p.nbands), block(NT);
#define MGI_STEMDW(NB_, R_)                                                                     \
    if (p.nb16 == NB_ && R == R_) {                                                             \
        auto k = stemdw_kernel<E, TIN, NB_, R_>;                                                \
        hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, \
                                           160 * 1024);                                         \
        if (e != hipSuccess) return e;                                                          \
        launch(k, grid, block, (unsigned)lds, st, p);                                           \
        return hipGetLastError();                                                               \
    }
    MGI_STEMDW(1, 4) MGI_STEMDW(1, 2) MGI_STEMDW(2, 4) MGI_STEMDW(2, 2)
    MGI_STEMDW(3, 4) MGI_STEMDW(3, 2) MGI_STEMDW(4, 4) MGI_STEMDW(4, 2)
#undef MGI_STEMDW
    return hipErrorInvalidValue;
}

}  // namespace

int stemdw_configs(const StemDwParams &p, int cfg, StemDwGeom *g, const char **name) {
    static const char *names[2] = {"band4", "band2"};
    if (p.nb16 < 1 || p.nb16 > 4 || p.K > 32 || p.S != 1 || p.SW != p.OW || p.SH != p.OH) return 0;
    int count = 0;
    for (int c = 0; c < 2; ++c) {
        StemDwGeom t{};
        if (!geometry(p, c, t)) continue;
        if (count == cfg) {
            if (g) *g = t;
            if (name) *name = names[c];
        }
        ++count;
    }
    return count;
}

hipError_t launch_stemdw(const StemDwParams &p, int cfg, bool fp16_in, hipStream_t st) {
    if (p.N <= 0) return hipSuccess;
    StemDwGeom g{};
    if (cfg < 0 || cfg >= stemdw_configs(p, -1, nullptr, nullptr) || !stemdw_configs(p, cfg, &g, nullptr))
        return hipErrorInvalidValue;
    StemDwParams q = p;
    im2col_offsets(q.koff, p.K, p.C, p.KW, p.dh, p.dw, g.rs);
    q.nbands = g.nbands;
    q.rs = g.rs;
    q.pstride = g.pstride;
    q.band_h8 = g.band_h8;
    if (p.bf16) return fp16_in ? launch_t<BF16, _Float16>(q, g.rows, g.lds, st) : launch_t<BF16, float>(q, g.rows, g.lds, st);
    return fp16_in ? launch_t<F16, _Float16>(q, g.rows, g.lds, st) : launch_t<F16, float>(q, g.rows, g.lds, st);
}

}  // namespace kern
}  // namespace mgi
