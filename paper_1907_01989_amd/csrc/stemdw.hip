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

// NB channel blocks of 16; R output rows per band; the stem and depthwise
// steps run over groups of G blocks at a time (planes for 2*G slices in LDS:
// G < NB trades a second pass over the band for less LDS, so that more
// workgroups share a compute unit); NT threads per workgroup.
template <typename E, typename TIN, int NB, int R, int G, int NT>
__global__ __launch_bounds__(NT) void stemdw_kernel(StemDwParams p) {
    constexpr int NSL = 2 * NB;                   // channel slices (8 channels each)
    constexpr int NSG = 2 * G;                    // slices of a group (planes in LDS)
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
    // LDS: planes [NSG][pstride] | input band [nrows][rs] halves | taps
    // [NSL][9] | depthwise bias [NSL * 8] fp32 | one zero element
    h8 *planes = lds;
    _Float16 *band = (_Float16 *)(lds + NSG * p.pstride);
    h8 *taps = lds + NSG * p.pstride + p.band_h8;
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

    const float lo = p.act2 == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act2 == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    const int fpr = (p.SW + 15) >> 4;
    const int nfr = nsr * fpr;
    const int sub = 4 * ((lane >> 4) & 1);        // half of a sliced element
#pragma unroll
    for (int g0 = 0; g0 < NB; g0 += G) {
        if (g0 > 0) __syncthreads();              // the previous group's planes are read
        // 2. stem outputs of rows [sr0, sr1) of blocks [g0, g0 + G) into the
        // planes: one 16-pixel fragment per wave step, one MFMA per block
        // over K <= 32 (accumulator = bias)
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
            for (int i = g0; i < g0 + G && i < NB; ++i) {
                const f4 acc = E::mma(a[i], b, c0[i]);
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[r], p.act1);
                if (sx < p.SW)
                    *(h4 *)((_Float16 *)(planes + (2 * (i - g0) + (lane >> 5)) * p.pstride + syl * p.SW + sx) +
                            sub) = E::pack4(v);
            }
        }
        __syncthreads();

        // 3. depthwise 3x3 (stride 1) from the planes: a thread owns one
        // output column of one slice of the group and the band's R rows
        const int sl0 = 2 * g0, nsg = min(NSG, p.ns - sl0);
        const int ntask = nsg * p.OW;
        for (int t = tid; t < ntask; t += NT) {
            const int sg = t / p.OW, ox = t - sg * p.OW;
            const int sl = sl0 + sg;
            const h8 *plane = planes + sg * p.pstride;
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
            float bias[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) bias[c] = dwb[sl * 8 + c];
            float acc[R][8];
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
                        for (int k = 0; k < 3; ++k) {  // (the first tap takes the bias as its addend)
                            if (ky == 0 && k == 0) E::fma8_from(acc[o], bias, w[0], v[0]);
                            else E::fma8(acc[o], w[ky * 3 + k], v[k]);
                        }
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
}

// configurations: band height, channel blocks per group (0 = all), threads
struct Cfg {
    int rows, group, threads;
    const char *name;
};
// (groups of one block with 256 threads, for more workgroups per compute
// unit, measured no faster on the 224 -> 112 stem: the node is bound by
// vector-ALU work, not latency)
constexpr Cfg kCfgs[] = {{4, 0, 512, "band4"}, {2, 0, 512, "band2"}};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

int stem_rs(const StemDwParams &p) {
    int rs = ((p.SW - 1) * p.sw + (p.KW - 1) * p.dw + 1) * p.C;
    rs = rs > (p.W + p.pl) * p.C ? rs : (p.W + p.pl) * p.C;
    return (rs + 7) & ~7;
}

bool geometry(const StemDwParams &p, int cfg, StemDwGeom &g) {
    if (cfg < 0 || cfg >= kNumCfgs) return false;
    const Cfg &c = kCfgs[cfg];
    if (c.group && c.group >= p.nb16) return false;               // same as the full group
    const int R = c.rows;
    const int nsl = 2 * p.nb16, nsg = 2 * (c.group ? c.group : p.nb16);
    const int rs = stem_rs(p);
    const int nsr = R + 2 < p.SH ? R + 2 : p.SH;                      // stem rows at most
    const int nrows = (nsr - 1) * p.sh + (p.KH - 1) * p.dh + 1;
    g.rows = R;
    g.group = c.group ? c.group : p.nb16;
    g.threads = c.threads;
    g.nbands = (p.OH + R - 1) / R;
    g.rs = rs;
    g.pstride = nsr * p.SW;
    g.band_h8 = (nrows * rs + 7) / 8;
    g.lds = ((size_t)nsg * g.pstride + g.band_h8 + nsl * 9) * 16 + (size_t)nsl * 8 * 4 + 16;
    return g.lds <= 160 * 1024;
}

template <typename E, typename TIN>
hipError_t launch_t(const StemDwParams &p, const StemDwGeom &g, hipStream_t st) {
    const dim3 grid(p.N * p.nbands);
#define MGI_STEMDW(NB_, R_, G_, NT_)                                                            \
    if (p.nb16 == NB_ && g.rows == R_ && g.group == G_ && g.threads == NT_) {                    \
        auto k = stemdw_kernel<E, TIN, NB_, R_, G_, NT_>;                                       \
        hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, \
                                           160 * 1024);                                         \
        if (e != hipSuccess) return e;                                                          \
        launch(k, grid, dim3(NT_), (unsigned)g.lds, st, p);                                     \
        return hipGetLastError();                                                               \
    }
#define MGI_STEMDW_NB(NB_) MGI_STEMDW(NB_, 4, NB_, 512) MGI_STEMDW(NB_, 2, NB_, 512)
    MGI_STEMDW_NB(1) MGI_STEMDW_NB(2) MGI_STEMDW_NB(3) MGI_STEMDW_NB(4)
#undef MGI_STEMDW_NB
#undef MGI_STEMDW
    return hipErrorInvalidValue;
}

}  // namespace

int stemdw_configs(const StemDwParams &p, int cfg, StemDwGeom *g, const char **name) {
    if (p.nb16 < 1 || p.nb16 > 4 || p.K > 32 || p.S != 1 || p.SW != p.OW || p.SH != p.OH) return 0;
    int count = 0;
    for (int c = 0; c < kNumCfgs; ++c) {
        StemDwGeom t{};
        if (!geometry(p, c, t)) continue;
        if (count == cfg) {
            if (g) *g = t;
            if (name) *name = kCfgs[c].name;
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
    if (p.bf16) return fp16_in ? launch_t<BF16, _Float16>(q, g, st) : launch_t<BF16, float>(q, g, st);
    return fp16_in ? launch_t<F16, _Float16>(q, g, st) : launch_t<F16, float>(q, g, st);
}

}  // namespace kern
}  // namespace mgi
