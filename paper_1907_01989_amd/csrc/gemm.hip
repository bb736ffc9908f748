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
//     4*(l/16)+r of pixel l%16, half a sliced element; it starts from the
//     bias (in every pointwise kernel, so all of them round alike), and the
//     epilogue applies the activation(s) and the residual and writes 8 bytes
//     per lane.
// Weight and activation tiles for four K slices (32 channels) per step are
// staged through LDS, double-buffered with one barrier per step, the next
// step's global loads issued before the current step's MFMAs.
#include <algorithm>
#include <cmath>

#include "device.h"

namespace mgi {
namespace kern {


template <typename E, int BM, int BN, bool TAPS, bool F32OUT>
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
    for (int i = 0; i < FN; ++i) {
        const f4 b0 = bias_frag(p.bias, nb0 + wn * FN + i, p.nb16, lane);
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = b0;
    }

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
                acc[i][j] = E::mma(a[i], b[j], acc[i][j]);
        if (more) lstore(cur ^ 1);
        __syncthreads();
    }

    // epilogue
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const int nb = nb0 + wn * FN + i;
        if (nb >= p.nb16) continue;
        const int nbase = nb * 16 + 4 * (lane >> 4);
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int m = m0 + wm * WM + j * 16 + (lane & 15);
            if (m >= p.M) continue;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r], p.act1);
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
                    for (int r = 0; r < 4; ++r) v[r] = act_apply(v[r] + E::get4(rv, r), p.act2);
                }
                *(h4 *)((_Float16 *)p.y + off) = E::pack4(v);
            }
        }
    }
}

template <typename E, int BM, int BN>
static hipError_t launch_bm_bn(const GemmParams &p, bool taps, bool f32out, hipStream_t st) {
    GemmParams q = p;
    q.mtiles = (p.M + BM - 1) / BM;
    q.ntiles = (p.nb16 * 16 + BN - 1) / BN;
    const dim3 grid(q.mtiles * q.ntiles), block(256);
    if (f32out) {
        if (taps) return hipErrorInvalidValue;
        launch((gemm_kernel<E, BM, BN, false, true>), grid, block, 0, st, q);
    } else if (taps) {
        launch((gemm_kernel<E, BM, BN, true, false>), grid, block, 0, st, q);
    } else {
        launch((gemm_kernel<E, BM, BN, false, false>), grid, block, 0, st, q);
    }
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmParams &p, int bm, int bn, bool taps, bool f32out,
                       hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
#define MGI_GEMM_CASE(BM_, BN_) \
    if (bm == BM_ && bn == BN_)     \
        return p.bf16 ? launch_bm_bn<BF16, BM_, BN_>(p, taps, f32out, st) : launch_bm_bn<F16, BM_, BN_>(p, taps, f32out, st);
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

// Global average pool of a GEMM tile (pipelined or weight-slab) that holds
// whole images: every output value is rounded to the storage type as a stored
// tensor would be (act1, then round) and staged in LDS as fp32, pixel-major
// [BM][BN] with the channel index XOR-swizzled by the pixel (4 * (px % 8); 4 *
// (px % 4) in a 16-channel tile) so that both the
// accumulator-layout writes and the per-channel reads are free of bank
// conflicts.  A thread then owns one (image, channel) and sums its pixels in
// the global-pool kernel's order (8 partial sums over pixels j, j + 8, ...,
// then pairs (0,4), (2,6), (1,5), (3,7) and their sums, times 1/hw), so the
// fused node equals the GEMM followed by the pool bit for bit; the lane of
// each 8 channels gathers the other seven by shuffles and stores the
// element.  Output: sliced pooled means [ns][nimg].
template <typename E, int BM, int BN, int FM, int FN>
__device__ __forceinline__ void pool_epilogue(const GemmParams &p, const f4 (&acc)[FN][FM], int mt, int nb0,
                                              int px0, int cb0, float *T, int tid, int lane) {
    static_assert(BN % 16 == 0, "whole channel blocks");
    // (the swizzle moves whole 4-channel groups inside their 32 channels, or
    // inside the tile's 16 channels when BN is 16)
    constexpr int PXM = BN >= 32 ? 7 : 3;
    auto at = [](int px, int ch) { return px * BN + (ch ^ (4 * (px & PXM))); };
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const int ch = (cb0 + i) * 16 + 4 * (lane >> 4);
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int px = px0 + j * 16 + (lane & 15);
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r], p.act1);
            const h4 h = E::pack4(v);
            f4 f;
#pragma unroll
            for (int r = 0; r < 4; ++r) f[r] = E::get4(h, r);
            *(f4 *)(T + at(px, ch)) = f;          // 4 channels stay contiguous under the swizzle
        }
    }
    __syncthreads();
    const float inv = 1.0f / (float)p.hw;
    for (int t0 = 0; t0 < p.ipt * BN; t0 += 256) {    // same trip count in every lane (shuffles)
        const int t = t0 + tid;
        const int k = t / BN, ch = t - k * BN;
        const bool live = t < p.ipt * BN;
        const int kk = live ? k : 0;
        float a[8];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
            float sum = 0.0f;
#pragma unroll
            for (int ii = 0; ii < 8; ++ii) {
                const int px = jj + 8 * ii;
                sum += px < p.hw ? T[at(kk * p.hw + min(px, p.hw - 1), ch)] : 0.0f;
            }
            a[jj] = sum;
        }
        const float q = (((a[0] + a[4]) + (a[2] + a[6])) + ((a[1] + a[5]) + (a[3] + a[7]))) * inv;
        float o[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) o[c] = __shfl(q, (lane & ~7) + c);
        const int img = mt * p.ipt + k, os = nb0 * 2 + ch / 8;
        if (live && (ch & 7) == 0 && img < p.nimg && os < p.ns) ((h8 *)p.y)[(size_t)os * p.nimg + img] = E::pack(o);
    }
}

// ---------------------------------------------------------------------------
// Pointwise GEMM, weight-slab variant.  The tile's whole weight slab
// (BN channels x all K, up to 64 KiB where several workgroups share a
// compute unit, up to the whole LDS for grids under one round) is loaded into
// LDS once, behind one barrier; each of the 4 waves then owns WM pixels and
// all BN channels, and
// streams its activation fragments straight from the sliced layout into
// registers, PF K-steps ahead of their use (a ring of PF register sets indexed
// statically by unrolling the K loop by PF).  The K loop has no barrier and no
// load other than the activation stream, so the in-order load counter lets
// PF steps of loads stay in flight.
// ---------------------------------------------------------------------------
// POOL: the output feeds only a global average pool over planes of p.hw <=
// BM pixels; an M-tile then holds p.ipt whole images and the epilogue writes
// the pooled means (pool_epilogue), as in the pipelined kernel.
template <typename E, int WM, int BN, int PF, bool POOL>
__global__ __launch_bounds__(256) void gemm_xs_kernel(GemmParams p) {
    constexpr int FM = WM / 16, FN = BN / 16, BM = 4 * WM;
    extern __shared__ h8 wsm[];                  // [FN][ksp][16]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int mt = tile / p.ntiles, nt = tile - mt * p.ntiles;
    const int m0 = (POOL ? mt * p.ipt * p.hw : mt * BM) + wave * WM, nb0 = nt * FN;
    const int ksteps = p.ksp >> 2;

    // Loads are branch-free (a load under a lane condition becomes an
    // exec-masked branch followed by a wait): a row past the end reads the
    // last row (its results are never stored); a K slice past the end (K not
    // a multiple of 32) reads the last real slice, whose products meet the
    // zero-padded weights of those K positions (exact for finite activations).
    int xm[FM], xmc[FM];
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        xm[j] = m0 + j * 16 + (lane & 15);
        xmc[j] = xm[j] < p.M ? xm[j] : p.M - 1;
    }
    const int xsl = lane >> 4;
    h8 xq[PF][FM];
    auto xload = [&](int kk, h8 *dst) {
        const int ks = min(kk * 4 + xsl, p.ksl - 1);
        const h8 *src = p.x + (size_t)ks * p.M;
#pragma unroll
        for (int j = 0; j < FM; ++j) dst[j] = src[xmc[j]];
    };
#pragma unroll
    for (int u = 0; u < PF; ++u)
        if (u < ksteps) xload(u, xq[u]);

    // accumulators start from the bias (loaded before the weight slab, whose
    // barrier then covers it)
    f4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const f4 b0 = bias_frag(p.bias, nb0 + i, p.nb16, lane);
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = b0;
    }

    // weight slab: FN blocks x ksp slices x 16 rows (blocks past the end are
    // clamped; their accumulators are never stored), 1 KiB per wave load by
    // direct global->LDS loads, all in flight together with the activation
    // prefetch; one wait and one barrier
    const int kq = p.ksp >> 2;                   // KiB loads per block
    for (int q = wave; q < FN * kq; q += 4) {
        const int f = q / kq, r = q - f * kq;
        const int nb = min(nb0 + f, p.nb16 - 1);
        load_lds16(p.w + ((size_t)nb * p.ksp + r * 4) * 16 + lane, wsm + q * 64);
    }
    wait_vm_lds<0>();
    __syncthreads();

    auto step = [&](int kk, const h8 *b) {
        h8 a[FN];
#pragma unroll
        for (int i = 0; i < FN; ++i) a[i] = wsm[(i * p.ksp + kk * 4) * 16 + lane];
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int j = 0; j < FM; ++j)
                acc[i][j] = E::mma(a[i], b[j], acc[i][j]);
    };
    // Main loop over whole groups of PF steps: every step issues exactly FM
    // loads (the prefetch index is clamped instead of skipped), so the wait
    // before each step's MFMAs can leave the newer PF-1 steps in flight.
    int kk0 = 0;
    for (; kk0 + PF <= ksteps; kk0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            step(kk0 + u, xq[u]);
            xload(min(kk0 + u + PF, ksteps - 1), xq[u]);
        }
    }
#pragma unroll
    for (int u = 0; u < PF - 1; ++u)
        if (kk0 + u < ksteps) step(kk0 + u, xq[u]);

    // epilogue tile after the weight slab: per wave, or the pooled tile
    float *stage = (float *)(wsm + FN * p.ksp * 16);
    if constexpr (POOL) {
        pool_epilogue<E, BM, BN, FM, FN>(p, acc, mt, nb0, wave * WM, 0, stage, tid, lane);
        return;
    }
    store_tile_c8<E, FM, FN>(p, acc, m0, nb0, stage + wave * (FN * FM * 256), lane);
}

// LDS bytes of the weight slab for a bn-wide tile (slab plus epilogue tile)
static size_t xs_stage_bytes(int wm, int bn) { return (size_t)4 * (wm / 16) * (bn / 16) * 256 * 4; }
size_t gemm_xs_lds_bytes(int ksp, int wm, int bn) {
    return (size_t)(bn / 16) * ksp * 256 + xs_stage_bytes(wm, bn);
}

constexpr size_t kXsMaxLds = 160 * 1024;

template <typename E, int WM, int BN, int PF, bool POOL>
static hipError_t launch_xs(const GemmParams &p, hipStream_t st) {
    GemmParams q = p;
    constexpr int BM = 4 * WM, FN = BN / 16;
    if (POOL) {
        q.ipt = BM / p.hw;
        q.mtiles = (p.nimg + q.ipt - 1) / q.ipt;
    } else {
        q.mtiles = (p.M + BM - 1) / BM;
    }
    q.ntiles = (p.nb16 + FN - 1) / FN;
    const size_t lds = gemm_xs_lds_bytes(p.ksp, WM, BN);
    if (lds > kXsMaxLds) return hipErrorInvalidValue;
    auto kern = gemm_xs_kernel<E, WM, BN, PF, POOL>;
    if (lds > 65536) {
        static const hipError_t attr =
            hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kXsMaxLds);
        if (attr != hipSuccess) return attr;
    }
    launch(kern, dim3(q.mtiles * q.ntiles), dim3(256), lds, st, q);
    return hipGetLastError();
}

hipError_t launch_gemm_xs(const GemmParams &p, int wm, int bn, int pf, bool pool, hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
    if (p.ksp % 4 != 0) return hipErrorInvalidValue;
    if (pool) {
        // pooled tiles: one image group of planes of at most 64 pixels per
        // 64-row tile (16 pixels per wave)
        if (p.hw < 1 || p.hw > 64 || p.M != p.nimg * p.hw || wm != 16) return hipErrorInvalidValue;
#define MGI_XSP_CASE(BN_, PF_) \
        if (bn == BN_ && pf == PF_) \
            return p.bf16 ? launch_xs<BF16, 16, BN_, PF_, true>(p, st) : launch_xs<F16, 16, BN_, PF_, true>(p, st);
        MGI_XSP_CASE(16, 2) MGI_XSP_CASE(16, 8) MGI_XSP_CASE(32, 2) MGI_XSP_CASE(32, 8)
        MGI_XSP_CASE(64, 2) MGI_XSP_CASE(64, 8)
#undef MGI_XSP_CASE
        return hipErrorInvalidValue;
    }
#define MGI_XS_CASE(WM_, BN_, PF_) \
    if (wm == WM_ && bn == BN_ && pf == PF_) \
        return p.bf16 ? launch_xs<BF16, WM_, BN_, PF_, false>(p, st) : launch_xs<F16, WM_, BN_, PF_, false>(p, st);
#define MGI_XS_PF(WM_, BN_) MGI_XS_CASE(WM_, BN_, 1) MGI_XS_CASE(WM_, BN_, 2) MGI_XS_CASE(WM_, BN_, 4) \
    MGI_XS_CASE(WM_, BN_, 8)
    MGI_XS_CASE(16, 16, 8)
    MGI_XS_PF(16, 32)
    MGI_XS_PF(16, 64)
    MGI_XS_PF(16, 128)
    MGI_XS_PF(32, 32)
    MGI_XS_PF(32, 64)
    MGI_XS_PF(32, 128)
    MGI_XS_PF(64, 32)
    MGI_XS_PF(64, 64)
#undef MGI_XS_PF
#undef MGI_XS_CASE
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Pointwise GEMM, pipelined variant for mid and long K.  Re-reading the
// activations for every 32-channel output block (the weight-slab kernel) costs
// more L2->CU traffic than the per-CU load path delivers once K and the number
// of output channels grow; here a workgroup owns a BM-pixel x BN-channel tile
// (2 x 2 waves of BM/2 x BN/2), so activations are read cout/BN times and
// weights M/BM times.  Both operands go through a ring of NST LDS stages of
// 4 K-slices each, filled by direct global->LDS loads (16 bytes per lane, no
// register staging): a stage's 64 consecutive sliced elements are one wave
// load, and its weight fragments keep the packed per-lane order.  Each
// iteration waits for its own stage (the newer NST-2 stages stay in flight),
// meets the other waves at a barrier, issues the load of the stage NST-1
// ahead into the slot freed by the previous iteration, and runs its MFMAs.
// The loop is unrolled by NST so every slot is a compile-time choice.
// ---------------------------------------------------------------------------
template <int BM, int BN, int KS_ = 4>
struct PipeTile {
    static constexpr int KS = KS_, NST = 4;       // K slices per stage (4 or 8: one or two MFMA K-steps)
    static constexpr int SUB = KS / 4;
    static constexpr int XE = BM * KS, WE = BN * KS;    // 16-byte elements per stage
    static constexpr int XL = XE / 256, WL = WE / 256;  // wave loads per wave per stage
    static constexpr int LPW = XL + WL;
    static_assert(XE % 256 == 0 && WE % 256 == 0, "tile must be a multiple of 64 both ways");
};

template <int BM, int BN, int KS>
__device__ __forceinline__ void pipe_issue(const GemmParams &p, int kk, h8 *st, int m0, int nb0,
                                           int wave, int lane) {
    using T = PipeTile<BM, BN, KS>;
    const int k0 = kk * T::KS;
#pragma unroll
    for (int i = 0; i < T::XL; ++i) {
        const int q = wave * T::XL + i;                  // wave load within the stage
        const int e0 = q * 64, sl = e0 / BM, px = e0 - sl * BM;
        const int ks = min(k0 + sl, p.ksl - 1);          // K tail meets zero weights
        const int m = min(m0 + px + lane, p.M - 1);      // rows past M are never stored
        load_lds16(p.x + (size_t)ks * p.M + m, st + e0);
    }
#pragma unroll
    for (int i = 0; i < T::WL; ++i) {
        const int L = wave * T::WL + i;                  // (output block, K-step) of the stage
        const int q = L / T::SUB, sub = L - q * T::SUB;
        const int nb = min(nb0 + q, p.nb16 - 1);
        load_lds16(p.w + ((size_t)nb * p.ksp + k0 + 4 * sub) * 16 + lane, st + T::XE + L * 64);
    }
}

// POOL: the output feeds only a global average pool over planes of p.hw <=
// BM pixels; an M-tile then holds p.ipt whole images (rows mt * ipt * hw
// on), and the epilogue writes the pooled means instead of the tile (see
// pool_epilogue).
template <typename E, int BM, int BN, bool POOL, int KS = 4>
__global__ __launch_bounds__(256) void gemm_pipe_kernel(GemmParams p) {
    using T = PipeTile<BM, BN, KS>;
    constexpr int WMP = BM / 2, WNC = BN / 2, FM = WMP / 16, FN = WNC / 16;
    static_assert(WMP * WNC * 4 <= (T::XE + T::WE) * 16, "epilogue tile must fit one stage");
    static_assert(!POOL || BM * BN * 4 <= 4 * (T::XE + T::WE) * 16, "pool tile must fit the ring");
    __shared__ h8 ring[4][T::XE + T::WE];
    h8 *st0 = ring[0], *st1 = ring[1], *st2 = ring[2], *st3 = ring[3];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = wave >> 1;
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int mt = tile / p.ntiles, nt = tile - mt * p.ntiles;
    const int m0 = POOL ? mt * p.ipt * p.hw : mt * BM, nb0 = nt * (BN / 16);
    const int nk = p.ksp / T::KS;

    f4 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i) {
        const f4 b0 = bias_frag(p.bias, nb0 + wn * FN + i, p.nb16, lane);
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = b0;
    }

    pipe_issue<BM, BN, KS>(p, 0, st0, m0, nb0, wave, lane);
    if (nk > 1) pipe_issue<BM, BN, KS>(p, 1, st1, m0, nb0, wave, lane);
    if (nk > 2) pipe_issue<BM, BN, KS>(p, 2, st2, m0, nb0, wave, lane);

    auto body = [&](int kk, const h8 *cur, h8 *nxt) {
        // stage kk has landed once at most min(2, nk-1-kk) newer stages are
        // pending; this wave's reads of the previous slot have returned, so
        // after the barrier no wave still reads the slot refilled below
        const int newer = min(2, nk - 1 - kk);
        if (newer >= 2) wait_vm_lds<2 * T::LPW>();
        else if (newer == 1) wait_vm_lds<T::LPW>();
        else wait_vm_lds<0>();
        __builtin_amdgcn_s_barrier();
        if (kk + 3 < nk) pipe_issue<BM, BN, KS>(p, kk + 3, nxt, m0, nb0, wave, lane);
#pragma unroll
        for (int sub = 0; sub < T::SUB; ++sub) {      // MFMA K-steps of the stage, in K order
            h8 a[FN], b[FM];
#pragma unroll
            for (int i = 0; i < FN; ++i) a[i] = cur[T::XE + ((wn * FN + i) * T::SUB + sub) * 64 + lane];
#pragma unroll
            for (int j = 0; j < FM; ++j)
                b[j] = cur[(4 * sub + (lane >> 4)) * BM + wm * WMP + j * 16 + (lane & 15)];
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    acc[i][j] = E::mma(a[i], b[j], acc[i][j]);
        }
    };
    for (int kk = 0; kk < nk; kk += 4) {
        body(kk, st0, st3);
        if (kk + 1 < nk) body(kk + 1, st1, st0);
        if (kk + 2 < nk) body(kk + 2, st2, st1);
        if (kk + 3 < nk) body(kk + 3, st3, st2);
    }

    __syncthreads();
    if (POOL) {
        pool_epilogue<E, BM, BN, FM, FN>(p, acc, mt, nb0, wm * WMP, wn * FN, (float *)&ring[0][0], tid, lane);
        return;
    }
    h8 *stage = wave == 0 ? st0 : wave == 1 ? st1 : wave == 2 ? st2 : st3;
    store_tile_c8<E, FM, FN>(p, acc, m0 + wm * WMP, nb0 + wn * FN, (float *)stage, lane);
}

template <typename E, int BM, int BN>
static hipError_t launch_pipe_t(const GemmParams &p, hipStream_t st) {
    GemmParams q = p;
    q.mtiles = (p.M + BM - 1) / BM;
    q.ntiles = (p.nb16 * 16 + BN - 1) / BN;
    launch((gemm_pipe_kernel<E, BM, BN, false>), dim3(q.mtiles * q.ntiles), dim3(256), 0, st, q);
    return hipGetLastError();
}

template <typename E, int BM, int BN>
static hipError_t launch_pipe_pool_t(const GemmParams &p, hipStream_t st) {
    GemmParams q = p;
    q.ipt = BM / p.hw;
    q.mtiles = (p.nimg + q.ipt - 1) / q.ipt;
    q.ntiles = (p.nb16 * 16 + BN - 1) / BN;
    launch((gemm_pipe_kernel<E, BM, BN, true>), dim3(q.mtiles * q.ntiles), dim3(256), 0, st, q);
    return hipGetLastError();
}

hipError_t launch_gemm_pool(const GemmParams &p, int bm, int bn, hipStream_t st) {
    if (p.nimg <= 0) return hipSuccess;
    if (p.ksp % 4 != 0 || p.Min != p.M || p.hw < 1 || p.hw > bm || p.hw > 64 || p.M != p.nimg * p.hw)
        return hipErrorInvalidValue;
    if (bm == 64 && bn == 64) return p.bf16 ? launch_pipe_pool_t<BF16, 64, 64>(p, st) : launch_pipe_pool_t<F16, 64, 64>(p, st);
    if (bm == 64 && bn == 128) return p.bf16 ? launch_pipe_pool_t<BF16, 64, 128>(p, st) : launch_pipe_pool_t<F16, 64, 128>(p, st);
    if (bm == 128 && bn == 64) return p.bf16 ? launch_pipe_pool_t<BF16, 128, 64>(p, st) : launch_pipe_pool_t<F16, 128, 64>(p, st);
    if (bm == 128 && bn == 128) return p.bf16 ? launch_pipe_pool_t<BF16, 128, 128>(p, st) : launch_pipe_pool_t<F16, 128, 128>(p, st);
    return hipErrorInvalidValue;
}

template <typename E>
static hipError_t launch_pipe_k8_t(const GemmParams &p, bool pool, hipStream_t st) {
    GemmParams q = p;
    q.ntiles = (p.nb16 * 16 + 63) / 64;
    if (pool) {
        q.ipt = 64 / p.hw;
        q.mtiles = (p.nimg + q.ipt - 1) / q.ipt;
        launch((gemm_pipe_kernel<E, 64, 64, true, 8>), dim3(q.mtiles * q.ntiles), dim3(256), 0, st, q);
    } else {
        q.mtiles = (p.M + 63) / 64;
        launch((gemm_pipe_kernel<E, 64, 64, false, 8>), dim3(q.mtiles * q.ntiles), dim3(256), 0, st, q);
    }
    return hipGetLastError();
}

// 64x64 tiles with 8 K slices (two MFMA K-steps) per ring stage: twice the
// bytes in flight per workgroup, for long-K GEMMs with few tiles
hipError_t launch_gemm_pipe_k8(const GemmParams &p, bool pool, hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
    if (p.ksp % 8 != 0 || p.Min != p.M) return hipErrorInvalidValue;
    if (pool && (p.hw < 1 || p.hw > 64 || p.M != p.nimg * p.hw)) return hipErrorInvalidValue;
    return p.bf16 ? launch_pipe_k8_t<BF16>(p, pool, st) : launch_pipe_k8_t<F16>(p, pool, st);
}

hipError_t launch_gemm_pipe(const GemmParams &p, int bm, int bn, hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
    if (p.ksp % 4 != 0 || p.Min != p.M) return hipErrorInvalidValue;
    if (bm == 64 && bn == 64) return p.bf16 ? launch_pipe_t<BF16, 64, 64>(p, st) : launch_pipe_t<F16, 64, 64>(p, st);
    if (bm == 64 && bn == 128) return p.bf16 ? launch_pipe_t<BF16, 64, 128>(p, st) : launch_pipe_t<F16, 64, 128>(p, st);
    if (bm == 128 && bn == 64) return p.bf16 ? launch_pipe_t<BF16, 128, 64>(p, st) : launch_pipe_t<F16, 128, 64>(p, st);
    if (bm == 128 && bn == 128) return p.bf16 ? launch_pipe_t<BF16, 128, 128>(p, st) : launch_pipe_t<F16, 128, 128>(p, st);
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Fully-connected layer (1x1 spatial input, fp32 logits out).  M (images) is
// small and K long, so a workgroup takes 16 output channels for up to 16*FM
// images and splits K over its 4 waves; each wave loads B K-steps of weight
// and activation fragments at once, straight from global memory, and the four
// fp32 partial tiles are summed through LDS in a fixed wave order.
// With SM, the softmax of the rows follows in the same launch: every
// workgroup publishes its logits (device-scope release fences) and counts
// itself in on its row tile's counter; the one that arrives last (the
// p.nb16-th) takes the acquire fence -- only it, so the others keep their
// cached weights -- puts the counter back to zero for the next launch and
// runs the softmax of the tile's rows with the standalone kernel's row
// routine.  No workgroup waits for another.
// ---------------------------------------------------------------------------
// s_waitcnt immediate that waits for every outstanding vector memory
// operation of the wave (vmcnt 0; expcnt and lgkmcnt left at their maxima)
constexpr int kWaitVmcnt0 = 0x0F70;

template <typename E, int FM, int B, bool SM>
__global__ __launch_bounds__(256) void fc_kernel(GemmParams p) {
    __shared__ f4 red[4][FM][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // the row tiles of one 16-channel weight block are neighbouring tiles,
    // which xcd_tile puts on one XCD: each weight block is read into one L2
    const int mtiles = gridDim.x / p.nb16, t = xcd_tile(blockIdx.x, gridDim.x);
    const int nb = t / mtiles, mt = t - nb * mtiles;
    const int m0 = mt * 16 * FM;
    const int ksteps = p.ksp >> 2;
    const int per = (ksteps + 3) >> 2;
    const int s0 = min(wave * per, ksteps), s1 = min(s0 + per, ksteps);
    int xmc[FM];
#pragma unroll
    for (int j = 0; j < FM; ++j) xmc[j] = min(m0 + j * 16 + (lane & 15), p.M - 1);
    const h8 *wrow = p.w + (size_t)nb * p.ksp * 16 + lane;
    f4 acc[FM];
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[j] = f4{0.f, 0.f, 0.f, 0.f};
    for (int s = s0; s < s1; s += B) {
        h8 xa[B][FM], wa[B];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int kk = min(s + b, s1 - 1);
            const int ks = min(kk * 4 + (lane >> 4), p.ksl - 1);
#pragma unroll
            for (int j = 0; j < FM; ++j) xa[b][j] = p.x[(size_t)ks * p.M + xmc[j]];
            wa[b] = wrow[(size_t)kk * 64];
        }
#pragma unroll
        for (int b = 0; b < B; ++b)
            if (s + b < s1) {
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    acc[j] = E::mma(wa[b], xa[b][j], acc[j]);
            }
    }
#pragma unroll
    for (int j = 0; j < FM; ++j) red[wave][j][lane] = acc[j];
    __syncthreads();
    for (int j = wave; j < FM; j += 4) {
        const f4 v = red[0][j][lane] + red[1][j][lane] + red[2][j][lane] + red[3][j][lane];
        const int m = m0 + j * 16 + (lane & 15);
        if (m >= p.M) continue;
        const int nbase = nb * 16 + 4 * (lane >> 4);
        float *y = (float *)p.y + (size_t)m * p.cout;
#pragma unroll
        for (int r = 0; r < 4; ++r)
            if (nbase + r < p.cout) y[nbase + r] = act_apply(v[r] + p.bias[nbase + r], p.act1);
    }
    if constexpr (SM) {
        __shared__ int last;
        // each wave waits for its logit stores to complete in the L2 (a
        // workgroup barrier alone does not wait for them); after the barrier
        // one release fence writes the L2 back for the whole workgroup, then
        // one arrival per workgroup
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (threadIdx.x == 0) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            last = atomicAdd(p.sm_cnt + mt, 1) == p.nb16 - 1;
        }
        __syncthreads();
        if (!last) return;
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");         // every logit of the tile is visible
        if (threadIdx.x == 0) atomicExch(p.sm_cnt + mt, 0);        // (every access to a counter is atomic)
        const float *z = (const float *)p.y + (size_t)m0 * p.cout;
        float *prob = p.sm_y + (size_t)m0 * p.cout;
        const int rows = min(16 * FM, p.M - m0);
        if (p.cout <= kSoftmaxRegCols) {
            // rows wave, wave + 4, ...: a wave loads up to four rows before
            // finishing any (one memory round trip per four rows)
            for (int r0 = wave; r0 < rows; r0 += 16) {
                float v[4][kSoftmaxPer];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (r0 + 4 * u < rows) softmax_load(z + (size_t)(r0 + 4 * u) * p.cout, p.cout, lane, v[u]);
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (r0 + 4 * u < rows) softmax_finish(v[u], prob + (size_t)(r0 + 4 * u) * p.cout, p.cout, lane);
            }
        } else {
            for (int r = wave; r < rows; r += 4)
                softmax_row(z + (size_t)r * p.cout, prob + (size_t)r * p.cout, p.cout, lane);
        }
    }
}

hipError_t launch_fc(const GemmParams &p, int fm, int kb, hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
    if (fm <= 0) fm = p.M <= 16 ? 1 : (p.M <= 32 ? 2 : 4);
    if (kb <= 0) kb = 4;
    const int mtiles = (p.M + 16 * fm - 1) / (16 * fm);
    const dim3 grid(mtiles * p.nb16), block(256);
    const bool sm = p.sm_y != nullptr;
    if (sm && !p.sm_cnt) return hipErrorInvalidValue;
#define MGI_FC_CASE(FM_, KB_)                                                              \
    if (fm == FM_ && kb == KB_) {                                                           \
        if (p.bf16 && sm) launch((fc_kernel<BF16, FM_, KB_, true>), grid, block, 0, st, p);  \
        else if (p.bf16) launch((fc_kernel<BF16, FM_, KB_, false>), grid, block, 0, st, p);  \
        else if (sm) launch((fc_kernel<F16, FM_, KB_, true>), grid, block, 0, st, p);        \
        else launch((fc_kernel<F16, FM_, KB_, false>), grid, block, 0, st, p);               \
        return hipGetLastError();                                                           \
    }
    MGI_FC_CASE(1, 4) MGI_FC_CASE(2, 4) MGI_FC_CASE(4, 4)
    MGI_FC_CASE(1, 8) MGI_FC_CASE(2, 8) MGI_FC_CASE(4, 8)
#undef MGI_FC_CASE
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Stem: a convolution that reads the NHWC graph input directly (no layout
// conversion of the input, Sec. 3.2), for windows with kh*kw*c <= 32 so the
// whole window is one MFMA K step.  A workgroup owns one image and a band of
// th output rows: it first stages the input rows of the band into LDS as
// fp16 (coalesced loads of whole input rows; rows outside the image and the
// padding columns are written as zeros), then each lane builds its B
// fragment -- im2col entries k = 8*(l/16) .. +7 of pixel l%16 -- from LDS and
// runs one MFMA per output block of 16 channels.  Entries k >= kh*kw*c read
// any staged value: their weights are zero.
// ---------------------------------------------------------------------------
template <typename E, typename TIN, int NB>
__global__ __launch_bounds__(256) void stem_kernel(StemParams p, int th, int rs, int nrows) {
    extern __shared__ _Float16 band[];           // [nrows][rs] 16-bit storage values
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int bands = (p.OH + th - 1) / th;
    const int n = blockIdx.x / bands, oy0 = (blockIdx.x - n * bands) * th;
    const int iy0 = oy0 * p.sh - p.pt;
    // weights and bias first, then the input rows of the band (all of the
    // workgroup's loads in flight together)
    h8 a[NB];
    f4 c0[NB];                                   // accumulators start from the bias
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        a[i] = p.w[(size_t)i * 64 + lane];
        c0[i] = bias_frag(p.bias, i, p.nb16, lane);
    }
    stage_input_band<E, TIN, 256, 4>(band, (const TIN *)p.x, n, p.H, p.W, p.C, iy0, nrows, rs, p.pl * p.C, tid);
    // offsets of the lane's 8 im2col entries inside a window
    int koff[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) koff[t] = p.koff[8 * (lane >> 4) + t];
    __syncthreads();

    // each wave parks a fragment's act1(acc) in its own LDS tile [2*NB
    // slices][16 pixels][8] fp32 behind the band, then re-reads it so that
    // consecutive lanes own consecutive pixels of one slice: residual reads
    // and output writes are whole 16-byte elements (a lane's 4 channels alone
    // would make half-masked writes)
    constexpr int NSL = 2 * NB;
    float *stg = (float *)(band + nrows * rs) + wave * (NSL * 16 * 8);
    const int fpr = (p.OW + 15) >> 4;            // 16-pixel fragments per output row
    const int nfr = min(th, p.OH - oy0) * fpr;
    int oyl = wave / fpr, fx = wave - oyl * fpr;  // fragment f = oyl * fpr + fx, stepped below
    for (int f = wave; f < nfr; f += 4, fx += 4) {
        while (fx >= fpr) {
            fx -= fpr;
            ++oyl;
        }
        const int ox0 = fx * 16;
        const int ox = ox0 + (lane & 15);
        const int base = oyl * p.sh * rs + min(ox, p.OW - 1) * p.sw * p.C;
        h8 b;
#pragma unroll
        for (int t = 0; t < 8; ++t) b[t] = band[base + koff[t]];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const f4 acc = E::mma(a[i], b, c0[i]);
            f4 v;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[r], p.act1);
            const int sl = 2 * i + (lane >> 5), half = 4 * ((lane >> 4) & 1);
            *(f4 *)(stg + (sl * 16 + (lane & 15)) * 8 + half) = v;
        }
        __builtin_amdgcn_wave_barrier();
        const size_t m0 = (size_t)(n * p.OH + oy0 + oyl) * p.OW + ox0;
#pragma unroll
        for (int t = 0; t < (NSL * 16 + 63) / 64; ++t) {
            const int e = lane + 64 * t;
            const int sl = e >> 4, px = e & 15;
            if (e >= NSL * 16 || sl >= p.ns || ox0 + px >= p.OW) continue;
            const f4 lo = *(const f4 *)(stg + e * 8), hi = *(const f4 *)(stg + e * 8 + 4);
            float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            const size_t off = (size_t)sl * p.M + m0 + px;
            if (p.res) {
                const h8 rv = p.res[off];
#pragma unroll
                for (int r = 0; r < 8; ++r) v[r] = act_apply(v[r] + E::get(rv, r), p.act2);
            }
            p.y[off] = E::pack(v);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

int stem_row_stride(int c, int w, int ow, int sw, int kh, int kw, int dw, int pl) {
    int rs = ((ow - 1) * sw + (kw - 1) * dw + 1) * c;
    rs = rs > (w + pl) * c ? rs : (w + pl) * c;
    if (stem_row_aligned(kh, kw, c, dw) && rs < (ow - 1) * sw * c + 10) rs = (ow - 1) * sw * c + 10;
    return (rs + 7) & ~7;
}

size_t stem_band_bytes(int th, int kh, int kw, int c, int w, int ow, int sh, int sw, int dh, int dw,
                       int pl) {
    const int nrows = (th - 1) * sh + (kh - 1) * dh + 1;
    return (size_t)nrows * stem_row_stride(c, w, ow, sw, kh, kw, dw, pl) * 2;
}

#ifndef MGI_STEM_ROWS
#define MGI_STEM_ROWS 4
#endif
constexpr int kStemRows = MGI_STEM_ROWS;

template <typename E, typename TIN>
static hipError_t launch_stem_t(const StemParams &p, hipStream_t st) {
    // band of th output rows: enough workgroups to fill the chip when possible
    // and a band that fits 64 KiB of LDS
    int th = kStemRows;
    while (th > 1 && (size_t)p.N * ((p.OH + th - 1) / th) < 1024) th >>= 1;
    while (th > 1 && stem_band_bytes(th, p.KH, p.KW, p.C, p.W, p.OW, p.sh, p.sw, p.dh, p.dw, p.pl) +
                             kStemStageBytes > 65536)
        th >>= 1;
    const int nrows = (th - 1) * p.sh + (p.KH - 1) * p.dh + 1;
    const int rs = stem_row_stride(p.C, p.W, p.OW, p.sw, p.KH, p.KW, p.dw, p.pl);
    const size_t lds = (size_t)nrows * rs * 2 + (size_t)4 * p.nb16 * 1024;   // band + per-wave staging
    if (lds > 65536 || p.K > 32) return hipErrorInvalidValue;
    StemParams q = p;
    im2col_offsets(q.koff, p.K, p.KH, p.C, p.KW, p.dh, p.dw, rs);
    const dim3 grid(p.N * ((p.OH + th - 1) / th)), block(256);
    switch (p.nb16) {
        case 1: launch((stem_kernel<E, TIN, 1>), grid, block, lds, st, q, th, rs, nrows); break;
        case 2: launch((stem_kernel<E, TIN, 2>), grid, block, lds, st, q, th, rs, nrows); break;
        case 3: launch((stem_kernel<E, TIN, 3>), grid, block, lds, st, q, th, rs, nrows); break;
        case 4: launch((stem_kernel<E, TIN, 4>), grid, block, lds, st, q, th, rs, nrows); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

bool stem_row_aligned(int KH, int KW, int C, int dw) { return KH == 3 && KW * C == 9 && dw == 1; }

int stem_kpos(int ky, int kx, int ci, int KH, int KW, int C, int dw) {
    const int e = kx * C + ci;                   // entry within the window row
    if (!stem_row_aligned(KH, KW, C, dw)) return ky * KW * C + e;
    return e < 8 ? 8 * ky + e : 24 + 2 * ky;
}

void im2col_offsets(int *koff, int K, int KH, int C, int KW, int dh, int dw, int rs) {
    const bool ra = stem_row_aligned(KH, KW, C, dw);
    for (int k = 0; k < 32; ++k) {
        int off = 0;
        if (ra) {
            // 8 values of row k / 8, or (from 24) the 9th and 10th value of
            // rows 0, 1, 2, 2
            const int ky = k < 24 ? k / 8 : std::min((k - 24) / 2, 2);
            const int e = k < 24 ? k % 8 : 8 + (k - 24) % 2;
            off = ky * dh * rs + e;
        } else if (k < K) {
            const int tap = k / C, ci = k - tap * C;
            const int ky = tap / KW, kx = tap - ky * KW;
            off = ky * dh * rs + kx * dw * C + ci;
        }
        koff[k] = off;
    }
}

hipError_t launch_stem(const StemParams &p, bool fp16_in, hipStream_t st) {
    if (p.M <= 0) return hipSuccess;
    if (p.bf16) return fp16_in ? launch_stem_t<BF16, _Float16>(p, st) : launch_stem_t<BF16, float>(p, st);
    return fp16_in ? launch_stem_t<F16, _Float16>(p, st) : launch_stem_t<F16, float>(p, st);
}

}  // namespace kern
}  // namespace mgi
