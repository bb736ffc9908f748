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
#include <type_traits>

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

// ---------------------------------------------------------------------------
// Rolling strips.  A workgroup owns a strip of `srows` output rows of one
// image and walks down it R output rows per step.  Stem rows live in a ring of
// Q = 2R + 2 row slots and input rows in a ring of `qi` slots, so each stem row
// of the strip is computed once (only the rows just above and below a strip
// are computed by both strips that read them) and each step needs one
// barrier.  Step k of the stem produces the rows the depthwise outputs of step
// k read for the first time; in the loop, phase j
//   - issues the global loads of the input rows stem step j + 2 adds,
//   - computes stem step j + 1 (input ring -> stem ring),
//   - computes the depthwise outputs of step j (stem ring -> output),
//   - stores the loaded input rows into the input ring,
// then waits at the barrier.  The rings are large enough that what a phase
// writes never overlaps what it reads.
//
// The stem window must be row-aligned (3 rows of 9 values, see
// stem_row_aligned) with an even number of values between neighbouring
// windows: a lane's 8 im2col values of one window row are 4 aligned 32-bit
// words of the staged row (the 9th values of the three rows, plus the value
// after each, are one word per row for the fourth lane group), so the
// gather is 4 LDS reads per fragment.  Arithmetic is that of the stem and
// depthwise kernels (same K positions, accumulation orders and rounding
// points), so results are bit-identical to the other configurations.
// ---------------------------------------------------------------------------
template <typename E, typename TIN, int NB, int NT, int R, int SH_, int UMAX>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(4))) void stemdw_roll_kernel(
    StemDwParams p) {   // 4 waves per SIMD: <= 128 VGPRs
    constexpr int NSL = 2 * NB, NWV = NT / 64, Q = 2 * R + 2;
    constexpr int QI = (2 * R - 1) * SH_ + 3;                // input rows held: two steps' worth
    constexpr int VN = 16 / sizeof(TIN);                     // input values per 16-byte load
    extern __shared__ h8 lds[];
    const int rs = p.rs, SW = p.SW;
    const bool vec = p.vec != 0;
    // stem-row ring: [NSL][Q][RW], row x at column x + dpl, the columns
    // around it zero (the depthwise step's horizontal padding)
    const int RW = SW + 2;
    h8 *ring = lds;
    _Float16 *inr = (_Float16 *)(lds + NSL * Q * RW);        // [QI][rs]
    h8 *taps = (h8 *)(inr + (size_t)QI * rs);                // [NSL][9]
    float *dwb = (float *)(taps + NSL * 9);                  // [NSL * 8]
    float *sbias = dwb + NSL * 8;                            // stem bias [NB * 16]
    h8 *zslot = (h8 *)(sbias + NB * 16);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int n = tile / p.nbands, strip = tile - n * p.nbands;
    const int o_lo = strip * p.srows, o_hi = min(p.OH, o_lo + p.srows);
    const int nsteps = (o_hi - o_lo + R - 1) / R;
    const int s_org = o_lo - p.dpt;                          // stem row of ring row 0
    const int s_cap = min(p.SH, o_hi - p.dpt + 2);           // no output of the strip reads past it
    const int i_org = s_org * SH_ - p.pt;                    // input row of input-ring row 0
    // stem step k: rows [sb(k), se(k)); input rows it reads: [ib(k), ie(k))
    auto ub = [&](int k) { return k == 0 ? s_org : s_org + k * R + 2; };   // rows written to the ring
    auto ue = [&](int k) { return s_org + (k + 1) * R + 2; };
    auto sb = [&](int k) { return max(0, ub(k)); };                         // rows computed
    auto se = [&](int k) { return min(s_cap, ue(k)); };
    auto ib = [&](int k) { return sb(k) * SH_ - p.pt; };
    auto ie = [&](int k) { return max(ib(k), (se(k) - 1) * SH_ - p.pt + 3); };
    const int rowlen = p.W * p.C, lead = p.pl * p.C;
    const int upr = vec ? rowlen / VN : rowlen;              // load units per input row
    const TIN *xin = (const TIN *)p.x + (size_t)n * p.H * rowlen;

    // weights (held in registers), taps and biases (in LDS: the stem bias
    // fragments are read again per fragment, which keeps the register count
    // at the 4-wave limit); zero columns of every input-ring slot
    h8 a[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) a[i] = p.w[(size_t)i * 64 + lane];
    if (tid < NSL * 9) taps[tid] = p.dw_w[tid];
    if (tid < NSL * 8) dwb[tid] = p.dw_b[tid];
    if (tid < NB * 16) sbias[tid] = p.bias[tid];
    if (tid == 0) *zslot = zero_h8();
    for (int e = tid; e < NSL * Q * 2; e += NT) {
        const int r = e >> 1, c = (e & 1) ? SW + p.dpl : 0;   // zero columns of ring row r
        for (int x = c; x < ((e & 1) ? RW : p.dpl); ++x) ring[r * RW + x] = zero_h8();
    }
    {
        uint16_t *b16 = (uint16_t *)inr;
        const int zc = rs - rowlen;                          // lead + tail columns per slot
        for (int e = tid; e < QI * zc; e += NT) {
            const int r = e / zc, c = e - r * zc;
            b16[r * rs + (c < lead ? c : rowlen + c)] = 0;
        }
    }

    // input staging: rows [r0, r1) into their ring slots; unit e of the range
    // = value group e % upr of row r0 + e / upr (a thread's units are e = tid
    // + u * NT, their row and column offsets computed once); rows outside the
    // image are zeros.  The first UMAX * NT units go through registers
    // (stage_issue, then stage_store) when they are 16-byte vectors; any rest,
    // and every single-value unit, is copied in stage_store.
    typedef TIN tv __attribute__((ext_vector_type(VN)));
    tv reg[UMAX];
    int urow[UMAX], ucol[UMAX];
#pragma unroll
    for (int u = 0; u < UMAX; ++u) {
        urow[u] = (tid + u * NT) / upr;
        ucol[u] = (tid + u * NT) - urow[u] * upr;
    }
    auto src_of = [&](int r, int c) {
        return xin + (size_t)min(max(r, 0), p.H - 1) * rowlen + (vec ? c * VN : c);
    };
    // fp16 input into fp16 planes: the conversion through fp32 is the identity
    // on finite values, so the 16 bytes are copied as they are
    constexpr bool raw = std::is_same<E, F16>::value && std::is_same<TIN, _Float16>::value;
    auto put = [&](int r, int c, const tv &v) {
        const bool inside = r >= 0 && r < p.H;
        _Float16 *dst = inr + ((unsigned)(r - i_org) % QI) * rs + lead;   // r >= i_org
        if (raw && vec) {
            const tv z = {};
            *(tv *)(dst + c * VN) = inside ? v : z;
        } else if (vec) {
            float f[VN];
#pragma unroll
            for (int i = 0; i < VN; ++i) f[i] = inside ? (float)v[i] : 0.0f;
            if constexpr (VN == 8) *(h8 *)(dst + c * 8) = E::pack(f);
            else *(h4 *)(dst + c * 4) = E::pack4(f);
        } else {
            ((uint16_t *)dst)[c] = E::bits(inside ? (float)v[0] : 0.0f);
        }
    };
    // (only 16-byte units go through registers: a load whose destination
    // depends on a run-time choice of unit size would be merged by register
    // copies right after it, which wait for the load to return)
    auto stage_issue = [&](int r0, int r1) {
        if (!vec) return;
#pragma unroll
        for (int u = 0; u < UMAX; ++u)
            if (urow[u] < r1 - r0) reg[u] = *(const tv *)src_of(r0 + urow[u], ucol[u]);
    };
    auto stage_store = [&](int r0, int r1) {
        if (vec) {
#pragma unroll
            for (int u = 0; u < UMAX; ++u)
                if (urow[u] < r1 - r0) put(r0 + urow[u], ucol[u], reg[u]);
        }
        const int total = (r1 - r0) * upr;
        for (int e = tid + (vec ? UMAX * NT : 0); e < total; e += NT) {
            const int rr = e / upr, c = e - rr * upr;
            const TIN *src = src_of(r0 + rr, c);
            tv v;
            if (vec) v = *(const tv *)src;
            else v[0] = *src;
            put(r0 + rr, c, v);
        }
    };

    // stem step: rows [s0, s1) into the ring, one 16-pixel fragment per wave
    // iteration (the last waves first: they have no depthwise task when
    // NSL * OW < NT), one MFMA per channel block; rows above and below the
    // stem output are written as zeros (the depthwise step's vertical
    // padding), rows that no stored output reads are skipped.  The
    // fragment's row and column are wave-uniform and stepped without division.
    const int fpr = (SW + 15) >> 4;
    const int q = lane >> 4;
    const int cstep = p.sw * p.C * 2;                        // bytes between neighbouring windows
    const int wv = NWV - 1 - wave;
    auto stem_step = [&](int s0, int s1) {
        int srow = s0 + wv / fpr, fx = wv - (wv / fpr) * fpr;
        for (; srow < s1; fx += NWV) {
            while (fx >= fpr) {
                fx -= fpr;
                ++srow;
            }
            if (srow >= s1) break;
            const int sxr = fx * 16 + (lane & 15);
            h4 *dst = (h4 *)((_Float16 *)(ring + ((lane >> 5) * Q + (srow - s_org) % Q) * RW + sxr + p.dpl) +
                             4 * (q & 1));
            if (srow < 0 || srow >= p.SH) {
                if (sxr < SW) {
                    float z[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int i = 0; i < NB; ++i) dst[(size_t)i * 2 * Q * RW * 2] = E::pack4(z);
                }
                continue;
            }
            if (srow >= s_cap) continue;
            const int r0 = srow * SH_ - p.pt - i_org;
            const int rb0 = (r0 % QI) * rs * 2, rb1 = ((r0 + 1) % QI) * rs * 2, rb2 = ((r0 + 2) % QI) * rs * 2;
            const char *base = (const char *)inr + min(sxr, SW - 1) * cstep;
            u4x w4;
            if (q < 3) {
                const uint32_t *src = (const uint32_t *)(base + (q == 0 ? rb0 : (q == 1 ? rb1 : rb2)));
                w4[0] = src[0]; w4[1] = src[1]; w4[2] = src[2]; w4[3] = src[3];
            } else {
                w4[0] = *(const uint32_t *)(base + rb0 + 16);
                w4[1] = *(const uint32_t *)(base + rb1 + 16);
                w4[2] = *(const uint32_t *)(base + rb2 + 16);
                w4[3] = w4[2];
            }
            const h8 b = __builtin_bit_cast(h8, w4);
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                const f4 acc = E::mma(a[i], b, *(const f4 *)(sbias + i * 16 + 4 * q));
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[r], p.act1);
                if (sxr < SW) dst[(size_t)i * 2 * Q * RW * 2] = E::pack4(v);
            }
        }
    };

    // the depthwise task of this thread (at most one: NSL * OW <= NT): slice
    // sg, output column ox, with its taps and bias held for the whole strip
    const float lo = p.act2 == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act2 == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    const int ntask = min(NSL, p.ns) * p.OW;
    const bool has_task = tid < ntask;
    const int sg = has_task ? tid / p.OW : 0, ox = tid - sg * p.OW;
    h8 w[9];
    float bias[8];
    if (has_task) {
#pragma unroll
        for (int kk = 0; kk < 9; ++kk) w[kk] = p.dw_w[sg * 9 + kk];
#pragma unroll
        for (int c = 0; c < 8; ++c) bias[c] = p.dw_b[sg * 8 + c];
    }
    const h8 *col = ring + (size_t)sg * Q * RW + ox;         // ring column ox = stem column ox - dpl
    h8 *yout = p.y + ((size_t)sg * p.N + n) * p.OH * p.OW + ox;
    auto dw_step = [&](int j) {
        if (!has_task) return;
        const int o0 = o_lo + j * R;
        const int slot0 = (j * R) % Q;
        float acc[R][8];
#pragma unroll
        for (int r = 0; r < R + 2; ++r) {
            const int slot = slot0 + r < Q ? slot0 + r : slot0 + r - Q;
            const h8 *row = col + slot * RW;
            h8 v[3];
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) v[kk] = row[kk];
#pragma unroll
            for (int ky = 0; ky < 3; ++ky) {
                const int o = r - ky;
                if (o >= 0 && o < R) {
#pragma unroll
                    for (int kk = 0; kk < 3; ++kk) {  // (the first tap takes the bias as its addend)
                        if (ky == 0 && kk == 0) E::fma8_from(acc[o], bias, w[0], v[0]);
                        else E::fma8(acc[o], w[ky * 3 + kk], v[kk]);
                    }
                }
            }
        }
#pragma unroll
        for (int o = 0; o < R; ++o) {
            if (o0 + o >= o_hi) break;
            float qv[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) qv[c] = __builtin_amdgcn_fmed3f(acc[o][c], lo, hi);
            yout[(size_t)(o0 + o) * p.OW] = E::pack(qv);
        }
    };

    // prologue: input rows of stem step 0; stem step 0 while the input rows
    // of step 1 load; those rows into the ring
    stage_issue(ib(0), ie(0));
    stage_store(ib(0), ie(0));
    if (nsteps > 1) stage_issue(ie(0), ie(1));
    __syncthreads();
    stem_step(ub(0), ue(0));
    __syncthreads();
    if (nsteps > 1) stage_store(ie(0), ie(1));
    // (every load of the prologue has returned here; waiting for them in so
    // many words keeps the loop's waits to the loads the loop issues, instead
    // of waits for the weight, tap and bias registers that the compiler
    // cannot prove loaded and so places after each step's row loads)
    wait_vm_lds<0>();
    __syncthreads();
    for (int j = 0; j < nsteps; ++j) {
        const bool more = j + 2 < nsteps;
        if (more) stage_issue(ie(j + 1), ie(j + 2));
        if (j + 1 < nsteps) stem_step(ub(j + 1), ue(j + 1));
        dw_step(j);
        if (more) stage_store(ie(j + 1), ie(j + 2));
        // (the staging registers count as read on every path, so that the
        // next step's loads into them wait for nothing)
#pragma unroll
        for (int u = 0; u < UMAX; ++u) asm volatile("" ::"v"(reg[u]));
        __syncthreads();
    }
}

// configurations: band height, channel blocks per group (0 = all), threads;
// or (roll) rolling strips of `rows` output rows walked R = `step` rows at a
// time (with `prod` waves that only compute stem rows while the others only
// compute depthwise outputs, or 0: every wave does both)
struct Cfg {
    int rows, group, threads, roll, step, prod;
    const char *name;
};
// (groups of one block with 256 threads, for more workgroups per compute
// unit, measured no faster on the 224 -> 112 stem: the node is bound by
// vector-ALU work, not latency)
constexpr Cfg kCfgs[] = {{4, 0, 512, 0, 0, 0, "band4"}, {2, 0, 512, 0, 0, 0, "band2"},
                         {14, 0, 512, 1, 2, 0, "roll14"}, {15, 0, 512, 1, 3, 0, "roll15r3"},
                         {28, 0, 512, 1, 2, 0, "roll28"}};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);
constexpr int kRollUnits = 2;      // input load units per thread held across a phase

int stem_rs(const StemDwParams &p) { return stem_row_stride(p.C, p.W, p.SW, p.sw, p.KH, p.KW, p.dw, p.pl); }

bool geometry(const StemDwParams &p, int cfg, bool fp16_in, StemDwGeom &g) {
    if (cfg < 0 || cfg >= kNumCfgs) return false;
    const Cfg &c = kCfgs[cfg];
    if (c.group && c.group >= p.nb16) return false;               // same as the full group
    const int nsl = 2 * p.nb16, nsg = 2 * (c.group ? c.group : p.nb16);
    const int rs = stem_rs(p);
    g.threads = c.threads;
    g.rs = rs;
    g.roll = c.roll;
    g.prod = c.prod;
    if (c.roll) {
        // row-aligned window, an even number of values between windows, and
        // strips of more than one step
        // the depthwise tasks of a row (slices x columns) fit the workgroup
        if (!stem_row_aligned(p.KH, p.KW, p.C, p.dw) || (p.sw * p.C) % 2 != 0 || c.rows < 2 * c.step ||
            p.OH <= c.step || p.sh != 2 || p.dh != 1 || std::min(nsl, p.ns) * p.OW > c.threads ||
            p.dpl < 0 || p.dpl > 2 || p.dpt < 0 || p.dpt > 2)
            return false;
        const int R = c.step, Q = 2 * R + 2;
        g.rows = R;
        g.group = p.nb16;
        g.srows = c.rows;
        g.nbands = (p.OH + c.rows - 1) / c.rows;
        g.qi = (2 * R - 1) * p.sh + 3;
        const int vn = fp16_in ? 8 : 4, rowlen = p.W * p.C, lead = p.pl * p.C;
        g.vec = rowlen % vn == 0 && lead % (fp16_in ? 8 : 4) == 0;
        g.pstride = 0;
        g.band_h8 = 0;
        g.lds = ((size_t)nsl * Q * (p.SW + 2) + nsl * 9) * 16 + (size_t)g.qi * rs * 2 + (size_t)nsl * 8 * 4 * 2 + 16;
        return g.lds <= 160 * 1024;
    }
    const int R = c.rows;
    const int nsr = R + 2 < p.SH ? R + 2 : p.SH;                      // stem rows at most
    const int nrows = (nsr - 1) * p.sh + (p.KH - 1) * p.dh + 1;
    g.rows = R;
    g.group = c.group ? c.group : p.nb16;
    g.nbands = (p.OH + R - 1) / R;
    g.pstride = nsr * p.SW;
    g.band_h8 = (nrows * rs + 7) / 8;
    g.srows = 0;
    g.qi = 0;
    g.vec = 0;
    g.lds = ((size_t)nsg * g.pstride + g.band_h8 + nsl * 9) * 16 + (size_t)nsl * 8 * 4 + 16;
    return g.lds <= 160 * 1024;
}

template <typename E, typename TIN>
hipError_t launch_t(const StemDwParams &p, const StemDwGeom &g, hipStream_t st) {
    const dim3 grid(p.N * p.nbands);
#define MGI_STEMDW(NB_, R_, G_, NT_)                                                            \
    if (!g.roll && p.nb16 == NB_ && g.rows == R_ && g.group == G_ && g.threads == NT_) {         \
        auto k = stemdw_kernel<E, TIN, NB_, R_, G_, NT_>;                                       \
        hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, \
                                           160 * 1024);                                         \
        if (e != hipSuccess) return e;                                                          \
        launch(k, grid, dim3(NT_), (unsigned)g.lds, st, p);                                     \
        return hipGetLastError();                                                               \
    }
#define MGI_STEMDW_ROLL(NB_, NT_, R_)                                                           \
    if (g.roll && p.nb16 == NB_ && g.threads == NT_ && g.rows == R_) {                           \
        auto k = stemdw_roll_kernel<E, TIN, NB_, NT_, R_, 2, kRollUnits>;                       \
        hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, \
                                           160 * 1024);                                         \
        if (e != hipSuccess) return e;                                                          \
        launch(k, grid, dim3(NT_), (unsigned)g.lds, st, p);                                     \
        return hipGetLastError();                                                               \
    }
#define MGI_STEMDW_NB(NB_) MGI_STEMDW(NB_, 4, NB_, 512) MGI_STEMDW(NB_, 2, NB_, 512) \
    MGI_STEMDW_ROLL(NB_, 512, 2) MGI_STEMDW_ROLL(NB_, 512, 3)
    MGI_STEMDW_NB(1) MGI_STEMDW_NB(2) MGI_STEMDW_NB(3) MGI_STEMDW_NB(4)
#undef MGI_STEMDW_NB
#undef MGI_STEMDW_ROLL
#undef MGI_STEMDW
    return hipErrorInvalidValue;
}

}  // namespace

int stemdw_configs(const StemDwParams &p, int cfg, StemDwGeom *g, const char **name) {
    if (p.nb16 < 1 || p.nb16 > 4 || p.K > 32 || p.S != 1 || p.SW != p.OW || p.SH != p.OH) return 0;
    int count = 0;
    for (int c = 0; c < kNumCfgs; ++c) {
        StemDwGeom t{};
        if (!geometry(p, c, p.fp16_in != 0, t)) continue;
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
    StemDwParams q = p;
    q.fp16_in = fp16_in;
    if (cfg < 0 || cfg >= stemdw_configs(q, -1, nullptr, nullptr) || !stemdw_configs(q, cfg, &g, nullptr))
        return hipErrorInvalidValue;
    im2col_offsets(q.koff, p.K, p.KH, p.C, p.KW, p.dh, p.dw, g.rs);
    q.nbands = g.nbands;
    q.rs = g.rs;
    q.pstride = g.pstride;
    q.band_h8 = g.band_h8;
    q.srows = g.srows;
    q.qi = g.qi;
    q.vec = g.vec;
    if (p.bf16) return fp16_in ? launch_t<BF16, _Float16>(q, g, st) : launch_t<BF16, float>(q, g, st);
    return fp16_in ? launch_t<F16, _Float16>(q, g, st) : launch_t<F16, float>(q, g, st);
}

}  // namespace kern
}  // namespace mgi
