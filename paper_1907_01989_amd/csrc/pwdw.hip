// Pointwise convolution fused with the depthwise 3x3 convolution that reads
// its output (an extension of the paper's fusion of the cheap operator into
// the expensive one, Sec. 3.2, to the pointwise -> depthwise pair inside a
// MobileNet stage).
//
// Unfused, the pointwise output is written to memory and read straight back by
// the depthwise kernel (on the 112 x 112 and 56 x 56 planes of a batch of 64
// that round trip is hundreds of MB), and each of the two kernels pays its own
// launch and ramp.  Here a workgroup owns 16*NBT output channels of the
// pointwise convolution (a channel tile; the last one may be partial) and
// either `ipt` whole images (at most 16*NW*FMW pixels) or a band of R output
// rows of one image together with the input rows those need (the halo rows
// are computed by both neighbouring bands), so the depthwise step over its
// channels needs nothing from other workgroups:
//   1. the weights (NBT channel blocks x all of K), the depthwise taps and
//      biases are copied into LDS by direct global->LDS loads (taps past the
//      input read a zero element kept in LDS);
//   2. each of the NW waves owns FMW fragments of 16 pixels and all NBT
//      channel blocks;
//      its activation fragments stream from the sliced layout into registers
//      PF K-steps ahead of use, and the MFMAs (v_mfma_f32_16x16x32, K
//      ascending, as in the GEMM kernels) read the weight fragments from LDS;
//   3. bias and activation are applied and the 16-bit pointwise output tile
//      is parked in LDS, slice-major, in place of the weights;
//   4. the depthwise convolution runs from LDS: one lane per output column, a
//      row of LPR lanes per (image, slice, strip of R output rows); the left
//      and right input columns come from the neighbouring lanes by wave-wide
//      DPP shifts (lanes past the row's end hold zeros, which is the zero
//      padding).
// Accumulation order, rounding points and activations are those of the
// separate GEMM and depthwise kernels, so the result is bit-identical to the
// unfused pair (and to the node's split form, which runs those kernels).
#include <algorithm>
#include <utility>

#include "device.h"

namespace mgi {
namespace kern {

constexpr int kPwDwLds = 160 * 1024;

template <typename E, int NW, int FMW, int NBT, int S_, int R, int LPR, int PF, bool DEEP>
__global__ __launch_bounds__(NW * 64, 2) void pwdw_kernel(PwDwParams p) {   // >= 2 waves per SIMD: <= 256 VGPRs
    const int PMAX = p.pstride;                   // pixel stride of the LDS output tile (>= a tile's pixels)
    constexpr int NCH = 16 * NBT;                 // output channels of a tile
    constexpr int NSL = 2 * NBT;                  // ... in sliced elements
    constexpr int GPI = NW * 64 / LPR;            // lane rows per pass of the depthwise step
    constexpr int CK = PF;                        // K-steps per weight chunk
    constexpr int SQ = NBT * CK;                  // 64-element wave loads per chunk
    constexpr int kTapQ = (NSL * 9 + 63) / 64, kTapH8 = 64 * kTapQ;   // taps [NSL][9], whole wave loads
    constexpr int kBiasQ = (NCH / 4 + 63) / 64;
    static_assert(LPR <= 64 && 64 % LPR == 0, "a lane row lies in one wave");
    static_assert(NW == 4 || NW == 8, "waves per workgroup");
    extern __shared__ h8 lds[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int grp = tile / p.ntiles, ct = tile - grp * p.ntiles;
    const int nb0 = ct * NBT;
    const int nbv = min(NBT, p.nb16 - nb0);       // channel blocks of this tile
    const int nsv = min(NSL, p.ns - 2 * nb0);     // ... and output slices (odd when channels = 8 mod 16)
    // pixels of the tile: whole images img0 .. img0+nimg-1, or the input rows
    // [ir0, ir1) of image img0 that output rows [oy_lo, oy_hi) read
    int img0, nimg, oy_lo, oy_hi, ir0, ir1;
    if (p.nbands) {
        img0 = grp / p.nbands;
        nimg = 1;
        oy_lo = (grp - img0 * p.nbands) * R;
        oy_hi = min(p.OH, oy_lo + R);
        ir0 = max(0, oy_lo * S_ - p.pt);
        ir1 = min(p.H, (oy_hi - 1) * S_ - p.pt + 3);
    } else {
        img0 = grp * p.ipt;
        nimg = min(p.ipt, p.N - img0);
        oy_lo = 0;
        oy_hi = p.OH;
        ir0 = 0;
        ir1 = p.H;
    }
    const int thw = (ir1 - ir0) * p.W;            // tile pixels per image
    const int P = nimg * thw;                     // valid pixels of the tile
    const int m0 = (img0 * p.H + ir0) * p.W;
    const int ksp = p.ksp, nk = ksp >> 2;
    const int nchunks = (nk + CK - 1) / CK;
    const int main_h8 = max(nchunks * SQ * 64, NSL * PMAX);
    const h8 *taps = lds + main_h8;                               // [NSL][9]
    const float *dwb = (const float *)(lds + main_h8 + kTapH8);  // [NCH]
    const f4 *pwb = (const f4 *)(lds + main_h8 + kTapH8 + 64 * kBiasQ);   // pointwise bias [NCH]
    h8 *zslot = lds + main_h8 + kTapH8 + 128 * kBiasQ;            // one zero element

    // 1. weights -> LDS in K order, chunk c = K-steps [c*CK, c*CK + CK) of the
    // NBT channel blocks, layout [chunk][NBT][CK][64]; wave load q of a chunk
    // is channel block q / CK, K-step q % CK (steps past K read the last one,
    // blocks past the tile's last read the last valid one: their results are
    // never stored); then the taps, depthwise and pointwise biases (sources
    // clamped to their last element; the copies past the end land in padding)
    {
        for (int c = 0; c < nchunks; ++c) {
            for (int q = wave; q < SQ; q += NW) {
                const int i = min(q / CK, nbv - 1), kk = min(c * CK + q % CK, nk - 1);
                load_lds16(p.w + ((size_t)(nb0 + i) * ksp + kk * 4) * 16 + lane, lds + (c * SQ + q) * 64);
            }
        }
        const h8 *tsrc = p.dw_w + (size_t)nb0 * 2 * 9;
        const h8 *bsrc = (const h8 *)(p.dw_b + nb0 * 16), *psrc = (const h8 *)(p.bias + nb0 * 16);
        const int tn = nsv * 9, dbn = nsv * 2, bn = nbv * 4;
        for (int q = wave; q < kTapQ + 2 * kBiasQ; q += NW) {
            if (q < kTapQ) {
                const int e = q * 64 + lane;
                load_lds16(tsrc + min(e, tn - 1), lds + main_h8 + e);
            } else if (q < kTapQ + kBiasQ) {
                const int e = (q - kTapQ) * 64 + lane;
                load_lds16(bsrc + min(e, dbn - 1), lds + main_h8 + kTapH8 + e);
            } else {
                const int e = (q - kTapQ - kBiasQ) * 64 + lane;
                load_lds16(psrc + min(e, bn - 1), lds + main_h8 + kTapH8 + 64 * kBiasQ + e);
            }
        }
    }

    // 2. this wave's pixel fragments: wave, wave + NW, ... (a fragment with no
    // valid pixel computes nothing; rows past the tile read its last pixel and
    // are never stored).  When K has more steps than the PF prefetch slots
    // (DEEP, chosen at launch), every K-step loads every fragment, valid or
    // not (an invalid one reads the tile's last pixel again), and the loop
    // issues the same loads whichever steps it computes: with no load under a
    // condition the compiler can count the loads in flight and wait only for
    // the one a step consumes, so the loads for the next PF-1 steps stay in
    // flight.  Otherwise the slots take all of K at once, each step once.
    int mj[FMW];
    bool fj[FMW];
#pragma unroll
    for (int j = 0; j < FMW; ++j) {
        const int f = wave + j * NW;
        fj[j] = f * 16 < P;
        mj[j] = m0 + min(f * 16 + (lane & 15), P - 1);
    }
    const int xsl = lane >> 4;
    h8 xq[PF][FMW];
    // (byte offsets from the tensor's base fit 32 bits: the host offers this
    // kernel only for inputs of at most 4 GiB)
    auto xload = [&](int kk, h8 *dst) {
        const uint32_t ks = min(kk * 4 + xsl, p.ksl - 1);   // K tail meets zero weights
        const uint32_t off = ks * (uint32_t)p.M;
#pragma unroll
        for (int j = 0; j < FMW; ++j) dst[j] = *(const h8 *)((const char *)p.x + (off + (uint32_t)mj[j]) * 16u);
    };
    if constexpr (DEEP) {
#pragma unroll
        for (int u = 0; u < PF; ++u) xload(u, xq[u]);
    } else {
#pragma unroll
        for (int u = 0; u < PF; ++u)
            if (u < nk) xload(u, xq[u]);
    }
    if (tid == 0) *zslot = zero_h8();
    wait_vm_lds<0>();                 // this wave's share of the weights has landed
    __builtin_amdgcn_s_barrier();     // ... and every other wave's

    // (accumulators start from the bias, as in every pointwise GEMM kernel;
    // the first K-step takes it from LDS as an operand, one channel block at
    // a time, so nothing is initialised and few registers hold it).  The
    // weight fragments are read right before their MFMAs: reading the next
    // step's ahead costs NBT*4 registers, and measured no faster, also where
    // the LDS already limits a compute unit to one workgroup.
    f4 acc[NBT][FMW];
    auto step = [&](int kk, const h8 *b, bool first) {
        const h8 *buf = lds + (kk / CK) * SQ * 64 + (kk % CK) * 64 + lane;
        h8 a[NBT];
#pragma unroll
        for (int i = 0; i < NBT; ++i) a[i] = buf[i * CK * 64];
        if (first) {
#pragma unroll
            for (int i = 0; i < NBT; ++i) {
                const f4 c0 = pwb[i * 4 + (lane >> 4)];
#pragma unroll
                for (int j = 0; j < FMW; ++j)
                    if (fj[j]) acc[i][j] = E::mma(a[i], b[j], c0);
            }
            return;
        }
#pragma unroll
        for (int j = 0; j < FMW; ++j)
            if (fj[j]) {
#pragma unroll
                for (int i = 0; i < NBT; ++i) acc[i][j] = E::mma(a[i], b[j], acc[i][j]);
            }
    };
    step(0, xq[0], true);
    if constexpr (DEEP) {
        for (int c = 0; c < nchunks; ++c) {
#pragma unroll
            for (int u = 0; u < CK; ++u) {
                const int kk = c * CK + u;
                if (kk > 0 && kk < nk) step(kk, xq[u], false);
                xload(min(kk + PF, nk - 1), xq[u]);   // (past the last step: a repeat of it, never used)
            }
        }
    } else {
#pragma unroll
        for (int u = 1; u < PF; ++u)
            if (u < nk) step(u, xq[u], false);
    }

    // 3. pointwise epilogue into LDS: tile [NSL][PMAX] of sliced elements
    // (lanes past the tile's last pixel computed that pixel again: they store
    // the same value to its place, so no store is under a lane mask)
    __syncthreads();
    int pxc[FMW];
#pragma unroll
    for (int j = 0; j < FMW; ++j) pxc[j] = min((wave + j * NW) * 16 + (lane & 15), P - 1);
#pragma unroll
    for (int i = 0; i < NBT; ++i) {
        if (i >= nbv) break;
        const int c = i * 16 + 4 * (lane >> 4);       // channel within the tile
        _Float16 *row = (_Float16 *)(lds + (c >> 3) * PMAX) + (c & 7);
#pragma unroll
        for (int j = 0; j < FMW; ++j) {
            if (!fj[j]) continue;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r], p.act1);
            *(h4 *)(row + pxc[j] * 8) = E::pack4(v);
        }
    }
    __syncthreads();

    // 4. depthwise 3x3 from LDS, taps and accumulation order of the separate
    // depthwise kernel
    constexpr int NR = (R - 1) * S_ + 3;          // input rows of a strip
    constexpr int NC = S_;                        // input columns loaded per lane
    // stride 2: lane ox loads columns 2*ox - pl and 2*ox - pl + 1; its third
    // tap column is its right neighbour's first
    const int cx0 = S_ == 2 ? -p.pl : 0;
    const int nsl = nsv;
    const int nstrips = p.nbands ? 1 : (p.OH + R - 1) / R;
    const int ngroups = nimg * nsl * nstrips;
    const int ox = tid % LPR;
    const float lo = p.act2 == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act2 == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    const int passes = (ngroups + GPI - 1) / GPI;
    for (int pass = 0; pass < passes; ++pass) {     // same count in every lane (DPP below)
        const int g = pass * GPI + tid / LPR;
        const bool gv = g < ngroups;
        const int gg = gv ? g : 0;
        // group gg = (t * nsl + sl) * nstrips + strip; a row band has one
        // image and one strip, so its groups are the slices (no division)
        int strip = 0, sl = gg, t = 0;
        if (nstrips != 1 || nimg != 1) {
            strip = gg % nstrips;
            const int rest = gg / nstrips;
            sl = rest % nsl;
            t = rest / nsl;
        }
        const int oy0 = oy_lo + strip * R, iy0 = oy0 * S_ - p.pt;
        const h8 *plane = lds + sl * PMAX + t * thw;
        h8 w[9];
#pragma unroll
        for (int k = 0; k < 9; ++k) w[k] = taps[sl * 9 + k];
        int cx[NC];
        bool cv[NC];
#pragma unroll
        for (int k = 0; k < NC; ++k) {
            cx[k] = ox * S_ + cx0 + k;
            cv[k] = gv && cx[k] >= 0 && cx[k] < p.W;
        }
        float bias2[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) bias2[c] = dwb[sl * 8 + c];
        float acc2[R][8];
        // row pointers advance by one plane row per input row (adds, not
        // per-row multiplies)
        const h8 *rowp[NC];
#pragma unroll
        for (int k = 0; k < NC; ++k) rowp[k] = plane + (iy0 - ir0) * p.W + cx[k];
        // every input row of the strip is read before the first FMA, so the
        // LDS latency of the later rows overlaps the arithmetic of the earlier
        h8 vr[NR][NC];
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int iy = iy0 + r;
            const bool rv = iy >= ir0 && iy < ir1;
#pragma unroll
            for (int k = 0; k < NC; ++k) {
                vr[r][k] = *((rv && cv[k]) ? rowp[k] : zslot);
                rowp[k] += p.W;
            }
        }
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const h8 *v = vr[r];
            h8 t3[3];
            if (S_ == 1) {          // columns ox-1, ox, ox+1 (left padding 1)
                t3[0] = wave_shift<kWaveShr1>(v[0]);
                t3[1] = v[0];
                t3[2] = wave_shift<kWaveShl1>(v[0]);
            } else {                // columns 2ox-pl, 2ox-pl+1, 2ox-pl+2
                t3[0] = v[0];
                t3[1] = v[NC - 1];
                t3[2] = wave_shift<kWaveShl1>(v[0]);
            }
#pragma unroll
            for (int ky = 0; ky < 3; ++ky) {
                const int tt = r - ky;
                if (tt >= 0 && tt % S_ == 0 && tt / S_ < R) {
#pragma unroll
                    for (int k = 0; k < 3; ++k) {      // (the first tap takes the bias as its addend)
                        if (ky == 0 && k == 0) E::fma8_from(acc2[tt / S_], bias2, w[0], t3[0]);
                        else E::fma8(acc2[tt / S_], w[ky * 3 + k], t3[k]);
                    }
                }
            }
        }
        if (gv && ox < p.OW) {
            const int gs = nb0 * 2 + sl;                 // global slice
            h8 *yout = p.y + (((size_t)gs * p.N + img0 + t) * p.OH + oy0) * p.OW + ox;
#pragma unroll
            for (int o = 0; o < R; ++o) {
                if (oy0 + o >= oy_hi) break;
                float q[8];
#pragma unroll
                for (int c = 0; c < 8; ++c) q[c] = __builtin_amdgcn_fmed3f(acc2[o][c], lo, hi);
                *yout = E::pack(q);
                yout += p.OW;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Instances.  A whole-image instance takes images of at most 16*NW*FMW pixels
// whose output rows fit a lane row (OW < LPR); a band instance takes R output
// rows per workgroup.  Each instance covers one stride and one lane-row width.
// ---------------------------------------------------------------------------
namespace {

struct Inst {
    bool band;
    int nw, fmw, nbt, s, r, lpr, pf;
    const char *name;
    int ipt = 0;   // image tiles: images per workgroup (0: as many as fit)
};

// the candidates, in preference order for a shape
constexpr Inst kInsts[] = {
    {false, 8, 2, 4, 1, 7, 16, 4, "img64"},   {false, 8, 2, 8, 1, 7, 16, 4, "img128"},
    {false, 8, 2, 4, 1, 7, 8, 4, "img64"},    {false, 8, 2, 8, 1, 7, 8, 4, "img128"},
    {false, 8, 2, 4, 2, 7, 16, 4, "img64"},   {false, 8, 2, 8, 2, 7, 16, 4, "img128"},
    {false, 8, 2, 4, 2, 7, 8, 4, "img64"},    {false, 8, 2, 8, 2, 7, 8, 4, "img128"},
    // row bands: 8 waves and 4-row bands, or 4 waves and 2-row bands (small
    // enough in LDS for two workgroups per compute unit)
    {true, 8, 2, 8, 2, 4, 16, 4, "band4x128"},  {true, 4, 3, 8, 2, 2, 16, 4, "band2x128w4"},  // 28 -> 14
    {true, 8, 2, 8, 1, 4, 32, 4, "band4x128"},  {true, 4, 3, 8, 1, 4, 32, 4, "band4x128w4"},  // 28 x 28
    {true, 8, 4, 8, 2, 4, 32, 4, "band4x128"},  {true, 4, 5, 8, 2, 2, 32, 2, "band2x128w4"},  // 56 -> 28
    {true, 8, 3, 8, 1, 4, 64, 2, "band4x128"},  {true, 4, 4, 8, 1, 2, 64, 2, "band2x128w4"},  // 56 x 56
    {true, 8, 8, 4, 2, 4, 64, 2, "band4x64"},   {true, 4, 9, 4, 2, 2, 64, 1, "band2x64w4"},   // 112 -> 56
    {true, 8, 4, 4, 1, 4, 64, 2, "band4x64"},   {true, 4, 4, 4, 1, 2, 64, 2, "band2x64w4"},   // 56 x 56, 64 channels
    // 32-channel tiles: half the LDS of the 64-channel ones, so more
    // workgroups share a compute unit (on the 112 and 56 planes, where K is
    // small, this pays for reading the activations twice as often; measured
    // slower on the deeper band layers, as were 16-channel tiles)
    {true, 4, 9, 2, 2, 2, 64, 1, "band2x32w4"},  {true, 4, 4, 2, 1, 2, 64, 2, "band2x32w4"},   // 112 -> 56, 56 x 56
    // 48- and 96-channel tiles: MobileNet-v2's expansions (96, 144, 192, 576,
    // 960 channels) are multiples of 48, so these leave no partial tile
    {true, 4, 9, 3, 2, 2, 64, 1, "band2x48w4"},  {true, 4, 4, 3, 1, 2, 64, 2, "band2x48w4"},   // 112 -> 56, 56 x 56
    {true, 4, 5, 3, 2, 2, 32, 2, "band2x48w4"},  {true, 4, 3, 3, 1, 4, 32, 4, "band4x48w4"},   // 56 -> 28, 28 x 28
    {true, 4, 3, 4, 2, 2, 16, 4, "band2x64w4"},  {true, 4, 3, 4, 1, 4, 32, 4, "band4x64w4"},   // 28 -> 14, 28 x 28
    {false, 8, 2, 6, 1, 7, 16, 4, "img96"},      {false, 8, 2, 6, 1, 7, 8, 4, "img96"},        // 14 x 14, 7 x 7
    {false, 8, 2, 6, 2, 7, 8, 4, "img96"},                                                     // 14 -> 7
    // four 7 x 7 images per workgroup instead of the five that fit: a batch
    // of 64 then makes 16 image groups, so 64-channel tiles of 960-1024
    // channels fill the 256 compute units in one round with fewer pixels per
    // workgroup (two images with 96- or 128-channel tiles measured slower)
    {false, 8, 2, 4, 1, 7, 8, 4, "img64i4", 4},
    // 64-channel image tiles of four pixel fragments per wave (two 14 x 14
    // images per workgroup): each weight fragment read from LDS serves four
    // pixel fragments instead of two, and the weight slab is half that of the
    // 128-channel tile (measured 1-3% faster than the 128-channel tile on
    // v1's 14 x 14 nodes; an 8-step activation prefetch was slower)
    {false, 8, 4, 4, 1, 7, 16, 4, "img64f4"},   {false, 8, 4, 4, 2, 7, 8, 4, "img64f4"},       // 14 x 14, 14 -> 7
    {true, 4, 5, 4, 2, 2, 32, 2, "band2x64w4"},  {true, 8, 4, 4, 2, 4, 32, 2, "band4x64"},     // 56 -> 28
    // 16- and 32-channel image tiles with 2-row depthwise strips, for small
    // batches: more workgroups, and the depthwise step spread over more lanes
    {false, 8, 2, 1, 1, 2, 16, 4, "img16"},      {false, 8, 2, 2, 1, 2, 16, 4, "img32"},       // 14 x 14
    {false, 8, 2, 1, 1, 2, 8, 4, "img16"},       {false, 8, 2, 2, 1, 2, 8, 4, "img32"},        // 7 x 7
    {false, 8, 2, 1, 2, 2, 8, 4, "img16"},       {false, 8, 2, 2, 2, 2, 8, 4, "img32"},        // 14 -> 7
    // ... with activations prefetched 8 K-steps ahead (at a batch of one the
    // K loop waits on the memory latency, not on the matrix cores)
    {false, 8, 2, 1, 1, 2, 16, 8, "img16p8"},    {false, 8, 2, 1, 1, 2, 8, 8, "img16p8"},      // 14 x 14, 7 x 7
    {false, 8, 2, 1, 2, 2, 8, 8, "img16p8"},                                                   // 14 -> 7
    // 16-channel bands for small batches
    {true, 4, 9, 1, 2, 2, 64, 1, "band2x16w4"},  {true, 4, 4, 1, 1, 2, 64, 2, "band2x16w4"},   // 112 -> 56, 56 x 56
    {true, 4, 5, 1, 2, 2, 32, 2, "band2x16w4"},  {true, 4, 3, 1, 1, 4, 32, 4, "band4x16w4"},   // 56 -> 28, 28 x 28
    {true, 4, 3, 1, 2, 2, 16, 4, "band2x16w4"},                                                // 28 -> 14
    // taller bands with 4 waves: less halo recomputation than 2- and 4-row
    // bands (a 7-row band computes 9 input rows of the pointwise output per
    // 7 output rows, a 2-row band 4 per 2), and 7 rows divide the 56 and 28
    // planes (measured on those planes at a batch of 64: 56 x 56 x 128 21.4
    // against 26.0 us for the best shorter band, 56 x 56 x 144 23.8 against
    // 30.4, 28 x 28 x 192 12.0 against 13.5; 6- and 8-row bands, 48-channel
    // tiles and 7-row bands of 14 x 14 planes measured slower)
    {true, 4, 6, 2, 1, 4, 64, 2, "band4x32w4"},  {true, 4, 8, 2, 1, 7, 64, 2, "band7x32w4"},   // 56 x 56
    {true, 4, 4, 4, 1, 7, 32, 4, "band7x64w4"},                                                // 28 x 28
};
constexpr int kNumInsts = sizeof(kInsts) / sizeof(kInsts[0]);

int lanes_for(int OW) { return OW < 8 ? 8 : OW < 16 ? 16 : OW < 32 ? 32 : OW < 64 ? 64 : 0; }

size_t tail_bytes(int nbt) {   // taps, two biases and a zero element behind the main region
    const size_t nsl = 2 * (size_t)nbt, nch = 16 * (size_t)nbt;
    return (64 * ((nsl * 9 + 63) / 64) + 128 * ((nch / 4 + 63) / 64) + 1) * 16;
}

size_t lds_bytes(const Inst &in, int ksp, int pstride) {
    const size_t nk = (size_t)ksp / 4, nchunks = (nk + in.pf - 1) / in.pf;
    const size_t slab = nchunks * in.nbt * in.pf * 64 * 16;                // weights, all of K
    const size_t otile = (size_t)2 * in.nbt * pstride * 16;                // pointwise output tile
    return (slab > otile ? slab : otile) + tail_bytes(in.nbt);
}

// geometry of instance `in` for a shape, or false if it does not apply
bool fits(const Inst &in, int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16,
          PwDwGeom *g) {
    if (S != in.s || lanes_for(OW) != in.lpr || pt < 0) return false;
    // the kernel addresses its input with 32-bit byte offsets
    if ((uint64_t)ksp * (uint64_t)N * (uint64_t)H * (uint64_t)W * 16u > 0xffffffffull) return false;
    // every input column a lane needs from a neighbour is held by a lane of the
    // same row, or is padding (the neighbour past the row's end holds zeros)
    if (S == 1 ? (pl != 1 || W >= in.lpr) : ((pl != 0 && pl != 1) || W > 2 * in.lpr - 1)) return false;
    const int pmax = 16 * in.nw * in.fmw;
    if (!in.band) {
        if (H * W > pmax) return false;
        g->ipt = pmax / (H * W);
        if (in.ipt) {
            // (not where it gives the same groups as the instance without a cap)
            if (in.ipt >= g->ipt || (N + in.ipt - 1) / in.ipt == (N + g->ipt - 1) / g->ipt) return false;
            g->ipt = in.ipt;
        }
        g->nbands = 0;
        g->groups = (N + g->ipt - 1) / g->ipt;
        g->pstride = g->ipt * H * W;
        // 16- and 32-channel image tiles read the activations 4x and 2x as
        // often as the 64-channel ones; they are for shapes whose 64-channel
        // tiles leave most compute units idle (a batch of one or a few)
        if (in.nbt < 4 && g->groups * ((nb16 + 3) / 4) >= 128) return false;
    } else {
        // a band's input rows: (R - 1) * S + 3 at most
        const int rows = std::min((in.r - 1) * S + 3, H);
        if (rows * W > pmax) return false;
        g->ipt = 1;
        g->nbands = (OH + in.r - 1) / in.r;
        g->groups = N * g->nbands;
        g->pstride = rows * W;
        // 16-channel bands: for shapes whose 64-channel bands leave most
        // compute units idle, as the small image tiles
        if (in.nbt == 1 && g->groups * ((nb16 + 3) / 4) >= 128) return false;
    }
    g->nbt = in.nbt;
    g->lds = lds_bytes(in, ksp, g->pstride);
    return g->lds <= (size_t)kPwDwLds;
}

template <typename E, int K>
hipError_t launch_t(const PwDwParams &p, size_t lds, hipStream_t st) {
    constexpr Inst in = kInsts[K];
    constexpr int NW = in.nw;
    auto deep = pwdw_kernel<E, NW, in.fmw, in.nbt, in.s, in.r, in.lpr, in.pf, true>;
    auto shallow = pwdw_kernel<E, NW, in.fmw, in.nbt, in.s, in.r, in.lpr, in.pf, false>;
    static const hipError_t attr = [&] {
        const hipError_t e =
            hipFuncSetAttribute((const void *)deep, hipFuncAttributeMaxDynamicSharedMemorySize, kPwDwLds);
        return e != hipSuccess
                   ? e
                   : hipFuncSetAttribute((const void *)shallow, hipFuncAttributeMaxDynamicSharedMemorySize, kPwDwLds);
    }();
    if (attr != hipSuccess) return attr;
    auto kern = (p.ksp >> 2) > in.pf ? deep : shallow;   // more K-steps than prefetch slots
    const int groups = p.nbands ? p.N * p.nbands : (p.N + p.ipt - 1) / p.ipt;
    launch(kern, dim3(groups * p.ntiles), dim3(NW * 64), (unsigned)lds, st, p);
    return hipGetLastError();
}

// instance k of the table (every entry is instantiated for both types)
template <typename E, size_t... K>
hipError_t launch_any(int k, const PwDwParams &p, size_t lds, hipStream_t st, std::index_sequence<K...>) {
    hipError_t r = hipErrorInvalidValue;
    (void)((k == (int)K && ((r = launch_t<E, (int)K>(p, lds, st)), true)) || ...);
    return r;
}

template <typename E>
hipError_t launch_inst(int k, const PwDwParams &p, size_t lds, hipStream_t st) {
    return launch_any<E>(k, p, lds, st, std::make_index_sequence<kNumInsts>{});
}

// the applicable instances of a shape, in table order
int applicable(int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16, int *idx,
               PwDwGeom *geo) {
    int n = 0;
    for (int k = 0; k < kNumInsts; ++k) {
        PwDwGeom g{};
        if (!fits(kInsts[k], N, H, W, OH, OW, S, pt, pl, ksp, nb16, &g)) continue;
        if (idx) idx[n] = k;
        if (geo) geo[n] = g;
        ++n;
    }
    return n;
}
}  // namespace

int pwdw_configs(int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16, int cfg,
                 PwDwGeom *g, const char **name) {
    int idx[kNumInsts];
    PwDwGeom geo[kNumInsts];
    const int n = applicable(N, H, W, OH, OW, S, pt, pl, ksp, nb16, idx, geo);
    if (cfg >= 0 && cfg < n) {
        if (g) *g = geo[cfg];
        if (name) *name = kInsts[idx[cfg]].name;
    }
    return n;
}

hipError_t launch_pwdw(const PwDwParams &p, int cfg, hipStream_t st) {
    int idx[kNumInsts];
    PwDwGeom geo[kNumInsts];
    const int n = applicable(p.N, p.H, p.W, p.OH, p.OW, p.S, p.pt, p.pl, p.ksp, p.nb16, idx, geo);
    if (cfg < 0 || cfg >= n || p.M != p.N * p.H * p.W || p.ksp % 4 != 0 || p.nb16 <= 0) return hipErrorInvalidValue;
    const PwDwGeom &g = geo[cfg];
    PwDwParams q = p;
    q.ipt = g.ipt;
    q.nbands = g.nbands;
    q.pstride = g.pstride;
    q.ntiles = (p.nb16 + g.nbt - 1) / g.nbt;
    if (p.N <= 0) return hipSuccess;
    return p.bf16 ? launch_inst<BF16>(idx[cfg], q, g.lds, st) : launch_inst<F16>(idx[cfg], q, g.lds, st);
}

}  // namespace kern
}  // namespace mgi
