// Pointwise convolution fused with the depthwise 3x3 convolution that reads
// its output (an extension of the paper's fusion of the cheap operator into
// the expensive one, Sec. 3.2, to the pointwise -> depthwise pair inside a
// MobileNet stage).
//
// Unfused, the pointwise output is written to memory and read straight back by
// the depthwise kernel, and each of the two kernels pays its own launch and
// ramp.  Here a workgroup owns `ipt` whole images (at most 256 pixels, planes of
// at most 16 x 16) and 16*NBT output channels of the pointwise convolution, so
// the depthwise step over those channels needs no halo from other workgroups:
//   1. the depthwise taps and biases are copied into LDS by direct
//      global->LDS loads;
//   2. each wave owns FMW fragments of 16 pixels and all NBT channel blocks;
//      its activation fragments stream from the sliced layout into registers
//      PF K-steps ahead of use, and the MFMAs (v_mfma_f32_16x16x32, K
//      ascending, as in the GEMM kernels) read the weight fragments from LDS.
//      The weights (NBT channel blocks x all of K) are copied into LDS by
//      direct global->LDS loads before the K loop.  (Waiting for them chunk by
//      chunk, or streaming them through a two-chunk ring, measured no faster:
//      the loop is bound by the L2->CU transfer of activations and weights,
//      about 324 KiB per workgroup at v1's 14x14 stage);
//   3. bias and activation are applied and the 16-bit pointwise output tile
//      is parked in LDS, slice-major, in place of the weights;
//   4. the depthwise convolution runs from LDS: one lane per output column, a
//      row of lanes per (image, slice, strip of R output rows); the left and
//      right input columns come from the neighbouring lanes by wave-wide DPP
//      shifts (lanes past the last column hold zeros, which is the zero
//      padding).
// Accumulation order, rounding points and activations are those of the
// separate GEMM and depthwise kernels, so the result is bit-identical to the
// unfused pair (and to the node's split form, which runs those kernels).
#include "device.h"

namespace mgi {
namespace kern {

// whole-wave lane shift of a 16-byte value: kWaveShr1 gives lane l the value
// of lane l-1 (lane 0 gets zero), kWaveShl1 that of lane l+1 (lane 63 gets zero)
constexpr int kWaveShl1 = 0x130, kWaveShr1 = 0x138;
template <int CTRL>
__device__ __forceinline__ h8 wave_shift(h8 v) {
    const u4x u = as_u4(v);
    u4x r;
#pragma unroll
    for (int d = 0; d < 4; ++d)
        r[d] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)u[d], CTRL, 0xf, 0xf, false);
    return __builtin_bit_cast(h8, r);
}

constexpr int kPwDwPixels = 256;   // pixel capacity of a tile (16 fragments)
constexpr int kPwDwLds = 160 * 1024;

template <typename E, int NW, int FMW, int NBT, int S_, int R, int LPR, int PF>
__global__ __launch_bounds__(NW * 64) void pwdw_kernel(PwDwParams p) {
    constexpr int PMAX = 16 * NW * FMW;
    constexpr int NCH = 16 * NBT;                 // output channels of the tile
    constexpr int NSL = 2 * NBT;                  // ... in sliced elements
    static_assert(PMAX == kPwDwPixels, "tile capacity");
    constexpr int CK = PF;                        // K-steps per weight chunk
    constexpr int SQ = NBT * CK;                  // 64-element wave loads per chunk
    static_assert(SQ % NW == 0, "weight chunk split");
    constexpr int DPW = SQ / NW;                  // ... per wave
    constexpr int GPI = NW * 64 / LPR;            // lane rows per pass of the depthwise step
    constexpr int kTapQ = (NSL * 9 + 63) / 64, kTapH8 = 64 * kTapQ;   // taps [NSL][9], whole wave loads
    constexpr int kBiasQ = (NCH / 4 + 63) / 64;
    extern __shared__ h8 lds[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int grp = tile / p.ntiles, ct = tile - grp * p.ntiles;
    const int hw = p.H * p.W;
    const int img0 = grp * p.ipt;
    const int nimg = min(p.ipt, p.N - img0);
    const int P = nimg * hw;                      // valid pixels of the tile
    const int m0 = img0 * hw;
    const int nb0 = ct * NBT;
    const int ksp = p.ksp, nk = ksp >> 2;
    const int nchunks = (nk + CK - 1) / CK;
    const int main_h8 = max(nchunks * SQ * 64, NSL * PMAX);
    const h8 *taps = lds + main_h8;                               // [NSL][9]
    const float *dwb = (const float *)(lds + main_h8 + kTapH8);  // [NSL][8]

    // 1. weights -> LDS in K order, chunk c = K-steps [c*CK, c*CK + CK) of the
    // NBT channel blocks, layout [chunk][NBT][CK][64]; wave load q of a chunk
    // is channel block q / CK, K-step q % CK (steps past K read the last one);
    // then the taps and depthwise biases (sources clamped to their last
    // element; the copies past the end land in padding)
    {
        for (int c = 0; c < nchunks; ++c) {
#pragma unroll
            for (int r = 0; r < DPW; ++r) {
                const int q = wave + NW * r, i = q / CK, kk = min(c * CK + q % CK, nk - 1);
                load_lds16(p.w + ((size_t)(nb0 + i) * ksp + kk * 4) * 16 + lane, lds + (c * SQ + q) * 64);
            }
        }
        const h8 *tsrc = p.dw_w + (size_t)nb0 * 2 * 9;
        const h8 *bsrc = (const h8 *)(p.dw_b + nb0 * 16);
        for (int q = wave; q < kTapQ + kBiasQ; q += NW) {
            const int e = (q < kTapQ ? q : q - kTapQ) * 64 + lane;
            if (q < kTapQ) load_lds16(tsrc + min(e, NSL * 9 - 1), lds + main_h8 + e);
            else load_lds16(bsrc + min(e, NCH / 4 - 1), lds + main_h8 + kTapH8 + e);
        }
    }

    // 2. this wave's pixel fragments: wave, wave + NW, ... (a fragment with no
    // valid pixel is skipped; rows past the tile read its last pixel and are
    // never stored)
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
    auto xload = [&](int kk, h8 *dst) {
        const int ks = min(kk * 4 + xsl, p.ksl - 1);   // K tail meets zero weights
        const h8 *src = p.x + (size_t)ks * p.M;
#pragma unroll
        for (int j = 0; j < FMW; ++j)
            if (fj[j]) dst[j] = src[mj[j]];
    };
#pragma unroll
    for (int u = 0; u < PF; ++u)
        if (u < nk) xload(u, xq[u]);
    wait_vm_lds<0>();                 // this wave's share of the weights has landed
    __builtin_amdgcn_s_barrier();     // ... and every other wave's

    f4 acc[NBT][FMW];
#pragma unroll
    for (int i = 0; i < NBT; ++i)
#pragma unroll
        for (int j = 0; j < FMW; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    auto step = [&](int kk, const h8 *b) {
        const h8 *buf = lds + (kk / CK) * SQ * 64 + (kk % CK) * 64 + lane;
        h8 a[NBT];
#pragma unroll
        for (int i = 0; i < NBT; ++i) a[i] = buf[i * CK * 64];
#pragma unroll
        for (int j = 0; j < FMW; ++j)
            if (fj[j]) {
#pragma unroll
                for (int i = 0; i < NBT; ++i) acc[i][j] = E::mma(a[i], b[j], acc[i][j]);
            }
    };
    for (int c = 0; c < nchunks; ++c) {
#pragma unroll
        for (int u = 0; u < CK; ++u) {
            const int kk = c * CK + u;
            if (kk < nk) {
                step(kk, xq[u]);
                xload(min(kk + PF, nk - 1), xq[u]);
            }
        }
    }

    // 3. pointwise epilogue into LDS: tile [NSL][PMAX] of sliced elements
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NBT; ++i) {
        const int c = i * 16 + 4 * (lane >> 4);       // channel within the tile
        float bv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) bv[r] = p.bias[nb0 * 16 + c + r];
#pragma unroll
        for (int j = 0; j < FMW; ++j) {
            const int px = (wave + j * NW) * 16 + (lane & 15);
            if (!fj[j] || px >= P) continue;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r] + bv[r], p.act1);
            *(h4 *)((_Float16 *)(lds + (c >> 3) * PMAX + px) + (c & 7)) = E::pack4(v);
        }
    }
    __syncthreads();

    // 4. depthwise 3x3 from LDS, taps and accumulation order of the separate
    // depthwise kernel
    constexpr int NR = (R - 1) * S_ + 3;          // input rows of a strip
    constexpr int NC = S_;                        // input columns loaded per lane
    const int nstrips = (p.OH + R - 1) / R;
    const int ngroups = nimg * NSL * nstrips;
    const int ox = tid % LPR;
    const float lo = p.act2 == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act2 == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    const int passes = (ngroups + GPI - 1) / GPI;
    for (int pass = 0; pass < passes; ++pass) {     // same count in every lane (DPP below)
        const int g = pass * GPI + tid / LPR;
        const bool gv = g < ngroups;
        const int gg = gv ? g : 0;
        const int strip = gg % nstrips, rest = gg / nstrips;
        const int sl = rest % NSL, t = rest / NSL;
        const int oy0 = strip * R, iy0 = oy0 * S_ - p.pt;
        const h8 *plane = lds + sl * PMAX + t * hw;
        h8 w[9];
#pragma unroll
        for (int k = 0; k < 9; ++k) w[k] = taps[sl * 9 + k];
        int cx[NC];
        bool cv[NC];
#pragma unroll
        for (int k = 0; k < NC; ++k) {
            cx[k] = ox * S_ + k;
            cv[k] = gv && cx[k] < p.W;
        }
        float acc2[R][8];
#pragma unroll
        for (int o = 0; o < R; ++o)
#pragma unroll
            for (int c = 0; c < 8; ++c) acc2[o][c] = dwb[sl * 8 + c];
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int iy = iy0 + r;
            const bool rv = iy >= 0 && iy < p.H;
            h8 v[NC];
#pragma unroll
            for (int k = 0; k < NC; ++k) v[k] = (rv && cv[k]) ? plane[iy * p.W + cx[k]] : zero_h8();
            h8 t3[3];
            if (S_ == 1) {          // columns ox-1, ox, ox+1 (left padding 1)
                t3[0] = wave_shift<kWaveShr1>(v[0]);
                t3[1] = v[0];
                t3[2] = wave_shift<kWaveShl1>(v[0]);
            } else if (p.pl == 0) { // columns 2ox, 2ox+1, 2ox+2
                t3[0] = v[0];
                t3[1] = v[NC - 1];
                t3[2] = wave_shift<kWaveShl1>(v[0]);
            } else {                // columns 2ox-1, 2ox, 2ox+1
                t3[0] = wave_shift<kWaveShr1>(v[NC - 1]);
                t3[1] = v[0];
                t3[2] = v[NC - 1];
            }
#pragma unroll
            for (int ky = 0; ky < 3; ++ky) {
                const int tt = r - ky;
                if (tt >= 0 && tt % S_ == 0 && tt / S_ < R) {
#pragma unroll
                    for (int k = 0; k < 3; ++k) E::fma8(acc2[tt / S_], w[ky * 3 + k], t3[k]);
                }
            }
        }
        if (gv && ox < p.OW) {
            const int gs = nb0 * 2 + sl;                 // global slice
            h8 *yout = p.y + ((size_t)gs * p.N + img0 + t) * p.OH * p.OW + ox;
#pragma unroll
            for (int o = 0; o < R; ++o) {
                if (oy0 + o >= p.OH) break;
                float q[8];
#pragma unroll
                for (int c = 0; c < 8; ++c) q[c] = __builtin_amdgcn_fmed3f(acc2[o][c], lo, hi);
                yout[(size_t)(oy0 + o) * p.OW] = E::pack(q);
            }
        }
    }
}

namespace {
constexpr int kPwDwNW = 8, kPwDwFMW = 2, kPwDwPF = 4, kPwDwR = 7;

int pwdw_nbt(int cfg) { return cfg == 0 ? 8 : 4; }

int pwdw_lpr(int OW) { return OW < 8 ? 8 : OW < 16 ? 16 : 0; }

size_t tail_bytes(int nbt) {   // taps and biases behind the main region
    const size_t nsl = 2 * (size_t)nbt;
    return (64 * ((nsl * 9 + 63) / 64) + 64 * ((nsl * 2 + 63) / 64)) * 16;
}

template <typename E, int NBT, int S_, int LPR>
hipError_t launch_pwdw_t(const PwDwParams &p, size_t lds, hipStream_t st) {
    auto kern = pwdw_kernel<E, kPwDwNW, kPwDwFMW, NBT, S_, kPwDwR, LPR, kPwDwPF>;
    static const hipError_t attr =
        hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kPwDwLds);
    if (attr != hipSuccess) return attr;
    const int groups = (p.N + p.ipt - 1) / p.ipt;
    launch(kern, dim3(groups * p.ntiles), dim3(kPwDwNW * 64), (unsigned)lds, st, p);
    return hipGetLastError();
}

size_t lds_bytes(int ksp, int nbt) {
    const size_t nk = (size_t)ksp / 4, nchunks = (nk + kPwDwPF - 1) / kPwDwPF;
    const size_t slab = nchunks * nbt * kPwDwPF * 64 * 16;   // weights, whole K in chunks
    const size_t otile = (size_t)2 * nbt * kPwDwPixels * 16;  // pointwise output tile
    return (slab > otile ? slab : otile) + tail_bytes(nbt);
}

template <typename E, int NBT>
hipError_t launch_pwdw_e(const PwDwParams &p, size_t lds, hipStream_t st) {
    const int lpr = pwdw_lpr(p.OW);
    if (p.S == 1) return lpr == 8 ? launch_pwdw_t<E, NBT, 1, 8>(p, lds, st) : launch_pwdw_t<E, NBT, 1, 16>(p, lds, st);
    return lpr == 8 ? launch_pwdw_t<E, NBT, 2, 8>(p, lds, st) : launch_pwdw_t<E, NBT, 2, 16>(p, lds, st);
}
}  // namespace

bool pwdw_supported(int H, int W, int OH, int OW, int S, int pt, int pl, int nb16, int ksp, int cfg, int *ipt) {
    if (cfg < 0 || cfg > 1 || H <= 0 || W <= 0 || OH <= 0 || OW <= 0 || (S != 1 && S != 2)) return false;
    const int hw = H * W;
    // whole images of at most 256 pixels per tile; an output row fits a row
    // of 8 or 16 lanes with a lane to spare, and every input column a lane
    // needs from a neighbour is held by a lane of the same row or is padding
    // (the neighbour past the row's end holds zeros): stride 1 with left
    // padding 1 and W < lanes, stride 2 with left padding 0 or 1 and
    // W <= 2 * lanes - 1
    const int lpr = pwdw_lpr(OW);
    if (hw > kPwDwPixels || lpr == 0 || pt < 0) return false;
    if (S == 1 ? (pl != 1 || W >= lpr) : ((pl != 0 && pl != 1) || W > 2 * lpr - 1)) return false;
    const int nbt = pwdw_nbt(cfg);
    if (nb16 % nbt != 0 || ksp % 4 != 0) return false;
    if (lds_bytes(ksp, nbt) > (size_t)kPwDwLds) return false;
    if (ipt) *ipt = kPwDwPixels / hw;
    return true;
}

hipError_t launch_pwdw(const PwDwParams &p, int cfg, hipStream_t st) {
    int ipt = 0;
    if (!pwdw_supported(p.H, p.W, p.OH, p.OW, p.S, p.pt, p.pl, p.nb16, p.ksp, cfg, &ipt) || p.ipt < 1 ||
        p.ipt > ipt || p.ntiles * pwdw_nbt(cfg) != p.nb16 || p.M != p.N * p.H * p.W)
        return hipErrorInvalidValue;
    if (p.N <= 0) return hipSuccess;
    const size_t lds = lds_bytes(p.ksp, pwdw_nbt(cfg));
    if (cfg == 0) return p.bf16 ? launch_pwdw_e<BF16, 8>(p, lds, st) : launch_pwdw_e<F16, 8>(p, lds, st);
    return p.bf16 ? launch_pwdw_e<BF16, 4>(p, lds, st) : launch_pwdw_e<F16, 4>(p, lds, st);
}

}  // namespace kern
}  // namespace mgi
