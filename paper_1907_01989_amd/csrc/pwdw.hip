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
//   3. bias and activation are applied, and the 16-bit pointwise output is
//      parked in LDS channel-planar: one zero-bordered plane per channel and
//      image, in place of the slab;
//   4. the depthwise convolution runs on the matrix cores.  For one channel and
//      one kernel row ky, the output plane (at most 16 x 16) is
//         out[oy][ox] += sum_ix in[oy*S + ky - pt][ix] * T[ix][ox],
//      T[ix][ox] = w[ky][ix - ox*S + pl] (zero off the three-tap band), one
//      v_mfma_f32_16x16x16: the A operand is four input columns of a row read
//      from the plane, the B operand is T, built per lane from the row's three
//      taps by a byte permute.  Three MFMAs per channel accumulate the kernel
//      rows; zero rows and columns of the plane are the zero padding.
// The pointwise part is bit-identical to the GEMM kernels; the depthwise sums
// are formed by the matrix core (fp32 accumulation) instead of nine
// sequential fp32 FMAs, so results agree with the separate depthwise kernel to
// fp32 rounding before the final 16-bit rounding.
#include "device.h"

namespace mgi {
namespace kern {

typedef uint32_t u2x __attribute__((ext_vector_type(2)));

constexpr int kPwDwPixels = 256;   // pixel capacity of a tile (16 fragments)
constexpr int kPwDwRow = 20;       // halves per plane row: 16 columns + bank padding
constexpr int kPwDwLds = 160 * 1024;

// halves per channel plane of an H-row input: a zero row above and below
__host__ __device__ constexpr int pwdw_plane(int H) { return (H + 2) * kPwDwRow + 4; }

template <typename E, int NW, int FMW, int NBT, int S_, int PF>
__global__ __launch_bounds__(NW * 64) void pwdw_kernel(PwDwParams p) {
    constexpr int PMAX = 16 * NW * FMW;
    constexpr int NCH = 16 * NBT;                 // output channels of the tile
    constexpr int NSL = 2 * NBT;                  // ... in sliced elements
    static_assert(PMAX == kPwDwPixels, "tile capacity");
    constexpr int CK = PF;                        // K-steps per weight chunk
    constexpr int SQ = NBT * CK;                  // 64-element wave loads per chunk
    static_assert(SQ % NW == 0, "weight chunk split");
    constexpr int DPW = SQ / NW;                  // ... per wave
    constexpr int kTapQ = (NCH * 3 / 2 + 63) / 64, kTapH8 = 64 * kTapQ;   // (w0,w1,w2,0) rows, whole wave loads
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
    const int pstr = pwdw_plane(p.H);
    const int nchunks = (nk + CK - 1) / CK;
    const int main_h8 = max(nchunks * SQ * 64, (p.ipt * NCH * pstr + 7) / 8);
    const h4 *taps = (const h4 *)(lds + main_h8);                 // [NCH][3]
    const float *dwb = (const float *)(lds + main_h8 + kTapH8);  // [NCH]

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
        const h8 *tsrc = (const h8 *)(p.dw_t + (size_t)nb0 * 16 * 3);
        const h8 *bsrc = (const h8 *)(p.dw_b + nb0 * 16);
        for (int q = wave; q < kTapQ + kBiasQ; q += NW) {
            const int e = (q < kTapQ ? q : q - kTapQ) * 64 + lane;
            if (q < kTapQ) load_lds16(tsrc + min(e, NCH * 3 / 2 - 1), lds + main_h8 + e);
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

    // 3. pointwise epilogue into channel planes [ipt][NCH][H + 2 rows][kPwDwRow]
    // (16-bit), zeroed first so that the border rows and the columns past W
    // read as zeros
    __syncthreads();
    _Float16 *planes = (_Float16 *)lds;
    {
        const int n4 = p.ipt * NCH * pstr / 4;
        h4 z;
#pragma unroll
        for (int i = 0; i < 4; ++i) z[i] = (_Float16)0.0f;
        for (int e = tid; e < n4; e += NW * 64) ((h4 *)planes)[e] = z;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < FMW; ++j) {
        const int px = (wave + j * NW) * 16 + (lane & 15);
        if (!fj[j] || px >= P) continue;
        const int t = px / hw, rem = px - t * hw;
        const int y = rem / p.W, x = rem - y * p.W;
        _Float16 *dst = planes + t * NCH * pstr + (y + 1) * kPwDwRow + x;
#pragma unroll
        for (int i = 0; i < NBT; ++i) {
            const int c = i * 16 + 4 * (lane >> 4);   // channel within the tile
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r] + p.bias[nb0 * 16 + c + r], p.act1);
            const h4 pv = E::pack4(v);
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(c + r) * pstr] = pv[r];
        }
    }
    __syncthreads();

    // 4. depthwise 3x3 on the matrix cores, one (image, slice) per wave at a time
    const int q4 = lane >> 4, ln = lane & 15;
    // B operand selectors: half i of this lane is T[4*q4 + i][ln], the tap
    // d = 4*q4 + i - ln*S + pl of the row, or zero (selector byte 0x0c)
    uint32_t sel[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        sel[h] = 0;
#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2) {
            const int d = 4 * q4 + 2 * h + b2 - ln * S_ + p.pl;
            const uint32_t pair = (d >= 0 && d <= 2) ? (uint32_t)(2 * d) | (uint32_t)(2 * d + 1) << 8 : 0x0c0cu;
            sel[h] |= pair << (16 * b2);
        }
    }
    const int prow = p.H + 1;                        // last plane row (a zero row)
    const float lo = p.act2 == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi = p.act2 == MGI_ACT_RELU6 ? 6.0f : INFINITY;
    const int units = nimg * NSL;
    for (int u = wave; u < units; u += NW) {
        const int t = u / NSL, sl = u - t * NSL;
        const _Float16 *plane = planes + (t * NCH + sl * 8) * pstr + 4 * q4;
        u2x tw[8][3];
#pragma unroll
        for (int ch = 0; ch < 8; ++ch)
#pragma unroll
            for (int ky = 0; ky < 3; ++ky) tw[ch][ky] = __builtin_bit_cast(u2x, taps[(sl * 8 + ch) * 3 + ky]);
        f4 dacc[8];
#pragma unroll
        for (int ch = 0; ch < 8; ++ch) dacc[ch] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ky = 0; ky < 3; ++ky) {
            // plane row of input row ln*S + ky - pt (rows of outputs past OH
            // are clamped; their results are never stored)
            const int rr = min(ln * S_ + ky - p.pt + 1, prow);
            h4 a[8];
#pragma unroll
            for (int ch = 0; ch < 8; ++ch) a[ch] = *(const h4 *)(plane + ch * pstr + rr * kPwDwRow);
#pragma unroll
            for (int ch = 0; ch < 8; ++ch) {
                u2x bw;
                bw[0] = __builtin_amdgcn_perm(tw[ch][ky][1], tw[ch][ky][0], sel[0]);
                bw[1] = __builtin_amdgcn_perm(tw[ch][ky][1], tw[ch][ky][0], sel[1]);
                dacc[ch] = E::mma16(a[ch], __builtin_bit_cast(h4, bw), dacc[ch]);
            }
        }
        // lane holds output column ln of rows 4*q4 .. 4*q4+3 for the 8 channels
        const int gs = nb0 * 2 + sl;
        h8 *yout = p.y + ((size_t)gs * p.N + img0 + t) * p.OH * p.OW;
        float bch[8];
#pragma unroll
        for (int ch = 0; ch < 8; ++ch) bch[ch] = dwb[sl * 8 + ch];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int oy = 4 * q4 + r;
            if (oy >= p.OH || ln >= p.OW) continue;
            float v[8];
#pragma unroll
            for (int ch = 0; ch < 8; ++ch) v[ch] = __builtin_amdgcn_fmed3f(dacc[ch][r] + bch[ch], lo, hi);
            yout[oy * p.OW + ln] = E::pack(v);
        }
    }
}

namespace {
constexpr int kPwDwNW = 8, kPwDwFMW = 2, kPwDwPF = 4;

int pwdw_nbt(int cfg) { return cfg == 0 ? 8 : 4; }

size_t tail_bytes(int nbt) {   // taps and biases behind the main region
    const size_t nch = 16 * (size_t)nbt;
    return (64 * ((nch * 3 / 2 + 63) / 64) + 64 * ((nch / 4 + 63) / 64)) * 16;
}

template <typename E, int NBT, int S_>
hipError_t launch_pwdw_t(const PwDwParams &p, size_t lds, hipStream_t st) {
    auto kern = pwdw_kernel<E, kPwDwNW, kPwDwFMW, NBT, S_, kPwDwPF>;
    static const hipError_t attr =
        hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kPwDwLds);
    if (attr != hipSuccess) return attr;
    const int groups = (p.N + p.ipt - 1) / p.ipt;
    launch(kern, dim3(groups * p.ntiles), dim3(kPwDwNW * 64), (unsigned)lds, st, p);
    return hipGetLastError();
}

size_t lds_bytes(int ksp, int H, int ipt, int nbt) {
    const size_t nk = (size_t)ksp / 4, nchunks = (nk + kPwDwPF - 1) / kPwDwPF;
    const size_t slab = nchunks * nbt * kPwDwPF * 64 * 16;   // weights, whole K in chunks
    const size_t planes = ((size_t)ipt * 16 * nbt * pwdw_plane(H) + 7) / 8 * 16;
    return (slab > planes ? slab : planes) + tail_bytes(nbt);
}
}  // namespace

bool pwdw_supported(int H, int W, int OH, int OW, int S, int pt, int pl, int nb16, int ksp, int cfg, int *ipt) {
    if (cfg < 0 || cfg > 1 || H <= 0 || W <= 0 || OH <= 0 || OW <= 0 || (S != 1 && S != 2)) return false;
    const int hw = H * W;
    // input and output planes of at most 16 x 16 (the MFMA tile); input
    // columns outside [0, 16) are padding (W <= 16) and drop out of the sum;
    // input rows read lie in [-1, H], the plane's zero border rows
    if (H > 16 || W > 16 || OH > 16 || OW > 16 || hw > kPwDwPixels) return false;
    if (pt < 0 || pt > 1 || pl < 0 || pl > 2 || (OH - 1) * S + 2 - pt > H) return false;
    const int nbt = pwdw_nbt(cfg);
    if (nb16 % nbt != 0 || ksp % 4 != 0) return false;
    int n = kPwDwPixels / hw;
    while (n > 0 && lds_bytes(ksp, H, n, nbt) > (size_t)kPwDwLds) --n;
    if (n == 0) return false;
    if (ipt) *ipt = n;
    return true;
}

hipError_t launch_pwdw(const PwDwParams &p, int cfg, hipStream_t st) {
    int ipt = 0;
    if (!pwdw_supported(p.H, p.W, p.OH, p.OW, p.S, p.pt, p.pl, p.nb16, p.ksp, cfg, &ipt) || p.ipt < 1 ||
        p.ipt > ipt || p.ntiles * pwdw_nbt(cfg) != p.nb16 || p.M != p.N * p.H * p.W)
        return hipErrorInvalidValue;
    if (p.N <= 0) return hipSuccess;
    const size_t lds = lds_bytes(p.ksp, p.H, p.ipt, pwdw_nbt(cfg));
    if (cfg == 0) {
        if (p.S == 1) return p.bf16 ? launch_pwdw_t<BF16, 8, 1>(p, lds, st) : launch_pwdw_t<F16, 8, 1>(p, lds, st);
        return p.bf16 ? launch_pwdw_t<BF16, 8, 2>(p, lds, st) : launch_pwdw_t<F16, 8, 2>(p, lds, st);
    }
    if (p.S == 1) return p.bf16 ? launch_pwdw_t<BF16, 4, 1>(p, lds, st) : launch_pwdw_t<F16, 4, 1>(p, lds, st);
    return p.bf16 ? launch_pwdw_t<BF16, 4, 2>(p, lds, st) : launch_pwdw_t<F16, 4, 2>(p, lds, st);
}

}  // namespace kern
}  // namespace mgi
