// MobileNet-v2's inverted residual block (pointwise expansion, depthwise 3x3,
// linear pointwise projection, residual add) as one kernel: the paper's
// fusion of cheap operators into the expensive one (Sec. 3.2) carried to the
// whole block.  Unfused, the expansion writes a tensor six times wider than
// the block's input and the projection reads the depthwise output of the same
// width back; here both stay in LDS and only the block input, the residual
// and the block output touch memory.
//
// A workgroup owns a band of R output rows of one image together with the
// input rows they read (halo rows are expanded by both neighbouring bands),
// or whole images, and walks the expansion channels in chunks of NBT blocks
// of 16.  Per chunk:
//   1. the chunk's expansion weights (all of K), depthwise taps, both biases
//      and the projection weights of the chunk's K range go to LDS by direct
//      global->LDS loads;
//   2. the expansion GEMM (v_mfma_f32_16x16x32, K ascending): the waves form
//      NW/CS pixel groups x CS channel parts, a wave owning FMW fragments of
//      16 pixels of its group and the NBT/CS blocks of its part; activations
//      stream from the sliced input PF K-steps ahead of use;
//   3. bias and act1 are applied and the 16-bit tile is parked in LDS;
//   4. the depthwise 3x3 (taps in the standalone kernel's order, neighbour
//      columns by wave-wide DPP shifts, act2 by v_med3) writes its 16-bit
//      results into a second LDS tile, sliced like memory; slices past the
//      expansion are zero;
//   5. the projection accumulates the chunk's K-steps: the waves form PG
//      pixel groups x NW/PG output-block groups; A fragments come from the
//      LDS copy of the projection weights, B fragments (16 pixels x 32
//      channels) are 16-byte reads of the depthwise tile.
// The projection accumulators start from its bias and run over K in steps of
// 32 channels in ascending order, exactly as the standalone GEMM kernels
// (chunks cover whole K-steps), and every stored intermediate is rounded as
// the separate kernels store it, so the result is bit-identical to the
// unfused expansion -> depthwise -> projection sequence.
#include <algorithm>
#include <utility>

#include "device.h"

namespace mgi {
namespace kern {

constexpr int kIrbLds = 160 * 1024;

template <typename E, int NW, int CS, int FMW, int NBT, int S_, int R, int LPR, int PF, bool DEEP, int PG, int FPW,
          int NBO, bool RES>
__global__ __launch_bounds__(NW * 64, 1) void irb_kernel(IrbParams p) {
    const int PMAX = p.pstride;                   // pixel stride of the expansion tile
    const int OPS = p.opstride;                   // pixel stride of the depthwise tile
    constexpr int NCH = 16 * NBT, NSL = 2 * NBT;  // channels and slices of a chunk
    constexpr int GPI = NW * 64 / LPR;            // lane rows per pass of the depthwise step
    constexpr int CK = PF;                        // K-steps per slab chunk
    constexpr int SQ = NBT * CK;                  // wave loads per slab chunk
    constexpr int kTapQ = (NSL * 9 + 63) / 64, kTapH8 = 64 * kTapQ;
    constexpr int kBiasQ = (NCH / 4 + 63) / 64;
    constexpr int NG = NW / CS, NBW = NBT / CS;   // expansion: pixel groups, blocks per wave
    constexpr int KSC = NSL / 4;                  // projection K-steps per chunk
    constexpr int OG = NW / PG;                   // projection: output-block groups
    constexpr int OBW = (NBO + OG - 1) / OG;      // ... output blocks per wave
    static_assert(LPR <= 64 && 64 % LPR == 0, "a lane row lies in one wave");
    static_assert(NW == 4 || NW == 8, "waves per workgroup");
    static_assert(NBT % 2 == 0 && NBT % CS == 0 && NW % CS == 0 && NW % PG == 0, "wave layout");
    static_assert(!(RES && DEEP), "resident weights hold all of K in the activation registers");
    extern __shared__ h8 lds[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = xcd_tile(blockIdx.x, gridDim.x);
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
    const int thw = (ir1 - ir0) * p.W;            // expansion pixels per image
    const int P = nimg * thw;
    const int m0 = (img0 * p.H + ir0) * p.W;
    const int orows = oy_hi - oy_lo;
    const int OP = nimg * orows * p.OW;           // output pixels of the tile (contiguous in memory)
    const int mo0 = (img0 * p.OH + oy_lo) * p.OW;
    const int NOF = (OP + 15) >> 4;
    const int ksp = p.ksp, nk = ksp >> 2;
    const int nkc = (nk + CK - 1) / CK;
    const int pks = p.pksp >> 2;                  // projection K-steps
    // LDS.  Per chunk (RES = false): slab / expansion tile (union), taps,
    // depthwise bias, expansion bias, zero element, depthwise tile, the
    // chunk's projection weights.  Resident (RES): every expansion weight
    // [nb16][nk][64], taps [2 nb16][9], both biases and every projection
    // weight [pnb16][pks][64] are loaded once; then the expansion tile, the
    // zero element and the depthwise tile.
    const int wq_all = p.nb16 * nk, tq_all = (2 * p.nb16 * 9 + 63) / 64, bq_all = (4 * p.nb16 + 63) / 64;
    const int main_h8 = RES ? wq_all * 64 : max(nkc * SQ * 64, NSL * PMAX);
    h8 *taps = lds + main_h8;
    float *dwb = (float *)(taps + (RES ? 64 * tq_all : kTapH8));
    const f4 *ewb = (const f4 *)((h8 *)dwb + (RES ? 64 * bq_all : 64 * kBiasQ));
    h8 *pres = (h8 *)ewb + (RES ? 64 * bq_all : 64 * kBiasQ);    // resident projection weights
    h8 *etile = RES ? pres + pks * p.pnb16 * 64 : lds;            // expansion tile [NSL][PMAX]
    h8 *zslot = RES ? etile + NSL * PMAX : pres;                  // one zero element
    h8 *dtile = zslot + 64;                                       // depthwise tile [NSL][OPS]
    h8 *ptile = RES ? pres : dtile + NSL * OPS;                   // projection weights

    // expansion: the wave's pixel fragments (group eg) and channel blocks
    const int eg = wave % NG, eb0 = (wave / NG) * NBW;
    int mj[FMW];
    bool fj[FMW];
#pragma unroll
    for (int j = 0; j < FMW; ++j) {
        const int f = eg + j * NG;
        fj[j] = f * 16 < P;
        mj[j] = m0 + min(f * 16 + (lane & 15), P - 1);
    }
    const int xsl = lane >> 4;
    h8 xq[PF][FMW];
    auto xload = [&](int kk, h8 *dst) {
        const uint32_t ks = min(kk * 4 + xsl, p.ksl - 1);   // K tail meets zero weights
        const uint32_t off = ks * (uint32_t)p.M;
#pragma unroll
        for (int j = 0; j < FMW; ++j) dst[j] = *(const h8 *)((const char *)p.x + (off + (uint32_t)mj[j]) * 16u);
    };

    // projection: the wave's output fragments (group pg) and output blocks
    // og, og + OG, ...; accumulators start from the bias
    const int pg = wave % PG, og = wave / PG;
    bool fo[FPW];
#pragma unroll
    for (int j = 0; j < FPW; ++j) fo[j] = pg + j * PG < NOF;
    f4 pacc[OBW][FPW];
#pragma unroll
    for (int i = 0; i < OBW; ++i) {
        const f4 b0 = bias_frag(p.pbias, og + i * OG, p.pnb16, lane);
#pragma unroll
        for (int j = 0; j < FPW; ++j) pacc[i][j] = b0;
    }

    constexpr int NR = (R - 1) * S_ + 3, NC = S_;
    const int cx0 = S_ == 2 ? -p.pl : 0;
    const int nstrips = p.nbands ? 1 : (p.OH + R - 1) / R;
    const int ox = tid % LPR;
    const float lo2 = p.act2 == MGI_ACT_NONE ? -INFINITY : 0.0f;
    const float hi2 = p.act2 == MGI_ACT_RELU6 ? 6.0f : INFINITY;

    if constexpr (RES) {
        // every weight, tap and bias once; all of K of the activations
        for (int q = wave; q < wq_all; q += NW) {
            const int nb = q / nk, kk = q - nb * nk;
            load_lds16(p.w + ((size_t)nb * ksp + kk * 4) * 16 + lane, lds + q * 64);
        }
        const int tn = 2 * p.nb16 * 9, bn = 4 * p.nb16;
        for (int q = wave; q < tq_all + 2 * bq_all; q += NW) {
            if (q < tq_all) {
                const int e = q * 64 + lane;
                load_lds16(p.dw_w + min(e, tn - 1), taps + e);
            } else if (q < tq_all + bq_all) {
                const int e = (q - tq_all) * 64 + lane;
                load_lds16((const h8 *)p.dw_b + min(e, bn - 1), (h8 *)dwb + e);
            } else {
                const int e = (q - tq_all - bq_all) * 64 + lane;
                load_lds16((const h8 *)p.bias + min(e, bn - 1), (const h8 *)ewb + e);
            }
        }
        for (int q = wave; q < p.pnb16 * pks; q += NW) {
            const int ob = q / pks, kg = q - ob * pks;
            load_lds16(p.pw + ((size_t)ob * p.pksp + kg * 4) * 16 + lane, pres + q * 64);
        }
#pragma unroll
        for (int u = 0; u < PF; ++u)
            if (u < nk) xload(u, xq[u]);
        if (tid == 0) *zslot = zero_h8();
        wait_vm_lds<0>();
        __syncthreads();
    }

    const int nct = (p.nb16 + NBT - 1) / NBT;     // expansion chunks
    for (int ct = 0; ct < nct; ++ct) {
        const int nb0 = ct * NBT;
        const int nbv = min(NBT, p.nb16 - nb0);
        const int nsv = min(NSL, p.ns - 2 * nb0);
        // (per-chunk loads: the previous chunk's projection reads are done)
        if (!RES && ct > 0) __syncthreads();

        // 1. weights, taps, biases and projection weights of the chunk -> LDS
        if constexpr (!RES) {
        for (int c = 0; c < nkc; ++c) {
            for (int q = wave; q < SQ; q += NW) {
                const int i = min(q / CK, nbv - 1), kk = min(c * CK + q % CK, nk - 1);
                load_lds16(p.w + ((size_t)(nb0 + i) * ksp + kk * 4) * 16 + lane, lds + (c * SQ + q) * 64);
            }
        }
        {
            const h8 *tsrc = p.dw_w + (size_t)nb0 * 2 * 9;
            const h8 *bsrc = (const h8 *)(p.dw_b + nb0 * 16), *esrc = (const h8 *)(p.bias + nb0 * 16);
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
                    load_lds16(esrc + min(e, bn - 1), lds + main_h8 + kTapH8 + 64 * kBiasQ + e);
                }
            }
            for (int q = wave; q < NBO * KSC; q += NW) {
                const int ob = min(q / KSC, p.pnb16 - 1), kg = min(ct * KSC + q % KSC, pks - 1);
                load_lds16(p.pw + ((size_t)ob * p.pksp + kg * 4) * 16 + lane, ptile + q * 64);
            }
        }

        // 2. expansion GEMM
        if constexpr (DEEP) {
#pragma unroll
            for (int u = 0; u < PF; ++u) xload(u, xq[u]);
        } else {
#pragma unroll
            for (int u = 0; u < PF; ++u)
                if (u < nk) xload(u, xq[u]);
        }
        if (tid == 0) *zslot = zero_h8();
        wait_vm_lds<0>();
        __syncthreads();
        }

        // (resident: block b of the chunk is expansion block min(nb0 + b, nb16 - 1))
        auto wblk = [&](int b) { return RES ? min(nb0 + b, p.nb16 - 1) : b; };
        f4 acc[NBW][FMW];
        auto step = [&](int kk, const h8 *b, bool first) {
            h8 a[NBW];
#pragma unroll
            for (int i = 0; i < NBW; ++i)
                a[i] = RES ? lds[(wblk(eb0 + i) * nk + kk) * 64 + lane]
                           : lds[(kk / CK) * SQ * 64 + (kk % CK) * 64 + lane + (eb0 + i) * CK * 64];
            if (first) {
#pragma unroll
                for (int i = 0; i < NBW; ++i) {
                    const f4 c0 = ewb[wblk(eb0 + i) * 4 + (lane >> 4)];
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
                    for (int i = 0; i < NBW; ++i) acc[i][j] = E::mma(a[i], b[j], acc[i][j]);
                }
        };
        step(0, xq[0], true);
        if constexpr (DEEP) {
            for (int c = 0; c < nkc; ++c) {
#pragma unroll
                for (int u = 0; u < CK; ++u) {
                    const int kk = c * CK + u;
                    if (kk > 0 && kk < nk) step(kk, xq[u], false);
                    xload(min(kk + PF, nk - 1), xq[u]);
                }
            }
        } else {
#pragma unroll
            for (int u = 1; u < PF; ++u)
                if (u < nk) step(u, xq[u], false);
        }

        // 3. expansion epilogue into LDS: [NSL][PMAX] (per-chunk weights:
        // in place of the slab, once every wave is done with it)
        if (!RES) __syncthreads();
#pragma unroll
        for (int i = 0; i < NBW; ++i) {
            if (eb0 + i >= nbv) break;
            const int c = (eb0 + i) * 16 + 4 * (lane >> 4);
            _Float16 *row = (_Float16 *)(etile + (c >> 3) * PMAX) + (c & 7);
#pragma unroll
            for (int j = 0; j < FMW; ++j) {
                if (!fj[j]) continue;
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = act_apply(acc[i][j][r], p.act1);
                *(h4 *)(row + (mj[j] - m0) * 8) = E::pack4(v);
            }
        }
        __syncthreads();

        // 4. depthwise 3x3 into the depthwise tile [NSL][OPS] (tile output
        // pixel t * orows * OW + (oy - oy_lo) * OW + ox); slices past the
        // expansion are zeroed, they meet zero projection weights
        {
            const int ngroups = nimg * nsv * nstrips;
            const int passes = (ngroups + GPI - 1) / GPI;
            for (int pass = 0; pass < passes; ++pass) {     // same count in every lane (DPP below)
                const int g = pass * GPI + tid / LPR;
                const bool gv = g < ngroups;
                const int gg = gv ? g : 0;
                int strip = 0, sl = gg, t = 0;
                if (nstrips != 1 || nimg != 1) {
                    strip = gg % nstrips;
                    const int rest = gg / nstrips;
                    sl = rest % nsv;
                    t = rest / nsv;
                }
                const int oy0 = oy_lo + strip * R, iy0 = oy0 * S_ - p.pt;
                const h8 *plane = etile + sl * PMAX + t * thw;
                const int tsl = RES ? 2 * nb0 + sl : sl;  // the slice's taps and bias
                h8 w[9];
#pragma unroll
                for (int k = 0; k < 9; ++k) w[k] = taps[tsl * 9 + k];
                int cx[NC];
                bool cv[NC];
#pragma unroll
                for (int k = 0; k < NC; ++k) {
                    cx[k] = ox * S_ + cx0 + k;
                    cv[k] = gv && cx[k] >= 0 && cx[k] < p.W;
                }
                float bias2[8];
#pragma unroll
                for (int c = 0; c < 8; ++c) bias2[c] = dwb[tsl * 8 + c];
                float acc2[R][8];
                const h8 *rowp[NC];      // advanced by one plane row per input row
#pragma unroll
                for (int k = 0; k < NC; ++k) rowp[k] = plane + (iy0 - ir0) * p.W + cx[k];
#pragma unroll
                for (int r = 0; r < NR; ++r) {
                    const int iy = iy0 + r;
                    const bool rv = iy >= ir0 && iy < ir1;
                    h8 v[NC];
#pragma unroll
                    for (int k = 0; k < NC; ++k) {
                        v[k] = *((rv && cv[k]) ? rowp[k] : zslot);
                        rowp[k] += p.W;
                    }
                    h8 t3[3];
                    if (S_ == 1) {
                        t3[0] = wave_shift<kWaveShr1>(v[0]);
                        t3[1] = v[0];
                        t3[2] = wave_shift<kWaveShl1>(v[0]);
                    } else {
                        t3[0] = v[0];
                        t3[1] = v[NC - 1];
                        t3[2] = wave_shift<kWaveShl1>(v[0]);
                    }
#pragma unroll
                    for (int ky = 0; ky < 3; ++ky) {
                        const int tt = r - ky;
                        if (tt >= 0 && tt % S_ == 0 && tt / S_ < R) {
#pragma unroll
                            for (int k = 0; k < 3; ++k) {
                                if (ky == 0 && k == 0) E::fma8_from(acc2[tt / S_], bias2, w[0], t3[0]);
                                else E::fma8(acc2[tt / S_], w[ky * 3 + k], t3[k]);
                            }
                        }
                    }
                }
                if (gv && ox < p.OW) {
                    h8 *dout = dtile + sl * OPS + t * orows * p.OW + (oy0 - oy_lo) * p.OW + ox;
#pragma unroll
                    for (int o = 0; o < R; ++o) {
                        if (oy0 + o >= oy_hi) break;
                        float q[8];
#pragma unroll
                        for (int c = 0; c < 8; ++c) q[c] = __builtin_amdgcn_fmed3f(acc2[o][c], lo2, hi2);
                        *dout = E::pack(q);
                        dout += p.OW;
                    }
                }
            }
            for (int e = tid; e < (NSL - nsv) * OPS; e += NW * 64) dtile[nsv * OPS + e] = zero_h8();
        }
        __syncthreads();

        // 5. projection over the chunk's K-steps
        for (int kl = 0; kl < KSC; ++kl) {
            if (ct * KSC + kl >= pks) break;
            h8 b[FPW];
#pragma unroll
            for (int j = 0; j < FPW; ++j)
                if (fo[j]) b[j] = dtile[(kl * 4 + (lane >> 4)) * OPS + (pg + j * PG) * 16 + (lane & 15)];
#pragma unroll
            for (int i = 0; i < OBW; ++i) {
                const int ob = og + i * OG;
                if (ob >= p.pnb16) break;
                const h8 a = RES ? ptile[(ob * pks + ct * KSC + kl) * 64 + lane] : ptile[(ob * KSC + kl) * 64 + lane];
#pragma unroll
                for (int j = 0; j < FPW; ++j)
                    if (fo[j]) pacc[i][j] = E::mma(a, b[j], pacc[i][j]);
            }
        }
    }

    // 6. projection epilogue: pact1, + residual, pact2, sliced store (each
    // lane writes 4 channels of one pixel; a wave's store covers two whole
    // 16-pixel slices)
#pragma unroll
    for (int i = 0; i < OBW; ++i) {
        const int ob = og + i * OG;
        if (ob >= p.pnb16) break;
        const int os = 2 * ob + ((lane >> 4) >> 1), half = 4 * ((lane >> 4) & 1);
#pragma unroll
        for (int j = 0; j < FPW; ++j) {
            if (!fo[j]) continue;
            const int q = (pg + j * PG) * 16 + (lane & 15);
            if (q >= OP || os >= p.ps) continue;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = act_apply(pacc[i][j][r], p.pact1);
            const size_t off = ((size_t)os * p.MO + mo0 + q) * 8 + half;   // in 16-bit values
            if (p.res) {
                const h4 rv = *(const h4 *)((const _Float16 *)p.res + off);
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = act_apply(v[r] + E::get4(rv, r), p.pact2);
            }
            *(h4 *)((_Float16 *)p.y + off) = E::pack4(v);
        }
    }
}

// ---------------------------------------------------------------------------
// Instances: the expansion tiling and depthwise geometry as in the fused
// pointwise -> depthwise kernel, plus the projection's wave layout (PG pixel
// groups of FPW fragments) and output blocks (at most NBO).
// ---------------------------------------------------------------------------
namespace {

struct Inst {
    bool band;
    int nw, cs, fmw, nbt, s, r, lpr, pf, pg, fpw, nbo;
    const char *name;
    bool res = false;    // every weight resident in LDS, loaded once (needs K <= 32 * pf)
};

constexpr Inst kInsts[] = {
    // (K-steps of activation prefetch: 1 for the 16..32-channel block inputs
    // of the wide planes, 2 for 64, 4 above)
    // 112 -> 56 (one output row per band), 56 x 56, 56 -> 28
    {true, 8, 1, 3, 2, 2, 1, 64, 1, 4, 1, 2, "irb1x64c32"},  {true, 8, 1, 3, 6, 2, 1, 64, 1, 4, 1, 2, "irb1x64c96"},
    {true, 8, 1, 2, 4, 1, 2, 64, 1, 8, 1, 2, "irb2x64c64"},  {true, 8, 1, 2, 2, 1, 2, 64, 1, 8, 1, 2, "irb2x64c32"},
    {true, 8, 1, 3, 4, 2, 2, 32, 1, 4, 1, 2, "irb2x32c64"},
    // 28 x 28, 28 -> 14
    {true, 8, 1, 2, 4, 1, 4, 32, 1, 8, 1, 2, "irb4x32c64"},  {true, 8, 1, 2, 4, 2, 4, 16, 1, 4, 1, 4, "irb4x16c64"},
    // resident weights: 112 -> 56, 56 x 56, 56 -> 28, 28 x 28, 28 -> 14, 14 x 14
    {true, 8, 1, 3, 2, 2, 1, 64, 1, 4, 1, 2, "irb1x64c32r", true},  {true, 8, 1, 3, 6, 2, 1, 64, 1, 4, 1, 2, "irb1x64c96r", true},
    {true, 8, 1, 2, 4, 1, 2, 64, 1, 8, 1, 2, "irb2x64c64r", true},  {true, 8, 1, 2, 2, 1, 2, 64, 1, 8, 1, 2, "irb2x64c32r", true},
    {true, 8, 1, 3, 4, 2, 2, 32, 1, 4, 1, 2, "irb2x32c64r", true},  {true, 8, 1, 2, 4, 1, 4, 32, 1, 8, 1, 2, "irb4x32c64r", true},
    {true, 8, 1, 2, 4, 2, 4, 16, 1, 4, 1, 4, "irb4x16c64r", true},
    {true, 8, 2, 2, 8, 1, 4, 16, 2, 4, 1, 2, "irb4x16c128r", true}, {true, 8, 2, 2, 8, 1, 4, 16, 2, 4, 1, 4, "irb4x16c128r", true},
    {true, 8, 2, 2, 8, 1, 4, 16, 2, 4, 1, 6, "irb4x16c128r", true},
    // 14 x 14 (up to 32, 64 and 96 output channels), 14 -> 7
    {true, 8, 2, 2, 8, 1, 4, 16, 4, 4, 1, 2, "irb4x16c128"}, {true, 8, 2, 2, 8, 1, 4, 16, 4, 4, 1, 4, "irb4x16c128"},
    {true, 8, 2, 2, 8, 1, 4, 16, 4, 4, 1, 6, "irb4x16c128"}, {true, 8, 2, 1, 8, 1, 2, 16, 4, 2, 1, 2, "irb2x16c128"},
    {true, 8, 2, 1, 8, 1, 2, 16, 4, 2, 1, 4, "irb2x16c128"}, {true, 8, 2, 1, 8, 1, 2, 16, 4, 2, 1, 6, "irb2x16c128"},
    {true, 8, 2, 2, 8, 2, 2, 8, 4, 1, 1, 10, "irb2x8c128"},
    // 7 x 7 (160 and 320 output channels)
    {true, 8, 8, 2, 8, 1, 2, 8, 4, 1, 1, 10, "irb2x8c128"},  {true, 8, 8, 2, 8, 1, 2, 8, 4, 1, 1, 20, "irb2x8c128"},
};
constexpr int kNumInsts = sizeof(kInsts) / sizeof(kInsts[0]);

int lanes_for(int OW) { return OW < 8 ? 8 : OW < 16 ? 16 : OW < 32 ? 32 : OW < 64 ? 64 : 0; }

struct Geom {
    int ipt, nbands, groups, pstride, opstride;
    size_t lds;
};

bool fits(const Inst &in, int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16, int pnb16,
          Geom *g) {
    if (S != in.s || lanes_for(OW) != in.lpr || pt < 0) return false;
    if (pnb16 > in.nbo || (in.nbo > 2 && pnb16 <= (in.nbo == 20 ? 10 : in.nbo == 10 ? 6 : in.nbo == 6 ? 4 : 2)))
        return false;   // the smallest instance whose output blocks cover the projection
    if ((uint64_t)ksp * (uint64_t)N * (uint64_t)H * (uint64_t)W * 16u > 0xffffffffull) return false;
    if (S == 1 ? (pl != 1 || W >= in.lpr) : ((pl != 0 && pl != 1) || W > 2 * in.lpr - 1)) return false;
    const int pmax = 16 * in.nw / in.cs * in.fmw;
    int op;
    if (!in.band) {
        if (H * W > pmax) return false;
        g->ipt = pmax / (H * W);
        g->nbands = 0;
        g->groups = (N + g->ipt - 1) / g->ipt;
        g->pstride = g->ipt * H * W;
        op = g->ipt * OH * OW;
    } else {
        const int rows = std::min((in.r - 1) * S + 3, H);
        if (rows * W > pmax) return false;
        g->ipt = 1;
        g->nbands = (OH + in.r - 1) / in.r;
        g->groups = N * g->nbands;
        g->pstride = rows * W;
        op = std::min(in.r, OH) * OW;
    }
    const int nof = (op + 15) / 16;
    if (nof > in.pg * in.fpw) return false;
    g->opstride = 16 * nof;
    const size_t nk = (size_t)ksp / 4, nkc = (nk + in.pf - 1) / in.pf;
    const size_t nsl = 2 * (size_t)in.nbt, nch = 16 * (size_t)in.nbt;
    const size_t etile = nsl * g->pstride * 16, dtile = nsl * g->opstride * 16;
    if (in.res) {
        // (the kernel's resident layout; projection K-steps at most ceil(2 nb16 / 4))
        if (nk > (size_t)in.pf) return false;
        const size_t pks = (2 * (size_t)nb16 + 3) / 4;
        g->lds = ((size_t)nb16 * nk * 64 + 64 * ((2 * (size_t)nb16 * 9 + 63) / 64) +
                  2 * 64 * ((4 * (size_t)nb16 + 63) / 64) + pks * pnb16 * 64 + 64) * 16 + etile + dtile;
    } else {
        const size_t slab = nkc * in.nbt * in.pf * 64 * 16;
        const size_t tail = (64 * ((nsl * 9 + 63) / 64) + 128 * ((nch / 4 + 63) / 64) + 64) * 16;
        g->lds = std::max(slab, etile) + tail + dtile + (size_t)in.nbo * (nsl / 4) * 64 * 16;
    }
    return g->lds <= (size_t)kIrbLds;
}

template <typename E, int K>
hipError_t launch_t(const IrbParams &p, size_t lds, hipStream_t st) {
    constexpr Inst in = kInsts[K];
    // (resident instances have no deep form: they run only when K fits the prefetch slots)
    auto deep = irb_kernel<E, in.nw, in.cs, in.fmw, in.nbt, in.s, in.r, in.lpr, in.pf, !in.res, in.pg, in.fpw, in.nbo,
                           in.res>;
    auto shallow = irb_kernel<E, in.nw, in.cs, in.fmw, in.nbt, in.s, in.r, in.lpr, in.pf, false, in.pg, in.fpw,
                              in.nbo, in.res>;
    static const hipError_t attr = [&] {
        const hipError_t e = hipFuncSetAttribute((const void *)deep, hipFuncAttributeMaxDynamicSharedMemorySize, kIrbLds);
        return e != hipSuccess
                   ? e
                   : hipFuncSetAttribute((const void *)shallow, hipFuncAttributeMaxDynamicSharedMemorySize, kIrbLds);
    }();
    if (attr != hipSuccess) return attr;
    auto kern = (p.ksp >> 2) > in.pf ? deep : shallow;
    const int groups = p.nbands ? p.N * p.nbands : (p.N + p.ipt - 1) / p.ipt;
    launch(kern, dim3(groups), dim3(in.nw * 64), (unsigned)lds, st, p);
    return hipGetLastError();
}

template <typename E, size_t... K>
hipError_t launch_any(int k, const IrbParams &p, size_t lds, hipStream_t st, std::index_sequence<K...>) {
    hipError_t r = hipErrorInvalidValue;
    (void)((k == (int)K && ((r = launch_t<E, (int)K>(p, lds, st)), true)) || ...);
    return r;
}

int applicable(int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16, int pnb16, int *idx,
               Geom *geo) {
    int n = 0;
    for (int k = 0; k < kNumInsts; ++k) {
        Geom g{};
        if (!fits(kInsts[k], N, H, W, OH, OW, S, pt, pl, ksp, nb16, pnb16, &g)) continue;
        if (idx) idx[n] = k;
        if (geo) geo[n] = g;
        ++n;
    }
    return n;
}
}  // namespace

int irb_configs(int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16, int pnb16, int cfg,
                const char **name, int *groups) {
    int idx[kNumInsts];
    Geom geo[kNumInsts];
    const int n = applicable(N, H, W, OH, OW, S, pt, pl, ksp, nb16, pnb16, idx, geo);
    if (cfg >= 0 && cfg < n) {
        if (name) *name = kInsts[idx[cfg]].name;
        if (groups) *groups = geo[cfg].groups;
    }
    return n;
}

hipError_t launch_irb(const IrbParams &p, int cfg, hipStream_t st) {
    int idx[kNumInsts];
    Geom geo[kNumInsts];
    const int n = applicable(p.N, p.H, p.W, p.OH, p.OW, p.S, p.pt, p.pl, p.ksp, p.nb16, p.pnb16, idx, geo);
    if (cfg < 0 || cfg >= n || p.M != p.N * p.H * p.W || p.MO != p.N * p.OH * p.OW || p.ksp % 4 != 0 ||
        p.pksp % 4 != 0 || p.nb16 <= 0 || p.pnb16 <= 0 || p.pksp < 2 * p.nb16 ||
        p.pksp > 4 * ((2 * p.nb16 + 3) / 4))
        return hipErrorInvalidValue;
    const Geom &g = geo[cfg];
    IrbParams q = p;
    q.ipt = g.ipt;
    q.nbands = g.nbands;
    q.pstride = g.pstride;
    q.opstride = g.opstride;
    if (p.N <= 0) return hipSuccess;
    return p.bf16 ? launch_any<BF16>(idx[cfg], q, g.lds, st, std::make_index_sequence<kNumInsts>{})
                  : launch_any<F16>(idx[cfg], q, g.lds, st, std::make_index_sequence<kNumInsts>{});
}

}  // namespace kern
}  // namespace mgi
