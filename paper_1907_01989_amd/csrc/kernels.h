// Kernel parameter blocks and launchers (internal to the engine).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "../../include/mgi.h"

namespace mgi {
namespace kern {

// Optional timestamps for the next kernel launch on this thread: when set,
// launches go through hipExtLaunchKernelGGL, which records `start` when the
// kernel begins and `stop` when it ends on the device.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents &launch_events();

template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, unsigned lds, hipStream_t st, Args... args) {
    const LaunchEvents &ev = launch_events();
    if (ev.start || ev.stop)
        hipExtLaunchKernelGGL(kernel, grid, block, lds, st, ev.start, ev.stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, st, args...);
}

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));

// C = act2(act1(W * X + bias) + residual): MFMA GEMM over sliced activations.
struct GemmParams {
    const h8 *x;         // sliced input, [slices][Min] of 8 halves
    const h8 *w;         // packed weights [nb16][ksp][16][8]
    const float *bias;   // [nb16 * 16]
    const h8 *res;       // sliced residual with the output's shape, or null
    void *y;             // sliced fp16 output, or fp32 (M x cout) for FC
    int M;               // output pixels (n * oh * ow)
    int Min;             // input pixels (n * h * w)
    int ksl, ksp;        // K slices, and padded to a multiple of 4
    int nb16, ns, cout;  // output blocks of 16, output slices, channels
    int act1, act2;
    int mtiles, ntiles;
    int bf16;            // storage type: 0 fp16, 1 bf16
    // implicit-GEMM window geometry
    int H, W, OH, OW, sin, kw, sh, sw, dh, dw, pt, pl;
    // pooled GEMM: pixels per image, images, images per M-tile (set by the launcher)
    int hw, nimg, ipt;
    // FC with the softmax of its rows (sm_y non-null): probabilities (M x cout)
    // and one arrival counter per tile of 16 * fm rows (zero before the launch,
    // zero after it)
    float *sm_y;
    int *sm_cnt;
};
hipError_t launch_gemm(const GemmParams &p, int bm, int bn, bool taps, bool f32out,
                       hipStream_t st);
// pointwise (1x1, stride 1) GEMM with fp16 sliced output: the tile's weight
// slab in LDS, activations streamed to registers; tile (4 * wm) pixels x bn
// channels, pf K steps of activation prefetch.  Needs
// gemm_xs_lds_bytes(ksp, wm, bn) <= 160 KiB and zero weights for padded K.
// pool: the output feeds only a global average pool (as launch_gemm_pool:
// hw, nimg set, M = nimg * hw, hw <= 64; wm 16, bn 16/32/64, pf 2/8); y
// receives the pooled means.
hipError_t launch_gemm_xs(const GemmParams &p, int wm, int bn, int pf, bool pool, hipStream_t st);
// pointwise GEMM with both operands in a 4-stage LDS ring fed by direct
// global->LDS loads; tile bm pixels x bn channels, bm, bn in {64, 128}
hipError_t launch_gemm_pipe(const GemmParams &p, int bm, int bn, hipStream_t st);
// the pipelined GEMM with 64x64 tiles and 8 K slices per ring stage (two
// MFMA K-steps; needs ksp % 8 == 0), plain or pooled (as launch_gemm_pool);
// same accumulation order as the 4-slice stages
hipError_t launch_gemm_pipe_k8(const GemmParams &p, bool pool, hipStream_t st);
// pointwise GEMM whose output feeds only a global average pool: M-tiles of
// bm rows hold bm / hw whole images (hw <= 64 pixels each, M = nimg * hw),
// and the pooled means are written, sliced [ns][nimg], bit-identical to the
// GEMM followed by the pool kernel
hipError_t launch_gemm_pool(const GemmParams &p, int bm, int bn, hipStream_t st);
// fully-connected layer, fp32 (M x cout) output; K split over the waves; a
// workgroup takes 16 * fm images (1, 2 or 4; 0 = by M) and loads kb K-steps
// (4 or 8; 0 = 4) at once.  Results do not depend on fm or kb.  With
// p.sm_y set, the softmax of every row follows in the same launch (p.sm_cnt:
// ceil(M / (16 * fm)) counters, zero on entry and left at zero).
hipError_t launch_fc(const GemmParams &p, int fm, int kb, hipStream_t st);
size_t gemm_xs_lds_bytes(int ksp, int wm, int bn);

// Depthwise 3x3 (stride 1 or 2, dilation 1) fused into the pointwise GEMM
// that consumes it: x is the depthwise input (sliced, N*H*W pixels per
// slice, K = g.ksl slices), g describes the pointwise GEMM (g.x unused).
struct DwPwParams {
    const h8 *x;
    const h8 *dww;       // fp16 taps [ksl][9][8]
    const float *dwb;    // [ksl * 8]
    const h8 *zero;      // one zeroed element
    int N, H, W, OH, OW, sh, sw, pt, pl, act;
    GemmParams g;
};
// Workgroup tile: RB whole output rows of one image (RB divides OH,
// RB * OW <= 64 * fmw); the input band of a chunk is NRB rows of WP elements
// for each of four slices, at most kDwPwBandMax elements.
constexpr int kDwPwBandMax = 2304;
struct DwPwTile {
    int RB = 0, nbands = 0, NRB = 0, WP = 0, fmw = 2;
    float inv_per = 0, inv_wp = 0, inv_ow = 0;
};
// band of at most max_px (64 or 128) pixels; false when no band fits
bool dwpw_tile(int OH, int OW, int S, int N, DwPwTile &t, int max_px = 128);
hipError_t launch_dwpw(const DwPwParams &p, const DwPwTile &t, hipStream_t st);
// channel blocks the kernel instance computes for nb16 output blocks (0: too many)
int dwpw_blocks(int nb16);

// Direct convolution of a small-channel NHWC graph input (kh*kw*c <= 32).
struct StemParams {
    const void *x;       // NHWC fp32 or fp16
    const h8 *w;         // packed [nb16][4][16][8], k = (ky*kw + kx)*c + ci
    const float *bias;
    const h8 *res;
    h8 *y;
    int N, H, W, C, OH, OW, M;
    int KH, KW, K, sh, sw, dh, dw, pt, pl;
    int nb16, ns, act1, act2;
    int bf16;            // storage type: 0 fp16, 1 bf16
    int koff[32];        // set by launch_stem: offset of im2col entry k in the LDS band
};
hipError_t launch_stem(const StemParams &p, bool fp16_in, hipStream_t st);
// LDS bytes the stem kernel stages for a band of th output rows, and at most
// for its output staging (4 waves x 4 channel blocks x 1 KiB)
constexpr size_t kStemStageBytes = 16384;
size_t stem_band_bytes(int th, int kh, int kw, int c, int w, int ow, int sh, int sw, int dh, int dw,
                       int pl);

// Stem convolution fused with the depthwise 3x3 convolution (stride 1,
// dilation 1) that reads its output: a workgroup owns R output rows of one
// image and computes the stem rows they read into LDS.
struct StemDwParams {
    const void *x;       // NHWC graph input, fp32 or fp16
    const h8 *w;         // stem weights [nb16][4][16][8], k = (ky*kw + kx)*c + ci
    const float *bias;   // [nb16 * 16]
    int N, H, W, C, SH, SW;          // input size and stem output size
    int KH, KW, K, sh, sw, dh, dw, pt, pl, nb16, act1;
    const h8 *dw_w;      // depthwise taps [2 * nb16][9][8]
    const float *dw_b;   // [16 * nb16]
    h8 *y;               // depthwise output, sliced [ns][N * OH * OW]
    int OH, OW, S, dpt, dpl, ns, act2;
    int nbands, rs, pstride, band_h8; // set by launch_stemdw from the configuration
    int srows, qi, vec;  // rolling strips: output rows per strip, input-ring slots, 16-byte input loads
    int fp16_in;         // the graph input is fp16 (else fp32)
    int bf16;            // storage type: 0 fp16, 1 bf16
    int koff[32];        // set by launch_stemdw: offset of im2col entry k in the LDS band
};
// A stem window (kh*kw*c <= 32 entries) is one MFMA K step of 32 positions.
// Entry (ky, kx, ci) sits at position (ky*kw + kx)*c + ci, except in
// row-aligned windows -- 3 rows of 9 entries (kw*c = 9, no horizontal
// dilation: the 3x3 stem over RGB) -- where row ky's first 8 entries take
// positions 8*ky .. 8*ky+7 and its 9th takes 24 + 2*ky (positions 25, 27,
// 29, 30, 31 hold zero weights): 8 consecutive positions are then 8
// consecutive values of one staged input row.
bool stem_row_aligned(int KH, int KW, int C, int dw);
int stem_kpos(int ky, int kx, int ci, int KH, int KW, int C, int dw);
// offset of the value that im2col position k < 32 reads inside an input band
// of row stride rs (positions with zero weights read values that are staged
// anyway: the next value of the same row, or the band's first)
void im2col_offsets(int *koff, int K, int KH, int C, int KW, int dh, int dw, int rs);
// row stride, in 16-bit values (a multiple of 8), of a staged input band for
// output width ow: every window value, and for row-aligned windows the value
// after each row's 9th, lies inside the row
int stem_row_stride(int c, int w, int ow, int sw, int kh, int kw, int dw, int pl);
struct StemDwGeom {
    int rows, group, threads, nbands, rs, pstride, band_h8;
    int roll, srows, qi, vec, prod;
    size_t lds;
};
// Number of fused configurations (band heights) that fit a shape (0: none);
// for 0 <= cfg < that number, its geometry and name.
int stemdw_configs(const StemDwParams &p, int cfg, StemDwGeom *g, const char **name);
hipError_t launch_stemdw(const StemDwParams &p, int cfg, bool fp16_in, hipStream_t st);

// reciprocals of a kernel's index divisors (see divmod_fast)
struct DivConsts {
    double inv_ow, inv_nstrips, inv_n;
};

struct DwParams {
    const h8 *x;
    const h8 *w;         // fp16 taps [S][kh*kw][8]
    const float *bias;   // [S*8]
    const h8 *zero;      // one zeroed 16-byte element (read for taps outside the input)
    h8 *y;
    int N, H, W, S, OH, OW, KH, KW, sh, sw, dh, dw, pt, pl, act;
    int bf16;            // storage type: 0 fp16, 1 bf16
};
// rows: output rows per thread of the 3x3 kernel (1, 2, 4 or 8; 0 = default)
hipError_t launch_depthwise(const DwParams &p, int rows, hipStream_t st);

// Pointwise convolution fused with the depthwise 3x3 convolution (dilation 1,
// stride 1 or 2) that consumes its output: a workgroup owns a channel tile and
// whole images or a band of output rows (with the input rows they read), so
// the depthwise step needs no data from other workgroups.
struct PwDwParams {
    const h8 *x;         // pointwise input, sliced [ksl][M]
    const h8 *w;         // packed pointwise weights [nb16][ksp][16][8]
    const float *bias;   // [nb16 * 16]
    int M, ksl, ksp, nb16, act1;
    const h8 *dw_w;      // depthwise taps [2 * nb16][9][8] (zero past the channels)
    const float *dw_b;   // [16 * nb16]
    h8 *y;               // depthwise output, sliced [ns][N * OH * OW]
    int ns;              // output slices: 2 * nb16, or one fewer (channels = 8 mod 16)
    int N, H, W, OH, OW, S, pt, pl, act2;
    int ipt, nbands, ntiles;   // set by launch_pwdw from the configuration
    int pstride;         // ... pixel stride of the LDS output tile
    int bf16;            // storage type: 0 fp16, 1 bf16
};
// Tiling of one configuration: images per tile (whole-image tiles) or bands
// per image, tile groups, channel blocks per tile, LDS bytes.
struct PwDwGeom {
    int ipt, nbands, groups, nbt, pstride;
    size_t lds;
};
// Number of fused-kernel configurations that cover a shape (0: none); for
// 0 <= cfg < that number, its geometry and name.
int pwdw_configs(int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16, int cfg,
                 PwDwGeom *g, const char **name);
hipError_t launch_pwdw(const PwDwParams &p, int cfg, hipStream_t st);

// MobileNet-v2 inverted residual block in one kernel: pointwise expansion
// (+ bias, act1), depthwise 3x3 (+ bias, act2) and pointwise projection
// (+ bias, pact1, + residual, pact2).  A workgroup owns a band of output rows
// of one image, or whole images, and walks all expansion channels in chunks;
// the expanded and depthwise tensors stay in LDS.
struct IrbParams {
    const h8 *x;         // block input, sliced [ksl][M]
    const h8 *w;         // packed expansion weights [nb16][ksp][16][8]
    const float *bias;   // [nb16 * 16]
    int M, ksl, ksp, nb16, act1;
    const h8 *dw_w;      // depthwise taps [2 * nb16][9][8]
    const float *dw_b;   // [16 * nb16]
    int ns, act2;        // expansion slices (2 * nb16, or one fewer), depthwise activation
    const h8 *pw;        // packed projection weights [pnb16][pksp][16][8], K = expansion channels
    const float *pbias;  // [pnb16 * 16]
    int pksp, pnb16, pact1, pact2;
    const h8 *res;       // residual, sliced like the output, or null
    h8 *y;               // output, sliced [ps][MO]
    int ps, MO;          // output slices and pixels
    int N, H, W, OH, OW, S, pt, pl;
    int ipt, nbands;     // set by launch_irb from the configuration
    int pstride;         // ... pixel stride of the LDS expansion tile
    int opstride;        // ... and of the LDS depthwise tile
    int bf16;            // storage type: 0 fp16, 1 bf16
};
// Number of configurations of the block kernel that cover a shape (0: none);
// for 0 <= cfg < that number, its name and workgroup count.  pnb16: output
// channel blocks of the projection.
int irb_configs(int N, int H, int W, int OH, int OW, int S, int pt, int pl, int ksp, int nb16, int pnb16, int cfg,
                const char **name, int *groups);
hipError_t launch_irb(const IrbParams &p, int cfg, hipStream_t st);

hipError_t launch_add(const h8 *a, const h8 *b, h8 *y, size_t count, int act, bool bf16, hipStream_t st);
// zero padding of a sliced tensor: (N, H, W) planes of S slices -> (N, OH, OW),
// input placed at row pt, column pl
hipError_t launch_pad(const h8 *x, h8 *y, int N, int S, int H, int W, int OH, int OW, int pt, int pl,
                      hipStream_t st);
hipError_t launch_act(const h8 *x, h8 *y, size_t count, int act, bool bf16, hipStream_t st);
hipError_t launch_gap(const h8 *x, h8 *y, const h8 *zero, int N, int HW, int S, bool bf16,
                      hipStream_t st);
hipError_t launch_softmax(const float *z, float *y, int rows, int cols, hipStream_t st);

struct ConcatParams {
    const h8 *src[8];
    int coff[9];
    int nin;
    int M, S, C;
    h8 *y;
};
hipError_t launch_concat(const ConcatParams &p, hipStream_t st);

struct ResizeParams {
    const h8 *x;
    void *y;             // sliced output, or int32 labels (argmax)
    int N, H, W, S, C, OH, OW;
    int align_corners;
    int bf16;            // storage type: 0 fp16, 1 bf16
};
hipError_t launch_resize(const ResizeParams &p, bool argmax, hipStream_t st);
hipError_t launch_argmax(const h8 *x, int *y, int M, int S, int C, bool bf16, hipStream_t st);

hipError_t launch_ingest(const void *x, bool fp16_in, h8 *y, int M, int C, bool bf16, hipStream_t st);
// sets `words` 32-bit words at dst to zero with a kernel (no memset node in a
// captured graph)
hipError_t launch_zero_words(unsigned *dst, size_t words, hipStream_t st);
hipError_t launch_export(const h8 *x, float *y, int M, int C, bool bf16, hipStream_t st);

}  // namespace kern
}  // namespace mgi
