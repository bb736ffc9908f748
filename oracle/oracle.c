/*
 * Plain CPU oracle for the forward pass of MobileNet-class networks.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header or helper with the
 * HIP engine.
 *
 * Every operator is written out from its plain definition, in double
 * precision, on NHWC tensors, with direct loops: no im2col, no blocking, no
 * BLAS, no intrinsics.  The only concession to speed is an OpenMP pragma on
 * the outermost (image, output-row) loop, which does not change any result
 * (each output element is still one sequential sum).
 *
 * Operators (what the paper's engine runs, Sec. 3 and Sec. 4.1):
 *   - 2D convolution over a (kernel_height x kernel_width) window, with
 *     stride, dilation and explicit four-sided zero padding (the paper folds a
 *     separate PAD op into the convolution, Sec. 3.1).
 *   - depthwise convolution (channel multiplier 1).
 *   - element-wise activations that the paper fuses into the preceding heavy
 *     op (Sec. 3.2): identity, ReLU, ReLU6.
 *   - element-wise ADD, CONCAT along channels, bilinear RESIZE (Sec. 3.1).
 *   - global average pool, fully-connected, softmax and per-pixel argmax (the
 *     classification / segmentation heads of the networks of Sec. 6).
 */
#include <math.h>
#include <omp.h>
#include <stddef.h>

/* Thread count of the OpenMP loops below (timing only; results do not depend
 * on it). */
void orc_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
int orc_max_threads(void) { return omp_get_max_threads(); }

#define IDX4(n, y, x, c, H, W, C) ((((size_t)(n) * (H) + (y)) * (W) + (x)) * (C) + (c))

/* y[n,oy,ox,co] = b[co] + sum_{ky,kx,ci} w[co,ky,kx,ci] * x~[n, oy*sh+ky*dh-pt, ox*sw+kx*dw-pl, ci]
 * where x~ is x with zeros outside [0,H) x [0,W).  w is OHWI. */
void orc_conv2d(const double *x, int N, int H, int W, int C,
                const double *w, const double *b, int CO, int KH, int KW,
                int sh, int sw, int dh, int dw, int pt, int pl,
                double *y, int OH, int OW)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int oy = 0; oy < OH; ++oy)
            for (int ox = 0; ox < OW; ++ox)
                for (int co = 0; co < CO; ++co) {
                    double acc = b ? b[co] : 0.0;
                    for (int ky = 0; ky < KH; ++ky) {
                        int iy = oy * sh + ky * dh - pt;
                        if (iy < 0 || iy >= H) continue;
                        for (int kx = 0; kx < KW; ++kx) {
                            int ix = ox * sw + kx * dw - pl;
                            if (ix < 0 || ix >= W) continue;
                            const double *xp = x + IDX4(n, iy, ix, 0, H, W, C);
                            const double *wp = w + (((size_t)co * KH + ky) * KW + kx) * C;
                            for (int ci = 0; ci < C; ++ci)
                                acc += wp[ci] * xp[ci];
                        }
                    }
                    y[IDX4(n, oy, ox, co, OH, OW, CO)] = acc;
                }
}

/* y[n,oy,ox,c] = b[c] + sum_{ky,kx} w[c,ky,kx] * x~[n, oy*sh+ky*dh-pt, ox*sw+kx*dw-pl, c] */
void orc_depthwise(const double *x, int N, int H, int W, int C,
                   const double *w, const double *b, int KH, int KW,
                   int sh, int sw, int dh, int dw, int pt, int pl,
                   double *y, int OH, int OW)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int oy = 0; oy < OH; ++oy)
            for (int ox = 0; ox < OW; ++ox)
                for (int c = 0; c < C; ++c) {
                    double acc = b ? b[c] : 0.0;
                    for (int ky = 0; ky < KH; ++ky) {
                        int iy = oy * sh + ky * dh - pt;
                        if (iy < 0 || iy >= H) continue;
                        for (int kx = 0; kx < KW; ++kx) {
                            int ix = ox * sw + kx * dw - pl;
                            if (ix < 0 || ix >= W) continue;
                            acc += w[((size_t)c * KH + ky) * KW + kx] * x[IDX4(n, iy, ix, c, H, W, C)];
                        }
                    }
                    y[IDX4(n, oy, ox, c, OH, OW, C)] = acc;
                }
}

/* act: 0 identity, 1 ReLU = max(v, 0), 2 ReLU6 = min(max(v, 0), 6); in place. */
void orc_activation(double *v, size_t count, int act)
{
    if (act == 0) return;
    for (size_t i = 0; i < count; ++i) {
        double t = v[i] > 0.0 ? v[i] : 0.0;
        if (act == 2 && t > 6.0) t = 6.0;
        v[i] = t;
    }
}

/* y = a + b, element-wise. */
void orc_add(const double *a, const double *b, double *y, size_t count)
{
    for (size_t i = 0; i < count; ++i) y[i] = a[i] + b[i];
}

/* y[n,c] = (1 / (H*W)) * sum_{h,w} x[n,h,w,c] */
void orc_global_avgpool(const double *x, int N, int H, int W, int C, double *y)
{
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c) {
            double s = 0.0;
            for (int h = 0; h < H; ++h)
                for (int w = 0; w < W; ++w)
                    s += x[IDX4(n, h, w, c, H, W, C)];
            y[(size_t)n * C + c] = s / ((double)H * W);
        }
}

/* y[n,j] = b[j] + sum_k w[j,k] * x[n,k]; w is COUT x CIN. */
void orc_fc(const double *x, int N, int CIN, const double *w, const double *b, int COUT, double *y)
{
    for (int n = 0; n < N; ++n)
        for (int j = 0; j < COUT; ++j) {
            double acc = b ? b[j] : 0.0;
            for (int k = 0; k < CIN; ++k)
                acc += w[(size_t)j * CIN + k] * x[(size_t)n * CIN + k];
            y[(size_t)n * COUT + j] = acc;
        }
}

/* Row-wise softmax over the last axis: exp(z - max z) / sum exp(z - max z). */
void orc_softmax(const double *z, int rows, int cols, double *y)
{
    for (int r = 0; r < rows; ++r) {
        const double *zr = z + (size_t)r * cols;
        double *yr = y + (size_t)r * cols;
        double m = zr[0];
        for (int j = 1; j < cols; ++j) if (zr[j] > m) m = zr[j];
        double s = 0.0;
        for (int j = 0; j < cols; ++j) { yr[j] = exp(zr[j] - m); s += yr[j]; }
        for (int j = 0; j < cols; ++j) yr[j] /= s;
    }
}

/* Channel concat of a (Ca channels) then b (Cb channels); equal N, H, W. */
void orc_concat2(const double *a, int Ca, const double *b, int Cb, size_t pixels, double *y)
{
    int C = Ca + Cb;
    for (size_t p = 0; p < pixels; ++p) {
        for (int c = 0; c < Ca; ++c) y[p * C + c] = a[p * Ca + c];
        for (int c = 0; c < Cb; ++c) y[p * C + Ca + c] = b[p * Cb + c];
    }
}

/* Source coordinate of output index d for a resize from `in` to `out` samples.
 * align_corners: the corner samples of input and output coincide,
 *   src = d * (in - 1) / (out - 1)  (0 when out == 1);
 * otherwise the plain scale src = d * in / out. */
static double src_coord(int d, int in, int out, int align_corners)
{
    if (align_corners) return out > 1 ? (double)d * (in - 1) / (out - 1) : 0.0;
    return (double)d * in / out;
}

/* Bilinear resize: 4-tap interpolation between floor(src) and floor(src)+1,
 * the upper neighbour clamped to the last sample. */
void orc_resize_bilinear(const double *x, int N, int H, int W, int C,
                         double *y, int OH, int OW, int align_corners)
{
    for (int n = 0; n < N; ++n)
        for (int oy = 0; oy < OH; ++oy) {
            double sy = src_coord(oy, H, OH, align_corners);
            int y0 = (int)floor(sy);
            if (y0 > H - 1) y0 = H - 1;
            int y1 = y0 + 1 < H ? y0 + 1 : H - 1;
            double fy = sy - y0;
            for (int ox = 0; ox < OW; ++ox) {
                double sx = src_coord(ox, W, OW, align_corners);
                int x0 = (int)floor(sx);
                if (x0 > W - 1) x0 = W - 1;
                int x1 = x0 + 1 < W ? x0 + 1 : W - 1;
                double fx = sx - x0;
                for (int c = 0; c < C; ++c) {
                    double v00 = x[IDX4(n, y0, x0, c, H, W, C)];
                    double v01 = x[IDX4(n, y0, x1, c, H, W, C)];
                    double v10 = x[IDX4(n, y1, x0, c, H, W, C)];
                    double v11 = x[IDX4(n, y1, x1, c, H, W, C)];
                    y[IDX4(n, oy, ox, c, OH, OW, C)] =
                        (1.0 - fy) * ((1.0 - fx) * v00 + fx * v01) +
                        fy * ((1.0 - fx) * v10 + fx * v11);
                }
            }
        }
}

/* Per-pixel index of the largest channel value; ties go to the lowest index. */
void orc_argmax(const double *x, size_t pixels, int C, int *y)
{
    for (size_t p = 0; p < pixels; ++p) {
        int best = 0;
        for (int c = 1; c < C; ++c)
            if (x[p * C + c] > x[p * C + best]) best = c;
        y[p] = best;
    }
}
