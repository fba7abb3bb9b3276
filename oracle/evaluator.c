/*
 * Oracle: plain direct evaluation of the operators of a CNN block.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * reference that the GPU library is checked against; the library never links,
 * loads or calls it.  Only tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.
 *
 * Every array is float64, NCHW, contiguous.  Each function is the textbook
 * definition written out as nested loops; there is no blocking, no
 * reordering and no fusion.  The paper runs its operators through cuDNN
 * (Sec. 5, implementation setup), so convolution is cross-correlation with
 * zero padding and floor output size.
 */
#include <math.h>
#include <stddef.h>

static int out_size(int in, int k, int s, int p) { return (in + 2 * p - k) / s + 1; }

/* Dense convolution ("Conv-Relu" schedule unit, Table 2):
 *   y[n,co,i,j] = b[co] + sum_{ci,u,v} w[co,ci,u,v] * xp[n,ci,i*sh+u-ph,j*sw+v-pw]
 * where xp is x with zeros outside its bounds; ReLU applied to x first if
 * pre_relu, and to y if post_relu. */
void oracle_conv2d(const double *x, int n, int c, int h, int w,
                   const double *wt, int cout, int kh, int kw,
                   int sh, int sw, int ph, int pw, const double *bias,
                   int pre_relu, int post_relu, double *y) {
  int ho = out_size(h, kh, sh, ph), wo = out_size(w, kw, sw, pw);
  for (int b = 0; b < n; ++b)
    for (int co = 0; co < cout; ++co)
      for (int i = 0; i < ho; ++i)
        for (int j = 0; j < wo; ++j) {
          double acc = bias ? bias[co] : 0.0;
          for (int ci = 0; ci < c; ++ci)
            for (int u = 0; u < kh; ++u)
              for (int v = 0; v < kw; ++v) {
                int r = i * sh + u - ph, q = j * sw + v - pw;
                if (r < 0 || r >= h || q < 0 || q >= w) continue;
                double xv = x[(((size_t)b * c + ci) * h + r) * w + q];
                if (pre_relu && xv < 0.0) xv = 0.0;
                acc += wt[(((size_t)co * c + ci) * kh + u) * kw + v] * xv;
              }
          if (post_relu && acc < 0.0) acc = 0.0;
          y[(((size_t)b * cout + co) * ho + i) * wo + j] = acc;
        }
}

/* Depthwise convolution (first half of "Relu-SepConv"): one kh x kw filter
 * per channel, stride 1, zero padding (ph, pw), no bias. */
void oracle_depthwise(const double *x, int n, int c, int h, int w,
                      const double *wt, int kh, int kw, int ph, int pw, double *y) {
  int ho = out_size(h, kh, 1, ph), wo = out_size(w, kw, 1, pw);
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch)
      for (int i = 0; i < ho; ++i)
        for (int j = 0; j < wo; ++j) {
          double acc = 0.0;
          for (int u = 0; u < kh; ++u)
            for (int v = 0; v < kw; ++v) {
              int r = i + u - ph, q = j + v - pw;
              if (r < 0 || r >= h || q < 0 || q >= w) continue;
              acc += wt[((size_t)ch * kh + u) * kw + v] *
                     x[(((size_t)b * c + ch) * h + r) * w + q];
            }
          y[(((size_t)b * c + ch) * ho + i) * wo + j] = acc;
        }
}

/* k x k pooling with stride s and padding p.  Max: maximum over the taps
 * that fall inside the input (padding never wins).  Average: sum of the taps
 * inside the input divided by k*k (padding counts as zero). */
void oracle_pool(const double *x, int n, int c, int h, int w,
                 int k, int s, int p, int is_max, double *y) {
  int ho = out_size(h, k, s, p), wo = out_size(w, k, s, p);
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch)
      for (int i = 0; i < ho; ++i)
        for (int j = 0; j < wo; ++j) {
          double acc = is_max ? -INFINITY : 0.0;
          for (int u = 0; u < k; ++u)
            for (int v = 0; v < k; ++v) {
              int r = i * s + u - p, q = j * s + v - p;
              if (r < 0 || r >= h || q < 0 || q >= w) continue;
              double xv = x[(((size_t)b * c + ch) * h + r) * w + q];
              if (is_max) { if (xv > acc) acc = xv; }
              else acc += xv;
            }
          y[(((size_t)b * c + ch) * ho + i) * wo + j] = is_max ? acc : acc / (double)(k * k);
        }
}
