/*
 * huge2_oracle.h -- CPU oracle for transposed and dilated 2-D convolution.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes,
 * links or calls this code; only the tests, the smoke check and the CPU
 * baseline leg of the benchmark do.  It shares no header, helper or table
 * with the GPU path.
 *
 * Everything is float64, NCHW, contiguous:
 *   x  [n][c_in][h][w]
 *   w  transposed conv: [c_in][c_out/groups][r][s]   (the paper's C x N x R x
 *                                              S of section 4.2 when groups = 1)
 *      dilated / strided conv: [c_out][c_in/groups][r][s]
 *   y  [n][c_out][h_out][w_out]
 *   bias  [c_out] or NULL
 *
 * Return value: 0 on success, -1 on an invalid descriptor.
 */
#ifndef HUGE2_ORACLE_H
#define HUGE2_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int n, c_in, h, w;
  int c_out, r, s;
  int stride_h, stride_w;
  int pad_h, pad_w;
  int out_pad_h, out_pad_w;
  int dil_h, dil_w;
  /* Grouped convolution (0 or 1: none): the channels split into `groups`
   * equal groups, and output channel k of group k / (c_out/groups) sums only
   * over the input channels of the same group (PyTorch's groups); the
   * weight gradients then join each weight element's input channel to the
   * output channels of its own group only. */
  int groups;
} oracle_conv;

/* Output size of the transposed conv: (h-1)*stride - 2*pad + dil*(r-1) + out_pad + 1. */
int oracle_transpose_out_dims(const oracle_conv* d, int* h_out, int* w_out);
/* Output size of the strided/dilated conv: floor((h + 2*pad - dil*(r-1) - 1)/stride) + 1. */
int oracle_conv_out_dims(const oracle_conv* d, int* h_out, int* w_out);

/* Algorithm 1 (section 2.1.1): materialise the zero-inserted input, then a
 * stride-1 correlation with the rotated, in/out-swapped kernel, multiplying
 * every term including the inserted zeros.  Parallel over (n, c_out) planes. */
int oracle_conv2d_transpose_alg1(const oracle_conv* d, const double* x, const double* w,
                                 const double* bias, double* y, int nthreads);

/* Algorithm 2 (section 2.1.1), generalised to padding and stride: a direct
 * gather with the dilated kernel; kernel zeros are never formed. */
int oracle_conv2d_dilated_alg2(const oracle_conv* d, const double* x, const double* w,
                               const double* bias, double* y, int nthreads);

/* The same two definitions evaluated one output element at a time, for
 * sampled checks at sizes where the full tensor is too costly.  idx holds
 * flat NCHW output indices; out[i] receives the value at idx[i]. */
int oracle_conv2d_transpose_points(const oracle_conv* d, const double* x, const double* w,
                                   const double* bias, const int64_t* idx, int64_t count,
                                   double* out, int nthreads);
int oracle_conv2d_dilated_points(const oracle_conv* d, const double* x, const double* w,
                                 const double* bias, const int64_t* idx, int64_t count,
                                 double* out, int nthreads);

/* Weight gradients for training (section 3.2.3), from the definitions
 * above by the chain rule; dy has the forward output's shape and dw the
 * weight's layout.
 *  transposed conv (the generator's layer):
 *    dw[c][k][m][q] = sum over (n, i, j) with oh = i*stride_h - pad_h + m*dil_h
 *                     and ow = j*stride_w - pad_w + q*dil_w inside the output
 *                     of x[n][c][i][j] * dy[n][k][oh][ow]
 *    (a strided correlation of the input with the output-error maps);
 *  dilated / strided conv (the discriminator's layer):
 *    dw[k][c][m][q] = sum over (n, oh, ow) with ih = oh*stride_h - pad_h +
 *                     m*dil_h and iw = ow*stride_w - pad_w + q*dil_w inside
 *                     the input of dy[n][k][oh][ow] * x[n][c][ih][iw]
 *    (the error maps, spread out by the stride, correlated with the input).
 * Parallel over (c, k) weight planes. */
int oracle_conv2d_transpose_wgrad(const oracle_conv* d, const double* x, const double* dy,
                                  double* dw, int nthreads);
int oracle_conv2d_dilated_wgrad(const oracle_conv* d, const double* x, const double* dy,
                                double* dw, int nthreads);

#ifdef __cplusplus
}
#endif
#endif
