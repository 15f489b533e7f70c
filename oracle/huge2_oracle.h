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
 *   w  transposed conv: [c_in][c_out][r][s]   (the paper's C x N x R x S,
 *                                              section 4.2)
 *      dilated / strided conv: [c_out][c_in][r][s]
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

#ifdef __cplusplus
}
#endif
#endif
