/*
 * huge2_oracle.c -- plain, slow, float64 CPU oracle for the transposed and
 * dilated convolutions of HUGE^2 (arXiv 1907.11210).
 *
 * TEST INFRASTRUCTURE ONLY: called by the tests, the smoke check and the
 * benchmark's CPU baseline leg, never by the product library.  It shares
 * no code with the GPU path.
 *
 * Readings of the paper taken here (the paper's loop bounds and indices in
 * Algorithms 1-2 are garbled; these are the readings used throughout):
 *  - Transposed conv is the zero-insertion emulation described right after
 *    Algorithm 2 (section 2.1.1): spread the input by inserting s-1 zeros
 *    between rows and columns, pad, then run a stride-1 convolution with
 *    the transposed kernel (rotated by 180 degrees, in/out channels
 *    swapped).  Padding, output padding and kernel dilation follow the
 *    usual deep-learning (PyTorch ConvTranspose2d) conventions, which the
 *    paper does not state.
 *  - Dilated conv is Algorithm 2 read as cross-correlation with a kernel
 *    whose taps are dil apart, extended by zero padding and a stride.
 *  - Accumulation is in double; nothing is rounded before the end.
 */
#include "huge2_oracle.h"

#include <pthread.h>
#include <stdlib.h>
#include <string.h>

static int ngroups(const oracle_conv* d) { return d->groups > 1 ? d->groups : 1; }

static int valid_common(const oracle_conv* d) {
  if (!d) return 0;
  if (d->groups < 0 || d->c_in % ngroups(d) != 0 || d->c_out % ngroups(d) != 0) return 0;
  if (d->n < 1 || d->c_in < 1 || d->h < 1 || d->w < 1) return 0;
  if (d->c_out < 1 || d->r < 1 || d->s < 1) return 0;
  if (d->stride_h < 1 || d->stride_w < 1 || d->dil_h < 1 || d->dil_w < 1) return 0;
  if (d->pad_h < 0 || d->pad_w < 0 || d->out_pad_h < 0 || d->out_pad_w < 0) return 0;
  return 1;
}

int oracle_transpose_out_dims(const oracle_conv* d, int* h_out, int* w_out) {
  if (!valid_common(d)) return -1;
  /* output padding must be smaller than either the stride or the dilation */
  int lim_h = d->stride_h > d->dil_h ? d->stride_h : d->dil_h;
  int lim_w = d->stride_w > d->dil_w ? d->stride_w : d->dil_w;
  if (d->out_pad_h >= lim_h || d->out_pad_w >= lim_w) return -1;
  long ho = (long)(d->h - 1) * d->stride_h - 2L * d->pad_h + (long)d->dil_h * (d->r - 1) +
            d->out_pad_h + 1;
  long wo = (long)(d->w - 1) * d->stride_w - 2L * d->pad_w + (long)d->dil_w * (d->s - 1) +
            d->out_pad_w + 1;
  if (ho < 1 || wo < 1) return -1;
  *h_out = (int)ho;
  *w_out = (int)wo;
  return 0;
}

int oracle_conv_out_dims(const oracle_conv* d, int* h_out, int* w_out) {
  if (!valid_common(d)) return -1;
  if (d->out_pad_h != 0 || d->out_pad_w != 0) return -1;
  long nh = (long)d->h + 2L * d->pad_h - (long)d->dil_h * (d->r - 1) - 1;
  long nw = (long)d->w + 2L * d->pad_w - (long)d->dil_w * (d->s - 1) - 1;
  if (nh < 0 || nw < 0) return -1;
  *h_out = (int)(nh / d->stride_h + 1);
  *w_out = (int)(nw / d->stride_w + 1);
  return 0;
}

/* ------------------------------------------------------------------ */
/* A tiny static work split over threads: planes tid, tid+T, tid+2T... */

typedef void (*plane_fn)(void* ctx, long plane);
typedef struct {
  plane_fn fn;
  void* ctx;
  long count;
  int tid, nthreads;
} worker_arg;

static void* worker_main(void* p) {
  worker_arg* a = (worker_arg*)p;
  for (long i = a->tid; i < a->count; i += a->nthreads) a->fn(a->ctx, i);
  return NULL;
}

static void run_parallel(plane_fn fn, void* ctx, long count, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (nthreads > count) nthreads = count > 0 ? (int)count : 1;
  pthread_t th[256];
  worker_arg args[256];
  for (int t = 0; t < nthreads; ++t) {
    args[t].fn = fn;
    args[t].ctx = ctx;
    args[t].count = count;
    args[t].tid = t;
    args[t].nthreads = nthreads;
  }
  int started = 0;
  for (int t = 1; t < nthreads; ++t) {
    if (pthread_create(&th[t], NULL, worker_main, &args[t]) != 0) break;
    started = t;
  }
  /* thread 0 runs here; any thread that failed to start is run inline */
  worker_main(&args[0]);
  for (int t = started + 1; t < nthreads; ++t) worker_main(&args[t]);
  for (int t = 1; t <= started; ++t) pthread_join(th[t], NULL);
}

/* ------------------------------------------------------------------ */
/* Algorithm 1: transposed conv by zero insertion.                      */

typedef struct {
  const oracle_conv* d;
  const double* xhat; /* [n][c_in][hh][wh] zero-inserted input */
  int hh, wh;         /* zero-inserted size: (h-1)*stride + 1 */
  int eh, ew;         /* virtual padding before: dil*(k-1) - pad (may be < 0: crop) */
  const double* w;
  const double* bias;
  double* y;
  int ho, wo;
} alg1_ctx;

/* One term source: the padded zero-inserted input at (ph, pw) of the padded
 * frame.  Positions outside the zero-inserted map are padding zeros. */
static double xhat_padded(const alg1_ctx* a, int n, int c, int ph, int pw) {
  int jh = ph - a->eh, jw = pw - a->ew;
  if (jh < 0 || jh >= a->hh || jw < 0 || jw >= a->wh) return 0.0;
  return a->xhat[(((long)n * a->d->c_in + c) * a->hh + jh) * a->wh + jw];
}

/* The input channels output channel k sums over: its group's [*c0, *c1), and
 * k's index inside the group (the weight array holds c_out/groups of them
 * for the transposed conv, c_in/groups for the conv). */
static void group_of(const oracle_conv* d, int k, int* c0, int* c1, int* k_in_group) {
  const int g = ngroups(d), cig = d->c_in / g, cog = d->c_out / g;
  *c0 = (k / cog) * cig;
  *c1 = *c0 + cig;
  *k_in_group = k % cog;
}

static double alg1_output(const alg1_ctx* a, int n, int k, int oh, int ow) {
  const oracle_conv* d = a->d;
  const int cog = d->c_out / ngroups(d);
  int c0, c1, kg;
  group_of(d, k, &c0, &c1, &kg);
  double acc = 0.0;
  for (int c = c0; c < c1; ++c)
    for (int m = 0; m < d->r; ++m)
      for (int q = 0; q < d->s; ++q) {
        /* the transposed kernel: rotated by 180 degrees, w[c][k] used as the
         * (k <- c) filter of the stride-1 convolution */
        double wv = a->w[(((long)c * cog + kg) * d->r + (d->r - 1 - m)) * d->s + (d->s - 1 - q)];
        acc += xhat_padded(a, n, c, oh + m * d->dil_h, ow + q * d->dil_w) * wv;
      }
  if (a->bias) acc += a->bias[k];
  return acc;
}

static void alg1_plane(void* p, long plane) {
  alg1_ctx* a = (alg1_ctx*)p;
  int n = (int)(plane / a->d->c_out), k = (int)(plane % a->d->c_out);
  double* yp = a->y + plane * (long)a->ho * a->wo;
  for (int oh = 0; oh < a->ho; ++oh)
    for (int ow = 0; ow < a->wo; ++ow) yp[(long)oh * a->wo + ow] = alg1_output(a, n, k, oh, ow);
}

static int alg1_setup(const oracle_conv* d, alg1_ctx* a, int* ho, int* wo) {
  if (oracle_transpose_out_dims(d, ho, wo) != 0) return -1;
  a->d = d;
  a->hh = (d->h - 1) * d->stride_h + 1;
  a->wh = (d->w - 1) * d->stride_w + 1;
  a->eh = d->dil_h * (d->r - 1) - d->pad_h;
  a->ew = d->dil_w * (d->s - 1) - d->pad_w;
  a->ho = *ho;
  a->wo = *wo;
  return 0;
}

int oracle_conv2d_transpose_alg1(const oracle_conv* d, const double* x, const double* w,
                                 const double* bias, double* y, int nthreads) {
  alg1_ctx a;
  int ho, wo;
  if (!x || !w || !y || alg1_setup(d, &a, &ho, &wo) != 0) return -1;
  /* materialise the zero-inserted input: x[i][j] lands at (i*stride_h, j*stride_w) */
  long nplanes_in = (long)d->n * d->c_in;
  double* xhat = (double*)calloc((size_t)nplanes_in * a.hh * a.wh, sizeof(double));
  if (!xhat) return -1;
  for (long pl = 0; pl < nplanes_in; ++pl)
    for (int i = 0; i < d->h; ++i)
      for (int j = 0; j < d->w; ++j)
        xhat[(pl * a.hh + (long)i * d->stride_h) * a.wh + (long)j * d->stride_w] =
            x[(pl * d->h + i) * d->w + j];
  a.xhat = xhat;
  a.w = w;
  a.bias = bias;
  a.y = y;
  run_parallel(alg1_plane, &a, (long)d->n * d->c_out, nthreads);
  free(xhat);
  return 0;
}

/* Per-element form: the zero-inserted input is read through its definition
 * instead of a materialised copy. */
typedef struct {
  alg1_ctx a;
  const double* x;
  const int64_t* idx;
  double* out;
  int64_t count;
} alg1_pts_ctx;

static double xhat_defined(const alg1_pts_ctx* p, int n, int c, int ph, int pw) {
  const oracle_conv* d = p->a.d;
  int jh = ph - p->a.eh, jw = pw - p->a.ew;
  if (jh < 0 || jh >= p->a.hh || jw < 0 || jw >= p->a.wh) return 0.0;
  if (jh % d->stride_h != 0 || jw % d->stride_w != 0) return 0.0; /* an inserted zero */
  return p->x[(((long)n * d->c_in + c) * d->h + jh / d->stride_h) * d->w + jw / d->stride_w];
}

static void alg1_point(void* ctx, long i) {
  alg1_pts_ctx* p = (alg1_pts_ctx*)ctx;
  const oracle_conv* d = p->a.d;
  int64_t f = p->idx[i];
  int ow = (int)(f % p->a.wo);
  f /= p->a.wo;
  int oh = (int)(f % p->a.ho);
  f /= p->a.ho;
  int k = (int)(f % d->c_out);
  int n = (int)(f / d->c_out);
  const int cog = d->c_out / ngroups(d);
  int c0, c1, kg;
  group_of(d, k, &c0, &c1, &kg);
  double acc = 0.0;
  for (int c = c0; c < c1; ++c)
    for (int m = 0; m < d->r; ++m)
      for (int q = 0; q < d->s; ++q) {
        double wv = p->a.w[(((long)c * cog + kg) * d->r + (d->r - 1 - m)) * d->s + (d->s - 1 - q)];
        acc += xhat_defined(p, n, c, oh + m * d->dil_h, ow + q * d->dil_w) * wv;
      }
  if (p->a.bias) acc += p->a.bias[k];
  p->out[i] = acc;
}

int oracle_conv2d_transpose_points(const oracle_conv* d, const double* x, const double* w,
                                   const double* bias, const int64_t* idx, int64_t count,
                                   double* out, int nthreads) {
  alg1_pts_ctx p;
  int ho, wo;
  if (!x || !w || (count > 0 && (!idx || !out)) || alg1_setup(d, &p.a, &ho, &wo) != 0) return -1;
  int64_t total = (int64_t)d->n * d->c_out * ho * wo;
  for (int64_t i = 0; i < count; ++i)
    if (idx[i] < 0 || idx[i] >= total) return -1;
  p.a.w = w;
  p.a.bias = bias;
  p.x = x;
  p.idx = idx;
  p.out = out;
  p.count = count;
  run_parallel(alg1_point, &p, (long)count, nthreads);
  return 0;
}

/* ------------------------------------------------------------------ */
/* Algorithm 2: dilated (and strided) conv as a direct gather.          */

typedef struct {
  const oracle_conv* d;
  const double* x;
  const double* w;
  const double* bias;
  double* y;
  int ho, wo;
  const int64_t* idx;
  double* out;
} alg2_ctx;

static double alg2_output(const alg2_ctx* a, int n, int k, int oh, int ow) {
  const oracle_conv* d = a->d;
  const int cig = d->c_in / ngroups(d);
  int c0, c1, kg;
  group_of(d, k, &c0, &c1, &kg);
  double acc = 0.0;
  for (int c = c0; c < c1; ++c)
    for (int m = 0; m < d->r; ++m)
      for (int q = 0; q < d->s; ++q) {
        int ih = oh * d->stride_h - d->pad_h + m * d->dil_h;
        int iw = ow * d->stride_w - d->pad_w + q * d->dil_w;
        if (ih < 0 || ih >= d->h || iw < 0 || iw >= d->w) continue; /* zero padding */
        acc += a->x[(((long)n * d->c_in + c) * d->h + ih) * d->w + iw] *
               a->w[(((long)k * cig + (c - c0)) * d->r + m) * d->s + q];
      }
  if (a->bias) acc += a->bias[k];
  return acc;
}

static void alg2_plane(void* p, long plane) {
  alg2_ctx* a = (alg2_ctx*)p;
  int n = (int)(plane / a->d->c_out), k = (int)(plane % a->d->c_out);
  double* yp = a->y + plane * (long)a->ho * a->wo;
  for (int oh = 0; oh < a->ho; ++oh)
    for (int ow = 0; ow < a->wo; ++ow) yp[(long)oh * a->wo + ow] = alg2_output(a, n, k, oh, ow);
}

int oracle_conv2d_dilated_alg2(const oracle_conv* d, const double* x, const double* w,
                               const double* bias, double* y, int nthreads) {
  alg2_ctx a;
  if (!x || !w || !y || oracle_conv_out_dims(d, &a.ho, &a.wo) != 0) return -1;
  a.d = d;
  a.x = x;
  a.w = w;
  a.bias = bias;
  a.y = y;
  run_parallel(alg2_plane, &a, (long)d->n * d->c_out, nthreads);
  return 0;
}

static void alg2_point(void* ctx, long i) {
  alg2_ctx* a = (alg2_ctx*)ctx;
  int64_t f = a->idx[i];
  int ow = (int)(f % a->wo);
  f /= a->wo;
  int oh = (int)(f % a->ho);
  f /= a->ho;
  int k = (int)(f % a->d->c_out);
  int n = (int)(f / a->d->c_out);
  a->out[i] = alg2_output(a, n, k, oh, ow);
}

int oracle_conv2d_dilated_points(const oracle_conv* d, const double* x, const double* w,
                                 const double* bias, const int64_t* idx, int64_t count,
                                 double* out, int nthreads) {
  alg2_ctx a;
  if (!x || !w || (count > 0 && (!idx || !out)) || oracle_conv_out_dims(d, &a.ho, &a.wo) != 0)
    return -1;
  int64_t total = (int64_t)d->n * d->c_out * a.ho * a.wo;
  for (int64_t i = 0; i < count; ++i)
    if (idx[i] < 0 || idx[i] >= total) return -1;
  a.d = d;
  a.x = x;
  a.w = w;
  a.bias = bias;
  a.y = NULL;
  a.idx = idx;
  a.out = out;
  run_parallel(alg2_point, &a, (long)count, nthreads);
  return 0;
}

/* ------------------------------------------------------------------ */
/* Weight gradients (section 3.2.3): the chain rule applied to the two  */
/* definitions above, one weight element at a time.  With groups, a     */
/* weight element joins input channel c only to the output channels of  */
/* c's group, so its gradient sums over that pair alone (groups = c_in  */
/* is the depthwise case: one input and one output map per element).    */

typedef struct {
  const oracle_conv* d;
  const double* x;
  const double* dy;
  double* dw;
  int ho, wo;
  int transposed;
} wgrad_ctx;

/* dw for one weight plane (all r x s taps): transposed, plane (c, k - first
 * output channel of c's group) of w [c_in][c_out/groups]; otherwise plane
 * (k, c - first input channel of k's group) of w [c_out][c_in/groups]. */
static void wgrad_plane(void* p, long plane) {
  wgrad_ctx* a = (wgrad_ctx*)p;
  const oracle_conv* d = a->d;
  const int g = ngroups(d), cig = d->c_in / g, cog = d->c_out / g;
  int c, k;
  if (a->transposed) {
    c = (int)(plane / cog);
    k = (c / cig) * cog + (int)(plane % cog);
  } else {
    k = (int)(plane / cig);
    c = (k / cog) * cig + (int)(plane % cig);
  }
  for (int m = 0; m < d->r; ++m)
    for (int q = 0; q < d->s; ++q) {
      double acc = 0.0;
      if (a->transposed) {
        /* every input pixel (i, j) and the output it reaches through tap (m, q) */
        for (int n = 0; n < d->n; ++n)
          for (int i = 0; i < d->h; ++i) {
            const int oh = i * d->stride_h - d->pad_h + m * d->dil_h;
            if (oh < 0 || oh >= a->ho) continue;
            for (int j = 0; j < d->w; ++j) {
              const int ow = j * d->stride_w - d->pad_w + q * d->dil_w;
              if (ow < 0 || ow >= a->wo) continue;
              acc += a->x[(((long)n * d->c_in + c) * d->h + i) * d->w + j] *
                     a->dy[(((long)n * d->c_out + k) * a->ho + oh) * a->wo + ow];
            }
          }
        a->dw[(((long)c * cog + k % cog) * d->r + m) * d->s + q] = acc;
      } else {
        /* every output pixel (oh, ow) and the input it reads through tap (m, q) */
        for (int n = 0; n < d->n; ++n)
          for (int oh = 0; oh < a->ho; ++oh) {
            const int ih = oh * d->stride_h - d->pad_h + m * d->dil_h;
            if (ih < 0 || ih >= d->h) continue;
            for (int ow = 0; ow < a->wo; ++ow) {
              const int iw = ow * d->stride_w - d->pad_w + q * d->dil_w;
              if (iw < 0 || iw >= d->w) continue;
              acc += a->dy[(((long)n * d->c_out + k) * a->ho + oh) * a->wo + ow] *
                     a->x[(((long)n * d->c_in + c) * d->h + ih) * d->w + iw];
            }
          }
        a->dw[(((long)k * cig + c % cig) * d->r + m) * d->s + q] = acc;
      }
    }
}

int oracle_conv2d_transpose_wgrad(const oracle_conv* d, const double* x, const double* dy,
                                  double* dw, int nthreads) {
  wgrad_ctx a;
  if (!x || !dy || !dw || oracle_transpose_out_dims(d, &a.ho, &a.wo) != 0) return -1;
  a.d = d;
  a.x = x;
  a.dy = dy;
  a.dw = dw;
  a.transposed = 1;
  run_parallel(wgrad_plane, &a, (long)d->c_in * (d->c_out / ngroups(d)), nthreads);
  return 0;
}

int oracle_conv2d_dilated_wgrad(const oracle_conv* d, const double* x, const double* dy,
                                double* dw, int nthreads) {
  wgrad_ctx a;
  if (!x || !dy || !dw || oracle_conv_out_dims(d, &a.ho, &a.wo) != 0) return -1;
  a.d = d;
  a.x = x;
  a.dy = dy;
  a.dw = dw;
  a.transposed = 0;
  run_parallel(wgrad_plane, &a, (long)d->c_out * (d->c_in / ngroups(d)), nthreads);
  return 0;
}
