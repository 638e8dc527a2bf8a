/*
 * ORACLE -- test infrastructure only.  Plain, slow, fp64 reference for the
 * convolution passes of the Conv2d+BN+SiLU block (paper Sec. 6.1, the
 * detector's conv blocks; Sec. 3 "reference-default semantics": convolution is
 * cross-correlation, zero padding, no bias before BN).
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may load
 * this file's library.  It shares no code with the HIP path.
 *
 * Layouts (dense, row-major):
 *   x  [N][H][W][Ci]       input activations (NHWC)
 *   w  [Co][kh][kw][Ci]    weights (OHWI)
 *   y  [N][Ho][Wo][Co]     output, Ho = floor((H + 2 ph - kh) / sh) + 1
 * Every element function below is the defining sum written out; the "full"
 * variants just evaluate the element function at every index.
 */
#include <stdint.h>

typedef struct {
  int32_t n, h, w, ci, co, kh, kw, sh, sw, ph, pw;
} ref_conv_dims;

static inline int32_t ref_ho(const ref_conv_dims* d) { return (d->h + 2 * d->ph - d->kh) / d->sh + 1; }
static inline int32_t ref_wo(const ref_conv_dims* d) { return (d->w + 2 * d->pw - d->kw) / d->sw + 1; }

static inline double xat(const double* x, const ref_conv_dims* d, int64_t n, int64_t h, int64_t w, int64_t c) {
  return x[((n * d->h + h) * d->w + w) * d->ci + c];
}
static inline double wat(const double* wt, const ref_conv_dims* d, int64_t o, int64_t r, int64_t s, int64_t c) {
  return wt[((o * d->kh + r) * d->kw + s) * d->ci + c];
}
static inline double yat(const double* y, const ref_conv_dims* d, int64_t n, int64_t p, int64_t q, int64_t o) {
  return y[((n * ref_ho(d) + p) * ref_wo(d) + q) * d->co + o];
}

/* Forward: y[n,p,q,o] = sum_{r,s,c} w[o,r,s,c] * x[n, p*sh - ph + r, q*sw - pw + s, c],
 * x taken as zero outside [0,H) x [0,W). */
double ref_conv_fwd_at(const double* x, const double* wt, const ref_conv_dims* d, int32_t n, int32_t p,
                       int32_t q, int32_t o) {
  double acc = 0.0;
  for (int32_t r = 0; r < d->kh; ++r) {
    int32_t ih = p * d->sh - d->ph + r;
    if (ih < 0 || ih >= d->h) continue;
    for (int32_t s = 0; s < d->kw; ++s) {
      int32_t iw = q * d->sw - d->pw + s;
      if (iw < 0 || iw >= d->w) continue;
      for (int32_t c = 0; c < d->ci; ++c) acc += wat(wt, d, o, r, s, c) * xat(x, d, n, ih, iw, c);
    }
  }
  return acc;
}

/* Data gradient (adjoint of the forward in x): dx[n,h,w,c] collects
 * w[o,r,s,c] * dy[n,p,q,o] over every (p,q,r,s,o) with p*sh - ph + r == h and
 * q*sw - pw + s == w. */
double ref_conv_dgrad_at(const double* dy, const double* wt, const ref_conv_dims* d, int32_t n, int32_t h,
                         int32_t w, int32_t c) {
  const int32_t ho = ref_ho(d), wo = ref_wo(d);
  double acc = 0.0;
  for (int32_t r = 0; r < d->kh; ++r) {
    int32_t tp = h + d->ph - r; /* = p * sh */
    if (tp < 0 || tp % d->sh != 0) continue;
    int32_t p = tp / d->sh;
    if (p >= ho) continue;
    for (int32_t s = 0; s < d->kw; ++s) {
      int32_t tq = w + d->pw - s;
      if (tq < 0 || tq % d->sw != 0) continue;
      int32_t q = tq / d->sw;
      if (q >= wo) continue;
      for (int32_t o = 0; o < d->co; ++o) acc += wat(wt, d, o, r, s, c) * yat(dy, d, n, p, q, o);
    }
  }
  return acc;
}

/* Weight gradient (adjoint of the forward in w):
 * dw[o,r,s,c] = sum_{n,p,q} dy[n,p,q,o] * x[n, p*sh - ph + r, q*sw - pw + s, c]. */
double ref_conv_wgrad_at(const double* x, const double* dy, const ref_conv_dims* d, int32_t o, int32_t r,
                         int32_t s, int32_t c) {
  const int32_t ho = ref_ho(d), wo = ref_wo(d);
  double acc = 0.0;
  for (int32_t n = 0; n < d->n; ++n)
    for (int32_t p = 0; p < ho; ++p) {
      int32_t ih = p * d->sh - d->ph + r;
      if (ih < 0 || ih >= d->h) continue;
      for (int32_t q = 0; q < wo; ++q) {
        int32_t iw = q * d->sw - d->pw + s;
        if (iw < 0 || iw >= d->w) continue;
        acc += yat(dy, d, n, p, q, o) * xat(x, d, n, ih, iw, c);
      }
    }
  return acc;
}

void ref_conv_fwd(const double* x, const double* wt, double* y, const ref_conv_dims* d) {
  const int32_t ho = ref_ho(d), wo = ref_wo(d);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int32_t n = 0; n < d->n; ++n)
    for (int32_t p = 0; p < ho; ++p)
      for (int32_t q = 0; q < wo; ++q)
        for (int32_t o = 0; o < d->co; ++o)
          y[(((int64_t)n * ho + p) * wo + q) * d->co + o] = ref_conv_fwd_at(x, wt, d, n, p, q, o);
}

void ref_conv_dgrad(const double* dy, const double* wt, double* dx, const ref_conv_dims* d) {
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int32_t n = 0; n < d->n; ++n)
    for (int32_t h = 0; h < d->h; ++h)
      for (int32_t w = 0; w < d->w; ++w)
        for (int32_t c = 0; c < d->ci; ++c)
          dx[(((int64_t)n * d->h + h) * d->w + w) * d->ci + c] = ref_conv_dgrad_at(dy, wt, d, n, h, w, c);
}

void ref_conv_wgrad(const double* x, const double* dy, double* dw, const ref_conv_dims* d) {
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int32_t o = 0; o < d->co; ++o)
    for (int32_t r = 0; r < d->kh; ++r)
      for (int32_t s = 0; s < d->kw; ++s)
        for (int32_t c = 0; c < d->ci; ++c)
          dw[(((int64_t)o * d->kh + r) * d->kw + s) * d->ci + c] = ref_conv_wgrad_at(x, dy, d, o, r, s, c);
}

/* Sampled variants: out[i] = the pass's element at flat index idx[i] of its output tensor. */
void ref_conv_fwd_sample(const double* x, const double* wt, const ref_conv_dims* d, const int64_t* idx,
                         int64_t count, double* out) {
  const int64_t ho = ref_ho(d), wo = ref_wo(d);
#pragma omp parallel for schedule(dynamic)
  for (int64_t i = 0; i < count; ++i) {
    int64_t t = idx[i];
    int32_t o = (int32_t)(t % d->co); t /= d->co;
    int32_t q = (int32_t)(t % wo); t /= wo;
    int32_t p = (int32_t)(t % ho); t /= ho;
    out[i] = ref_conv_fwd_at(x, wt, d, (int32_t)t, p, q, o);
  }
}

void ref_conv_dgrad_sample(const double* dy, const double* wt, const ref_conv_dims* d, const int64_t* idx,
                           int64_t count, double* out) {
#pragma omp parallel for schedule(dynamic)
  for (int64_t i = 0; i < count; ++i) {
    int64_t t = idx[i];
    int32_t c = (int32_t)(t % d->ci); t /= d->ci;
    int32_t w = (int32_t)(t % d->w); t /= d->w;
    int32_t h = (int32_t)(t % d->h); t /= d->h;
    out[i] = ref_conv_dgrad_at(dy, wt, d, (int32_t)t, h, w, c);
  }
}

void ref_conv_wgrad_sample(const double* x, const double* dy, const ref_conv_dims* d, const int64_t* idx,
                           int64_t count, double* out) {
#pragma omp parallel for schedule(dynamic)
  for (int64_t i = 0; i < count; ++i) {
    int64_t t = idx[i];
    int32_t c = (int32_t)(t % d->ci); t /= d->ci;
    int32_t s = (int32_t)(t % d->kw); t /= d->kw;
    int32_t r = (int32_t)(t % d->kh); t /= d->kh;
    out[i] = ref_conv_wgrad_at(x, dy, d, (int32_t)t, r, s, c);
  }
}

/* One output channel of the forward over all N*Ho*Wo rows (for per-channel
 * statistics at sizes where the full output is too costly). */
void ref_conv_fwd_channel(const double* x, const double* wt, const ref_conv_dims* d, int32_t o, double* col) {
  const int32_t ho = ref_ho(d), wo = ref_wo(d);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int32_t n = 0; n < d->n; ++n)
    for (int32_t p = 0; p < ho; ++p)
      for (int32_t q = 0; q < wo; ++q)
        col[((int64_t)n * ho + p) * wo + q] = ref_conv_fwd_at(x, wt, d, n, p, q, o);
}

/* Threads the OpenMP loops above use (reported beside timings). */
#include <omp.h>
int ref_num_threads(void) { return omp_get_max_threads(); }
