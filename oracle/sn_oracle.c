/*
 * Oracle: plain, slow, obviously correct float64 reference of the layer
 * operations that a SoftNeuro net computes.  TEST INFRASTRUCTURE ONLY: it is
 * called by the tests, by the smoke check and by the CPU-baseline leg of the
 * benchmark, never by the product path, and it shares no code with it.
 *
 * Every routine the GPU path offers for a layer (direct, implicit GEMM,
 * Winograd, in any tensor layout) must compute the same function of the
 * inputs; the routines differ only in rounding.  The paper states that
 * routines are interchangeable implementations of one layer computation
 * (Sec. III-A, III-C), so the oracle is the plain definition of each layer:
 *
 *   conv2d   y[n,k,p,q] = b[k] + sum_{c in group(k), r, s}
 *                         w[k, c - c0(k), r, s] * x[n, c, p*st - pad + r, q*st - pad + s]
 *            cross-correlation (no kernel flip), zero padding, optional
 *            fused activation (the importer fuses ReLU into the previous
 *            layer, Sec. III-A).  Groups: 1 (dense) or C (depthwise).
 *   maxpool  max over the window restricted to valid input positions.
 *   gap      mean over H x W.
 *   add      a + b, optional activation (residual merge layer).
 *   fc       y = W x + b; the paper's dense routine is the same function
 *            computed as a 1x1 convolution (Sec. III-D).
 *
 * Tensors are NCHW, weights OIHW, all float64.  Storage rounding (or_round)
 * rounds a float64 value once, to nearest-even, to the storage format of the
 * run dtype.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>

enum { OR_ACT_NONE = 0, OR_ACT_RELU = 1, OR_ACT_RELU6 = 2 };
enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2 };

static double act_apply(double v, int act) {
  if (act == OR_ACT_RELU) return v > 0.0 ? v : 0.0;
  if (act == OR_ACT_RELU6) return v < 0.0 ? 0.0 : (v > 6.0 ? 6.0 : v);
  return v;
}

static int out_dim(int in, int k, int stride, int pad) {
  return (in + 2 * pad - k) / stride + 1;
}

/* One output element of a (grouped) convolution, straight from the definition. */
static double conv_point(const double* x, int C, int H, int W, const double* w, int K, int R,
                         int S, int stride, int pad, int groups, const double* b, int n, int k,
                         int p, int q) {
  int cg = C / groups;               /* input channels per group  */
  int kg = K / groups;               /* output channels per group */
  int c0 = (k / kg) * cg;            /* first input channel of k's group */
  double acc = b ? b[k] : 0.0;
  for (int c = 0; c < cg; ++c) {
    for (int r = 0; r < R; ++r) {
      int h = p * stride - pad + r;
      if (h < 0 || h >= H) continue;
      for (int s = 0; s < S; ++s) {
        int ww = q * stride - pad + s;
        if (ww < 0 || ww >= W) continue;
        double xv = x[(((size_t)n * C + (c0 + c)) * H + h) * W + ww];
        double wv = w[(((size_t)k * cg + c) * R + r) * S + s];
        acc += wv * xv;
      }
    }
  }
  return acc;
}

void or_conv2d(const double* x, int N, int C, int H, int W, const double* w, int K, int R,
               int S, int stride, int pad, int groups, const double* b, int act, double* y) {
  int P = out_dim(H, R, stride, pad), Q = out_dim(W, S, stride, pad);
  long nk = (long)N * K;
#pragma omp parallel for schedule(dynamic, 1)
  for (long t = 0; t < nk; ++t) {
    int n = (int)(t / K), k = (int)(t % K);
    for (int p = 0; p < P; ++p)
      for (int q = 0; q < Q; ++q)
        y[(((size_t)n * K + k) * P + p) * Q + q] =
            act_apply(conv_point(x, C, H, W, w, K, R, S, stride, pad, groups, b, n, k, p, q), act);
  }
}

/* Sampled outputs: idx holds npts quadruples (n, k, p, q). */
void or_conv2d_points(const double* x, int N, int C, int H, int W, const double* w, int K, int R,
                      int S, int stride, int pad, int groups, const double* b, int act,
                      const int64_t* idx, int64_t npts, double* out) {
  (void)N;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < npts; ++i) {
    const int64_t* t = idx + 4 * i;
    out[i] = act_apply(conv_point(x, C, H, W, w, K, R, S, stride, pad, groups, b, (int)t[0],
                                  (int)t[1], (int)t[2], (int)t[3]),
                       act);
  }
}

void or_maxpool(const double* x, int N, int C, int H, int W, int k, int stride, int pad,
                double* y) {
  int P = out_dim(H, k, stride, pad), Q = out_dim(W, k, stride, pad);
  long nc = (long)N * C;
#pragma omp parallel for schedule(static)
  for (long t = 0; t < nc; ++t) {
    const double* xp = x + (size_t)t * H * W;
    for (int p = 0; p < P; ++p)
      for (int q = 0; q < Q; ++q) {
        double m = -INFINITY;
        for (int r = 0; r < k; ++r) {
          int h = p * stride - pad + r;
          if (h < 0 || h >= H) continue;
          for (int s = 0; s < k; ++s) {
            int ww = q * stride - pad + s;
            if (ww < 0 || ww >= W) continue;
            double v = xp[(size_t)h * W + ww];
            if (v > m) m = v;
          }
        }
        y[((size_t)t * P + p) * Q + q] = m;
      }
  }
}

void or_gap(const double* x, int N, int C, int H, int W, double* y) {
  long nc = (long)N * C;
  for (long t = 0; t < nc; ++t) {
    double s = 0.0;
    for (long i = 0; i < (long)H * W; ++i) s += x[(size_t)t * H * W + i];
    y[t] = s / ((double)H * W);
  }
}

void or_add(const double* a, const double* b, int64_t n, int act, double* y) {
  for (int64_t i = 0; i < n; ++i) y[i] = act_apply(a[i] + b[i], act);
}

void or_fc(const double* x, int N, int Cin, const double* w, int K, const double* b, double* y) {
#pragma omp parallel for schedule(static)
  for (long t = 0; t < (long)N * K; ++t) {
    int n = (int)(t / K), k = (int)(t % K);
    double acc = b ? b[k] : 0.0;
    for (int c = 0; c < Cin; ++c) acc += w[(size_t)k * Cin + c] * x[(size_t)n * Cin + c];
    y[t] = acc;
  }
}

/* Round v once to a binary format with p significant bits, minimum normal
 * exponent emin and largest finite value maxv; ties to even. */
static double round_format(double v, int p, int emin, double maxv) {
  if (v == 0.0 || !isfinite(v)) return v;
  int e = ilogb(v);                       /* |v| in [2^e, 2^(e+1)) */
  if (e < emin) e = emin;                 /* subnormal range: fixed quantum */
  double quantum = ldexp(1.0, e - (p - 1));
  double r = nearbyint(v / quantum) * quantum; /* default rounding mode: nearest-even */
  if (fabs(r) > maxv) r = copysign(INFINITY, v);
  return r;
}

double or_round1(double v, int dtype) {
  switch (dtype) {
    case OR_F32:  return round_format(v, 24, -126, 3.4028234663852886e38);
    case OR_F16:  return round_format(v, 11, -14, 65504.0);
    case OR_BF16: return round_format(v, 8, -126, 3.3895313892515355e38);
  }
  return v;
}

void or_round(double* v, int64_t n, int dtype) {
  for (int64_t i = 0; i < n; ++i) v[i] = or_round1(v[i], dtype);
}

int or_num_threads(void) {
#ifdef _OPENMP
  extern int omp_get_max_threads(void);
  return omp_get_max_threads();
#else
  return 1;
#endif
}
