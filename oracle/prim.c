/*
 * Test infrastructure: the CPU oracle's layer primitives, fp64, direct loops.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg use this file.  It shares
 * nothing with the GPU path.  The paper names its layers (convolution, batch normalisation,
 * ReLU, max pooling; Sec. 4.1, Tables vgg / resnet) without formulas; these are the standard
 * definitions:
 *
 *   conv      y[n,p,q,o] = sum_{r,s,c} w[o,r,s,c] * x[n, p*st + r - pad, q*st + s - pad, c]
 *             (cross-correlation, zeros outside the image, no bias)
 *   maxpool   y[n,p,q,c] = max over the k x k window at (p*st - pad, q*st - pad); positions
 *             outside the image never win; the gradient goes to the first maximum in row-major
 *             window order
 *   BN        training mode: per channel mean and biased variance over (n, h, w)
 *
 * All tensors are NHWC (filters [o][r][s][c]).  Every output element is a fixed-order sum, so
 * results do not depend on the thread count.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#define IDX4(a, b, c, d, B_, C_, D_) ((((size_t)(a) * (B_) + (b)) * (C_) + (c)) * (D_) + (d))

/* y[B,Ho,Wo,K] = conv(x[B,H,W,C], w[K,k,k,C]) */
void pnn_oracle_conv_fwd(const double* x, int B, int H, int W, int C, const double* w, int K,
                         int k, int st, int pad, double* y, int Ho, int Wo) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < B; n++)
    for (int p = 0; p < Ho; p++)
      for (int q = 0; q < Wo; q++) {
        double* out = y + IDX4(n, p, q, 0, Ho, Wo, K);
        for (int o = 0; o < K; o++) {
          double acc = 0.0;
          for (int r = 0; r < k; r++) {
            int ih = p * st + r - pad;
            if (ih < 0 || ih >= H) continue;
            for (int s = 0; s < k; s++) {
              int iw = q * st + s - pad;
              if (iw < 0 || iw >= W) continue;
              const double* xv = x + IDX4(n, ih, iw, 0, H, W, C);
              const double* wv = w + IDX4(o, r, s, 0, k, k, C);
              for (int c = 0; c < C; c++) acc += wv[c] * xv[c];
            }
          }
          out[o] = acc;
        }
      }
}

/* gx[B,H,W,C] = dL/dx for the convolution above, from gy[B,Ho,Wo,K]:
 * gx[n,h,v,c] = sum over (r,s,o) with h = p*st + r - pad, v = q*st + s - pad of gy[n,p,q,o] w[o,r,s,c] */
void pnn_oracle_conv_bwd_data(const double* gy, int B, int H, int W, int C, const double* w, int K,
                              int k, int st, int pad, double* gx, int Ho, int Wo) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < B; n++)
    for (int h = 0; h < H; h++)
      for (int v = 0; v < W; v++) {
        double* out = gx + IDX4(n, h, v, 0, H, W, C);
        for (int c = 0; c < C; c++) out[c] = 0.0;
        for (int r = 0; r < k; r++) {
          int t = h + pad - r;
          if (t < 0 || t % st) continue;
          int p = t / st;
          if (p >= Ho) continue;
          for (int s = 0; s < k; s++) {
            int u = v + pad - s;
            if (u < 0 || u % st) continue;
            int q = u / st;
            if (q >= Wo) continue;
            const double* g = gy + IDX4(n, p, q, 0, Ho, Wo, K);
            for (int o = 0; o < K; o++) {
              const double* wv = w + IDX4(o, r, s, 0, k, k, C);
              double go = g[o];
              for (int c = 0; c < C; c++) out[c] += go * wv[c];
            }
          }
        }
      }
}

/* gw[K,k,k,C] = dL/dw: gw[o,r,s,c] = sum_{n,p,q} gy[n,p,q,o] x[n, p*st + r - pad, q*st + s - pad, c] */
void pnn_oracle_conv_bwd_weight(const double* x, int B, int H, int W, int C, const double* gy, int K,
                                int k, int st, int pad, double* gw, int Ho, int Wo) {
#pragma omp parallel for collapse(3) schedule(static)
  for (int o = 0; o < K; o++)
    for (int r = 0; r < k; r++)
      for (int s = 0; s < k; s++) {
        double* out = gw + IDX4(o, r, s, 0, k, k, C);
        for (int c = 0; c < C; c++) out[c] = 0.0;
        for (int n = 0; n < B; n++)
          for (int p = 0; p < Ho; p++) {
            int ih = p * st + r - pad;
            if (ih < 0 || ih >= H) continue;
            for (int q = 0; q < Wo; q++) {
              int iw = q * st + s - pad;
              if (iw < 0 || iw >= W) continue;
              double g = gy[IDX4(n, p, q, o, Ho, Wo, K)];
              const double* xv = x + IDX4(n, ih, iw, 0, H, W, C);
              for (int c = 0; c < C; c++) out[c] += g * xv[c];
            }
          }
      }
}

/* max pool, k x k window, stride st, padding pad (padding never selected) */
void pnn_oracle_maxpool_fwd(const double* x, int B, int H, int W, int C, int k, int st, int pad,
                            double* y, int Ho, int Wo) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < B; n++)
    for (int p = 0; p < Ho; p++)
      for (int q = 0; q < Wo; q++)
        for (int c = 0; c < C; c++) {
          double m = -INFINITY;
          for (int r = 0; r < k; r++) {
            int ih = p * st + r - pad;
            if (ih < 0 || ih >= H) continue;
            for (int s = 0; s < k; s++) {
              int iw = q * st + s - pad;
              if (iw < 0 || iw >= W) continue;
              double v = x[IDX4(n, ih, iw, c, H, W, C)];
              if (v > m) m = v;
            }
          }
          y[IDX4(n, p, q, c, Ho, Wo, C)] = m;
        }
}

/* gx += routed gy: each output's gradient goes to the first maximum of its window */
void pnn_oracle_maxpool_bwd(const double* x, int B, int H, int W, int C, int k, int st, int pad,
                            const double* gy, double* gx, int Ho, int Wo) {
#pragma omp parallel for schedule(static)
  for (int n = 0; n < B; n++)
    for (int p = 0; p < Ho; p++)
      for (int q = 0; q < Wo; q++)
        for (int c = 0; c < C; c++) {
          double m = -INFINITY;
          size_t arg = 0;
          int found = 0;
          for (int r = 0; r < k; r++) {
            int ih = p * st + r - pad;
            if (ih < 0 || ih >= H) continue;
            for (int s = 0; s < k; s++) {
              int iw = q * st + s - pad;
              if (iw < 0 || iw >= W) continue;
              size_t i = IDX4(n, ih, iw, c, H, W, C);
              if (!found || x[i] > m) { m = x[i]; arg = i; found = 1; }
            }
          }
          if (found) gx[arg] += gy[IDX4(n, p, q, c, Ho, Wo, C)];
        }
}

/* batch statistics over the M rows of x[M,C]: mean and biased variance (two passes) */
void pnn_oracle_bn_stats(const double* x, long M, int C, double* mean, double* var) {
#pragma omp parallel for schedule(static)
  for (int c = 0; c < C; c++) {
    double s = 0.0;
    for (long m = 0; m < M; m++) s += x[(size_t)m * C + c];
    double mu = s / (double)M;
    double v = 0.0;
    for (long m = 0; m < M; m++) {
      double d = x[(size_t)m * C + c] - mu;
      v += d * d;
    }
    mean[c] = mu;
    var[c] = v / (double)M;
  }
}

/* per-channel sums over the M rows of a[M,C] and of a*b (BN backward reductions) */
void pnn_oracle_colsum2(const double* a, const double* b, long M, int C, double* sa, double* sab) {
#pragma omp parallel for schedule(static)
  for (int c = 0; c < C; c++) {
    double s = 0.0, t = 0.0;
    for (long m = 0; m < M; m++) {
      double v = a[(size_t)m * C + c];
      s += v;
      t += v * b[(size_t)m * C + c];
    }
    sa[c] = s;
    sab[c] = t;
  }
}

/* round to the nearest bfloat16 (8 significant bits, ties to even); normal range only */
void pnn_oracle_round_bf16(double* x, size_t n) {
#pragma omp parallel for schedule(static)
  for (size_t i = 0; i < n; i++) {
    double v = x[i];
    if (v == 0.0 || !isfinite(v)) continue;
    int e;
    double m = frexp(v, &e);          /* v = m * 2^e, 0.5 <= |m| < 1 */
    m = nearbyint(m * 256.0) / 256.0; /* 8 significant bits, current (nearest-even) mode */
    x[i] = ldexp(m, e);
  }
}

#ifdef _OPENMP
#include <omp.h>
int pnn_oracle_threads(void) { return omp_get_max_threads(); }
#else
int pnn_oracle_threads(void) { return 1; }
#endif

/* The three convolution definitions above, evaluated only at the flat output indices idx[0..n)
 * (for checks at full size where whole tensors are too costly in fp64). */
void pnn_oracle_conv_fwd_at(const double* x, int B, int H, int W, int C, const double* w, int K,
                            int k, int st, int pad, int Ho, int Wo, const long* idx, long n,
                            double* out) {
  (void)B;
#pragma omp parallel for schedule(static)
  for (long i = 0; i < n; i++) {
    long t = idx[i];
    int o = (int)(t % K); t /= K;
    int q = (int)(t % Wo); t /= Wo;
    int p = (int)(t % Ho);
    int nb = (int)(t / Ho);
    double acc = 0.0;
    for (int r = 0; r < k; r++) {
      int ih = p * st + r - pad;
      if (ih < 0 || ih >= H) continue;
      for (int s = 0; s < k; s++) {
        int iw = q * st + s - pad;
        if (iw < 0 || iw >= W) continue;
        const double* xv = x + IDX4(nb, ih, iw, 0, H, W, C);
        const double* wv = w + IDX4(o, r, s, 0, k, k, C);
        for (int c = 0; c < C; c++) acc += wv[c] * xv[c];
      }
    }
    out[i] = acc;
  }
}

void pnn_oracle_conv_bwd_data_at(const double* gy, int B, int H, int W, int C, const double* w,
                                 int K, int k, int st, int pad, int Ho, int Wo, const long* idx,
                                 long n, double* out) {
  (void)B;
#pragma omp parallel for schedule(static)
  for (long i = 0; i < n; i++) {
    long t = idx[i];
    int c = (int)(t % C); t /= C;
    int v = (int)(t % W); t /= W;
    int h = (int)(t % H);
    int nb = (int)(t / H);
    double acc = 0.0;
    for (int r = 0; r < k; r++) {
      int th = h + pad - r;
      if (th < 0 || th % st) continue;
      int p = th / st;
      if (p >= Ho) continue;
      for (int s = 0; s < k; s++) {
        int tw = v + pad - s;
        if (tw < 0 || tw % st) continue;
        int q = tw / st;
        if (q >= Wo) continue;
        const double* g = gy + IDX4(nb, p, q, 0, Ho, Wo, K);
        for (int o = 0; o < K; o++) acc += g[o] * w[IDX4(o, r, s, c, k, k, C)];
      }
    }
    out[i] = acc;
  }
}

void pnn_oracle_conv_bwd_weight_at(const double* x, int B, int H, int W, int C, const double* gy,
                                   int K, int k, int st, int pad, int Ho, int Wo, const long* idx,
                                   long n, double* out) {
#pragma omp parallel for schedule(static)
  for (long i = 0; i < n; i++) {
    long t = idx[i];
    int c = (int)(t % C); t /= C;
    int s = (int)(t % k); t /= k;
    int r = (int)(t % k);
    int o = (int)(t / k);
    double acc = 0.0;
    for (int nb = 0; nb < B; nb++)
      for (int p = 0; p < Ho; p++) {
        int ih = p * st + r - pad;
        if (ih < 0 || ih >= H) continue;
        for (int q = 0; q < Wo; q++) {
          int iw = q * st + s - pad;
          if (iw < 0 || iw >= W) continue;
          acc += gy[IDX4(nb, p, q, o, Ho, Wo, K)] * x[IDX4(nb, ih, iw, c, H, W, C)];
        }
      }
    out[i] = acc;
  }
}
