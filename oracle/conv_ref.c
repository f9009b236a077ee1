/*
 * Oracle for the forward convolution of Eq. (1) -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests, the smoke check and the benchmark's cpu_baseline leg may load
 * this file's library.  The product path (the HIP library) never links,
 * calls or falls back to it.
 *
 * What it computes (Sec. 1, Eq. (1); loop bounds of Listing 2 in Sec. 2.2):
 *
 *   Out[n][k][h][w] = sum over c < C, r < R, s < S of
 *                     In[n][c][h + r][w + s] * Ker[k][c][r][s]
 *
 * for h < P = H - R + 1 and w < Q = W - S + 1 (H, W are the *input* height
 * and width, as in the caption of Table 1; the output extents follow from
 * the index h + r staying inside the input: a valid correlation, no kernel
 * flip, no padding, stride 1).  Out is written, not accumulated into: the
 * equation defines Out as the sum, Listing 2's "+=" presumes a zeroed Out.
 *
 * Layouts (Sec. 9 and the artifact appendix): In is NCHW, Ker is KCRS, Out
 * is NKPQ, all dense and row-major.  Inputs arrive as float (fp32, or bf16
 * values widened to fp32, which is exact); every product and every partial
 * sum is formed in double.  A float times a float is exact in double, so
 * the only rounding is the fp64 summation, ~1e-16 relative.
 *
 * The loop order (n, k, h, w outside; c, r, s inside) is the plain order of
 * the definition; nothing is blocked, fused or reordered.  The outer (n, k)
 * pairs are independent, so an OpenMP pragma may run them on several host
 * threads; each output is still one sequential sum in c, r, s order.
 */
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One output element, Eq. (1) written out. */
static double conv_point(int C, int H, int W, int R, int S,
                         const float *In_n, const float *Ker_k, int h, int w) {
  double acc = 0.0;
  for (int c = 0; c < C; ++c)
    for (int r = 0; r < R; ++r)
      for (int s = 0; s < S; ++s)
        acc += (double)In_n[((size_t)c * H + (h + r)) * W + (w + s)] *
               (double)Ker_k[((size_t)c * R + r) * S + s];
  return acc;
}

/* Full output tensor Out[N][K][P][Q] (fp64).  Returns 0, or -1 on a shape
 * that Eq. (1) does not define (a non-positive extent, or R > H, S > W). */
int oracle_conv_fwd(int N, int C, int K, int H, int W, int R, int S,
                    const float *In, const float *Ker, double *Out) {
  if (N <= 0 || C <= 0 || K <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 ||
      R > H || S > W)
    return -1;
  const int P = H - R + 1, Q = W - S + 1;
  const long long NK = (long long)N * K;
#pragma omp parallel for schedule(dynamic, 1)
  for (long long nk = 0; nk < NK; ++nk) {
    const int n = (int)(nk / K), k = (int)(nk % K);
    const float *In_n = In + (size_t)n * C * H * W;
    const float *Ker_k = Ker + (size_t)k * C * R * S;
    double *Out_nk = Out + (size_t)nk * P * Q;
    for (int h = 0; h < P; ++h)
      for (int w = 0; w < Q; ++w)
        Out_nk[(size_t)h * Q + w] = conv_point(C, H, W, R, S, In_n, Ker_k, h, w);
  }
  return 0;
}

/* Selected outputs only: idx[i] is a flat NKPQ index into Out; out[i]
 * receives that element (fp64).  For full-size shapes where the whole
 * tensor would take too long on the host. */
int oracle_conv_fwd_points(int N, int C, int K, int H, int W, int R, int S,
                           const float *In, const float *Ker,
                           const int64_t *idx, int64_t npts, double *out) {
  if (N <= 0 || C <= 0 || K <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 ||
      R > H || S > W)
    return -1;
  const int P = H - R + 1, Q = W - S + 1;
  const int64_t total = (int64_t)N * K * P * Q;
  for (int64_t i = 0; i < npts; ++i)
    if (idx[i] < 0 || idx[i] >= total) return -2;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < npts; ++i) {
    int64_t e = idx[i];
    const int w = (int)(e % Q); e /= Q;
    const int h = (int)(e % P); e /= P;
    const int k = (int)(e % K); e /= K;
    const int n = (int)e;
    out[i] = conv_point(C, H, W, R, S, In + (size_t)n * C * H * W,
                        Ker + (size_t)k * C * R * S, h, w);
  }
  return 0;
}

/*
 * Strided and zero-padded correlation (row f2).  The paper presents Eq. (1)
 * without stride or dilation and notes that its method carries over to the
 * general case (Sec. 3.1, footnote 1); Table 1 includes stride-2 layers.
 * The general form used here (the usual definition of a strided, padded
 * correlation, as in PyTorch's conv2d):
 *
 *   Out[n][k][h][w] = sum over c < C, r < R, s < S of
 *                     X[n][c][h*sh + r - ph][w*sw + s - pw] * Ker[k][c][r][s]
 *
 * where X is In inside [0, H) x [0, W) and zero outside (ph, pw rows and
 * columns of zero padding on each side), for h < P = (H + 2 ph - R) / sh + 1
 * and w < Q = (W + 2 pw - S) / sw + 1 (integer division).  With sh = sw = 1
 * and ph = pw = 0 it is Eq. (1) above.
 */
static double conv_point_ex(int C, int H, int W, int R, int S, int sh, int sw, int ph, int pw,
                            const float *In_n, const float *Ker_k, int h, int w) {
  double acc = 0.0;
  for (int c = 0; c < C; ++c)
    for (int r = 0; r < R; ++r)
      for (int s = 0; s < S; ++s) {
        const int y = h * sh + r - ph, x = w * sw + s - pw; /* input row and column */
        if (y < 0 || y >= H || x < 0 || x >= W) continue;   /* zero padding */
        acc += (double)In_n[((size_t)c * H + y) * W + x] *
               (double)Ker_k[((size_t)c * R + r) * S + s];
      }
  return acc;
}

static int ex_extents(int H, int W, int R, int S, int sh, int sw, int ph, int pw, int *P, int *Q) {
  if (sh <= 0 || sw <= 0 || ph < 0 || pw < 0 || H + 2 * ph < R || W + 2 * pw < S) return -1;
  *P = (H + 2 * ph - R) / sh + 1;
  *Q = (W + 2 * pw - S) / sw + 1;
  return 0;
}

/* Full output [N][K][P][Q] of the strided, padded form (fp64).  Returns 0,
 * or -1 on an undefined shape. */
int oracle_conv_fwd_ex(int N, int C, int K, int H, int W, int R, int S, int sh, int sw, int ph,
                       int pw, const float *In, const float *Ker, double *Out) {
  int P, Q;
  if (N <= 0 || C <= 0 || K <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 ||
      ex_extents(H, W, R, S, sh, sw, ph, pw, &P, &Q))
    return -1;
  const long long NK = (long long)N * K;
#pragma omp parallel for schedule(dynamic, 1)
  for (long long nk = 0; nk < NK; ++nk) {
    const int n = (int)(nk / K), k = (int)(nk % K);
    const float *In_n = In + (size_t)n * C * H * W;
    const float *Ker_k = Ker + (size_t)k * C * R * S;
    double *Out_nk = Out + (size_t)nk * P * Q;
    for (int h = 0; h < P; ++h)
      for (int w = 0; w < Q; ++w)
        Out_nk[(size_t)h * Q + w] = conv_point_ex(C, H, W, R, S, sh, sw, ph, pw, In_n, Ker_k, h, w);
  }
  return 0;
}

/* Selected outputs of the strided, padded form (flat NKPQ indices). */
int oracle_conv_fwd_ex_points(int N, int C, int K, int H, int W, int R, int S, int sh, int sw,
                              int ph, int pw, const float *In, const float *Ker,
                              const int64_t *idx, int64_t npts, double *out) {
  int P, Q;
  if (N <= 0 || C <= 0 || K <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 ||
      ex_extents(H, W, R, S, sh, sw, ph, pw, &P, &Q))
    return -1;
  const int64_t total = (int64_t)N * K * P * Q;
  for (int64_t i = 0; i < npts; ++i)
    if (idx[i] < 0 || idx[i] >= total) return -2;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < npts; ++i) {
    int64_t e = idx[i];
    const int w = (int)(e % Q); e /= Q;
    const int h = (int)(e % P); e /= P;
    const int k = (int)(e % K); e /= K;
    const int n = (int)e;
    out[i] = conv_point_ex(C, H, W, R, S, sh, sw, ph, pw, In + (size_t)n * C * H * W,
                           Ker + (size_t)k * C * R * S, h, w);
  }
  return 0;
}

/* Sets the number of host threads later OpenMP regions of this library use
   (n >= 1); returns the previous number. */
int oracle_set_num_threads(int n) {
#ifdef _OPENMP
  const int prev = omp_get_max_threads();
  if (n >= 1) omp_set_num_threads(n);
  return prev;
#else
  (void)n;
  return 1;
#endif
}

/* Number of host threads an OpenMP region of this library would use. */
int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
