/*
 * kred oracle: plain, slow, fp64 CPU evaluation of the symbolic-matrix
 * reductions.  TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the
 * benchmark's CPU-baseline leg call it to check and to time the GPU library.
 * The GPU library never includes, links or calls anything in this directory,
 * and this file shares no code with it.
 *
 * What is computed follows Charlier, Feydy, Glaunes, Collin, Durif, "Kernel
 * Operations on the GPU, with Autodiff, without Memory Overflows"
 * (arXiv:2004.11127):
 *   - Eq. (1): a_i = sum_j exp(-|x_i - y_j|^2 / (2 sigma^2)) b_j, i = 1..M;
 *   - Eq. (2), Sec. 2: a_i = Reduction_{j=1..N} F(p, x_i, y_j) for a formula F
 *     and a reduction among those Sec. 2 lists (sum, log-sum-exp, min, max,
 *     arg-min, arg-K-min; arg-max by symmetry with arg-min);
 *   - Sec. 2 "Backpropagation": the gradient of a reduction is again a
 *     reduction of the same form; here d a_i / d x_i of Eq. (1), and the
 *     vector-Jacobian product of Eq. (1) in x for a cotangent of its output.
 *
 * Every routine is the definition written out: a double loop over (i, j) in
 * fp64 with a sequential j loop, libm exp/log/sqrt, no blocking and no
 * reordering beyond what the definition states.  Rows are 0-based; the
 * paper's i = 1..M is i = 0..M-1 here.  Inputs arrive already converted to
 * double by the caller.  OpenMP splits the independent rows i across threads.
 *
 * Readings of the paper that these routines encode (the paper is silent on
 * them):
 *   - Laplacian kernel: exp(-|x - y| / sigma), no normalising constant.
 *   - Gaussian kernel: exactly Eq. (1), no (2 pi sigma^2)^(-D/2) factor.
 *   - Log-sum-exp formula (Sinkhorn form): s_ij = g_j - |x_i - y_j|^2 / eps,
 *     a_i = log sum_j exp(s_ij), natural log.
 *   - Arg-K-min: the indices of the K smallest |x_i - y_j|^2, ascending by
 *     (distance, index); equal distances are ordered by the lower index.
 *
 * Parity unpinned: none of the routines below (each has closed-form or
 * brute-force checks in the test suite).
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <omp.h>

#define ORACLE_GAUSS 0
#define ORACLE_LAPLACE 1
#define ORACLE_SQDIST 2

/* |x_i - y_j|^2 in the direct form sum_k (x_ik - y_jk)^2. */
static double sq_dist(const double* xi, const double* yj, int D) {
  double d = 0.0;
  for (int k = 0; k < D; ++k) {
    double t = xi[k] - yj[k];
    d += t * t;
  }
  return d;
}

/* The scalar kernel value F(d) for the sum formulas, d = |x - y|^2. */
static double kernel_value(int formula, double d, double sigma) {
  switch (formula) {
    case ORACLE_GAUSS: return exp(-d / (2.0 * sigma * sigma));   /* Eq. (1) */
    case ORACLE_LAPLACE: return exp(-sqrt(d) / sigma);
    default: return d;                                             /* squared distance */
  }
}

static int64_t row_of(const int64_t* rows, int64_t r) { return rows ? rows[r] : r; }

/*
 * Sum reduction of Eq. (2) with F = kernel(x_i, y_j) * b_j (Eq. (1) when the
 * kernel is the Gaussian):  out[r, e] = sum_j F(|x_i - y_j|^2) b_je,
 * norm[r, e] = sum_j |F(|x_i - y_j|^2) b_je|, i = rows[r] (or r if rows is
 * NULL).  x: M x D, y: N x D, b: N x E, out and norm: nrows x E, row-major.
 * Returns 0, or -1 on a bad argument.
 */
int oracle_kernel_sum(int formula, double sigma, int64_t M, int64_t N, int D, int E,
                      const double* x, const double* y, const double* b,
                      const int64_t* rows, int64_t nrows, double* out, double* norm) {
  if (formula < ORACLE_GAUSS || formula > ORACLE_SQDIST || D < 1 || E < 1 || nrows < 0) return -1;
  if (formula != ORACLE_SQDIST && !(sigma > 0.0)) return -1;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t i = row_of(rows, r);
    const double* xi = x + i * D;
    for (int e = 0; e < E; ++e) { out[r * E + e] = 0.0; norm[r * E + e] = 0.0; }
    for (int64_t j = 0; j < N; ++j) {
      const double kij = kernel_value(formula, sq_dist(xi, y + j * D, D), sigma);
      for (int e = 0; e < E; ++e) {
        const double term = kij * b[j * E + e];
        out[r * E + e] += term;
        norm[r * E + e] += fabs(term);
      }
    }
  }
  (void)M;
  return 0;
}

/*
 * Gaussian sum of Eq. (1) with E = 1 and its gradient with respect to x_i
 * (the derivative reduction of Sec. 2, "Backpropagation"):
 *   out[r, 0]   = a_i   = sum_j k_ij b_j,            k_ij = exp(-|x_i-y_j|^2 / (2 sigma^2))
 *   out[r, 1+k] = g_ik  = sum_j k_ij b_j (y_jk - x_ik) / sigma^2
 * which is d a_i / d x_ik, since d k_ij / d x_ik = -k_ij (x_ik - y_jk) / sigma^2.
 * norm holds the matching sums of absolute values of the summands.
 * out and norm: nrows x (1 + D).
 */
int oracle_gauss_gradx(double sigma, int64_t M, int64_t N, int D,
                       const double* x, const double* y, const double* b,
                       const int64_t* rows, int64_t nrows, double* out, double* norm) {
  if (D < 1 || nrows < 0 || !(sigma > 0.0)) return -1;
  const int W = 1 + D;
  const double s2 = sigma * sigma;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t i = row_of(rows, r);
    const double* xi = x + i * D;
    for (int c = 0; c < W; ++c) { out[r * W + c] = 0.0; norm[r * W + c] = 0.0; }
    for (int64_t j = 0; j < N; ++j) {
      const double* yj = y + j * D;
      const double w = exp(-sq_dist(xi, yj, D) / (2.0 * s2)) * b[j];
      out[r * W] += w;
      norm[r * W] += fabs(w);
      for (int k = 0; k < D; ++k) {
        const double term = w * (yj[k] - xi[k]) / s2;
        out[r * W + 1 + k] += term;
        norm[r * W + 1 + k] += fabs(term);
      }
    }
  }
  (void)M;
  return 0;
}

/*
 * Vector-Jacobian product of the Gaussian kernel sum in x (Sec. 2,
 * "Backpropagation": the gradient of a reduction is again a reduction of the
 * form of Eq. (2)).  For the output a_i = sum_j k_ij b_j of Eq. (1) with E
 * signal columns, k_ij = exp(-|x_i - y_j|^2 / (2 sigma^2)), and a cotangent
 * e (M x E), the scalar L = sum_i <e_i, a_i> has
 *   dL/dx_ik = sum_j k_ij <e_i, b_j> (y_jk - x_ik) / sigma^2.
 * The y-gradient is this same reduction with the roles of (x, e) and (y, b)
 * exchanged; dL/db_j = sum_i k_ij e_i is the Gaussian sum with x and y
 * exchanged.  norm holds the sums of absolute values of the summands.
 * out and norm: nrows x D.
 */
int oracle_gauss_vjp(double sigma, int64_t M, int64_t N, int D, int E,
                     const double* x, const double* y, const double* b, const double* e,
                     const int64_t* rows, int64_t nrows, double* out, double* norm) {
  if (D < 1 || E < 1 || nrows < 0 || !(sigma > 0.0)) return -1;
  const double s2 = sigma * sigma;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t i = row_of(rows, r);
    const double* xi = x + i * D;
    const double* ei = e + i * E;
    for (int k = 0; k < D; ++k) { out[r * D + k] = 0.0; norm[r * D + k] = 0.0; }
    for (int64_t j = 0; j < N; ++j) {
      const double* yj = y + j * D;
      const double* bj = b + j * E;
      double dot = 0.0;
      for (int c = 0; c < E; ++c) dot += ei[c] * bj[c];
      const double w = exp(-sq_dist(xi, yj, D) / (2.0 * s2)) * dot;
      for (int k = 0; k < D; ++k) {
        const double term = w * (yj[k] - xi[k]) / s2;
        out[r * D + k] += term;
        norm[r * D + k] += fabs(term);
      }
    }
  }
  (void)M;
  return 0;
}

/*
 * Log-sum-exp reduction of Eq. (2) with the Sinkhorn-style formula
 *   s_ij = g_j - |x_i - y_j|^2 / eps,  a_i = log sum_j exp(s_ij),
 * evaluated in two passes: m_i = max_j s_ij, then a_i = m_i + log sum_j
 * exp(s_ij - m_i).  With N = 0 the empty sum gives a_i = -infinity.
 * out[r] also returns m_i in maxv[r] when maxv is not NULL.
 */
int oracle_sinkhorn_lse(double eps, int64_t M, int64_t N, int D,
                        const double* x, const double* y, const double* g,
                        const int64_t* rows, int64_t nrows, double* out, double* maxv) {
  if (D < 1 || nrows < 0 || !(eps > 0.0)) return -1;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t i = row_of(rows, r);
    const double* xi = x + i * D;
    double m = -INFINITY;
    for (int64_t j = 0; j < N; ++j) {
      const double s = g[j] - sq_dist(xi, y + j * D, D) / eps;
      if (s > m) m = s;
    }
    double acc = 0.0;
    for (int64_t j = 0; j < N; ++j) {
      const double s = g[j] - sq_dist(xi, y + j * D, D) / eps;
      acc += exp(s - m);
    }
    out[r] = (N > 0) ? m + log(acc) : -INFINITY;
    if (maxv) maxv[r] = m;
  }
  (void)M;
  return 0;
}

/*
 * Log-sum-exp reduction of Eq. (2) for the log-domain kernel sums: with
 * weights g_j in the log domain,
 *   a_i = log sum_j k_ij exp(g_j) = log sum_j exp(s_ij),  s_ij = g_j + log k_ij,
 * for the Gaussian (log k = -d / (2 sigma^2), formula 0) and the Laplacian
 * (log k = -sqrt(d) / sigma, formula 1) kernels, d = |x_i - y_j|^2.  Two
 * passes as in the Sinkhorn-form routine above: the row maximum m_i, then
 * m_i + log sum_j exp(s_ij - m_i).  out, maxv (may be NULL): nrows.
 */
int oracle_kernel_lse(int formula, double sigma, int64_t M, int64_t N, int D,
                      const double* x, const double* y, const double* g,
                      const int64_t* rows, int64_t nrows, double* out, double* maxv) {
  if (D < 1 || nrows < 0 || !(sigma > 0.0)) return -1;
  if (formula != ORACLE_GAUSS && formula != ORACLE_LAPLACE) return -1;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t i = row_of(rows, r);
    const double* xi = x + i * D;
    double m = -INFINITY;
    for (int64_t j = 0; j < N; ++j) {
      const double d = sq_dist(xi, y + j * D, D);
      const double s = g[j] + (formula == ORACLE_GAUSS ? -d / (2.0 * sigma * sigma) : -sqrt(d) / sigma);
      if (s > m) m = s;
    }
    double acc = 0.0;
    for (int64_t j = 0; j < N; ++j) {
      const double d = sq_dist(xi, y + j * D, D);
      const double s = g[j] + (formula == ORACLE_GAUSS ? -d / (2.0 * sigma * sigma) : -sqrt(d) / sigma);
      acc += exp(s - m);
    }
    out[r] = (N > 0) ? m + log(acc) : -INFINITY;
    if (maxv) maxv[r] = m;
  }
  (void)M;
  return 0;
}

/*
 * Min, max, arg-min and arg-max reductions of Eq. (2) (Sec. 2 lists .min(),
 * .max() and .argmin() beside the sum): for each selected row i and each
 * component e of the formula, the extreme value over j of F_ije and the
 * lowest index j where it is reached.  Formulas:
 *   formula 0..2 (Gauss, Laplace, squared distance) with b: F_ije = kernel(d_ij) b_je;
 *   formula 2 with b == NULL:                               F_ij  = d_ij (E = 1);
 *   formula 4 (log-sum-exp formula):                         F_ij  = b_j - d_ij / param (E = 1).
 * param is sigma (Gauss, Laplace) or eps (formula 4).  op: 0 = min, 1 = max.
 * val, idx (idx may be NULL) and scale: nrows x E; scale holds max_j |F_ije|,
 * the size of the row's values.  With N = 0: val = +inf (min) or -inf (max),
 * idx = -1, scale = 0.
 */
int oracle_extreme(int formula, int op, double param, int64_t M, int64_t N, int D, int E,
                   const double* x, const double* y, const double* b,
                   const int64_t* rows, int64_t nrows, double* val, int64_t* idx, double* scale) {
  if (D < 1 || E < 1 || nrows < 0 || (op != 0 && op != 1)) return -1;
  if (formula == 3 || formula < 0 || formula > 4) return -1;
  if (formula != ORACLE_SQDIST && !(param > 0.0)) return -1;
  if ((formula == 4 || b == NULL) && E != 1) return -1;
  if (b == NULL && formula != ORACLE_SQDIST) return -1;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t i = row_of(rows, r);
    const double* xi = x + i * D;
    for (int e = 0; e < E; ++e) {
      val[r * E + e] = op == 0 ? INFINITY : -INFINITY;
      if (idx) idx[r * E + e] = -1;
      scale[r * E + e] = 0.0;
    }
    for (int64_t j = 0; j < N; ++j) {
      const double d = sq_dist(xi, y + j * D, D);
      for (int e = 0; e < E; ++e) {
        double f;
        if (formula == 4) f = b[j] - d / param;
        else if (b == NULL) f = d;
        else f = kernel_value(formula, d, param) * b[j * E + e];
        const int better = op == 0 ? f < val[r * E + e] : f > val[r * E + e];
        if (better) {   /* strict: the first (lowest) j keeps a tie */
          val[r * E + e] = f;
          if (idx) idx[r * E + e] = j;
        }
        if (fabs(f) > scale[r * E + e]) scale[r * E + e] = fabs(f);
      }
    }
  }
  (void)M;
  return 0;
}

/* (d, j) strictly before (d', j') in the ascending (distance, index) order. */
static int before(double d, int64_t j, double d2, int64_t j2) {
  return d < d2 || (d == d2 && j < j2);
}

/*
 * Arg-K-min reduction of Eq. (2) (Sec. 2, argKmin): for each selected row i,
 * the indices of the K smallest |x_i - y_j|^2 over j, ascending by
 * (distance, index).  Plain selection: keep a sorted list of the K best
 * (distance, index) pairs seen so far and insert each new pair in order.
 * idx: nrows x K (int64), dist: nrows x K (may be NULL).  Requires 1 <= K <= N.
 */
int oracle_argkmin(int64_t M, int64_t N, int D, int K,
                   const double* x, const double* y,
                   const int64_t* rows, int64_t nrows, int64_t* idx, double* dist) {
  if (D < 1 || K < 1 || K > N || nrows < 0) return -1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const int64_t i = row_of(rows, r);
    const double* xi = x + i * D;
    int64_t* bj = idx + r * K;
    double bd[1024];
    double* bdp = (K <= 1024) ? bd : NULL;
    if (!bdp) continue;  /* K is capped well below this by the caller */
    int count = 0;
    for (int64_t j = 0; j < N; ++j) {
      const double d = sq_dist(xi, y + j * D, D);
      if (count == K && !before(d, j, bdp[K - 1], bj[K - 1])) continue;
      int pos = (count < K) ? count : K - 1;   /* slot freed at the end */
      while (pos > 0 && before(d, j, bdp[pos - 1], bj[pos - 1])) {
        bdp[pos] = bdp[pos - 1];
        bj[pos] = bj[pos - 1];
        --pos;
      }
      bdp[pos] = d;
      bj[pos] = j;
      if (count < K) ++count;
    }
    if (dist)
      for (int k = 0; k < K; ++k) dist[r * K + k] = bdp[k];
  }
  (void)M;
  return 0;
}

/* Number of OpenMP threads the routines above use. */
int oracle_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    n = omp_get_num_threads();
  }
  return n;
}
