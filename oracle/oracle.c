/*
 * ChebBooster online stage: slow, plain fp64 CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file; only the test suite, the smoke check and the CPU baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with
 * the HIP library.
 *
 * What it computes (paper, Section 3.2 "Chebyshev-Inspired Extrapolation",
 * Section 3.3 "ChebBooster", Appendix A):
 *
 *   - barycentric weights rho_j = 1 / omega'(x_j) for arbitrary distinct
 *     nodes (Appendix A, general-weights equation),
 *   - interpolation coefficients w_j(x) = (rho_j / (x - x_j)) /
 *     sum_i rho_i / (x - x_i)  (Section 3.2, coefficient equation; Appendix A,
 *     second barycentric form), with nodes and target first mapped affinely
 *     onto [-1, 1] (Section 3.3, weight precomputation),
 *   - the skipped-step prediction f_t = sum_j w_j f_{s_j} (Section 3.3,
 *     forward application equation; Algorithm 1, online stage), evaluated
 *     per element in fp64 with the terms added oldest to newest.
 *
 * Floating-point storage formats are decoded exactly from their IEEE-754
 * definitions.  All accumulation is fp64.  No blocking, no reordering, no
 * fused shortcuts: one element at a time, one history entry at a time.
 *
 * Every function has pins in the CPU test suite against closed forms,
 * exact rational Lagrange weights and the paper's equispaced-node formula.
 */
#include "oracle.h"

#include <math.h>
#include <stdint.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Threads (the per-element loop is independent across elements).            */
/* ------------------------------------------------------------------------ */

int oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Node checks and normalisation (Section 3.3: timesteps mapped to [-1,1]).   */
/* ------------------------------------------------------------------------ */

/* Returns 0 when every node is finite and no two are equal, else a negative
 * code: -1 bad count, -2 non-finite node, -3 repeated node. */
int oracle_check_nodes(const double *x, int n) {
  if (n < 1) return -1;
  for (int j = 0; j < n; ++j)
    if (!isfinite(x[j])) return -2;
  for (int j = 0; j < n; ++j)
    for (int k = j + 1; k < n; ++k)
      if (x[j] == x[k]) return -3;
  return 0;
}

/* Affine map of the node span [min x, max x] onto [-1, 1]; the target goes
 * through the same map, so |y*| > 1 means extrapolation.  With a single node
 * there is no span and everything maps to 0. */
void oracle_normalise(const double *x, int n, double xstar, double *y,
                      double *ystar) {
  double a = x[0], b = x[0];
  for (int j = 1; j < n; ++j) {
    if (x[j] < a) a = x[j];
    if (x[j] > b) b = x[j];
  }
  if (n == 1 || b == a) {
    for (int j = 0; j < n; ++j) y[j] = 0.0;
    *ystar = 0.0;
    return;
  }
  for (int j = 0; j < n; ++j) y[j] = (2.0 * x[j] - (a + b)) / (b - a);
  *ystar = (2.0 * xstar - (a + b)) / (b - a);
}

/* ------------------------------------------------------------------------ */
/* Barycentric weights (Appendix A).                                          */
/* ------------------------------------------------------------------------ */

/* rho_j = 1 / omega'(y_j), omega'(y_j) = prod_{k != j} (y_j - y_k). */
void oracle_barycentric_rho(const double *y, int n, double *rho) {
  for (int j = 0; j < n; ++j) {
    double d = 1.0;
    for (int k = 0; k < n; ++k)
      if (k != j) d *= (y[j] - y[k]);
    rho[j] = 1.0 / d;
  }
}

/* One row of interpolation coefficients for one target.  Returns 0 or the
 * negative code of oracle_check_nodes.  A target equal to a node gets the
 * unit vector of that node (the second form is 0/0 there, its limit is the
 * node value). */
int oracle_weights_row(const double *x, int n, double xstar, double *w) {
  int rc = oracle_check_nodes(x, n);
  if (rc) return rc;
  if (!isfinite(xstar)) return -2;
  for (int j = 0; j < n; ++j) {
    if (xstar == x[j]) {
      for (int k = 0; k < n; ++k) w[k] = (k == j) ? 1.0 : 0.0;
      return 0;
    }
  }
  double y[ORACLE_MAX_NODES], rho[ORACLE_MAX_NODES], q[ORACLE_MAX_NODES];
  if (n > ORACLE_MAX_NODES) return -1;
  double ystar;
  oracle_normalise(x, n, xstar, y, &ystar);
  if (n == 1) { /* degree-0 interpolant: the single cached value */
    w[0] = 1.0;
    return 0;
  }
  oracle_barycentric_rho(y, n, rho);
  double denom = 0.0;
  for (int j = 0; j < n; ++j) {
    double diff = ystar - y[j];
    if (diff == 0.0) { /* distinct x collapsed by the map: take the limit */
      for (int k = 0; k < n; ++k) w[k] = (k == j) ? 1.0 : 0.0;
      return 0;
    }
    q[j] = rho[j] / diff;
    denom += q[j];
  }
  for (int j = 0; j < n; ++j) w[j] = q[j] / denom;
  return 0;
}

/* Table of rows: w[m * n + j] for target m, node j (oldest to newest). */
int oracle_weights(const double *x, int n, const double *xstar, int m,
                   double *w) {
  for (int i = 0; i < m; ++i) {
    int rc = oracle_weights_row(x, n, xstar[i], w + (size_t)i * n);
    if (rc) return rc;
  }
  return 0;
}

/* Lagrange product form l_j(x) = prod_{k != j} (x - x_k) / (x_j - x_k)
 * (Appendix A, Lagrange basis).  Evaluated on the raw nodes; used by the
 * tests as a second, independent route to the same coefficients. */
int oracle_lagrange_row(const double *x, int n, double xstar, double *w) {
  int rc = oracle_check_nodes(x, n);
  if (rc) return rc;
  for (int j = 0; j < n; ++j) {
    double l = 1.0;
    for (int k = 0; k < n; ++k)
      if (k != j) l *= (xstar - x[k]) / (x[j] - x[k]);
    w[j] = l;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Exact decoding of storage formats (IEEE-754 definitions).                  */
/* ------------------------------------------------------------------------ */

/* bfloat16 is the upper half of an IEEE binary32 pattern. */
double oracle_bf16_to_f64(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Correct rounding of a binary64 value to bfloat16, ties to even, written
 * from the format definition: 8 significand bits, exponent range of
 * binary32 (normal down to 2^-126, subnormal spacing 2^-133). */
uint16_t oracle_round_bf16(double v) {
  if (isnan(v)) return (uint16_t)0x7FC0;
  uint16_t sign = signbit(v) ? 0x8000 : 0x0000;
  double a = fabs(v);
  if (a == 0.0) return sign;
  if (isinf(a)) return (uint16_t)(sign | 0x7F80);
  int ex;
  (void)frexp(a, &ex);          /* a = m * 2^ex, m in [0.5, 1) */
  int e = ex - 1;               /* a in [2^e, 2^(e+1)) */
  int qexp = (e < -126) ? -133 : e - 7;
  double units = ldexp(a, -qexp);          /* exact: power-of-two scaling */
  double r = floor(units);
  double frac = units - r;                 /* exact: units < 2^9 */
  if (frac > 0.5 || (frac == 0.5 && fmod(r, 2.0) != 0.0)) r += 1.0;
  double rounded = ldexp(r, qexp);
  if (rounded >= ldexp(1.0, 128)) return (uint16_t)(sign | 0x7F80);
  float f = (float)rounded;                /* exact: fits in binary32 */
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return (uint16_t)(sign | (uint16_t)((u >> 16) & 0x7FFF));
}

/* Correct rounding of binary64 to binary32, ties to even: the C cast under
 * the default rounding mode is exactly that operation. */
float oracle_round_f32(double v) { return (float)v; }

/* Array forms of the two bfloat16 conversions. */
void oracle_decode_bf16(const uint16_t *h, int64_t count, double *out) {
  for (int64_t i = 0; i < count; ++i) out[i] = oracle_bf16_to_f64(h[i]);
}

void oracle_encode_bf16(const double *v, int64_t count, uint16_t *out) {
  for (int64_t i = 0; i < count; ++i) out[i] = oracle_round_bf16(v[i]);
}

/* ------------------------------------------------------------------------ */
/* The skipped-step prediction, element by element (Section 3.3, Alg. 1).    */
/* ------------------------------------------------------------------------ */

/* out[i] = sum_{k=0}^{n-1} w[k] * F_k[i], k from oldest to newest, fp64.
 * When absmag is not NULL it receives sum_k |w[k]| * |F_k[i]|, the size of
 * the terms that cancel, which the parity bound is stated against. */
void oracle_extrapolate_bf16(const uint16_t *const *F, int n, const double *w,
                             int64_t count, double *out, double *absmag) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    double s = 0.0, m = 0.0;
    for (int k = 0; k < n; ++k) {
      double f = oracle_bf16_to_f64(F[k][i]);
      s += w[k] * f;
      m += fabs(w[k]) * fabs(f);
    }
    out[i] = s;
    if (absmag) absmag[i] = m;
  }
}

void oracle_extrapolate_f32(const float *const *F, int n, const double *w,
                            int64_t count, double *out, double *absmag) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    double s = 0.0, m = 0.0;
    for (int k = 0; k < n; ++k) {
      double f = (double)F[k][i];
      s += w[k] * f;
      m += fabs(w[k]) * fabs(f);
    }
    out[i] = s;
    if (absmag) absmag[i] = m;
  }
}

void oracle_extrapolate_f64(const double *const *F, int n, const double *w,
                            int64_t count, double *out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    double s = 0.0;
    for (int k = 0; k < n; ++k) s += w[k] * F[k][i];
    out[i] = s;
  }
}

/* ------------------------------------------------------------------------ */
/* Full-computation schedule (Section 3.3, weight precomputation).           */
/* ------------------------------------------------------------------------ */

/* is_full[s] = 1 when step s of 0..T-1 runs the full network: s outside
 * [s0, T-1-s1], or r divides (s - s0).  Returns the number of full steps. */
int oracle_full_schedule(int T, int s0, int s1, int r, uint8_t *is_full) {
  if (T < 1 || s0 < 0 || s1 < 0 || r < 1) return -1;
  int count = 0;
  for (int s = 0; s < T; ++s) {
    int outside = (s < s0) || (s > T - 1 - s1);
    int on_grid = ((s - s0) % r) == 0;
    is_full[s] = (uint8_t)(outside || on_grid);
    count += is_full[s];
  }
  return count;
}

/* ------------------------------------------------------------------------ */
/* Offline table by simulating the online stage (Algorithm 1).               */
/* ------------------------------------------------------------------------ */

/* What step `step` does under a full-step mask full[0..T-1] (or, in
 * oracle_table_row, under the schedule (T, s0, s1, r)) with history size n,
 * found by running Algorithm 1's loop from step 0: a full step appends
 * itself to the history H (dropping the oldest once H holds n entries); a
 * skipped step with |H| = n gets the coefficients of the abscissae of H at
 * its own abscissa.  A skipped step with |H| < n follows `policy`: 0 runs
 * the full network instead (and so enters H), 1 uses the |H| entries it has
 * (a lower-degree interpolant), or a full step if H is empty.
 *   *kind     0 full, 1 predicted
 *   *n_used   entries the prediction uses (0 for a full step)
 *   nodes[]   their steps, oldest to newest;  w[] their coefficients.
 * Returns 0, or a negative code (bad arguments, or oracle_weights_row's). */
int oracle_table_row_mask(int T, const uint8_t *full, int n, const double *abscissa,
                          int policy, int step, int *kind, int *n_used, int *nodes,
                          double *w) {
  if (T < 1 || n < 1 || n > ORACLE_MAX_NODES || step < 0 || step >= T) return -1;
  if (policy != 0 && policy != 1) return -1;
  int hist[ORACLE_MAX_NODES];
  int count = 0;
  for (int s = 0; s <= step; ++s) {
    int runs_full = full[s] || count == 0 || (count < n && policy == 0);
    if (s == step) {
      if (runs_full) {
        *kind = 0;
        *n_used = 0;
        return 0;
      }
      double x[ORACLE_MAX_NODES];
      for (int j = 0; j < count; ++j) {
        nodes[j] = hist[j];
        x[j] = abscissa[hist[j]];
      }
      *kind = 1;
      *n_used = count;
      return oracle_weights_row(x, count, abscissa[s], w);
    }
    if (runs_full) {
      if (count == n) {           /* drop the oldest */
        for (int j = 1; j < n; ++j) hist[j - 1] = hist[j];
        count -= 1;
      }
      hist[count++] = s;
    }
  }
  return -1; /* not reached */
}

int oracle_table_row(int T, int s0, int s1, int r, int n, const double *abscissa,
                     int policy, int step, int *kind, int *n_used, int *nodes,
                     double *w) {
  uint8_t full[4096];
  if (T < 1 || T > 4096) return -1;
  if (oracle_full_schedule(T, s0, s1, r, full) < 0) return -1;
  return oracle_table_row_mask(T, full, n, abscissa, policy, step, kind, n_used, nodes, w);
}

/* ------------------------------------------------------------------------ */
/* Residual application on a skipped step (Section 3.1, block equation).     */
/* ------------------------------------------------------------------------ */

/* A DiT block adds its module outputs to the residual stream:
 * x_{l+1} = x_l + S^l + C^l + M^l.  On a skipped step every module output
 * is the prediction sum_k w_k F_k[segment], so after all blocks
 *     x_out[j] = x_in[j] + sum over segments s covering j of
 *                sum_k w_k F_k[slot_offset[s] + (j - res_offset[s])].
 * F_k are n history entries of slot_numel elements (bfloat16 bit patterns),
 * segment s holds seg_numel[s] elements at slot_offset[s] and adds into
 * residual elements res_offset[s] .. res_offset[s] + seg_numel[s] - 1
 * (res_offset[s] < 0: the segment is not added).  x_in may be NULL (zero).
 * absmag (may be NULL) receives |x_in[j]| + the sum of |w_k| |F_k[.]| over
 * the same terms.  Everything in fp64, segment by segment, oldest entry
 * first.  Returns 0, or -1 if a segment leaves the residual. */
int oracle_residual_bf16(const uint16_t *const *F, int n, const double *w,
                         const int64_t *slot_offset, const int64_t *seg_numel,
                         const int64_t *res_offset, int n_segs, const double *x_in,
                         int64_t res_numel, double *x_out, double *absmag) {
  for (int s = 0; s < n_segs; ++s)
    if (res_offset[s] >= 0 && res_offset[s] + seg_numel[s] > res_numel) return -1;
  for (int64_t j = 0; j < res_numel; ++j) {
    x_out[j] = x_in ? x_in[j] : 0.0;
    if (absmag) absmag[j] = x_in ? fabs(x_in[j]) : 0.0;
  }
  for (int s = 0; s < n_segs; ++s) {
    if (res_offset[s] < 0) continue;
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < seg_numel[s]; ++e) {
      double acc = 0.0, mag = 0.0;
      for (int k = 0; k < n; ++k) {
        double f = oracle_bf16_to_f64(F[k][slot_offset[s] + e]);
        acc += w[k] * f;
        mag += fabs(w[k]) * fabs(f);
      }
      x_out[res_offset[s] + e] += acc;
      if (absmag) absmag[res_offset[s] + e] += mag;
    }
  }
  return 0;
}

/* The same with binary32 history entries. */
int oracle_residual_f32(const float *const *F, int n, const double *w,
                        const int64_t *slot_offset, const int64_t *seg_numel,
                        const int64_t *res_offset, int n_segs, const double *x_in,
                        int64_t res_numel, double *x_out, double *absmag) {
  for (int s = 0; s < n_segs; ++s)
    if (res_offset[s] >= 0 && res_offset[s] + seg_numel[s] > res_numel) return -1;
  for (int64_t j = 0; j < res_numel; ++j) {
    x_out[j] = x_in ? x_in[j] : 0.0;
    if (absmag) absmag[j] = x_in ? fabs(x_in[j]) : 0.0;
  }
  for (int s = 0; s < n_segs; ++s) {
    if (res_offset[s] < 0) continue;
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < seg_numel[s]; ++e) {
      double acc = 0.0, mag = 0.0;
      for (int k = 0; k < n; ++k) {
        double f = (double)F[k][slot_offset[s] + e];
        acc += w[k] * f;
        mag += fabs(w[k]) * fabs(f);
      }
      x_out[res_offset[s] + e] += acc;
      if (absmag) absmag[res_offset[s] + e] += mag;
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Node and weight variants (Section 3.2).                                    */
/* ------------------------------------------------------------------------ */

/* Chebyshev points on [a, b], largest first.  kind 1: the roots of T_n,
 * cos((2j-1) pi / (2n)), j = 1..n (Section 3.2, node equation); kind 2: the
 * extrema cos((j-1) pi / (n-1)), j = 1..n (n >= 2).  Returns 0 or -1. */
int oracle_chebyshev_nodes(int n, int kind, double a, double b, double *x) {
  if (n < 1 || (kind != 1 && kind != 2) || (kind == 2 && n < 2)) return -1;
  const double pi = 3.14159265358979323846;
  for (int j = 1; j <= n; ++j) {
    double c = (kind == 1) ? cos((2.0 * j - 1.0) * pi / (2.0 * n))
                           : cos((j - 1.0) * pi / (n - 1.0));
    x[j - 1] = 0.5 * (a + b) + 0.5 * (b - a) * c;
  }
  return 0;
}

/* Coefficients from the alternating weights printed in Section 3.2,
 * rho_j = (-1)^j * (1/2 at j = 1 and j = n, 1 otherwise), put into the
 * coefficient equation of Section 3.2 at the given nodes.  A target on a
 * node gets that node's unit row.  Returns 0 or the node-check code. */
int oracle_weights_row_alternating(const double *x, int n, double xstar, double *w) {
  int rc = oracle_check_nodes(x, n);
  if (rc) return rc;
  if (!isfinite(xstar)) return -2;
  for (int j = 0; j < n; ++j) {
    if (xstar == x[j]) {
      for (int k = 0; k < n; ++k) w[k] = (k == j) ? 1.0 : 0.0;
      return 0;
    }
  }
  if (n == 1) {
    w[0] = 1.0;
    return 0;
  }
  double denom = 0.0;
  for (int j = 0; j < n; ++j) {
    double rho = ((j % 2) ? -1.0 : 1.0) * ((j == 0 || j == n - 1) ? 0.5 : 1.0);
    w[j] = rho / (xstar - x[j]);
    denom += w[j];
  }
  for (int j = 0; j < n; ++j) w[j] /= denom;
  return 0;
}

/* Taylor expansion about the newest node x_{n-1} (the comparison of
 * Section 3.2's Runge-function study, whose text gives no formula; the
 * reading taken here): the i-th derivative over i! is estimated by the
 * divided difference over the newest i+1 nodes, so
 *     P(x*) = sum_{i=0}^{n-1} f[x_{n-1}, ..., x_{n-1-i}] (x* - x_{n-1})^i.
 * On equispaced nodes f[...] is the i-th backward difference over i! h^i.
 * The coefficient of every f_j comes from the recursive divided-difference
 * table run on the unit vector e_j.  Returns 0 or a negative code. */
int oracle_weights_row_taylor(const double *x, int n, double xstar, double *w) {
  int rc = oracle_check_nodes(x, n);
  if (rc) return rc;
  if (!isfinite(xstar)) return -2;
  if (n > ORACLE_MAX_NODES) return -1;
  const double d = xstar - x[n - 1];
  for (int j = 0; j < n; ++j) {
    /* table[k] holds the divided difference over nodes k-i .. k of e_j */
    double table[ORACLE_MAX_NODES];
    for (int k = 0; k < n; ++k) table[k] = (k == j) ? 1.0 : 0.0;
    double sum = table[n - 1];     /* i = 0: f[x_{n-1}] */
    double power = 1.0;
    for (int i = 1; i < n; ++i) {
      for (int k = n - 1; k >= i; --k) table[k] = (table[k] - table[k - 1]) / (x[k] - x[k - i]);
      power *= d;
      sum += table[n - 1] * power;
    }
    w[j] = sum;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* IEEE-754 binary16 storage (the same prediction for fp16-stored caches).    */
/* ------------------------------------------------------------------------ */

/* Exact value of a binary16 pattern: 1 sign bit, 5 exponent bits (bias 15),
 * 10 fraction bits; exponent 0 holds zero and the subnormals m * 2^-24,
 * exponent 31 holds the infinities and NaNs. */
double oracle_f16_to_f64(uint16_t h) {
  const int sign = (h >> 15) & 1;
  const int expo = (h >> 10) & 0x1F;
  const int frac = h & 0x3FF;
  double v;
  if (expo == 0) {
    v = ldexp((double)frac, -24);
  } else if (expo == 31) {
    v = frac ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + frac), expo - 25);
  }
  return sign ? -v : v;
}

/* Nearest binary16 value, ties to even; magnitudes that round to 2^16 or
 * more become infinity; NaN becomes the quiet NaN 0x7E00. */
uint16_t oracle_round_f16(double v) {
  if (isnan(v)) return (uint16_t)0x7E00;
  const uint16_t sign = signbit(v) ? 0x8000 : 0x0000;
  const double a = fabs(v);
  if (a == 0.0) return sign;
  if (isinf(a)) return (uint16_t)(sign | 0x7C00);
  int ex;
  (void)frexp(a, &ex);                     /* a in [2^(ex-1), 2^ex) */
  const int e = ex - 1;
  const int qexp = (e < -14) ? -24 : e - 10;   /* spacing of binary16 there */
  const double units = ldexp(a, -qexp);    /* exact */
  double r = floor(units);
  const double frac = units - r;           /* exact */
  if (frac > 0.5 || (frac == 0.5 && fmod(r, 2.0) != 0.0)) r += 1.0;
  const double rounded = ldexp(r, qexp);
  if (rounded >= 65536.0) return (uint16_t)(sign | 0x7C00);
  if (rounded < ldexp(1.0, -14)) return (uint16_t)(sign | (uint16_t)ldexp(rounded, 24));
  int ex2;
  (void)frexp(rounded, &ex2);
  const int e2 = ex2 - 1;
  const uint16_t mant = (uint16_t)((ldexp(rounded, -e2) - 1.0) * 1024.0);
  return (uint16_t)(sign | (uint16_t)((e2 + 15) << 10) | mant);
}

void oracle_decode_f16(const uint16_t *h, int64_t count, double *out) {
  for (int64_t i = 0; i < count; ++i) out[i] = oracle_f16_to_f64(h[i]);
}

void oracle_encode_f16(const double *v, int64_t count, uint16_t *out) {
  for (int64_t i = 0; i < count; ++i) out[i] = oracle_round_f16(v[i]);
}

/* Section 3.3 forward application over binary16 history entries, as
 * oracle_extrapolate_bf16. */
void oracle_extrapolate_f16(const uint16_t *const *F, int n, const double *w,
                            int64_t count, double *out, double *absmag) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    double s = 0.0, m = 0.0;
    for (int k = 0; k < n; ++k) {
      double f = oracle_f16_to_f64(F[k][i]);
      s += w[k] * f;
      m += fabs(w[k]) * fabs(f);
    }
    out[i] = s;
    if (absmag) absmag[i] = m;
  }
}

/* Residual application over binary16 history entries, as
 * oracle_residual_bf16. */
int oracle_residual_f16(const uint16_t *const *F, int n, const double *w,
                        const int64_t *slot_offset, const int64_t *seg_numel,
                        const int64_t *res_offset, int n_segs, const double *x_in,
                        int64_t res_numel, double *x_out, double *absmag) {
  for (int s = 0; s < n_segs; ++s)
    if (res_offset[s] >= 0 && res_offset[s] + seg_numel[s] > res_numel) return -1;
  for (int64_t j = 0; j < res_numel; ++j) {
    x_out[j] = x_in ? x_in[j] : 0.0;
    if (absmag) absmag[j] = x_in ? fabs(x_in[j]) : 0.0;
  }
  for (int s = 0; s < n_segs; ++s) {
    if (res_offset[s] < 0) continue;
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < seg_numel[s]; ++e) {
      double acc = 0.0, mag = 0.0;
      for (int k = 0; k < n; ++k) {
        double f = oracle_f16_to_f64(F[k][slot_offset[s] + e]);
        acc += w[k] * f;
        mag += fabs(w[k]) * fabs(f);
      }
      x_out[res_offset[s] + e] += acc;
      if (absmag) absmag[res_offset[s] + e] += mag;
    }
  }
  return 0;
}
