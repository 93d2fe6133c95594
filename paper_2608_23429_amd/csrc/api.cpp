// Host side of libcheb: error reporting, launch shape, weight
// precomputation and the stateless combination entry point.
#include <float.h>
#include <limits.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "internal.h"

namespace cheb {

namespace {
thread_local char g_error[512] = "";

std::mutex g_shape_mutex;
cheb_launch_config g_shape = {64, 1, 1, 0, 0};

constexpr int kMaxDevices = 64;
int g_cus[kMaxDevices] = {0};
int g_lds[kMaxDevices] = {0};
std::mutex g_cus_mutex;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
}  // namespace

int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_error, sizeof g_error, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_error[0] = '\0';
  return CHEB_OK;
}

cheb_launch_config launch_shape() {
  std::lock_guard<std::mutex> lock(g_shape_mutex);
  return g_shape;
}

int device_info(int *cus, int *lds_per_cu) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CHEB_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev >= 0 && dev < kMaxDevices) {
    std::lock_guard<std::mutex> lock(g_cus_mutex);
    if (g_cus[dev] > 0) {
      *cus = g_cus[dev];
      *lds_per_cu = g_lds[dev];
      return CHEB_OK;
    }
  }
  int n = 0, lds = 0;
  e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess || n <= 0)
    return fail(CHEB_E_HIP, "compute unit count: %s", hipGetErrorString(e));
  e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev);
  if (e != hipSuccess || lds < 0)
    return fail(CHEB_E_HIP, "LDS per compute unit: %s", hipGetErrorString(e));
  if (dev >= 0 && dev < kMaxDevices) {
    std::lock_guard<std::mutex> lock(g_cus_mutex);
    g_cus[dev] = n;
    g_lds[dev] = lds;
  }
  *cus = n;
  *lds_per_cu = lds;
  return CHEB_OK;
}

// A computed row is refused when a weight is not finite, or when the
// rounding error of the second form, bounded by about n 2^-53 sum_j |w_j|
// relative to each weight, could exceed the fp32 resolution (2^-24) at which
// the bf16 kernel consumes the row: past that point fp64 no longer delivers
// the coefficients to the precision they are used at.
static int check_row(const double *w, int n, double target) {
  double mass = 0.0;
  for (int j = 0; j < n; ++j) {
    if (!isfinite(w[j]))
      return fail(CHEB_E_NONFINITE, "weight %d is not finite (target %.17g)", j, target);
    mass += fabs(w[j]);
  }
  if (double(n) * mass * 0x1p-53 > 0x1p-24)
    return fail(CHEB_E_NONFINITE,
                "weights too ill-conditioned for fp64 (sum |w| = %.3g, target %.17g)", mass,
                target);
  return CHEB_OK;
}

// Barycentric coefficients of one target (Section 3.2, coefficient
// equation; Appendix A, rho_j = 1 / omega'(x_j) and the second form).
// The abscissae are first mapped affinely so their span becomes [-1, 1]
// (Section 3.3); Lagrange coefficients are unchanged by any affine map, and
// the map keeps the products in omega' near unit scale.
int weights_row(const double *x, int n, double target, double *w) {
  if (n < 1 || n > CHEB_MAX_NODES)
    return fail(CHEB_E_INVAL, "history size %d outside 1..%d", n, CHEB_MAX_NODES);
  if (!isfinite(target)) return fail(CHEB_E_NONFINITE, "target abscissa is not finite");
  double lo = x[0], hi = x[0];
  for (int j = 0; j < n; ++j) {
    if (!isfinite(x[j])) return fail(CHEB_E_NONFINITE, "history abscissa %d is not finite", j);
    lo = fmin(lo, x[j]);
    hi = fmax(hi, x[j]);
  }
  for (int j = 0; j < n; ++j)
    for (int k = 0; k < j; ++k)
      if (x[j] == x[k])
        return fail(CHEB_E_DUPNODE, "history abscissae %d and %d are equal (%.17g)", k, j, x[j]);
  // Target on a node: the interpolant takes the node's value.
  for (int j = 0; j < n; ++j) {
    if (target == x[j]) {
      for (int k = 0; k < n; ++k) w[k] = (k == j) ? 1.0 : 0.0;
      return CHEB_OK;
    }
  }
  if (n == 1) {
    w[0] = 1.0;
    return CHEB_OK;
  }
  const double mid = 0.5 * (lo + hi);
  const double inv_half = 2.0 / (hi - lo);
  double y[CHEB_MAX_NODES];
  for (int j = 0; j < n; ++j) y[j] = (x[j] - mid) * inv_half;
  const double yt = (target - mid) * inv_half;
  // term_j = 1 / (omega'(y_j) (yt - y_j)).  The product is carried as a
  // mantissa in [0.5, 1) and a power of two, so nodes clustered closely
  // enough for omega' to leave the double range still give their weights:
  // the second form is unchanged by a common factor, and every term is
  // scaled by the same power of two before the sum.  Where nothing leaves
  // the range the result is bit for bit that of the plain product.
  double inv[CHEB_MAX_NODES];
  long expo[CHEB_MAX_NODES];
  long top = LONG_MIN;
  for (int j = 0; j < n; ++j) {
    const double gap = yt - y[j];
    if (gap == 0.0) {  // distinct abscissae that the map rounded together
      for (int k = 0; k < n; ++k) w[k] = (k == j) ? 1.0 : 0.0;
      return CHEB_OK;
    }
    double m = 1.0;
    long e = 0;
    for (int k = 0; k < n; ++k) {
      if (k == j) continue;
      const double d = y[j] - y[k];
      if (d == 0.0)
        return fail(CHEB_E_DUPNODE,
                    "history abscissae %d and %d coincide once mapped onto [-1, 1]", k, j);
      int ex = 0;
      m = frexp(m * d, &ex);
      e += ex;
    }
    int ex = 0;
    m = frexp(m * gap, &ex);
    e += ex;
    inv[j] = 1.0 / m;  // magnitude in (1, 2]
    expo[j] = -e;
    top = expo[j] > top ? expo[j] : top;
  }
  double terms[CHEB_MAX_NODES];
  double total = 0.0;
  for (int j = 0; j < n; ++j) {
    const long shift = expo[j] - top;  // <= 0
    terms[j] = ldexp(inv[j], shift < -2000 ? -2000 : int(shift));
    total += terms[j];
  }
  for (int j = 0; j < n; ++j) w[j] = terms[j] / total;
  return check_row(w, n, target);
}

// Coefficients from the alternating weights printed in Section 3.2,
// rho_j = (-1)^j (1/2 at the first and last node, 1 otherwise), in the
// coefficient equation.  They are the barycentric weights of Chebyshev
// extrema; at other nodes they give a rational interpolant.
int weights_row_alternating(const double *x, int n, double target, double *w) {
  if (n < 1 || n > CHEB_MAX_NODES)
    return fail(CHEB_E_INVAL, "history size %d outside 1..%d", n, CHEB_MAX_NODES);
  if (!isfinite(target)) return fail(CHEB_E_NONFINITE, "target abscissa is not finite");
  for (int j = 0; j < n; ++j) {
    if (!isfinite(x[j])) return fail(CHEB_E_NONFINITE, "history abscissa %d is not finite", j);
    for (int k = 0; k < j; ++k)
      if (x[j] == x[k])
        return fail(CHEB_E_DUPNODE, "history abscissae %d and %d are equal (%.17g)", k, j, x[j]);
  }
  for (int j = 0; j < n; ++j) {
    if (target == x[j]) {
      for (int k = 0; k < n; ++k) w[k] = (k == j) ? 1.0 : 0.0;
      return CHEB_OK;
    }
  }
  double total = 0.0;
  for (int j = 0; j < n; ++j) {
    const double sign = (j & 1) ? -1.0 : 1.0;
    const double end = (n > 1 && (j == 0 || j == n - 1)) ? 0.5 : 1.0;
    w[j] = sign * end / (target - x[j]);
    total += w[j];
  }
  for (int j = 0; j < n; ++j) w[j] /= total;
  return check_row(w, n, target);
}

// Taylor expansion about the newest abscissa x_{n-1} (the comparison in
// Section 3.2's Runge-function study; the text gives no formula): the i-th
// derivative over i! is estimated by the divided difference over the newest
// i + 1 abscissae,
//     P(t) = sum_{i<n} f[x_{n-1-i}, ..., x_{n-1}] (t - x_{n-1})^i,
// and the divided difference over the set S is sum_{j in S} f_j / prod_{m in
// S, m != j} (x_j - x_m).  On equispaced abscissae it is the i-th backward
// difference over i! h^i.
int weights_row_taylor(const double *x, int n, double target, double *w) {
  if (n < 1 || n > CHEB_MAX_NODES)
    return fail(CHEB_E_INVAL, "history size %d outside 1..%d", n, CHEB_MAX_NODES);
  if (!isfinite(target)) return fail(CHEB_E_NONFINITE, "target abscissa is not finite");
  for (int j = 0; j < n; ++j) {
    if (!isfinite(x[j])) return fail(CHEB_E_NONFINITE, "history abscissa %d is not finite", j);
    for (int k = 0; k < j; ++k)
      if (x[j] == x[k])
        return fail(CHEB_E_DUPNODE, "history abscissae %d and %d are equal (%.17g)", k, j, x[j]);
  }
  for (int j = 0; j < n; ++j) w[j] = 0.0;
  const double d = target - x[n - 1];
  double power = 1.0;  // d^i
  for (int i = 0; i < n; ++i) {
    const int first = n - 1 - i;
    for (int j = first; j < n; ++j) {
      double den = 1.0;
      for (int m = first; m < n; ++m)
        if (m != j) den *= x[j] - x[m];
      w[j] += power / den;
    }
    power *= d;
  }
  return check_row(w, n, target);
}

}  // namespace cheb

using namespace cheb;

extern "C" {

const char *cheb_last_error(void) { return g_error; }

int cheb_version(void) { return CHEB_VERSION; }

int cheb_get_launch_config(cheb_launch_config *cfg) {
  if (!cfg) return fail(CHEB_E_INVAL, "cfg is NULL");
  *cfg = launch_shape();
  return ok();
}

int cheb_set_launch_config(const cheb_launch_config *cfg) {
  if (!cfg) return fail(CHEB_E_INVAL, "cfg is NULL");
  if (cfg->block != 64 && cfg->block != 256 && cfg->block != 512 && cfg->block != 1024)
    return fail(CHEB_E_INVAL, "block must be 64, 256, 512 or 1024 (got %d)", cfg->block);
  if (cfg->unroll != 1 && cfg->unroll != 2 && cfg->unroll != 4)
    return fail(CHEB_E_INVAL, "unroll must be 1, 2 or 4 (got %d)", cfg->unroll);
  if (cfg->block == 64 && cfg->unroll != 1)
    return fail(CHEB_E_INVAL, "block 64 takes unroll 1 (got %d)", cfg->unroll);
  if (cfg->block * cfg->unroll > 1024)
    return fail(CHEB_E_INVAL, "block x unroll must not exceed 1024 (got %d x %d)", cfg->block,
                cfg->unroll);
  if (cfg->nontemporal != 0 && cfg->nontemporal != 1)
    return fail(CHEB_E_INVAL, "nontemporal must be 0 or 1 (got %d)", cfg->nontemporal);
  if (cfg->blocks_per_cu < 0 || cfg->blocks_per_cu > 64)
    return fail(CHEB_E_INVAL, "blocks_per_cu must be 0..64 (got %d)", cfg->blocks_per_cu);
  if (cfg->waves_per_cu < -1 || cfg->waves_per_cu > 32)
    return fail(CHEB_E_INVAL, "waves_per_cu must be -1..32 (got %d)", cfg->waves_per_cu);
  std::lock_guard<std::mutex> lock(g_shape_mutex);
  g_shape = *cfg;
  return ok();
}

int cheb_precompute_weights(const double *hist_t, int32_t n_hist, const double *target_t,
                            int32_t n_target, double *w_out) {
  if (!hist_t) return fail(CHEB_E_INVAL, "hist_t is NULL");
  if (n_target < 0) return fail(CHEB_E_INVAL, "n_target is negative");
  if (n_target > 0 && (!target_t || !w_out)) return fail(CHEB_E_INVAL, "target_t or w_out is NULL");
  if (n_hist < 1 || n_hist > CHEB_MAX_NODES)
    return fail(CHEB_E_INVAL, "n_hist %d outside 1..%d", n_hist, CHEB_MAX_NODES);
  // Validate every row before writing any, so w_out is untouched on error.
  double row[CHEB_MAX_NODES];
  for (int32_t m = 0; m < n_target; ++m) {
    int rc = weights_row(hist_t, n_hist, target_t[m], row);
    if (rc != CHEB_OK) return rc;
  }
  if (n_target == 0) {
    int rc = weights_row(hist_t, n_hist, hist_t[0], row);  // node checks only
    if (rc != CHEB_OK) return rc;
  }
  for (int32_t m = 0; m < n_target; ++m) {
    weights_row(hist_t, n_hist, target_t[m], row);
    memcpy(w_out + size_t(m) * n_hist, row, sizeof(double) * n_hist);
  }
  return ok();
}

int cheb_precompute_weights_variant(const double *hist_t, int32_t n_hist,
                                    const double *target_t, int32_t n_target, int32_t variant,
                                    double *w_out) {
  if (variant == CHEB_RHO_GENERAL)
    return cheb_precompute_weights(hist_t, n_hist, target_t, n_target, w_out);
  if (variant != CHEB_RHO_ALTERNATING && variant != CHEB_TAYLOR)
    return fail(CHEB_E_INVAL, "unknown weight variant %d", variant);
  auto row_of = variant == CHEB_TAYLOR ? weights_row_taylor : weights_row_alternating;
  if (!hist_t) return fail(CHEB_E_INVAL, "hist_t is NULL");
  if (n_target < 0) return fail(CHEB_E_INVAL, "n_target is negative");
  if (n_target > 0 && (!target_t || !w_out)) return fail(CHEB_E_INVAL, "target_t or w_out is NULL");
  double row[CHEB_MAX_NODES];
  for (int32_t m = 0; m < n_target; ++m) {
    int rc = row_of(hist_t, n_hist, target_t[m], row);
    if (rc != CHEB_OK) return rc;
  }
  if (n_target == 0) {
    int rc = row_of(hist_t, n_hist, hist_t[0], row);
    if (rc != CHEB_OK) return rc;
  }
  for (int32_t m = 0; m < n_target; ++m) {
    row_of(hist_t, n_hist, target_t[m], row);
    memcpy(w_out + size_t(m) * n_hist, row, sizeof(double) * n_hist);
  }
  return ok();
}

int cheb_chebyshev_nodes(int32_t n, int32_t kind, double a, double b, double *x_out) {
  if (!x_out) return fail(CHEB_E_INVAL, "x_out is NULL");
  if (n < 1 || n > CHEB_MAX_NODES) return fail(CHEB_E_INVAL, "n %d outside 1..%d", n, CHEB_MAX_NODES);
  if (kind != 1 && kind != 2) return fail(CHEB_E_INVAL, "kind must be 1 or 2");
  if (kind == 2 && n < 2) return fail(CHEB_E_INVAL, "Chebyshev extrema need n >= 2");
  if (!isfinite(a) || !isfinite(b)) return fail(CHEB_E_NONFINITE, "interval is not finite");
  const double mid = 0.5 * (a + b), half = 0.5 * (b - a);
  for (int32_t j = 0; j < n; ++j) {
    const double angle = kind == 1 ? M_PI * (2.0 * j + 1.0) / (2.0 * n) : M_PI * j / (n - 1.0);
    x_out[j] = mid + half * cos(angle);
  }
  return ok();
}

int cheb_combine_multi(const void *const *src, int32_t n_src, const double *w, int32_t n_out,
                       void *const *out, int64_t numel, int32_t dtype, void *stream) {
  return combine_checked(src, n_src, w, n_out, out, numel, dtype, kChunkVecs, stream);
}

int cheb_combine(const void *const *src, int32_t n_src, const double *w, void *out,
                 int64_t numel, int32_t dtype, void *stream) {
  void *outs[1] = {out};
  if (numel > 0 && !out) return fail(CHEB_E_INVAL, "out is NULL");
  return cheb_combine_multi(src, n_src, w, 1, outs, numel, dtype, stream);
}

}  // extern "C"

namespace cheb {

int combine_checked(const void *const *src, int32_t n_src, const double *w, int32_t n_out,
                    void *const *out, int64_t numel, int32_t dtype, int64_t super_vecs,
                    void *stream) {
  const bool contiguous = super_vecs == kChunkVecs;
  if (!valid_dtype(dtype)) return fail(CHEB_E_DTYPE, "unknown dtype %d", dtype);
  if (n_src < 1 || n_src > CHEB_MAX_SLOTS)
    return fail(CHEB_E_INVAL, "n_src %d outside 1..%d", n_src, CHEB_MAX_SLOTS);
  if (n_out < 1 || n_out > CHEB_MAX_OUTPUTS)
    return fail(CHEB_E_INVAL, "n_out %d outside 1..%d", n_out, CHEB_MAX_OUTPUTS);
  if (!src || !w || !out) return fail(CHEB_E_INVAL, "src, w or out is NULL");
  if (numel < 0) return fail(CHEB_E_INVAL, "numel is negative");
  if (numel / elems_per_vec(dtype) >= kMaxVecs)
    return fail(CHEB_E_INVAL, "numel %lld too large for one launch", (long long)numel);
  for (int m = 0; m < n_out * n_src; ++m) {
    if (!isfinite(w[m])) return fail(CHEB_E_NONFINITE, "weight %d is not finite", m);
    // The bf16 and fp16 kernels take their weights as fp32.
    if (dtype != CHEB_F32 && fabs(w[m]) > double(FLT_MAX))
      return fail(CHEB_E_NONFINITE, "weight %d (%.17g) overflows fp32", m, w[m]);
  }
  if (!contiguous && numel % elems_per_vec(dtype) != 0)
    return fail(CHEB_E_INVAL, "interleaved sources need whole 16-byte vectors");
  if (numel == 0) return ok();
  const uintptr_t bytes = uintptr_t(numel) * elem_bytes(dtype);
  auto overlap = [bytes](const void *a, const void *b) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + bytes && y < x + bytes;
  };
  for (int k = 0; k < n_src; ++k) {
    if (!src[k]) return fail(CHEB_E_INVAL, "src[%d] is NULL", k);
    if (!aligned16(src[k])) return fail(CHEB_E_ALIGN, "src[%d] is not 16-byte aligned", k);
  }
  for (int m = 0; m < n_out; ++m) {
    if (!out[m]) return fail(CHEB_E_INVAL, "out[%d] is NULL", m);
    if (!aligned16(out[m])) return fail(CHEB_E_ALIGN, "out[%d] is not 16-byte aligned", m);
    // Interleaved sources spread over their arena; the cache checks the
    // outputs against the whole arena instead.
    if (contiguous)
      for (int k = 0; k < n_src; ++k)
        if (overlap(out[m], src[k])) return fail(CHEB_E_INVAL, "out[%d] overlaps src[%d]", m, k);
    for (int j = 0; j < m; ++j)
      if (overlap(out[m], out[j])) return fail(CHEB_E_INVAL, "out[%d] overlaps out[%d]", m, j);
  }
  return launch_combine(dtype, src, n_src, w, n_out, out, numel, super_vecs,
                        static_cast<hipStream_t>(stream));
}

}  // namespace cheb
