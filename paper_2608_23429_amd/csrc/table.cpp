// Offline stage: the full-computation schedule and the table of weight rows
// for every step the schedule skips (paper, Section 3.3, weight
// precomputation; Algorithm 1, offline stage), its serialisation (the
// "prepackaged" tables of Section 3.3), and the row-checked prediction of
// the online stage.
#include <errno.h>
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "internal.h"

struct cheb_table {
  int32_t T = 0, s0 = 0, s1 = 0, r = 1, n_hist = 1, policy = 0;
  std::vector<double> abscissa;  // [T]
  std::vector<uint8_t> predicted;  // [T]: 1 when the step is predicted
  std::vector<int32_t> n_used;     // [T]
  std::vector<int32_t> nodes;      // [T][n_hist], oldest to newest
  std::vector<double> w;           // [T][n_hist]
};

using namespace cheb;

namespace {

constexpr int32_t kMaxSteps = 1 << 20;
constexpr const char *kMagic = "chebtable";
constexpr int kFormat = 1;

bool schedule_args_ok(int32_t T, int32_t s0, int32_t s1, int32_t r) {
  return T >= 1 && T <= kMaxSteps && s0 >= 0 && s1 >= 0 && r >= 1;
}

// Membership of step s in the schedule F: s outside [s0, T-1-s1], or r
// divides s - s0.
bool in_schedule(int32_t T, int32_t s0, int32_t s1, int32_t r, int32_t s) {
  if (s < s0 || s > T - 1 - s1) return true;
  return (s - s0) % r == 0;
}

// Rows of every step given which steps the schedule runs in full.
int fill_rows(cheb_table *t, const uint8_t *scheduled) {
  const int32_t T = t->T, n = t->n_hist;
  t->predicted.assign(size_t(T), 0);
  t->n_used.assign(size_t(T), 0);
  t->nodes.assign(size_t(T) * n, -1);
  t->w.assign(size_t(T) * n, 0.0);
  // Steps that run the network: the schedule's, plus (policy 0) any step
  // reached before n full steps exist, plus any step reached with none.
  std::vector<int32_t> full_steps;
  for (int32_t s = 0; s < T; ++s) {
    const int32_t have = int32_t(full_steps.size());
    const bool runs = scheduled[s] || have == 0 || (t->policy == 0 && have < n);
    if (runs) full_steps.push_back(s);
  }
  double x[CHEB_MAX_NODES];
  for (int32_t s = 0; s < T; ++s) {
    auto it = std::lower_bound(full_steps.begin(), full_steps.end(), s);
    if (it != full_steps.end() && *it == s) continue;  // full step
    const int32_t before = int32_t(it - full_steps.begin());
    const int32_t used = std::min(before, n);
    t->predicted[size_t(s)] = 1;
    t->n_used[size_t(s)] = used;
    for (int32_t j = 0; j < used; ++j) {
      const int32_t node = full_steps[size_t(before - used + j)];
      t->nodes[size_t(s) * n + j] = node;
      x[j] = t->abscissa[size_t(node)];
    }
    int rc = weights_row(x, used, t->abscissa[size_t(s)], &t->w[size_t(s) * n]);
    if (rc != CHEB_OK) return rc;
  }
  return CHEB_OK;
}

}  // namespace

extern "C" {

int cheb_schedule(int32_t T, int32_t s0, int32_t s1, int32_t r, uint8_t *is_full) {
  if (!schedule_args_ok(T, s0, s1, r))
    return fail(CHEB_E_INVAL, "schedule needs 1 <= T <= %d, s0 >= 0, s1 >= 0, r >= 1", kMaxSteps);
  if (!is_full) return fail(CHEB_E_INVAL, "is_full is NULL");
  for (int32_t s = 0; s < T; ++s) is_full[s] = in_schedule(T, s0, s1, r, s) ? 1 : 0;
  return ok();
}

int cheb_table_build(cheb_table **out, int32_t T, int32_t s0, int32_t s1, int32_t r,
                     int32_t n_hist, const double *abscissa, int32_t policy) {
  if (!out) return fail(CHEB_E_INVAL, "out is NULL");
  *out = nullptr;
  if (!schedule_args_ok(T, s0, s1, r))
    return fail(CHEB_E_INVAL, "schedule needs 1 <= T <= %d, s0 >= 0, s1 >= 0, r >= 1", kMaxSteps);
  if (n_hist < 1 || n_hist > CHEB_MAX_SLOTS)
    return fail(CHEB_E_INVAL, "n_hist %d outside 1..%d", n_hist, CHEB_MAX_SLOTS);
  if (policy != CHEB_SHORT_FULL && policy != CHEB_SHORT_LOWER)
    return fail(CHEB_E_INVAL, "unknown short-history policy %d", policy);
  if (!abscissa) return fail(CHEB_E_INVAL, "abscissa is NULL");
  for (int32_t s = 0; s < T; ++s)
    if (!isfinite(abscissa[s])) return fail(CHEB_E_NONFINITE, "abscissa of step %d", s);
  cheb_table *t = new (std::nothrow) cheb_table();
  if (!t) return fail(CHEB_E_INVAL, "out of host memory");
  t->T = T;
  t->s0 = s0;
  t->s1 = s1;
  t->r = r;
  t->n_hist = n_hist;
  t->policy = policy;
  t->abscissa.assign(abscissa, abscissa + T);
  std::vector<uint8_t> scheduled(static_cast<size_t>(T), 0);
  for (int32_t s = 0; s < T; ++s) scheduled[size_t(s)] = in_schedule(T, s0, s1, r, s) ? 1 : 0;
  int rc = fill_rows(t, scheduled.data());
  if (rc != CHEB_OK) {
    delete t;
    return rc;
  }
  *out = t;
  return ok();
}

int cheb_table_build_mask(cheb_table **out, int32_t T, const uint8_t *is_full, int32_t n_hist,
                          const double *abscissa, int32_t policy) {
  if (!out) return fail(CHEB_E_INVAL, "out is NULL");
  *out = nullptr;
  if (T < 1 || T > kMaxSteps) return fail(CHEB_E_INVAL, "T %d outside 1..%d", T, kMaxSteps);
  if (!is_full || !abscissa) return fail(CHEB_E_INVAL, "is_full or abscissa is NULL");
  if (n_hist < 1 || n_hist > CHEB_MAX_SLOTS)
    return fail(CHEB_E_INVAL, "n_hist %d outside 1..%d", n_hist, CHEB_MAX_SLOTS);
  if (policy != CHEB_SHORT_FULL && policy != CHEB_SHORT_LOWER)
    return fail(CHEB_E_INVAL, "unknown short-history policy %d", policy);
  for (int32_t s = 0; s < T; ++s)
    if (!isfinite(abscissa[s])) return fail(CHEB_E_NONFINITE, "abscissa of step %d", s);
  cheb_table *t = new (std::nothrow) cheb_table();
  if (!t) return fail(CHEB_E_INVAL, "out of host memory");
  // A mask table records no (s0, s1, r); saved tables carry r = 0 to say so.
  t->T = T;
  t->s0 = 0;
  t->s1 = 0;
  t->r = 0;
  t->n_hist = n_hist;
  t->policy = policy;
  t->abscissa.assign(abscissa, abscissa + T);
  std::vector<uint8_t> scheduled(is_full, is_full + T);
  for (uint8_t &v : scheduled) v = v ? 1 : 0;
  int rc = fill_rows(t, scheduled.data());
  if (rc != CHEB_OK) {
    delete t;
    return rc;
  }
  *out = t;
  return ok();
}

int cheb_table_destroy(cheb_table *t) {
  delete t;
  return ok();
}

int cheb_table_info(const cheb_table *t, int32_t *T, int32_t *n_hist, int32_t *policy,
                    int32_t *n_full) {
  if (!t) return fail(CHEB_E_INVAL, "table is NULL");
  if (T) *T = t->T;
  if (n_hist) *n_hist = t->n_hist;
  if (policy) *policy = t->policy;
  if (n_full) {
    int32_t c = 0;
    for (uint8_t p : t->predicted) c += p ? 0 : 1;
    *n_full = c;
  }
  return ok();
}

int cheb_table_step(const cheb_table *t, int32_t step, int32_t *predicted, int32_t *n_used,
                    int32_t *node_steps, double *w) {
  if (!t || !predicted || !n_used) return fail(CHEB_E_INVAL, "table or outputs NULL");
  if (step < 0 || step >= t->T) return fail(CHEB_E_INVAL, "step %d outside 0..%d", step, t->T - 1);
  *predicted = t->predicted[size_t(step)];
  *n_used = t->n_used[size_t(step)];
  const size_t base = size_t(step) * t->n_hist;
  for (int32_t j = 0; j < *n_used; ++j) {
    if (node_steps) node_steps[j] = t->nodes[base + j];
    if (w) w[j] = t->w[base + j];
  }
  return ok();
}

int cheb_table_save(const cheb_table *t, const char *path) {
  if (!t || !path) return fail(CHEB_E_INVAL, "table or path is NULL");
  FILE *f = fopen(path, "w");
  if (!f) return fail(CHEB_E_IO, "cannot open %s: %s", path, strerror(errno));
  // Hexadecimal floating point round-trips every double exactly.
  fprintf(f, "%s %d\n", kMagic, kFormat);
  fprintf(f, "T %d s0 %d s1 %d r %d n_hist %d policy %d\n", t->T, t->s0, t->s1, t->r,
          t->n_hist, t->policy);
  for (int32_t s = 0; s < t->T; ++s) {
    fprintf(f, "step %d %a", s, t->abscissa[size_t(s)]);
    if (!t->predicted[size_t(s)]) {
      fprintf(f, " full\n");
      continue;
    }
    const size_t base = size_t(s) * t->n_hist;
    fprintf(f, " predict %d", t->n_used[size_t(s)]);
    for (int32_t j = 0; j < t->n_used[size_t(s)]; ++j)
      fprintf(f, " %d %a", t->nodes[base + j], t->w[base + j]);
    fprintf(f, "\n");
  }
  const bool bad = ferror(f) != 0;
  if (fclose(f) != 0 || bad) return fail(CHEB_E_IO, "write to %s failed", path);
  return ok();
}

int cheb_table_load(cheb_table **out, const char *path) {
  if (!out || !path) return fail(CHEB_E_INVAL, "out or path is NULL");
  *out = nullptr;
  FILE *f = fopen(path, "r");
  if (!f) return fail(CHEB_E_IO, "cannot open %s: %s", path, strerror(errno));
  auto bad = [&](const char *what) {
    fclose(f);
    return fail(CHEB_E_IO, "%s: malformed table (%s)", path, what);
  };
  char magic[32] = {0};
  int format = 0;
  if (fscanf(f, "%31s %d", magic, &format) != 2 || strcmp(magic, kMagic) != 0 ||
      format != kFormat)
    return bad("header");
  cheb_table tmp;
  if (fscanf(f, " T %d s0 %d s1 %d r %d n_hist %d policy %d", &tmp.T, &tmp.s0, &tmp.s1,
             &tmp.r, &tmp.n_hist, &tmp.policy) != 6)
    return bad("parameters");
  const bool mask_table = tmp.r == 0 && tmp.s0 == 0 && tmp.s1 == 0;
  if ((!mask_table && !schedule_args_ok(tmp.T, tmp.s0, tmp.s1, tmp.r)) ||
      (mask_table && (tmp.T < 1 || tmp.T > kMaxSteps)) || tmp.n_hist < 1 ||
      tmp.n_hist > CHEB_MAX_SLOTS || (tmp.policy != 0 && tmp.policy != 1))
    return bad("parameters out of range");
  const int32_t T = tmp.T, n = tmp.n_hist;
  tmp.abscissa.assign(size_t(T), 0.0);
  tmp.predicted.assign(size_t(T), 0);
  tmp.n_used.assign(size_t(T), 0);
  tmp.nodes.assign(size_t(T) * n, -1);
  tmp.w.assign(size_t(T) * n, 0.0);
  char kind[16];
  for (int32_t s = 0; s < T; ++s) {
    int idx = -1;
    if (fscanf(f, " step %d %la %15s", &idx, &tmp.abscissa[size_t(s)], kind) != 3 || idx != s)
      return bad("step line");
    if (!isfinite(tmp.abscissa[size_t(s)])) return bad("abscissa");
    if (strcmp(kind, "full") == 0) continue;
    if (strcmp(kind, "predict") != 0) return bad("step kind");
    int used = 0;
    if (fscanf(f, "%d", &used) != 1 || used < 1 || used > n) return bad("entry count");
    tmp.predicted[size_t(s)] = 1;
    tmp.n_used[size_t(s)] = used;
    for (int32_t j = 0; j < used; ++j) {
      int node = -1;
      double wj = 0.0;
      if (fscanf(f, "%d %la", &node, &wj) != 2) return bad("entry");
      if (node < 0 || node >= s || !isfinite(wj)) return bad("entry value");
      if (j > 0 && node <= tmp.nodes[size_t(s) * n + j - 1]) return bad("entry order");
      tmp.nodes[size_t(s) * n + j] = node;
      tmp.w[size_t(s) * n + j] = wj;
    }
  }
  fclose(f);
  cheb_table *t = new (std::nothrow) cheb_table(std::move(tmp));
  if (!t) return fail(CHEB_E_INVAL, "out of host memory");
  *out = t;
  return ok();
}

int cheb_extrapolate_steps(cheb_cache *c, const cheb_table *t, int32_t first_step,
                           int32_t n_steps, void *const *out, void *stream) {
  if (!c || !t || !out) return fail(CHEB_E_INVAL, "cache, table or out is NULL");
  if (n_steps < 1 || n_steps > CHEB_MAX_OUTPUTS)
    return fail(CHEB_E_INVAL, "n_steps %d outside 1..%d", n_steps, CHEB_MAX_OUTPUTS);
  if (first_step < 0 || first_step + n_steps > t->T)
    return fail(CHEB_E_INVAL, "steps %d..%d outside the table", first_step,
                first_step + n_steps - 1);
  const int32_t n = t->n_hist;
  const size_t b0 = size_t(first_step) * n;
  const int32_t used = t->n_used[size_t(first_step)];
  for (int32_t m = 0; m < n_steps; ++m) {
    const int32_t s = first_step + m;
    if (!t->predicted[size_t(s)]) return fail(CHEB_E_INVAL, "step %d is a full step", s);
    if (t->n_used[size_t(s)] != used ||
        memcmp(&t->nodes[size_t(s) * n], &t->nodes[b0], sizeof(int32_t) * size_t(used)) != 0)
      return fail(CHEB_E_MISMATCH, "steps %d and %d use different histories", first_step, s);
  }
  // The newest `used` entries of the ring must be the row's nodes.
  double held[CHEB_MAX_SLOTS];
  int32_t count = 0;
  int rc = cheb_cache_history(c, held, &count);
  if (rc != CHEB_OK) return rc;
  if (count < used)
    return fail(CHEB_E_NOTREADY, "history holds %d entries, step %d needs %d", count,
                first_step, used);
  for (int32_t j = 0; j < used; ++j) {
    const double want = t->abscissa[size_t(t->nodes[b0 + j])];
    if (held[count - used + j] != want)
      return fail(CHEB_E_MISMATCH, "history entry %d holds abscissa %.17g, step %d needs %.17g",
                  count - used + j, held[count - used + j], first_step, want);
  }
  double w[CHEB_MAX_OUTPUTS * CHEB_MAX_SLOTS];
  for (int32_t m = 0; m < n_steps; ++m)
    memcpy(w + size_t(m) * used, &t->w[size_t(first_step + m) * n], sizeof(double) * size_t(used));
  return extrapolate_newest(c, used, w, n_steps, out, stream);
}

}  // extern "C"
