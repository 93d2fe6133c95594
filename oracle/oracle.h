/*
 * ChebBooster online stage: fp64 CPU oracle (TEST INFRASTRUCTURE ONLY).
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this.  It shares nothing with the HIP library.  Definitions and
 * paper citations are in oracle.c.
 */
#ifndef CHEB_ORACLE_H
#define CHEB_ORACLE_H

#include <stdint.h>

#define ORACLE_MAX_NODES 64

#ifdef __cplusplus
extern "C" {
#endif

int oracle_set_threads(int n);
int oracle_max_threads(void);

int oracle_check_nodes(const double *x, int n);
void oracle_normalise(const double *x, int n, double xstar, double *y,
                      double *ystar);
void oracle_barycentric_rho(const double *y, int n, double *rho);
int oracle_weights_row(const double *x, int n, double xstar, double *w);
int oracle_weights(const double *x, int n, const double *xstar, int m,
                   double *w);
int oracle_lagrange_row(const double *x, int n, double xstar, double *w);

double oracle_bf16_to_f64(uint16_t h);
uint16_t oracle_round_bf16(double v);
float oracle_round_f32(double v);
void oracle_decode_bf16(const uint16_t *h, int64_t count, double *out);
void oracle_encode_bf16(const double *v, int64_t count, uint16_t *out);

void oracle_extrapolate_bf16(const uint16_t *const *F, int n, const double *w,
                             int64_t count, double *out, double *absmag);
void oracle_extrapolate_f32(const float *const *F, int n, const double *w,
                            int64_t count, double *out, double *absmag);
void oracle_extrapolate_f64(const double *const *F, int n, const double *w,
                            int64_t count, double *out);

int oracle_full_schedule(int T, int s0, int s1, int r, uint8_t *is_full);
int oracle_table_row_mask(int T, const uint8_t *full, int n, const double *abscissa,
                          int policy, int step, int *kind, int *n_used, int *nodes,
                          double *w);
int oracle_table_row(int T, int s0, int s1, int r, int n, const double *abscissa,
                     int policy, int step, int *kind, int *n_used, int *nodes,
                     double *w);

int oracle_chebyshev_nodes(int n, int kind, double a, double b, double *x);
int oracle_weights_row_alternating(const double *x, int n, double xstar, double *w);
int oracle_weights_row_taylor(const double *x, int n, double xstar, double *w);
int oracle_residual_bf16(const uint16_t *const *F, int n, const double *w,
                         const int64_t *slot_offset, const int64_t *seg_numel,
                         const int64_t *res_offset, int n_segs, const double *x_in,
                         int64_t res_numel, double *x_out, double *absmag);
double oracle_f16_to_f64(uint16_t h);
uint16_t oracle_round_f16(double v);
void oracle_decode_f16(const uint16_t *h, int64_t count, double *out);
void oracle_encode_f16(const double *v, int64_t count, uint16_t *out);
void oracle_extrapolate_f16(const uint16_t *const *F, int n, const double *w,
                            int64_t count, double *out, double *absmag);
int oracle_residual_f16(const uint16_t *const *F, int n, const double *w,
                        const int64_t *slot_offset, const int64_t *seg_numel,
                        const int64_t *res_offset, int n_segs, const double *x_in,
                        int64_t res_numel, double *x_out, double *absmag);
int oracle_residual_f32(const float *const *F, int n, const double *w,
                        const int64_t *slot_offset, const int64_t *seg_numel,
                        const int64_t *res_offset, int n_segs, const double *x_in,
                        int64_t res_numel, double *x_out, double *absmag);

#ifdef __cplusplus
}
#endif

#endif
