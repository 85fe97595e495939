/*
 * fp64 reference recurrences for the oracle (TEST INFRASTRUCTURE ONLY).
 *
 * Plain C twin of oracle.gated_delta_recurrence / oracle.decay_recurrence:
 * one value head, token by token, in the paper's orientation (S is d_v x d_k,
 * S_0 given).  Nothing here is shared with, or linked into, the HIP library;
 * the oracle's Python side calls it through ctypes and runs heads on several
 * host threads (each call is single-threaded and touches only its own S).
 *
 * Gated DeltaNet (Section 2.1, Eq. recurrence, decay combined with a rank-one
 * erase):
 *     S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 * evaluated as u = S_{t-1} k_t, then
 *     S_t[i][j] = alpha_t (S_{t-1}[i][j] - beta_t u[i] k_t[j]) + beta_t v_t[i] k_t[j].
 *
 * Per-head decay without the erase (the Mamba2 form Section 2.1 names), with
 * the same write:
 *     S_t = alpha_t S_{t-1} + beta_t v_t k_t^T.
 *
 * Arguments (all host memory, row-major):
 *   k      row t at k + t * k_stride, d_k values
 *   v      row t at v + t * v_stride, d_v values
 *   alpha, beta   element t at [t * ab_stride]
 *   S      [d_v][d_k], the initial state on entry and S_L on return
 *   work   d_v doubles of scratch (the gated recurrence only)
 */
#include <stdint.h>

void oracle_gdn_head(int64_t L, int32_t dk, int32_t dv, const double* k, int64_t k_stride, const double* v,
                     int64_t v_stride, const double* alpha, const double* beta, int64_t ab_stride, double* S,
                     double* work) {
  for (int64_t t = 0; t < L; ++t) {
    const double* kt = k + t * k_stride;
    const double* vt = v + t * v_stride;
    const double a = alpha[t * ab_stride];
    const double b = beta[t * ab_stride];
    for (int32_t i = 0; i < dv; ++i) {
      double u = 0.0;
      for (int32_t j = 0; j < dk; ++j) u += S[(int64_t)i * dk + j] * kt[j];
      work[i] = u;
    }
    for (int32_t i = 0; i < dv; ++i) {
      double* row = S + (int64_t)i * dk;
      const double bu = b * work[i];
      const double bv = b * vt[i];
      for (int32_t j = 0; j < dk; ++j) row[j] = a * (row[j] - bu * kt[j]) + bv * kt[j];
    }
  }
}

void oracle_decay_head(int64_t L, int32_t dk, int32_t dv, const double* k, int64_t k_stride, const double* v,
                       int64_t v_stride, const double* alpha, const double* beta, int64_t ab_stride, double* S) {
  for (int64_t t = 0; t < L; ++t) {
    const double* kt = k + t * k_stride;
    const double* vt = v + t * v_stride;
    const double a = alpha[t * ab_stride];
    const double b = beta[t * ab_stride];
    for (int32_t i = 0; i < dv; ++i) {
      double* row = S + (int64_t)i * dk;
      const double bv = b * vt[i];
      for (int32_t j = 0; j < dk; ++j) row[j] = a * row[j] + bv * kt[j];
    }
  }
}

/* Gated DeltaNet with the per-token read-out of the layer's output
 * (o_t = S_t q_t, the state after token t applied to that token's query):
 * as oracle_gdn_head, and row t of the output at o + t * o_stride (d_v
 * values), with q row t at q + t * q_stride (d_k values). */
void oracle_gdn_head_out(int64_t L, int32_t dk, int32_t dv, const double* k, int64_t k_stride, const double* v,
                         int64_t v_stride, const double* alpha, const double* beta, int64_t ab_stride, double* S,
                         double* work, const double* q, int64_t q_stride, double* o, int64_t o_stride) {
  for (int64_t t = 0; t < L; ++t) {
    oracle_gdn_head(1, dk, dv, k + t * k_stride, k_stride, v + t * v_stride, v_stride, alpha + t * ab_stride,
                    beta + t * ab_stride, ab_stride, S, work);
    const double* qt = q + t * q_stride;
    double* ot = o + t * o_stride;
    for (int32_t i = 0; i < dv; ++i) {
      double acc = 0.0;
      for (int32_t j = 0; j < dk; ++j) acc += S[(int64_t)i * dk + j] * qt[j];
      ot[i] = acc;
    }
  }
}
