/*
 * attn_oracle.c -- plain, slow fp64 reference for scaled dot-product attention,
 * forward and backward, one head at a time.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The product path
 * (the HIP kernels behind libdash) never calls it, and the two share no code.
 *
 * What it computes (the paper's Background section and Algorithm 1, "Exact
 * Algorithm and Modifications" appendix), written out as definitions in fp64:
 *
 *   S_ij = scale * <q_i, k_j>                     scores (Alg. 1, S = Q K^T;
 *                                                  the softmax scale is implicit
 *                                                  in the paper, explicit here)
 *   key j is visible from query i  iff  !causal or j <= i
 *   L_i  = log sum_{visible j} exp(S_ij)           logsumexp vector L (Alg. 1 inputs)
 *   P_ij = exp(S_ij - L_i), 0 where not visible    (Alg. 1, P = exp(S - L))
 *   O_i  = sum_j P_ij v_j
 *   D_i  = <dO_i, O_i>                             (Alg. 1 preprocessing, rowsum(dO o O))
 *   dP_ij = <dO_i, v_j>                            (Alg. 1, dP = dO V^T)
 *   dS_ij = P_ij (dP_ij - D_i)                     (Alg. 1, dS = P o (dP - D))
 *   dV_j = sum_i P_ij dO_i                         (Alg. 1, dV += P^T dO)
 *   dK_j = scale * sum_i dS_ij q_i                 (Alg. 1, dK += dS^T Q, times scale)
 *   dQ_i = scale * sum_j dS_ij k_j                 (Alg. 1, dQ = dS K, times scale)
 *
 * Every array is one head, row-major [N][d] doubles.  Rows are independent in
 * the forward and in dQ; columns are independent in dK/dV, so each entry point
 * takes the set of rows (or columns) it should produce: this lets the tests
 * sample single outputs of very large problems without computing the rest.
 * OpenMP parallelises over those rows/columns only; every sum runs in index
 * order inside one thread, so results do not depend on the thread count.
 */
#include <math.h>
#include <stdlib.h>

static double dotd(const double *a, const double *b, int d) {
  double s = 0.0;
  for (int t = 0; t < d; t++) s += a[t] * b[t];
  return s;
}

/* number of keys visible from query row i */
static int n_visible(int i, int N, int causal) { return causal ? (i + 1 < N ? i + 1 : N) : N; }

/* Row i of the forward: fills lse_i and o_i (d doubles).  s_row has N slots. */
static void fwd_row(const double *q, const double *k, const double *v, int N, int d, int causal,
                    double scale, int i, double *s_row, double *o_i, double *lse_i) {
  int nv = n_visible(i, N, causal);
  double m = -INFINITY;
  for (int j = 0; j < nv; j++) {
    s_row[j] = scale * dotd(q + (size_t)i * d, k + (size_t)j * d, d);
    if (s_row[j] > m) m = s_row[j];
  }
  double z = 0.0;
  for (int j = 0; j < nv; j++) z += exp(s_row[j] - m);
  double L = m + log(z);
  for (int t = 0; t < d; t++) o_i[t] = 0.0;
  for (int j = 0; j < nv; j++) {
    double p = exp(s_row[j] - L);
    const double *vj = v + (size_t)j * d;
    for (int t = 0; t < d; t++) o_i[t] += p * vj[t];
  }
  *lse_i = L;
}

/*
 * Forward for the query rows listed in rows[0..nrows).  Writes o[r][:] and
 * lse[r] at the absolute row index r (o is [N][d], lse is [N]).
 */
void oracle_fwd_rows(const double *q, const double *k, const double *v, int N, int d, int causal,
                     double scale, const int *rows, int nrows, double *o, double *lse) {
#pragma omp parallel
  {
    double *s_row = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
#pragma omp for schedule(dynamic, 1)
    for (int r = 0; r < nrows; r++) {
      int i = rows[r];
      fwd_row(q, k, v, N, d, causal, scale, i, s_row, o + (size_t)i * d, lse + i);
    }
    free(s_row);
  }
}

/*
 * dQ for the query rows listed in rows[].  Row i needs only its own L_i and
 * D_i, which are recomputed here from the definitions (forward row, then
 * D_i = <dO_i, O_i>).  Also writes lse[i] and D[i] for those rows.
 */
void oracle_bwd_dq_rows(const double *q, const double *k, const double *v, const double *dO,
                        int N, int d, int causal, double scale, const int *rows, int nrows,
                        double *dq, double *lse, double *D) {
#pragma omp parallel
  {
    double *s_row = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
    double *o_i = (double *)malloc(sizeof(double) * (size_t)(d > 0 ? d : 1));
#pragma omp for schedule(dynamic, 1)
    for (int r = 0; r < nrows; r++) {
      int i = rows[r];
      double L;
      fwd_row(q, k, v, N, d, causal, scale, i, s_row, o_i, &L);
      const double *dOi = dO + (size_t)i * d;
      double Di = dotd(dOi, o_i, d);
      double *dqi = dq + (size_t)i * d;
      for (int t = 0; t < d; t++) dqi[t] = 0.0;
      int nv = n_visible(i, N, causal);
      for (int j = 0; j < nv; j++) {
        double p = exp(s_row[j] - L);
        double dp = dotd(dOi, v + (size_t)j * d, d);
        double ds = p * (dp - Di);
        const double *kj = k + (size_t)j * d;
        for (int t = 0; t < d; t++) dqi[t] += ds * kj[t];
      }
      for (int t = 0; t < d; t++) dqi[t] *= scale;
      lse[i] = L;
      D[i] = Di;
    }
    free(o_i);
    free(s_row);
  }
}

/*
 * dK and dV for the key rows listed in cols[].  Column j of P and dS needs
 * L_i and D_i of every query row that sees key j; the caller passes them
 * (lse[N], D[N]) -- normally produced by oracle_bwd_dq_rows over all rows.
 */
void oracle_bwd_dkdv_cols(const double *q, const double *k, const double *v, const double *dO,
                          int N, int d, int causal, double scale, const double *lse,
                          const double *D, const int *cols, int ncols, double *dk, double *dv) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int c = 0; c < ncols; c++) {
    int j = cols[c];
    double *dkj = dk + (size_t)j * d;
    double *dvj = dv + (size_t)j * d;
    for (int t = 0; t < d; t++) { dkj[t] = 0.0; dvj[t] = 0.0; }
    const double *kj = k + (size_t)j * d;
    const double *vj = v + (size_t)j * d;
    for (int i = causal ? j : 0; i < N; i++) {
      const double *qi = q + (size_t)i * d;
      const double *dOi = dO + (size_t)i * d;
      double p = exp(scale * dotd(qi, kj, d) - lse[i]);
      double dp = dotd(dOi, vj, d);
      double ds = p * (dp - D[i]);
      for (int t = 0; t < d; t++) {
        dvj[t] += p * dOi[t];
        dkj[t] += ds * qi[t];
      }
    }
    for (int t = 0; t < d; t++) dkj[t] *= scale;
  }
}

/*
 * The full probability matrix P (N x N, zeros where masked), for tiny
 * problems only: lets the tests check identities such as
 * rowsum(dO o O) == rowsum(P o dP) against an independently formed dP.
 */
void oracle_probs(const double *q, const double *k, int N, int d, int causal, double scale,
                  double *P) {
  for (int i = 0; i < N; i++) {
    int nv = n_visible(i, N, causal);
    double m = -INFINITY;
    for (int j = 0; j < nv; j++) {
      double s = scale * dotd(q + (size_t)i * d, k + (size_t)j * d, d);
      if (s > m) m = s;
    }
    double z = 0.0;
    for (int j = 0; j < nv; j++) z += exp(scale * dotd(q + (size_t)i * d, k + (size_t)j * d, d) - m);
    double L = m + log(z);
    for (int j = 0; j < N; j++)
      P[(size_t)i * N + j] = j < nv ? exp(scale * dotd(q + (size_t)i * d, k + (size_t)j * d, d) - L) : 0.0;
  }
}
