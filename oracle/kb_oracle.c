/*
 * kb_oracle.c -- plain CPU oracle for relation-set following on a reified KB.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header, table or helper with the HIP path.
 *
 * What it computes (Sec. 2.3, Eq. 4 and its minibatch form in App. C):
 *
 *   follow(X, R) = (X M_subj^T  (.)  R M_rel^T) M_obj
 *
 * with M_subj[l, m] = 1 iff m is the subject of triple l, M_obj[l, m] = 1 iff
 * m is its object, and M_rel[l, m] = w_l iff m is its relation (w_l = 1 for a
 * hard KB; the soft-KB extension of App. A stores the triple's confidence in
 * M_rel).  Unrolling the three products, example beta of the output is
 *
 *   Y[beta][j] = sum over triples l with obj_l == j of
 *                w_l * X[beta][subj_l] * R[beta][rel_l].
 *
 * The gradients follow from the chain rule on this bilinear map (the paper
 * states the operation is differentiable but prints no formulas):
 *
 *   dX[beta][i] = sum over l with subj_l == i of w_l * dY[beta][obj_l] * R[beta][rel_l]
 *   dR[beta][k] = sum over l with rel_l  == k of w_l * X[beta][subj_l] * dY[beta][obj_l]
 *
 * Conventions: the paper's batch-major orientation, X, Y, dY, dX as [b][N_E]
 * and R, dR as [b][N_R], row-major.  Ids are 0-based (the paper's are 1-based).
 * The triple list is walked in the caller's order; duplicate triples each
 * count.  Products and running sums are taken in double precision and every
 * output is rounded to float once.  Examples (beta) are independent and are
 * shared out across OpenMP threads; each example's sum order is fixed, so the
 * result does not depend on the thread count.
 *
 * Parity is pinned by the tests against dense evaluations of Eq. 1-4, the
 * brute-force neighbour sets of Claim 1, linearity, the adjoint identity,
 * exact finite differences, the triple-shard identity of App. D and the grid
 * KB's closed form.
 *
 * Return value of every entry point: 0 on success, -1 on bad arguments,
 * -2 on allocation failure.
 */
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORA_OK 0
#define ORA_EINVAL (-1)
#define ORA_ENOMEM (-2)

static int check_ids(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
                     const int32_t *rel, const int32_t *obj) {
  if (n_e < 0 || n_r < 0 || n_t < 0) return ORA_EINVAL;
  if (n_t > 0 && (!subj || !rel || !obj)) return ORA_EINVAL;
  for (int64_t l = 0; l < n_t; ++l) {
    if (subj[l] < 0 || subj[l] >= n_e) return ORA_EINVAL;
    if (obj[l] < 0 || obj[l] >= n_e) return ORA_EINVAL;
    if (rel[l] < 0 || rel[l] >= n_r) return ORA_EINVAL;
  }
  return ORA_OK;
}

static int pick_threads(int nthreads, int b) {
  int t = nthreads > 0 ? nthreads : omp_get_max_threads();
  if (t > b) t = b;
  return t < 1 ? 1 : t;
}

static double weight_of(const float *w, int64_t l) { return w ? (double)w[l] : 1.0; }

/* Forward, Eq. 4: Y[b][n_e]. */
int ora_follow(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
               const int32_t *rel, const int32_t *obj, const float *w, int32_t b,
               const float *X, const float *R, float *Y, int32_t nthreads) {
  if (b < 0 || (b > 0 && (!X || !R || !Y))) return ORA_EINVAL;
  int rc = check_ids(n_e, n_r, n_t, subj, rel, obj);
  if (rc) return rc;
  int err = 0;
#pragma omp parallel num_threads(pick_threads(nthreads, b))
  {
    double *acc = (double *)malloc(sizeof(double) * (size_t)(n_e > 0 ? n_e : 1));
    if (!acc) {
#pragma omp atomic write
      err = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int32_t beta = 0; beta < b; ++beta) {
      if (!acc) continue;
      const float *x = X + (size_t)beta * n_e;
      const float *r = R + (size_t)beta * n_r;
      for (int64_t j = 0; j < n_e; ++j) acc[j] = 0.0;
      for (int64_t l = 0; l < n_t; ++l)
        acc[obj[l]] += weight_of(w, l) * (double)x[subj[l]] * (double)r[rel[l]];
      float *y = Y + (size_t)beta * n_e;
      for (int64_t j = 0; j < n_e; ++j) y[j] = (float)acc[j];
    }
    free(acc);
  }
  return err ? ORA_ENOMEM : ORA_OK;
}

/* Backward: dX[b][n_e] and dR[b][n_r]; either output may be NULL to skip it. */
int ora_follow_backward(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
                        const int32_t *rel, const int32_t *obj, const float *w,
                        int32_t b, const float *X, const float *R, const float *dY,
                        float *dX, float *dR, int32_t nthreads) {
  if (b < 0 || (b > 0 && (!dY || (dX && !R) || (dR && !X)))) return ORA_EINVAL;
  int rc = check_ids(n_e, n_r, n_t, subj, rel, obj);
  if (rc) return rc;
  int err = 0;
#pragma omp parallel num_threads(pick_threads(nthreads, b))
  {
    double *ax = (double *)malloc(sizeof(double) * (size_t)(n_e > 0 ? n_e : 1));
    double *ar = (double *)malloc(sizeof(double) * (size_t)(n_r > 0 ? n_r : 1));
    if (!ax || !ar) {
#pragma omp atomic write
      err = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int32_t beta = 0; beta < b; ++beta) {
      if (!ax || !ar) continue;
      const float *dy = dY + (size_t)beta * n_e;
      if (dX) {
        const float *r = R + (size_t)beta * n_r;
        for (int64_t i = 0; i < n_e; ++i) ax[i] = 0.0;
        for (int64_t l = 0; l < n_t; ++l)
          ax[subj[l]] += weight_of(w, l) * (double)dy[obj[l]] * (double)r[rel[l]];
        float *dx = dX + (size_t)beta * n_e;
        for (int64_t i = 0; i < n_e; ++i) dx[i] = (float)ax[i];
      }
      if (dR) {
        const float *x = X + (size_t)beta * n_e;
        for (int64_t k = 0; k < n_r; ++k) ar[k] = 0.0;
        for (int64_t l = 0; l < n_t; ++l)
          ar[rel[l]] += weight_of(w, l) * (double)x[subj[l]] * (double)dy[obj[l]];
        float *dr = dR + (size_t)beta * n_r;
        for (int64_t k = 0; k < n_r; ++k) dr[k] = (float)ar[k];
      }
    }
    free(ax);
    free(ar);
  }
  return err ? ORA_ENOMEM : ORA_OK;
}

/*
 * Sampled outputs for KBs too large to evaluate whole.  `which` selects the
 * quantity and the index space of `ids`:
 *   0: Y  at objects   ids[q]  (forward)
 *   1: dX at subjects  ids[q]
 *   2: dR at relations ids[q]
 * out is [b][n_ids].  Each requested value is the same per-triple sum as above,
 * taken over the whole triple list in caller order (ids must be distinct).
 */
int ora_sampled(int32_t which, int64_t n_e, int64_t n_r, int64_t n_t,
                const int32_t *subj, const int32_t *rel, const int32_t *obj,
                const float *w, int32_t b, const float *X, const float *R,
                const float *dY, int32_t n_ids, const int32_t *ids, float *out,
                int32_t nthreads) {
  if (which < 0 || which > 2 || b < 0 || n_ids < 0 || (n_ids > 0 && (!ids || !out)))
    return ORA_EINVAL;
  if (b > 0 && ((which == 0 && (!X || !R)) || (which == 1 && (!dY || !R)) ||
                (which == 2 && (!X || !dY))))
    return ORA_EINVAL;
  int rc = check_ids(n_e, n_r, n_t, subj, rel, obj);
  if (rc) return rc;
  int64_t space = which == 2 ? n_r : n_e;
  int32_t *slot = (int32_t *)malloc(sizeof(int32_t) * (size_t)(space > 0 ? space : 1));
  if (!slot) return ORA_ENOMEM;
  for (int64_t e = 0; e < space; ++e) slot[e] = -1;
  for (int32_t q = 0; q < n_ids; ++q) {
    if (ids[q] < 0 || ids[q] >= space || slot[ids[q]] >= 0) {
      free(slot);
      return ORA_EINVAL;
    }
    slot[ids[q]] = q;
  }
  int err = 0;
#pragma omp parallel num_threads(pick_threads(nthreads, b))
  {
    double *acc = (double *)malloc(sizeof(double) * (size_t)(n_ids > 0 ? n_ids : 1));
    if (!acc) {
#pragma omp atomic write
      err = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int32_t beta = 0; beta < b; ++beta) {
      if (!acc) continue;
      for (int32_t q = 0; q < n_ids; ++q) acc[q] = 0.0;
      for (int64_t l = 0; l < n_t; ++l) {
        int32_t key = which == 0 ? obj[l] : (which == 1 ? subj[l] : rel[l]);
        int32_t q = slot[key];
        if (q < 0) continue;
        double a, c;
        if (which == 0) {
          a = (double)X[(size_t)beta * n_e + subj[l]];
          c = (double)R[(size_t)beta * n_r + rel[l]];
        } else if (which == 1) {
          a = (double)dY[(size_t)beta * n_e + obj[l]];
          c = (double)R[(size_t)beta * n_r + rel[l]];
        } else {
          a = (double)X[(size_t)beta * n_e + subj[l]];
          c = (double)dY[(size_t)beta * n_e + obj[l]];
        }
        acc[q] += weight_of(w, l) * a * c;
      }
      for (int32_t q = 0; q < n_ids; ++q) out[(size_t)beta * n_ids + q] = (float)acc[q];
    }
    free(acc);
  }
  free(slot);
  return err ? ORA_ENOMEM : ORA_OK;
}

/* Forward in double end to end (no rounding to float), for multi-hop chains. */
int ora_follow_f64(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
                   const int32_t *rel, const int32_t *obj, const double *w, int32_t b,
                   const double *X, const double *R, double *Y) {
  if (b < 0 || (b > 0 && (!X || !R || !Y))) return ORA_EINVAL;
  int rc = check_ids(n_e, n_r, n_t, subj, rel, obj);
  if (rc) return rc;
  for (int32_t beta = 0; beta < b; ++beta) {
    const double *x = X + (size_t)beta * n_e;
    const double *r = R + (size_t)beta * n_r;
    double *y = Y + (size_t)beta * n_e;
    for (int64_t j = 0; j < n_e; ++j) y[j] = 0.0;
    for (int64_t l = 0; l < n_t; ++l)
      y[obj[l]] += (w ? w[l] : 1.0) * x[subj[l]] * r[rel[l]];
  }
  return ORA_OK;
}

/* Backward in double end to end; dX or dR may be NULL. */
int ora_follow_backward_f64(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
                            const int32_t *rel, const int32_t *obj, const double *w,
                            int32_t b, const double *X, const double *R,
                            const double *dY, double *dX, double *dR) {
  if (b < 0 || (b > 0 && (!dY || (dX && !R) || (dR && !X)))) return ORA_EINVAL;
  int rc = check_ids(n_e, n_r, n_t, subj, rel, obj);
  if (rc) return rc;
  for (int32_t beta = 0; beta < b; ++beta) {
    const double *dy = dY + (size_t)beta * n_e;
    if (dX) {
      const double *r = R + (size_t)beta * n_r;
      double *dx = dX + (size_t)beta * n_e;
      for (int64_t i = 0; i < n_e; ++i) dx[i] = 0.0;
      for (int64_t l = 0; l < n_t; ++l)
        dx[subj[l]] += (w ? w[l] : 1.0) * dy[obj[l]] * r[rel[l]];
    }
    if (dR) {
      const double *x = X + (size_t)beta * n_e;
      double *dr = dR + (size_t)beta * n_r;
      for (int64_t k = 0; k < n_r; ++k) dr[k] = 0.0;
      for (int64_t l = 0; l < n_t; ++l)
        dr[rel[l]] += (w ? w[l] : 1.0) * x[subj[l]] * dy[obj[l]];
    }
  }
  return ORA_OK;
}

/*
 * Residual follow, the hop of the KB-completion chains (Sec. 3.2, App. E):
 *   Y[beta][j]  = follow(X, R)[beta][j] + gamma * X[beta][j]
 * and its backward for upstream dY:
 *   dX[beta][i] = (gradient of follow w.r.t. X)[beta][i] + gamma * dY[beta][i]
 *   dR          = gradient of follow w.r.t. R (the residual term has none).
 * The per-triple sum is taken first (caller order, double), then gamma * X
 * (or gamma * dY) is added in double and the result rounded to float once.
 */
int ora_follow_residual(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
                        const int32_t *rel, const int32_t *obj, const float *w, int32_t b,
                        const float *X, const float *R, float gamma, float *Y,
                        int32_t nthreads) {
  if (b < 0 || (b > 0 && (!X || !R || !Y))) return ORA_EINVAL;
  int rc = check_ids(n_e, n_r, n_t, subj, rel, obj);
  if (rc) return rc;
  int err = 0;
#pragma omp parallel num_threads(pick_threads(nthreads, b))
  {
    double *acc = (double *)malloc(sizeof(double) * (size_t)(n_e > 0 ? n_e : 1));
    if (!acc) {
#pragma omp atomic write
      err = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int32_t beta = 0; beta < b; ++beta) {
      if (!acc) continue;
      const float *x = X + (size_t)beta * n_e;
      const float *r = R + (size_t)beta * n_r;
      for (int64_t j = 0; j < n_e; ++j) acc[j] = 0.0;
      for (int64_t l = 0; l < n_t; ++l)
        acc[obj[l]] += weight_of(w, l) * (double)x[subj[l]] * (double)r[rel[l]];
      float *y = Y + (size_t)beta * n_e;
      for (int64_t j = 0; j < n_e; ++j) y[j] = (float)(acc[j] + (double)gamma * (double)x[j]);
    }
    free(acc);
  }
  return err ? ORA_ENOMEM : ORA_OK;
}

/*
 * Accumulating follow: Y[beta][j] = follow(X, R)[beta][j] + gamma * Z[beta][j]
 * for any Z of Y's shape (Z = X is the residual hop above; Z = the old Y
 * adds a hop's result into an existing output).  The per-triple sum first
 * (caller order, double), then gamma * Z added in double, one rounding.  Y
 * may be Z itself.  The gradient is follow's for X and R and gamma * dY for
 * Z.
 */
int ora_follow_accumulate(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
                          const int32_t *rel, const int32_t *obj, const float *w, int32_t b,
                          const float *X, const float *R, const float *Z, float gamma, float *Y,
                          int32_t nthreads) {
  if (b < 0 || (b > 0 && (!X || !R || !Z || !Y))) return ORA_EINVAL;
  int rc = check_ids(n_e, n_r, n_t, subj, rel, obj);
  if (rc) return rc;
  int err = 0;
#pragma omp parallel num_threads(pick_threads(nthreads, b))
  {
    double *acc = (double *)malloc(sizeof(double) * (size_t)(n_e > 0 ? n_e : 1));
    if (!acc) {
#pragma omp atomic write
      err = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int32_t beta = 0; beta < b; ++beta) {
      if (!acc) continue;
      const float *x = X + (size_t)beta * n_e;
      const float *r = R + (size_t)beta * n_r;
      const float *z = Z + (size_t)beta * n_e;
      for (int64_t j = 0; j < n_e; ++j) acc[j] = 0.0;
      for (int64_t l = 0; l < n_t; ++l)
        acc[obj[l]] += weight_of(w, l) * (double)x[subj[l]] * (double)r[rel[l]];
      float *y = Y + (size_t)beta * n_e;
      for (int64_t j = 0; j < n_e; ++j) y[j] = (float)(acc[j] + (double)gamma * (double)z[j]);
    }
    free(acc);
  }
  return err ? ORA_ENOMEM : ORA_OK;
}

int ora_follow_backward_residual(int64_t n_e, int64_t n_r, int64_t n_t, const int32_t *subj,
                                 const int32_t *rel, const int32_t *obj, const float *w,
                                 int32_t b, const float *X, const float *R, const float *dY,
                                 float gamma, float *dX, float *dR, int32_t nthreads) {
  int rc = ora_follow_backward(n_e, n_r, n_t, subj, rel, obj, w, b, X, R, dY, NULL, dR, nthreads);
  if (rc || !dX) return rc;
  if (!R) return ORA_EINVAL;
  int err = 0;
#pragma omp parallel num_threads(pick_threads(nthreads, b))
  {
    double *ax = (double *)malloc(sizeof(double) * (size_t)(n_e > 0 ? n_e : 1));
    if (!ax) {
#pragma omp atomic write
      err = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int32_t beta = 0; beta < b; ++beta) {
      if (!ax) continue;
      const float *dy = dY + (size_t)beta * n_e;
      const float *r = R + (size_t)beta * n_r;
      for (int64_t i = 0; i < n_e; ++i) ax[i] = 0.0;
      for (int64_t l = 0; l < n_t; ++l)
        ax[subj[l]] += weight_of(w, l) * (double)dy[obj[l]] * (double)r[rel[l]];
      float *dx = dX + (size_t)beta * n_e;
      for (int64_t i = 0; i < n_e; ++i) dx[i] = (float)(ax[i] + (double)gamma * (double)dy[i]);
    }
    free(ax);
  }
  return err ? ORA_ENOMEM : ORA_OK;
}
