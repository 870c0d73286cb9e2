/* The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer: every
 * entry point on random KBs (hard and soft), sampled outputs against the full
 * ones, the double-precision and residual variants against the float ones,
 * and the error paths.  Exit status 0 when every check holds (sanitizer
 * reports abort the program).  Built and run by tests/test_host_sanitizers.py
 * together with oracle/kb_oracle.c. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int ora_follow(int64_t, int64_t, int64_t, const int32_t *, const int32_t *, const int32_t *,
               const float *, int32_t, const float *, const float *, float *, int32_t);
int ora_follow_backward(int64_t, int64_t, int64_t, const int32_t *, const int32_t *,
                        const int32_t *, const float *, int32_t, const float *, const float *,
                        const float *, float *, float *, int32_t);
int ora_sampled(int32_t, int64_t, int64_t, int64_t, const int32_t *, const int32_t *,
                const int32_t *, const float *, int32_t, const float *, const float *,
                const float *, int32_t, const int32_t *, float *, int32_t);
int ora_follow_f64(int64_t, int64_t, int64_t, const int32_t *, const int32_t *, const int32_t *,
                   const double *, int32_t, const double *, const double *, double *);
int ora_follow_backward_f64(int64_t, int64_t, int64_t, const int32_t *, const int32_t *,
                            const int32_t *, const double *, int32_t, const double *,
                            const double *, const double *, double *, double *);
int ora_follow_residual(int64_t, int64_t, int64_t, const int32_t *, const int32_t *,
                        const int32_t *, const float *, int32_t, const float *, const float *,
                        float, float *, int32_t);
int ora_follow_backward_residual(int64_t, int64_t, int64_t, const int32_t *, const int32_t *,
                                 const int32_t *, const float *, int32_t, const float *,
                                 const float *, const float *, float, float *, float *, int32_t);

static int failures = 0;
#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

static uint64_t rng = 20020615u;
static uint32_t next_u32(void) {
  rng ^= rng << 13;
  rng ^= rng >> 7;
  rng ^= rng << 17;
  return (uint32_t)(rng >> 11);
}
static float next_float(void) { return (float)(next_u32() % 2001) / 1000.0f - 1.0f; }

static void run_case(int64_t n_e, int64_t n_r, int64_t n_t, int32_t b, int weighted) {
  int32_t *s = malloc(sizeof(int32_t) * (size_t)(n_t ? n_t : 1));
  int32_t *r = malloc(sizeof(int32_t) * (size_t)(n_t ? n_t : 1));
  int32_t *o = malloc(sizeof(int32_t) * (size_t)(n_t ? n_t : 1));
  float *w = weighted ? malloc(sizeof(float) * (size_t)(n_t ? n_t : 1)) : NULL;
  for (int64_t l = 0; l < n_t; ++l) {
    s[l] = (int32_t)(next_u32() % (uint32_t)n_e);
    r[l] = (int32_t)(next_u32() % (uint32_t)n_r);
    o[l] = (int32_t)(next_u32() % (uint32_t)n_e);
    if (w) w[l] = 0.25f + (float)(next_u32() % 8);
  }
  const size_t ne = (size_t)b * (size_t)n_e, nr = (size_t)b * (size_t)n_r;
  float *X = malloc(sizeof(float) * ne), *R = malloc(sizeof(float) * nr);
  float *dY = malloc(sizeof(float) * ne), *Y = malloc(sizeof(float) * ne);
  float *dX = malloc(sizeof(float) * ne), *dR = malloc(sizeof(float) * nr);
  float *Yr = malloc(sizeof(float) * ne), *dXr = malloc(sizeof(float) * ne);
  float *dRr = malloc(sizeof(float) * nr);
  double *Xd = malloc(sizeof(double) * ne), *Rd = malloc(sizeof(double) * nr);
  double *dYd = malloc(sizeof(double) * ne), *Yd = malloc(sizeof(double) * ne);
  double *dXd = malloc(sizeof(double) * ne), *dRd = malloc(sizeof(double) * nr);
  double *wd = weighted ? malloc(sizeof(double) * (size_t)(n_t ? n_t : 1)) : NULL;
  for (size_t k = 0; k < ne; ++k) {
    X[k] = next_float();
    dY[k] = next_float();
    Xd[k] = X[k];
    dYd[k] = dY[k];
  }
  for (size_t k = 0; k < nr; ++k) Rd[k] = R[k] = next_float();
  for (int64_t l = 0; w && l < n_t; ++l) wd[l] = w[l];

  CHECK(ora_follow(n_e, n_r, n_t, s, r, o, w, b, X, R, Y, 3) == 0);
  CHECK(ora_follow_backward(n_e, n_r, n_t, s, r, o, w, b, X, R, dY, dX, dR, 2) == 0);
  CHECK(ora_follow_f64(n_e, n_r, n_t, s, r, o, wd, b, Xd, Rd, Yd) == 0);
  CHECK(ora_follow_backward_f64(n_e, n_r, n_t, s, r, o, wd, b, Xd, Rd, dYd, dXd, dRd) == 0);
  /* The float outputs are the double results rounded once. */
  for (size_t k = 0; k < ne; ++k) CHECK(Y[k] == (float)Yd[k] && dX[k] == (float)dXd[k]);
  for (size_t k = 0; k < nr; ++k) CHECK(dR[k] == (float)dRd[k]);
  /* Residual hop with gamma = 0 is the plain hop; with gamma it adds gamma * X. */
  CHECK(ora_follow_residual(n_e, n_r, n_t, s, r, o, w, b, X, R, 0.0f, Yr, 1) == 0);
  for (size_t k = 0; k < ne; ++k) CHECK(Yr[k] == Y[k]);
  CHECK(ora_follow_residual(n_e, n_r, n_t, s, r, o, w, b, X, R, 0.5f, Yr, 0) == 0);
  for (size_t k = 0; k < ne; ++k) CHECK(Yr[k] == (float)(Yd[k] + 0.5 * Xd[k]));
  CHECK(ora_follow_backward_residual(n_e, n_r, n_t, s, r, o, w, b, X, R, dY, 0.5f, dXr, dRr, 4) ==
        0);
  for (size_t k = 0; k < ne; ++k) CHECK(dXr[k] == (float)(dXd[k] + 0.5 * dYd[k]));
  for (size_t k = 0; k < nr; ++k) CHECK(dRr[k] == dR[k]);
  /* Sampled outputs equal the full ones. */
  for (int32_t which = 0; which < 3; ++which) {
    const int64_t space = which == 2 ? n_r : n_e;
    const int32_t n_ids = (int32_t)(space < 5 ? space : 5);
    int32_t ids[5];
    for (int32_t q = 0; q < n_ids; ++q) ids[q] = (int32_t)(space - 1 - q);
    float *out = malloc(sizeof(float) * (size_t)b * (size_t)(n_ids ? n_ids : 1));
    CHECK(ora_sampled(which, n_e, n_r, n_t, s, r, o, w, b, X, R, dY, n_ids, ids, out, 2) == 0);
    const float *full = which == 0 ? Y : (which == 1 ? dX : dR);
    for (int32_t beta = 0; beta < b; ++beta)
      for (int32_t q = 0; q < n_ids; ++q)
        CHECK(out[(size_t)beta * n_ids + q] == full[(size_t)beta * space + ids[q]]);
    free(out);
  }
  /* Error paths: an id out of range, a repeated sampled id, a bad pass. */
  if (n_t > 0) {
    const int32_t keep = s[0];
    s[0] = (int32_t)n_e;
    CHECK(ora_follow(n_e, n_r, n_t, s, r, o, w, b, X, R, Y, 1) == -1);
    s[0] = keep;
  }
  {
    int32_t dup[2] = {0, 0};
    float out[2 * 64];
    if (b <= 64) CHECK(ora_sampled(0, n_e, n_r, n_t, s, r, o, w, b, X, R, dY, 2, dup, out, 1) == -1);
    CHECK(ora_sampled(3, n_e, n_r, n_t, s, r, o, w, b, X, R, dY, 0, NULL, NULL, 1) == -1);
  }
  free(s), free(r), free(o), free(w), free(X), free(R), free(dY), free(Y), free(dX), free(dR);
  free(Yr), free(dXr), free(dRr), free(Xd), free(Rd), free(dYd), free(Yd), free(dXd), free(dRd);
  free(wd);
}

int main(void) {
  run_case(40, 3, 600, 5, 0);
  run_case(40, 3, 600, 4, 1);
  run_case(1, 1, 50, 3, 1);
  run_case(30, 2, 0, 2, 0);
  run_case(300, 17, 5000, 9, 1);
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("oracle checks passed\n");
  return 0;
}
