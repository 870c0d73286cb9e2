/*
 * abi_check.c -- uses libkbfollow from plain C (no Python, no torch).
 *
 * Builds the toy KB below, runs kb_follow and kb_follow_backward on the GPU
 * with hipMalloc'd buffers, and checks the results against values worked out
 * by hand from Eq. 4 and its gradients.  Exit status 0 on success.
 *
 * KB (0-based ids): entities 0..4, relations 0..1, triples (s, r, o):
 *   (0,0,1) (0,1,2) (1,0,2) (2,0,3) (2,0,3) (4,1,0)     -- (2,0,3) twice
 * One example (b = 1): X = e0 + 2 e2, R = (1, 3).
 *   Y[1] = X0 R0 = 1; Y[2] = X0 R1 = 3; Y[3] = 2 X2 R0 = 4; Y[0] = X4 R1 = 0; Y[4] = 0.
 * With dY = (1, 2, 3, 4, 5):
 *   dX[0] = dY1 R0 + dY2 R1 = 2 + 9 = 11; dX[1] = dY2 R0 = 3; dX[2] = 2 dY3 R0 = 8;
 *   dX[3] = 0; dX[4] = dY0 R1 = 3.
 *   dR[0] = X0 dY1 + X1 dY2 + 2 X2 dY3 = 2 + 0 + 16 = 18; dR[1] = X0 dY2 + X4 dY0 = 3.
 */
#include <hip/hip_runtime_api.h>
#include <stdio.h>

#include "kbfollow.h"

#define CHECK_HIP(x)                                                        \
  do {                                                                      \
    if ((x) != hipSuccess) {                                                \
      fprintf(stderr, "HIP error at line %d\n", __LINE__);                 \
      return 2;                                                             \
    }                                                                       \
  } while (0)

static int expect(const char *what, const float *got, const float *want, int n) {
  int bad = 0;
  for (int i = 0; i < n; ++i)
    if (got[i] != want[i]) {
      fprintf(stderr, "%s[%d] = %g, expected %g\n", what, i, got[i], want[i]);
      bad = 1;
    }
  return bad;
}

int main(void) {
  const int32_t subj[] = {0, 0, 1, 2, 2, 4}, rel[] = {0, 1, 0, 0, 0, 1}, obj[] = {1, 2, 2, 3, 3, 0};
  const float X[5] = {1, 0, 2, 0, 0}, R[2] = {1, 3}, dY[5] = {1, 2, 3, 4, 5};
  const float Y_want[5] = {0, 1, 3, 4, 0}, dX_want[5] = {11, 3, 8, 0, 3}, dR_want[2] = {18, 3};
  kb_t *kb = NULL;
  kb_status st = kb_create(5, 2, 6, subj, rel, obj, NULL, NULL, &kb);
  if (st != KB_OK) {
    fprintf(stderr, "kb_create: %s: %s\n", kb_status_str(st), kb_last_error());
    return 1;
  }
  /* An id out of range is refused before any device work. */
  const int32_t bad_obj[] = {1, 2, 2, 3, 3, 5};
  kb_t *kb_bad = NULL;
  if (kb_create(5, 2, 6, subj, rel, bad_obj, NULL, NULL, &kb_bad) != KB_ERANGE || kb_bad) {
    fprintf(stderr, "out-of-range object id was accepted\n");
    return 1;
  }
  float *dX_ = NULL, *dR_ = NULL, *dY_ = NULL, *dXin = NULL, *dRin = NULL, *dYout = NULL;
  void *ws = NULL;
  size_t ws_bytes = kb_workspace_size(kb, 1);
  CHECK_HIP(hipMalloc((void **)&dXin, sizeof X));
  CHECK_HIP(hipMalloc((void **)&dRin, sizeof R));
  CHECK_HIP(hipMalloc((void **)&dYout, sizeof X));
  CHECK_HIP(hipMalloc((void **)&dY_, sizeof dY));
  CHECK_HIP(hipMalloc((void **)&dX_, sizeof X));
  CHECK_HIP(hipMalloc((void **)&dR_, sizeof R));
  if (ws_bytes) CHECK_HIP(hipMalloc(&ws, ws_bytes));
  CHECK_HIP(hipMemcpy(dXin, X, sizeof X, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dRin, R, sizeof R, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dY_, dY, sizeof dY, hipMemcpyHostToDevice));
  if ((st = kb_follow(kb, 1, dXin, dRin, dYout, ws, ws_bytes, NULL)) != KB_OK ||
      (st = kb_follow_backward(kb, 1, dXin, dRin, dY_, dX_, dR_, ws, ws_bytes, NULL)) != KB_OK) {
    fprintf(stderr, "compute call: %s: %s\n", kb_status_str(st), kb_last_error());
    return 1;
  }
  float Y[5], dXh[5], dRh[2];
  CHECK_HIP(hipMemcpy(Y, dYout, sizeof Y, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(dXh, dX_, sizeof dXh, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(dRh, dR_, sizeof dRh, hipMemcpyDeviceToHost));
  int bad = expect("Y", Y, Y_want, 5) | expect("dX", dXh, dX_want, 5) | expect("dR", dRh, dR_want, 2);
  kb_destroy(kb);
  hipFree(dXin);
  hipFree(dRin);
  hipFree(dYout);
  hipFree(dY_);
  hipFree(dX_);
  hipFree(dR_);
  hipFree(ws);
  if (!bad) printf("abi_check ok\n");
  return bad;
}
