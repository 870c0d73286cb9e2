/*
 * kbchain.h -- C ABI of the multi-hop chain glue (gfx950), a harness library
 * beside kbfollow.h.
 *
 * The multi-hop question-answering model of Sec. 3.2 chains follow steps,
 * x^t = follow(x^{t-1}, r^t), takes a softmax of the last hop's entity
 * weights and a cross-entropy loss against the answer set written as a
 * distribution.  Between the follow calls the chain needs a few column-wise
 * operations, provided here so that a whole chain, forward and backward, runs
 * in this project's kernels:
 *   r^t = softmax(rho^t) over the relations (and its backward),
 *   x^t = u^t / sum(u^t) over the entities, one sum per example (and its
 *         backward),
 *   the softmax cross-entropy of the last hop (loss and gradient).
 *
 * Layout: every array is entity-major (or relation-major) and
 * batch-contiguous float32 [n][b], element (i, beta) at i * b + beta, as in
 * kbfollow.h; each of the b columns is one example and every reduction runs
 * over the n rows of a column.  Reductions are taken in double, in a fixed
 * order (bitwise reproducible), and every float output is rounded once.
 *
 * Streams and memory: every call only enqueues work on `stream` (hipStream_t,
 * NULL = null stream), allocates nothing and returns.  All pointers are
 * DEVICE pointers; input and output arrays must not overlap unless stated.
 * The kernels are sized for chain-harness shapes: one 1024-thread workgroup
 * reduces 16 columns over all n rows (64 rows at a time, four deep in
 * flight), so a launch spans ceil(b / 16) workgroups.
 *
 * Errors: arguments are checked before anything is enqueued; on failure
 * nothing is launched.  Returns KBC_OK, KBC_EINVAL (null pointer, n < 1 or
 * b < 1) or KBC_EHIP (launch failure).
 */
#ifndef KBCHAIN_H
#define KBCHAIN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { KBC_OK = 0, KBC_EINVAL = 1, KBC_EHIP = 4 } kbc_status;

/* p[:, beta] = softmax(z[:, beta]) over the n rows:
 * exp(z - max) / sum(exp(z - max)), in double.  z, p: [n][b]. */
kbc_status kbc_softmax(int64_t n, int32_t b, const float *z, float *p, void *stream);

/* Backward of kbc_softmax: dz = p (.) (dp - <dp, p>), the inner product per
 * column.  p is softmax's output; dp the upstream gradient.  All [n][b]. */
kbc_status kbc_softmax_backward(int64_t n, int32_t b, const float *p, const float *dp, float *dz,
                                void *stream);

/* L1 normalisation per column: sums[beta] = sum_i u[i, beta] (double), and
 * x = u / sums.  u, x: [n][b]; sums: DEVICE double[b], written.  For
 * non-negative u (entity weights). */
kbc_status kbc_l1_normalize(int64_t n, int32_t b, const float *u, float *x, double *sums,
                            void *stream);

/* Backward of kbc_l1_normalize: du = (dx - <dx, x>) / sums, per column.
 * x: the normalised output; sums: as written by kbc_l1_normalize. */
kbc_status kbc_l1_normalize_backward(int64_t n, int32_t b, const float *x, const double *sums,
                                     const float *dx, float *du, void *stream);

/* Softmax cross-entropy of logits z against targets t (both [n][b]),
 * averaged over the b examples:
 *   col_loss[beta] = -sum_i t[i, beta] * log softmax(z[:, beta])[i]   (double[b])
 *   loss[0]        = (sum over beta of col_loss, in order) / b         (double[1])
 *   dz             = (softmax(z) * sum_i t[i, beta] - t) / b            ([n][b])
 * (dz is the gradient of loss[0]; with targets summing to 1 per column it is
 * (softmax(z) - t) / b). */
kbc_status kbc_softmax_xent(int64_t n, int32_t b, const float *z, const float *t,
                            double *col_loss, double *loss, float *dz, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* KBCHAIN_H */
