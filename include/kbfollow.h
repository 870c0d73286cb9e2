/*
 * kbfollow.h -- C ABI of the MI355X (gfx950) relation-set following library.
 *
 * A reified KB (Sec. 2.3) stores N_T triples (s_l, r_l, o_l): subject entity,
 * relation and object entity of fact l.  With M_subj, M_obj, M_rel the N_T x N_E,
 * N_T x N_E and N_T x N_R matrices that map triple l to its subject, object and
 * relation (M_rel holding the triple's weight w_l for a soft KB, App. A), the
 * library evaluates for a minibatch of b examples (Eq. 4, App. C)
 *
 *     Y = follow(X, R) = (X M_subj^T  (.)  R M_rel^T) M_obj
 *
 * and the two gradients of a scalar loss with upstream gradient dY = dL/dY:
 *
 *     dX[i] = sum over triples l with s_l == i of  w_l * dY[o_l] (.) R[r_l]
 *     dR[k] = sum over triples l with r_l == k of  w_l * X[s_l]  (.) dY[o_l]
 *
 * Layout of every activation (this library's own choice, the transpose of the
 * paper's b x N row-vector view): entity-major, batch-contiguous float32.
 *     X, Y, dY, dX : [N_E][b]   element (i, beta) at i * b + beta
 *     R, dR        : [N_R][b]   element (k, beta) at k * b + beta
 * Ids are 0-based (the paper's are 1-based, Sec. 2.1).
 *
 * Numerics: products and sums are taken in double precision on the GPU and
 * every output element is rounded to float once.  Sums run in a fixed order,
 * so two calls with the same inputs give bitwise-equal results.  Duplicate
 * triples each count.  An output row no triple reaches is +0.0.  No clamping
 * and no NaN checks: IEEE values propagate.
 *
 * Streams: every compute call only enqueues work on `stream` (a hipStream_t;
 * NULL = the null stream) and returns; it never synchronises the host and
 * never allocates device memory.  Scratch space comes from the caller's
 * `workspace`, sized with kb_workspace_size().  On KBs of 2^20 triples or
 * more, at b <= 32, kb_follow_backward runs its dR pass on a stream the KB owns, forked
 * from `stream` with an event and joined back into it before returning, so
 * that work enqueued on `stream` afterwards still follows both passes (and
 * a graph captured on `stream` contains both).
 *
 * Errors: argument checks run on the host before anything is enqueued; on
 * failure nothing is launched and no output is touched.  The status says what
 * went wrong and kb_last_error() gives a message (per calling thread).
 * No C++ exception ever crosses this interface.
 *
 * Thread safety: a kb_t is immutable after kb_create (profiling counters
 * excepted, see kb_profile_*), so calls on different streams, each with its
 * own workspace and outputs, may run concurrently.
 */
#ifndef KBFOLLOW_H
#define KBFOLLOW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kb_t kb_t; /* opaque handle to a KB resident on one GPU */

typedef enum {
  KB_OK = 0,
  KB_EINVAL = 1,  /* bad argument: null pointer, size, alignment, overlap, workspace */
  KB_ERANGE = 2,  /* a triple id outside [0, N_E) or [0, N_R) */
  KB_ENOMEM = 3,  /* device or host allocation failed */
  KB_EHIP = 4,    /* a HIP runtime call or kernel launch failed */
  KB_ENOTSUP = 5  /* valid request this build does not implement */
} kb_status;

/*
 * Build a KB on the current HIP device from host triple arrays (Sec. 2.3: the
 * reified KB M_subj, M_obj, M_rel, one nonzero per row).
 *
 *   n_entities, n_relations : 0 <= N_E, N_R <= 2^30.
 *   n_triples               : N_T, 0 <= N_T < 2^31.
 *   subj, rel, obj          : HOST int32 arrays of N_T ids (may be NULL when
 *                             N_T == 0); copied, the caller keeps ownership.
 *   weight                  : HOST float array of N_T triple weights w_l
 *                             (soft KB, App. A) or NULL for a hard KB (w = 1).
 *   stream                  : hipStream_t used for the uploads.  kb_create
 *                             waits for them before it returns.
 *   out                     : receives the handle; set to NULL on failure.
 *
 * The three sorted layouts (by object, by subject, by relation) and their
 * work plans are built on the host and uploaded; the host copies are freed.
 * Device memory held: 8 bytes per triple per layout (24 per triple; 36 with
 * weights) plus about 8 bytes per non-empty row per layout.  Building sorts
 * the triples three ways (radix sorts of one 64-bit key per triple when
 * 2 * bits(N_E - 1) + bits(N_R - 1) <= 64, else chained counting sorts) on
 * up to 16 host threads (the calling thread plus threads it starts and joins
 * before returning).
 * Errors: KB_EINVAL (sizes, null pointers), KB_ERANGE (an id out of range;
 * checked before any device work), KB_ENOMEM, KB_EHIP.
 *
 * Environment variables read here, for tests and tuning (results are the
 * same up to the summation order of split rows, or bitwise the same):
 *   KBFOLLOW_CHUNK, KBFOLLOW_REL_CHUNK  entries per chunk of the entity and
 *                                       relation layouts (default 256 and
 *                                       128, less for small KBs; rounded up
 *                                       to 8);
 *   KBFOLLOW_FAN_IN                     partials per combine task (32);
 *   KBFOLLOW_PLAIN_LOADS=1              plain loads instead of raw buffer
 *                                       loads (bitwise the same);
 *   KBFOLLOW_B_IN_LDS=0                 the second operand (R, or X for dR)
 *                                       read into registers per run even
 *                                       where its table fits LDS (bitwise
 *                                       the same);
 *   KBFOLLOW_LAYOUT_SORT=counting       the chained counting sorts for
 *                                       every KB (bitwise the same);
 *   KBFOLLOW_OVERLAP_BACKWARD=0|1       dR concurrent with dX on the KB's
 *                                       own stream (default: from 2^20
 *                                       triples at b <= 32; 1 also forces it
 *                                       on small KBs; bitwise the same);
 *   KBFOLLOW_HOST_THREADS               host threads for the layout sorts
 *                                       (default: the hardware's, at most 16;
 *                                       the same layouts for any count);
 *   KBFOLLOW_XCD                        chunk lists, one per XCD (8; 1 keeps
 *                                       one list in row order);
 *   KBFOLLOW_HUB_MIN                    triples from which a row is split
 *                                       into one segment per class of its
 *                                       gathered ids (256);
 *   KBFOLLOW_BAND=0                     hub chunks in stream order instead of
 *                                       by first gathered id;
 *   KBFOLLOW_DR_CLASS_B=0|1             dR's chunk lists classed by the
 *                                       gathered object id (0) or by the
 *                                       subject id held per run (1); default:
 *                                       by subject when the top 1 % of
 *                                       objects hold a quarter of the triples;
 *   KBFOLLOW_DR_BLOCKS                  blocks of the object id leading
 *                                       dR's hub segments (64; 0 or 1: none);
 *   KBFOLLOW_MAX_LPT                    widest lane group of the register
 *                                       variant, every pass (default: 32, 8
 *                                       for dR from b = 128; bitwise the
 *                                       same);
 *   KBFOLLOW_STREAM_STAMPS=0            phase timing of the stream kernels by
 *                                       event records instead of their
 *                                       dispatch timestamps.
 */
kb_status kb_create(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                    const int32_t *subj, const int32_t *rel, const int32_t *obj,
                    const float *weight, void *stream, kb_t **out);

/* Free a KB and its device memory.  NULL-safe.  The caller must make sure no
 * enqueued work still uses it (synchronise its streams first). */
void kb_destroy(kb_t *kb);

/* Bytes of device workspace that kb_follow and kb_follow_backward need for
 * batch size b (scratch for the partial sums of rows that cross chunks).  May
 * be 0.  Returns 0 for a NULL kb or b < 1. */
size_t kb_workspace_size(const kb_t *kb, int32_t b);

/*
 * Forward pass, Eq. 4:  Y[j] = sum over triples l with o_l == j of
 * w_l * X[s_l] (.) R[r_l]   (b-wide rows).
 *
 *   b          : batch size, b >= 1.
 *   X          : DEVICE float [N_E][b], read only.
 *   R          : DEVICE float [N_R][b], read only.
 *   Y          : DEVICE float [N_E][b], fully overwritten; must not overlap X or R.
 *   workspace  : DEVICE scratch of at least kb_workspace_size(kb, b) bytes,
 *                256-byte aligned (may be NULL when that size is 0; at
 *                least 16-byte alignment is enforced).  It must not overlap
 *                X, R or Y.  Its contents on entry are ignored.  Calls
 *                running at the same time must not share one.
 *   ws_bytes   : size of workspace in bytes.
 *   stream     : hipStream_t on which the work is enqueued.
 *
 * Pointers must be 4-byte aligned; when b % 4 == 0 the fast path also needs
 * X, R and Y 16-byte aligned (otherwise KB_EINVAL).
 */
kb_status kb_follow(const kb_t *kb, int32_t b, const float *X, const float *R, float *Y,
                    void *workspace, size_t ws_bytes, void *stream);

/*
 * Backward pass of Eq. 4 for upstream gradient dY:
 *   dX[i] = sum over l with s_l == i of w_l * dY[o_l] (.) R[r_l]
 *   dR[k] = sum over l with r_l == k of w_l * X[s_l] (.) dY[o_l]
 *
 *   X, R, dY : DEVICE float [N_E][b], [N_R][b], [N_E][b], read only.  X may be
 *              NULL when dR is NULL, R may be NULL when dX is NULL.
 *   dX       : DEVICE float [N_E][b], overwritten, or NULL to skip it.
 *   dR       : DEVICE float [N_R][b], overwritten, or NULL to skip it.
 *   Outputs must not overlap each other or any input, and the workspace
 *   overlaps none of the arrays.  Workspace and stream as for kb_follow (dX
 *   and dR use disjoint parts of the workspace, since on a large KB the two
 *   passes run concurrently; see Streams above).
 */
kb_status kb_follow_backward(const kb_t *kb, int32_t b, const float *X, const float *R,
                             const float *dY, float *dX, float *dR, void *workspace,
                             size_t ws_bytes, void *stream);

/*
 * kb_follow for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops, harnesses that forbid hipMalloc): the same
 * forward pass, kernels and bitwise the same Y, but the split-row partials go
 * to a fixed scratch array inside the library instead of a caller workspace,
 * so neither the call nor the caller allocates anything.
 *
 *   X, R, Y, stream : as for kb_follow (Y fully overwritten).
 *
 * The scratch holds KB_NOALLOC_SCRATCH_BYTES (64 MiB) per GPU, taken on the
 * first call on that GPU and held until the process ends.  A KB and batch
 * size whose kb_workspace_size exceeds it are refused with KB_EINVAL before
 * anything is enqueued (the 10 M-entity / 50 M-triple KB needs about 61 MiB
 * at b = 32).  Every call on one GPU shares that GPU's scratch, and the
 * scratch keeps the last call's partials (each call writes every partial it
 * reads, so nothing needs clearing): calls that overlap in time on one GPU --
 * on two streams, or from two host threads -- race and must not be issued.
 * Other errors as for kb_follow.
 */
#define KB_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
kb_status kb_follow_noalloc(const kb_t *kb, int32_t b, const float *X, const float *R, float *Y,
                            void *stream);

/*
 * Residual hop of the KB-completion chains (Sec. 3.2, App. E), which add each
 * hop's input back:  Y = follow(X, R) + gamma * X  (gamma = 1 in the paper).
 * Arguments, layout and rules as for kb_follow; each element of Y is the
 * double-precision sum plus gamma * X, rounded to float once.
 */
kb_status kb_follow_residual(const kb_t *kb, int32_t b, const float *X, const float *R,
                             float gamma, float *Y, void *workspace, size_t ws_bytes,
                             void *stream);

/*
 * Backward of kb_follow_residual for upstream gradient dY:
 *   dX = (dX of kb_follow_backward) + gamma * dY,   dR as in kb_follow_backward.
 * Arguments and rules as for kb_follow_backward.
 */
kb_status kb_follow_backward_residual(const kb_t *kb, int32_t b, const float *X, const float *R,
                                      const float *dY, float gamma, float *dX, float *dR,
                                      void *workspace, size_t ws_bytes, void *stream);

/*
 * Accumulating follow (the residual hop's added term from any array; the
 * KB-completion hop of Sec. 3.2 / App. E is Z = X):
 *   Y[j][beta] = follow(X, R)[j][beta] + gamma * Z[j][beta]
 * summed in double and rounded to float once, like kb_follow.
 *   Z : DEVICE [N_E][b] floats, aligned like X.  Z == Y adds the hop's
 *       result into Y in place (each row of Z is read by the thread that
 *       then writes that row of Y); otherwise Z must not overlap Y.  Z may
 *       be X or overlap X or R (it is only read).
 * Other arguments, the workspace and the errors as for kb_follow (KB_EINVAL
 * also for a NULL Z or a Z that overlaps Y without being Y).  Raw buffer
 * loads need the added rows to come from X, so with any other Z the
 * forward pass takes the plain-load path (a few percent slower).  The
 * gradient is kb_follow_backward's for X and R and gamma * dY for Z.
 */
kb_status kb_follow_accumulate(const kb_t *kb, int32_t b, const float *X, const float *R,
                               const float *Z, float gamma, float *Y, void *workspace,
                               size_t ws_bytes, void *stream);

/* Static description of a status code. */
const char *kb_status_str(kb_status s);

/* Message describing the last failure on the calling thread ("" if none). */
const char *kb_last_error(void);

/* ------------------------------------------------------------------------
 * Inspection (host side; none of these touch the GPU)
 * ------------------------------------------------------------------------ */

/* Sizes and plan statistics of a built KB. */
typedef struct {
  int64_t n_entities, n_relations, n_triples;
  int32_t weighted;         /* 1 if built with per-triple weights */
  int32_t chunk_len[3];     /* triples per chunk, one chunk per lane group (obj, subj, rel) */
  int64_t n_chunks[3];      /* chunks per layout: by object, by subject, by relation */
  int64_t n_split_rows[3];  /* rows that cross a chunk boundary */
  int64_t n_slots[3];       /* partial-sum slots (all combine levels) */
  int32_t n_levels[3];      /* combine levels */
  int64_t n_empty_rows[3];  /* rows with no triple (written as zeros) */
  int64_t max_row_len[3];   /* longest row (triples) */
  int64_t device_bytes;     /* device memory the KB holds */
} kb_info_t;

kb_status kb_get_info(const kb_t *kb, kb_info_t *info);

/*
 * The sorted layout kb_create builds, computed on the host only (no GPU needed).
 *   which = 0: by object   (rows = objects,   key order (o, r, s)), col_a = subj, col_b = rel
 *   which = 1: by subject  (rows = subjects,  key order (s, r, o)), col_a = obj,  col_b = rel
 *   which = 2: by relation (rows = relations, key order (r, s, o)), col_a = obj,  col_b = subj
 *   (col_a is the id gathered for every triple, col_b the id read once per run
 *   of equal col_b inside a row)
 *   offsets : HOST int32 [rows + 1]; row q's triples are positions offsets[q] .. offsets[q+1]-1
 *   col_a, col_b, perm : HOST int32 [N_T]; perm[p] = caller index of the triple at position p
 * Any output pointer may be NULL.  Same validation and errors as kb_create.
 */
kb_status kb_layout_host(int64_t n_entities, int64_t n_relations, int64_t n_triples,
                         const int32_t *subj, const int32_t *rel, const int32_t *obj,
                         int32_t which, int32_t *offsets, int32_t *col_a, int32_t *col_b,
                         int32_t *perm);

/* ------------------------------------------------------------------------
 * Checked builds (for testing)
 * ------------------------------------------------------------------------ */

/*
 * A build compiled with KBFOLLOW_CHECKED validates, inside the kernels, every
 * row, workspace-slot and combine index against its table before using it.
 * An index outside its table is replaced by a valid one and counted; the
 * computation goes on (results are then wrong, but no access leaves its
 * buffer).  This returns the count on the current device since the last
 * reset (and resets it when `reset` is nonzero).  Normal builds return
 * KB_ENOTSUP with *count = 0.
 */
kb_status kb_checked_violations(uint64_t *count, int32_t reset);

/* ------------------------------------------------------------------------
 * Kernel timing with HIP events (for benchmarks; not thread safe)
 * ------------------------------------------------------------------------ */

/* Phases whose GPU time is recorded when profiling is on.  Per pass: STREAM
 * is the stream kernel; TAIL the one launch that does the first combine
 * level (rows split over several chunks) and writes the rows without
 * triples; COMBINE the further combine levels (rows split over many chunks). */
typedef enum {
  KB_PH_FWD_STREAM = 0, KB_PH_FWD_TAIL, KB_PH_FWD_COMBINE,
  KB_PH_DX_STREAM, KB_PH_DX_TAIL, KB_PH_DX_COMBINE,
  KB_PH_DR_STREAM, KB_PH_DR_TAIL, KB_PH_DR_COMBINE,
  KB_PH_COUNT
} kb_phase;

/* Turn event recording around each phase's launches on (1) or off (0).
 * Turning it on clears the accumulated times. */
kb_status kb_profile_enable(kb_t *kb, int32_t on);

/* Record only the phases whose bit (1u << kb_phase) is set in phase_mask
 * (0 turns recording off); clears the accumulated times like
 * kb_profile_enable.  A STREAM phase (one kernel) is timed by its kernel's
 * own start and end timestamps (hipExtLaunchKernel), which adds nothing to
 * the stream; TAIL and COMBINE phases add two events each, and each event
 * costs a few microseconds of GPU time (and, recorded between the dX pass's
 * launches, holds back the concurrent dR pass), so a benchmark that times
 * whole steps records only the phases it needs. */
kb_status kb_profile_select(kb_t *kb, uint32_t phase_mask);

/* Wait for the recorded events, add their elapsed times into ms[KB_PH_COUNT]
 * and their launch counts into launches[KB_PH_COUNT] (either may be NULL),
 * then clear the record. */
kb_status kb_profile_read(kb_t *kb, double *ms, int64_t *launches);

/* The kernel a phase launches for this KB at batch size b, as profilers
 * print it (e.g. "stream_kernel<4, 8, true, false, false, true>"), written
 * NUL-terminated into name[len] (truncated if longer); "" when the phase
 * launches nothing.  residual != 0 describes kb_follow_residual and
 * kb_follow_backward_residual instead of kb_follow and kb_follow_backward.
 * Uses the runtime's occupancy calculator on the KB's device (which must be
 * current) but enqueues nothing.  KB_EINVAL for a NULL kb or name, len = 0,
 * b < 1 or a phase outside [0, KB_PH_COUNT). */
kb_status kb_phase_kernel(const kb_t *kb, int32_t b, int32_t phase, int32_t residual, char *name,
                          size_t len);

#ifdef __cplusplus
}
#endif

#endif /* KBFOLLOW_H */
