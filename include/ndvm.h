/*
 * ndvm.h -- C ABI of the MI355X NDVM hot path.
 *
 * The method (arXiv 2607.03574, "Differentiate the Evaluator, Not the
 * Program"): a fixed evaluator walks a program held as runtime data together
 * with numeric parameters theta and returns y = E(P, theta); the goal is
 * dy/dtheta (Section 2).  Structure (control, locals, loop counters) stays
 * on the host; numeric payloads live in dense batched buffers whose leading
 * axis is the lane (parameter-vector) axis (Section 3.1, Definition "Payload
 * table"); reverse mode is a define-by-run tape over numeric primitives only,
 * replayed in reverse with vectorised loops over the batch axis (Section
 * 3.4); one structural walk serves B parameter vectors (Section 3.5); the
 * result is each lane's loss and its exact gradient on the realized trace
 * (Section 4, Property 1).
 *
 * Here the structural walk happens once per program on the host
 * (ndvm_tape_build) and yields a lane-invariant tape in which numeric
 * branches are per-lane selects.  ndvm_tape_upload schedules the tape for the
 * GPU; ndvm_forward / ndvm_grad replay it on the device for L lanes (16
 * lanes per wave, each lane's independent operations spread over 4 threads),
 * and ndvm_grad_many does so for many programs in a single launch.
 * ndvm_adam_step is the optimiser step of a calibration loop driven by
 * ndvm_grad.
 *
 * Conventions for every entry point:
 *  - All functions return ndvm_status; on a non-OK status a message is
 *    available from ndvm_last_error() (per calling thread).  No C++
 *    exception crosses this boundary.
 *  - Argument and size errors are reported synchronously, before any GPU
 *    work is enqueued (NDVM_E_ARG).
 *  - Device pointers are plain HIP device addresses (for example a torch
 *    tensor's data_ptr()).  `stream` is a hipStream_t passed as void*; NULL
 *    means the default stream.  Compute calls (ndvm_forward, ndvm_grad,
 *    ndvm_grad_many, ndvm_adam_step) only enqueue work on `stream`: they never
 *    schedule on the host, allocate or synchronise.  The device program of a
 *    gradient launch depends on the lane count (it sets each lane's register
 *    budget) and is scheduled and copied to the device by the sizing calls
 *    ndvm_workspace_bytes / ndvm_workspace_bytes_many, which a caller needs
 *    anyway to size the workspace; a compute call for a lane count that was
 *    never sized returns NDVM_E_ARG.  Faults inside a kernel surface at the
 *    caller's next synchronisation, launch failures as NDVM_E_DEVICE.
 *  - The caller owns every buffer it passes and must keep it alive until the
 *    enqueued work has completed.  The library keeps no caller pointer after
 *    a call returns.  Tape handles are owned by the library until
 *    ndvm_tape_free().
 *  - Numerics are fp64.  Non-finite lane results are values, not errors; a
 *    lane never influences another lane.
 *  - A tape handle may be used from several streams at once; a workspace must
 *    not be shared by calls that can run concurrently.
 */
#ifndef NDVM_H
#define NDVM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ndvm_tape ndvm_tape;

typedef enum {
    NDVM_OK = 0,
    NDVM_E_ARG = 1,             /* bad pointer, size, stride or count */
    NDVM_E_BYTECODE = 2,        /* malformed bytecode or a program that cannot be traced */
    NDVM_E_STRUCT_DIVERGE = 3,  /* numeric branch arms leave different structure */
    NDVM_E_TAPE = 4,            /* malformed tape bytes */
    NDVM_E_NOMEM = 5,           /* host or device allocation failed / workspace too small */
    NDVM_E_DEVICE = 6,          /* HIP runtime error */
    NDVM_E_UNSUPPORTED = 7,     /* valid input outside what this build handles */
    NDVM_E_INTERNAL = 8         /* a fault inside the library (a bug), not a caller error */
} ndvm_status;

/* Save policies for the reverse sweep (argument `policy` of ndvm_tape_upload;
 * Section 3.4: the tape keeps the payloads the reverse sweep reads).  Both
 * give the same bits: a recomputed value is computed by the same operations
 * on the same inputs as the stored one. */
#define NDVM_POLICY_SAVE 1       /* store every value an adjoint rule reads when the forward sweep computes it;
                                    the reverse sweep restores them and recomputes nothing */
#define NDVM_POLICY_RECOMPUTE 2  /* store segment inputs only; each segment's reverse sweep recomputes the
                                    values its rules read from them */
/* Option OR'd into `policy`: wave-level branch skipping (Section 6 lane
 * masking, decided per wave).  The arm of a numeric branch that only that
 * arm's select reads is laid out behind a skip test; a wave in which every
 * lane decides the branch the other way does not run the arm, in the forward
 * sweep or the reverse sweep.  Results are bit for bit those without the
 * option (a skipped arm would only have produced values the selects discard
 * and adjoint contributions of exactly zero).  It pays when the lanes of a
 * wave (64 / slots consecutive lanes) tend to decide alike, e.g. a population
 * ordered by the branch's predicate; with lanes that decide at random it
 * costs a few percent (the skip tests, and arms packed apart). */
#define NDVM_BRANCH_SKIP 0x100

typedef struct {
    uint32_t n_params;    /* P: parameters per lane */
    uint32_t n_obs;       /* observations the program reads */
    uint32_t n_ops;       /* tape ops (leaves included) */
    uint32_t n_consts;    /* tape constant pool entries */
    uint32_t loss_slot;   /* tape slot holding the loss */
    uint32_t n_selects;   /* per-lane select ops (numeric branches) */
    uint64_t tape_bytes;  /* size of the serialized tape */
} ndvm_tape_info;

/*
 * Trace producer (host only; Section 3.3 control as realized trace, Section
 * 3.4 payload-only tape, Section 6 lane-masked divergent control).
 * Walks the stack bytecode once with symbolic values and returns the
 * serialized lane-invariant tape in *tape (malloc'd by the library; release
 * with ndvm_free).  Counted loops are unrolled; a numeric IFLT traces both
 * arms and merges differing stack positions and locals with SELECT ops; an
 * IFLT on two constants resolves here.  No folding or CSE is performed.
 * Errors: NDVM_E_ARG (null pointers), NDVM_E_BYTECODE, NDVM_E_STRUCT_DIVERGE.
 */
ndvm_status ndvm_tape_build(const uint8_t *bytecode, size_t bytecode_len,
                            uint8_t **tape, size_t *tape_len);

/*
 * Validate a serialized tape (host bytes), schedule it for the device and
 * copy the device program to GPU memory on `stream` (Section 3.4 replay;
 * the schedule decides register placement, checkpoint segments and what is
 * recomputed in the reverse sweep).  `policy` is NDVM_POLICY_SAVE or
 * NDVM_POLICY_RECOMPUTE, optionally OR'd with NDVM_BRANCH_SKIP.
 * On success *out receives a handle owned by the library.
 * Errors: NDVM_E_ARG, NDVM_E_TAPE (malformed tape), NDVM_E_NOMEM,
 * NDVM_E_DEVICE, NDVM_E_UNSUPPORTED (unknown policy).
 */
ndvm_status ndvm_tape_upload(const uint8_t *tape, size_t tape_len, int policy,
                             void *stream, ndvm_tape **out);

/*
 * ndvm_tape_upload for a population of n tapes (tape i: host bytes tapes[i],
 * lens[i] of them), all with one `policy`: the tapes are validated and their
 * forward programs scheduled on all host threads, then copied to GPU memory on
 * `stream` in order.  On success out[i] receives tape i's handle (each
 * released with ndvm_tape_free); on any error every out[i] is NULL, nothing is
 * left allocated and the message names the first failing tape.  n = 0 is a
 * no-op.  Library infrastructure for program populations (the replay of
 * Section 3.4 applied to many candidate programs).
 * Errors: as ndvm_tape_upload; NDVM_E_ARG for n < 0 or null arrays or tapes.
 */
ndvm_status ndvm_tape_upload_many(const uint8_t *const *tapes, const size_t *lens, int n, int policy,
                                  void *stream, ndvm_tape **out);

/* Sizes of an uploaded tape.  Library infrastructure (no passage of the
 * paper defines it): counts the caller may want for logging or sizing.
 * Errors: NDVM_E_ARG. */
ndvm_status ndvm_tape_info_get(const ndvm_tape *tape, ndvm_tape_info *out);

/*
 * Bytes of device workspace ndvm_forward (with_grad = 0) or ndvm_grad
 * (with_grad = 1) needs for L lanes.  Library infrastructure (no passage of
 * the paper defines it): the workspace holds segment checkpoints and any lane
 * registers that do not fit in LDS.  This is the preparation call of a lane
 * count: with with_grad = 1 it schedules the tape for that launch shape and
 * copies the device program to the GPU (synchronously; once per tape and
 * register budget, then cached), so that ndvm_grad itself only enqueues.
 * Errors: NDVM_E_ARG (null handle/pointer, L < 0), NDVM_E_NOMEM,
 * NDVM_E_DEVICE, NDVM_E_UNSUPPORTED (program too large for the device format).
 */
ndvm_status ndvm_workspace_bytes(const ndvm_tape *tape, int64_t L, int with_grad,
                                 size_t *bytes);

/*
 * Batched forward replay (Section 3.5): loss[l] = E(P, theta_l) for
 * l = 0..L-1.
 *   params : device fp64, element (l, p) at params[l*ld_p + p], ld_p >= P
 *   obs    : device fp64 [n_obs]; n_obs must equal the tape's n_obs
 *   loss   : device fp64 [L]
 *   workspace : device buffer of at least ndvm_workspace_bytes(tape, L, 0)
 *               bytes (may be NULL when that size is 0), 256-byte aligned
 * L = 0 is a no-op.  Errors: NDVM_E_ARG (null tape or buffer, L < 0,
 * ld_p < P, n_obs different from the tape's), NDVM_E_NOMEM (workspace too
 * small), NDVM_E_DEVICE.
 */
ndvm_status ndvm_forward(const ndvm_tape *tape, const double *params, int64_t L,
                         int64_t ld_p, const double *obs, int64_t n_obs, double *loss,
                         void *workspace, size_t workspace_bytes, void *stream);

/*
 * Batched forward replay plus the exact reverse-mode sweep (Section 3.4,
 * Appendix C table tab:adjoints; Property 1 for branches): loss[l] as above
 * and grad[l*ld_g + p] = d loss_l / d theta_{l,p}.  Branch predicates carry
 * no gradient; a node whose incoming adjoint is exactly zero contributes
 * nothing, so untaken select arms cannot poison gradients.
 * Same argument rules as ndvm_forward plus ld_g >= P; the workspace must
 * hold ndvm_workspace_bytes(tape, L, 1) bytes, and that call must have been
 * made for this L (else NDVM_E_ARG).
 */
ndvm_status ndvm_grad(const ndvm_tape *tape, const double *params, int64_t L,
                      int64_t ld_p, const double *obs, int64_t n_obs, double *loss,
                      double *grad, int64_t ld_g, void *workspace, size_t workspace_bytes,
                      void *stream);

/*
 * ndvm_grad without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  The call allocates nothing (no hipMalloc, hipFree
 * or allocating library routine): the launch's checkpoint, trash and spill
 * rows live in a static device array of NDVM_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends.  Arguments,
 * results and errors as ndvm_grad, with the same preparation
 * (ndvm_workspace_bytes(tape, L, 1) for this L, made beforehand, where
 * allocation is allowed); a launch whose workspace would exceed the array is
 * rejected with NDVM_E_NOMEM before anything is enqueued.  Nothing in the
 * array needs to start at zero (every row is written before it is read), and
 * it keeps the last call's contents.  All calls on one GPU share the array:
 * calls that can overlap on one GPU (several streams, several threads) race
 * and must be serialised by the caller.
 */
#define NDVM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
ndvm_status ndvm_grad_noalloc(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p,
                              const double *obs, int64_t n_obs, double *loss, double *grad, int64_t ld_g,
                              void *stream);

/*
 * Flattened data axis (Section 3.5, named axes flattened into the batch
 * dimension): for a loss that is a scaled sum over N data points of a
 * per-point term, `tape` is the per-point term program, reading its point's
 * observation row (the tape's n_obs values), and the launch runs one lane
 * per (parameter vector, data point), L*N lanes.  Then
 *   loss[l]         = scale * ((((0 + t_0) + t_1) + ...) + t_{N-1})
 *   grad[l*ld_g+p]  = scale * ((((0 + g_0p) + g_1p) + ...) + g_{N-1,p})
 * with t_i and g_i the term and its gradient along lane (l, i)'s realized
 * trace: a left fold over the points in ascending order, then one
 * multiplication (a second, small kernel on `stream`).
 *   params : device fp64, element (l, p) at params[l*ld_p + p], ld_p >= P
 *   points : device fp64, observation k of point i at points[i*ld_pt + k],
 *            ld_pt >= the tape's n_obs
 *   loss   : device fp64 [L];  grad : element (l, p) at grad[l*ld_g + p]
 *   workspace : ndvm_workspace_bytes_points(tape, L, n_points) bytes (the
 *               replay's rows for L*N lanes plus the per-point terms and term
 *               gradients); that call prepares the launch and must precede
 * L = 0 is a no-op.  Errors: NDVM_E_ARG (null tape or buffer, L < 0,
 * n_points < 1, a stride too small, L*N overflowing, a lane count never
 * prepared), NDVM_E_NOMEM (workspace too small), NDVM_E_DEVICE.
 */
ndvm_status ndvm_grad_points(const ndvm_tape *tape, const double *params, int64_t L, int64_t ld_p,
                             const double *points, int64_t n_points, int64_t ld_pt, double scale, double *loss,
                             double *grad, int64_t ld_g, void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes of ndvm_grad_points for L parameter vectors and n_points
 * data points; the preparation call of that launch shape (schedules the term
 * program for L*n_points lanes and copies it to the GPU).  Library
 * infrastructure.  Errors: NDVM_E_ARG, NDVM_E_NOMEM, NDVM_E_DEVICE,
 * NDVM_E_UNSUPPORTED. */
ndvm_status ndvm_workspace_bytes_points(const ndvm_tape *tape, int64_t L, int64_t n_points, size_t *bytes);

/*
 * Many programs in one launch (candidate-level parallelism of Section 6,
 * "Across cores", mapped onto the GPU grid): program q uses
 *   params : params + q*prog_stride_p, element (l, p) at [l*ld_p + p]
 *   loss   : loss + q*L
 *   grad   : grad + q*prog_stride_g, element (l, p) at [l*ld_g + p]
 * All programs read the same obs[n_obs] and must declare that n_obs; ld_p and
 * ld_g must cover the largest P.  Workspace: ndvm_workspace_bytes_many, which
 * must have been called for the same program list and L (else NDVM_E_ARG).
 * More than 65,535 programs are enqueued as several launches on `stream`.
 * Errors: as ndvm_grad, plus NDVM_E_ARG for n_prog < 0, a null tape or
 * program strides smaller than L*ld_p / L*ld_g.
 */
ndvm_status ndvm_grad_many(const ndvm_tape *const *tapes, int n_prog, const double *params,
                           int64_t L, int64_t ld_p, int64_t prog_stride_p, const double *obs,
                           int64_t n_obs, double *loss, double *grad, int64_t ld_g,
                           int64_t prog_stride_g, void *workspace, size_t workspace_bytes,
                           void *stream);

/* Workspace bytes for ndvm_grad_many; the preparation call of a program set
 * and lane count (schedules every program for the launch's register budget
 * and copies the programs and the launch's program table to the GPU).
 * Errors: NDVM_E_ARG, NDVM_E_NOMEM, NDVM_E_DEVICE, NDVM_E_UNSUPPORTED. */
ndvm_status ndvm_workspace_bytes_many(const ndvm_tape *const *tapes, int n_prog, int64_t L,
                                      size_t *bytes);

/*
 * Device walker (Section 9, "What remains designed and unbuilt", and
 * Appendix A: the structural walk on the device under wave-ballot lane
 * masks; Section 3.4 define-by-run tape; Section 6 lane masking; Appendix C
 * adjoints).  No tape is built and nothing is scheduled on the host: the
 * host only validates the bytecode and measures its structure (stack depth,
 * locals, nesting, a bound on the nodes a walk records) without unrolling
 * it, then copies the program set to the GPU once.  One wave walks a program
 * for 64 lanes; a numeric IFLT runs each arm under the mask of the lanes that
 * take it (one ballot; an arm no lane takes is not walked) and merges what
 * the two arms left different, per lane.  Per lane the result is the loss
 * and exact gradient of that lane's realized trace (Section 4, Property 1),
 * the values ndvm_grad returns for the same program.
 *
 * Scalar programs only: bytecode with a matrix word (DOT, MATMUL, TRANSPOSE,
 * INV, DET, LOGDET, TRACE, OUTER, PACK, INDEX) is NDVM_E_UNSUPPORTED.  Every
 * IFLT's arms must leave the same stack depth and set the same locals
 * (NDVM_E_STRUCT_DIVERGE), also where both operands are constants (the tape
 * path resolves such a branch on the host and accepts any arms).
 */
typedef struct ndvm_walk ndvm_walk;

/* Validate `n_prog` bytecode programs (bytecodes[q], lens[q] bytes each, all
 * with the same observation count) and copy them to the current device on
 * `stream` (synchronised before returning).  *out receives a handle owned by
 * the library (ndvm_walk_free).  Errors: NDVM_E_ARG (null pointers, n_prog
 * <= 0, differing observation counts), NDVM_E_BYTECODE, NDVM_E_STRUCT_DIVERGE,
 * NDVM_E_UNSUPPORTED (matrix words; limits: stack depth 64, 32 locals,
 * nesting 32, 2^24 nodes, and the wave's structural state -- value rows of
 * the parameters and of the stack and locals, node numbers, frames and two
 * flag bits per node -- within 64 KiB of LDS), NDVM_E_NOMEM, NDVM_E_DEVICE;
 * the message names the program. */
ndvm_status ndvm_walk_prepare(const uint8_t *const *bytecodes, const size_t *lens, int n_prog, void *stream,
                              ndvm_walk **out);

typedef struct {
    uint32_t n_params, n_obs;
    uint64_t n_nodes;     /* bound on the nodes one wave's walk records (parameters included) */
    uint32_t depth;       /* largest operand stack depth */
    uint32_t n_locals;    /* locals referenced */
    uint32_t n_frames;    /* deepest IFLT nesting */
    uint32_t n_loops;     /* deepest LOOP nesting */
} ndvm_walk_info;

/* Host only: the validation and structural measurement ndvm_walk_prepare
 * applies to one program, without touching a device.  Library
 * infrastructure.  Errors: as ndvm_walk_prepare for one program. */
ndvm_status ndvm_walk_measure(const uint8_t *bytecode, size_t len, ndvm_walk_info *out);

/* Workspace bytes of ndvm_walk_grad for L lanes per program: a status word
 * and, per wave slot of the launch (enough waves to fill the GPU, at most one
 * per 64 lanes of every program), 1,048 bytes per node the largest program
 * can record (values and adjoints of 64 lanes, the node record).  Host only.
 * Errors: NDVM_E_ARG. */
ndvm_status ndvm_walk_workspace_bytes(const ndvm_walk *w, int64_t L, size_t *bytes);

/* The walk of every program of the set for L lanes each, on `stream`.
 * params: program q, lane l, parameter p at params[q*prog_stride_p + l*ld_p
 * + p]; ld_p and ld_g at least the largest parameter count; the strides are
 * read only when the set has more than one program.  obs[n_obs] is shared.
 * loss[q*L + l]; grad as params with ld_g, prog_stride_g (columns beyond a
 * program's own parameter count are not written).  workspace: device memory
 * of ndvm_walk_workspace_bytes bytes (its status word is cleared on
 * `stream`).  Enqueues only.  Errors: NDVM_E_ARG (null pointers, L < 0,
 * n_obs mismatch, leading dimensions or strides too small, another current
 * device), NDVM_E_NOMEM (workspace too small), NDVM_E_DEVICE. */
ndvm_status ndvm_walk_grad(const ndvm_walk *w, const double *params, int64_t L, int64_t ld_p,
                           int64_t prog_stride_p, const double *obs, int64_t n_obs, double *loss, double *grad,
                           int64_t ld_g, int64_t prog_stride_g, void *workspace, size_t workspace_bytes,
                           void *stream);

/* Synchronise `stream` and read the status word of a workspace ndvm_walk_grad
 * used: NDVM_E_INTERNAL if a wave met a bound the validation should have
 * excluded (its lanes then hold NaN), else NDVM_OK.  Library
 * infrastructure.  Errors: NDVM_E_ARG, NDVM_E_DEVICE, NDVM_E_INTERNAL. */
ndvm_status ndvm_walk_status(const void *workspace, void *stream);

/* Release a walker program set (NULL is ignored); as ndvm_tape_free. */
void ndvm_walk_free(ndvm_walk *w);

/* Release a tape handle (NULL is ignored).  Waits for nothing: the caller
 * must not free a tape while work that uses it is still pending. */
void ndvm_tape_free(ndvm_tape *tape);

/* Release memory returned by ndvm_tape_build (NULL is ignored). */
void ndvm_free(void *p);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char *ndvm_last_error(void);

/*
 * One Adam step for a population of parameter vectors (calibration: an
 * optimiser fits every lane's parameters with the exact gradients of
 * ndvm_grad, as in the paper's Kalman maximum-likelihood fit, Section "From
 * buckets to phases").  Adam with bias correction (Kingma and Ba, 2015):
 *   m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g*g;
 *   p = p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * evaluated in that order in fp64; beta1^t and beta2^t are computed on the
 * host with pow.
 *   params : device fp64, element (l, k) at params[l*ld_p + k], updated in place
 *   grad   : device fp64, element (l, k) at grad[l*ld_g + k] (ndvm_grad's output)
 *   m, v   : device fp64 moment buffers, [L, P] contiguous, zero before step t = 1;
 *            owned by the caller, updated in place
 *   t      : step number, >= 1
 * Errors (synchronous): NDVM_E_ARG for a null buffer with L*P > 0, L < 0, P < 0,
 * ld_p < P, ld_g < P, t < 1, or beta1, beta2 outside [0, 1); NDVM_E_DEVICE for a
 * launch failure.
 */
ndvm_status ndvm_adam_step(double *params, const double *grad, double *m, double *v, int64_t L, int64_t P,
                           int64_t ld_p, int64_t ld_g, int64_t t, double lr, double beta1, double beta2,
                           double eps, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* NDVM_H */
