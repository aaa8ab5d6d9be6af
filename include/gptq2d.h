/*
 * gptq2d.h -- C ABI of the MI355X (gfx950) GPTQ-2D library.
 *
 * Two-sided adaptive rounding (Chen, Hoefler, Alistarh, "GPTQ-2D: Cubic-Time
 * Two-Sided Adaptive Rounding", arXiv 2607.27042). Given a real matrix X
 * (m x n) and nonsingular bases A (m x m) and B (n x n), the library rounds X
 * to an integer matrix Z under the metric ||A (Z - X) B||_F^2 (Sec. 3.2,
 * Eq. objective) with the greedy fixed-order trajectory of one-dimensional
 * adaptive rounding (Algorithm 1) on the column-major vectorisation of X,
 * computed anti-diagonal by anti-diagonal (Sec. 4.2, Algorithm 3; blocked as
 * in Sec. 4.3, Algorithm 4). Theorem 2 makes the result identical to the
 * vectorised sweep.
 *
 * Conventions shared by every entry point
 *   - Matrices are row-major with a leading dimension counted in elements
 *     (ld >= number of columns).
 *   - Matrix pointers are DEVICE pointers on the current HIP device, unless an
 *     argument says "host".
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream). Work
 *     is enqueued on it; calls return before the GPU finishes unless a call is
 *     documented to synchronise.
 *   - Every call returns a gptq2d_status; nothing throws across the ABI. On an
 *     error, gptq2d_last_error() returns a message for the calling thread.
 *   - Internally all factors and all accumulation are in double precision,
 *     whatever the input type; GPTQ2D_F32 only selects the type of X, A, B and
 *     of the returned corrected values.
 *   - Rounding breaks ties to even (the paper asks for any deterministic rule,
 *     Theorem 1).
 */
#ifndef GPTQ2D_H
#define GPTQ2D_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gptq2d_factors_s* gptq2d_factors_t; /* opaque factor handle */

typedef enum { GPTQ2D_F32 = 0, GPTQ2D_F64 = 1 } gptq2d_dtype;

typedef enum {
  GPTQ2D_OK = 0,
  GPTQ2D_ERR_INVALID_ARG = -1, /* bad shape, stride, pointer or dtype */
  GPTQ2D_ERR_SINGULAR = -2,    /* A or B singular: a Gram pivot was not positive and finite */
  GPTQ2D_ERR_NONFINITE = -3,   /* X held a NaN or an infinity */
  GPTQ2D_ERR_OOM = -4,         /* device allocation failed */
  GPTQ2D_ERR_HIP = -5,         /* a HIP runtime call failed */
  GPTQ2D_ERR_WORKSPACE = -6,   /* workspace missing or too small */
  GPTQ2D_ERR_OVERFLOW = -7,    /* a rounded value does not fit in int32 */
  GPTQ2D_ERR_TIMEOUT = -8      /* an internal wait between waves exceeded its bound */
} gptq2d_status;

/* ---------------------------------------------------------------------------
 * Factor handle: L, U and the diagonal scales of the two inverse Grams.
 *
 * The feedback factors are fixed by the bases (Sec. 3.1 and Sec. 4.1):
 *   G = A^T A,  H = B B^T                                     (Eq. GH)
 *   G^{-1} = L diag(lamL) L^T,  L unit lower triangular
 *   H^{-1} = U^T diag(lamU) U,  U unit upper triangular
 * They are computed once and reused for any number of X (Sec. 4.2: the
 * one-time factorisation). A handle owns its device storage until
 * gptq2d_factors_destroy; it is immutable while gptq2d_round uses it.
 * ------------------------------------------------------------------------- */

/* Allocates device storage for an m x n problem on the current device.
 * 1 <= m, n <= 65536. *out receives the handle. Errors: INVALID_ARG, OOM. */
gptq2d_status gptq2d_factors_create(int m, int n, gptq2d_factors_t* out);

/* Frees the handle (NULL is ignored). The caller must ensure no enqueued work
 * still uses it. */
void gptq2d_factors_destroy(gptq2d_factors_t f);

/* Problem shape of a handle. */
gptq2d_status gptq2d_factors_shape(gptq2d_factors_t f, int* m, int* n);

/* Rounding order of handle f. The paper's sweep visits vec(X) from its first
 * entry on (GPTQ's direction); Sec. 2 notes that YAQA rounds in the opposite
 * direction, from the last column on. reverse = 0 (the default) selects the
 * first, reverse != 0 the second: the entries are visited in the reverse of
 * the forward order, which is the forward sweep of the index-reversed problem
 * (P X P, A P, P B; P the reversal permutation of matching size) with its Z
 * and Y reversed back. Z, Y and the objective are returned in X's own
 * indexing either way. The factors a handle holds belong to its order: in
 * reverse order they are those of the index-reversed problem, and
 * gptq2d_factors_export / gptq2d_factors_import exchange them in that form.
 * Set the order before gptq2d_factor_compute or gptq2d_factors_import;
 * factors already in the handle are not converted. Enqueues nothing.
 * Errors: INVALID_ARG on a NULL handle. */
gptq2d_status gptq2d_factors_set_order(gptq2d_factors_t f, int reverse);

/* Enqueues the factorisation of A (m x m, lda) and B (n x n, ldb), both of
 * type dt, into f: Gram formation, Cholesky of the index-reversed Grams,
 * triangular inversion and normalisation (the LDL factors of the inverse
 * Grams, Sec. 3.1 / first two steps of Algorithm 3). Allocates nothing and
 * does not synchronise; a pivot failure is recorded on the device and
 * reported by gptq2d_factor_check. A and B are only read. */
gptq2d_status gptq2d_factor_compute(gptq2d_factors_t f, gptq2d_dtype dt, const void* A,
                                    int64_t lda, const void* B, int64_t ldb, void* stream);

/* Synchronises `stream` and returns SINGULAR if the last factorisation into f
 * met a non-positive or non-finite pivot, OK otherwise. */
gptq2d_status gptq2d_factor_check(gptq2d_factors_t f, void* stream);

/* Bytes of device workspace gptq2d_factor_batched needs for `count` problems
 * (0 if count < 1). */
size_t gptq2d_factor_batched_workspace_size(int count);

/* Enqueues the factorisation of `count` problems at once: problem p as
 * gptq2d_factor_compute(f[p], dt, A[p], lda[p], B[p], ldb[p], stream) would,
 * with the same bits. f, A, lda, B, ldb are host arrays (A[p], B[p] device
 * pointers); a handle may appear only once. Problems of one shape (m, n) are
 * factorised in common launches: every step of the factorisation runs for
 * all of them in one launch, so small problems, whose factorisation is a
 * chain of short launches, share each launch instead of queueing. Groups of
 * different shapes run side by side, each on a stream of the group's first
 * handle (created on its first batched use), ordered after the work already
 * on `stream`; `stream` then waits for all of them. workspace: device memory
 * of at least gptq2d_factor_batched_workspace_size(count) bytes, 256-byte
 * aligned, owned by the caller (the batch's argument table); overlapping
 * calls need distinct workspaces. Allocates no device memory; does not
 * synchronise. Errors: INVALID_ARG, WORKSPACE, HIP. */
gptq2d_status gptq2d_factor_batched(int count, const gptq2d_factors_t* f, gptq2d_dtype dt,
                                    const void* const* A, const int64_t* lda, const void* const* B,
                                    const int64_t* ldb, void* workspace, size_t ws_bytes,
                                    void* stream);

/* Synchronises `stream` and returns SINGULAR if the last factorisation of any
 * of the handles f[0 .. count-1] met a non-positive or non-finite pivot. */
gptq2d_status gptq2d_factor_batched_check(int count, const gptq2d_factors_t* f, void* stream);

/* Convenience: create + compute + check (one synchronisation). On error no
 * handle is returned. */
gptq2d_status gptq2d_factor(int m, int n, gptq2d_dtype dt, const void* A, int64_t lda,
                            const void* B, int64_t ldb, void* stream, gptq2d_factors_t* out);

/* Copies the factors to caller memory (device pointers, fp64): L (m x m,
 * ldl), U (n x n, ldu), lamL (m), lamU (n). Any pointer may be NULL to skip
 * it. Enqueued on `stream`. */
gptq2d_status gptq2d_factors_export(gptq2d_factors_t f, double* L, int64_t ldl, double* U,
                                    int64_t ldu, double* lamL, double* lamU, void* stream);

/* Loads factors computed elsewhere (device pointers, fp64) into f, replacing
 * its contents: L unit lower (m x m), U unit upper (n x n), lamL, lamU > 0.
 * Only the strictly lower part of L and strictly upper part of U are read;
 * their diagonals are taken as one. Enqueued on `stream`. */
gptq2d_status gptq2d_factors_import(gptq2d_factors_t f, const double* L, int64_t ldl,
                                    const double* U, int64_t ldu, const double* lamL,
                                    const double* lamU, void* stream);

/* ---------------------------------------------------------------------------
 * Rounding sweep (Sec. 4.2, Algorithm 3, blocked as Algorithm 4).
 * ------------------------------------------------------------------------- */

/* Bytes of device workspace gptq2d_round needs for handle f (0 on a NULL
 * handle). */
size_t gptq2d_round_workspace_size(gptq2d_factors_t f);

/* Enqueues the rounding of X (m x n, type dt, ldx) with the factors in f.
 *   Z   (required, int32, m x n, ldz): the rounded matrix.
 *   Y   (nullable, type dt, m x n, ldy): the corrected value of every entry at
 *       the moment it was rounded (Algorithm 3's Y); Z = rint(Y).
 *   objective (nullable, device fp64 scalar): ||A (Z - X) B||_F^2, evaluated
 *       as sum_ij (Z - Y)_ij^2 / (lamL_i lamU_j), which equals the objective
 *       for the factors in f (Z - X = L E U with E = Z - Y, Eq. Y-LEU).
 *   workspace: device memory of at least gptq2d_round_workspace_size(f)
 *       bytes, 256-byte aligned, owned by the caller; it holds the deferred
 *       feedback buffers and the error flags. Concurrent calls need distinct
 *       workspaces and outputs.
 * Asynchronous: a non-finite X or an int32 overflow is recorded in the
 * workspace and reported by gptq2d_round_check. */
gptq2d_status gptq2d_round(gptq2d_factors_t f, gptq2d_dtype dt, const void* X, int64_t ldx,
                           int32_t* Z, int64_t ldz, void* Y, int64_t ldy, double* objective,
                           void* workspace, size_t ws_bytes, void* stream);

/* Synchronises `stream` and returns NONFINITE, OVERFLOW or TIMEOUT if the
 * last gptq2d_round that used `workspace` met one, OK otherwise. */
gptq2d_status gptq2d_round_check(gptq2d_factors_t f, const void* workspace, void* stream);

/* gptq2d_round for callers that cannot allocate (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same kernels and
 * results as gptq2d_round(f, dt, X, ldx, Z, ldz, Y, ldy, objective, ...), but
 * the workspace is a fixed 64 MiB array of device memory inside the library
 * (one per device, held from the first use on that device until the process
 * ends), so the caller passes no workspace and the call allocates nothing.
 *   status_word (required, device int32, owned by the caller): the error bits
 *       of this call; gptq2d_round_check(f, status_word, stream) turns them
 *       into NONFINITE, OVERFLOW or TIMEOUT as for gptq2d_round.
 * Limit: gptq2d_round_workspace_size(f) <= 64 MiB, about 4 x 8 bytes per
 * entry of X padded to multiples of 64 (e.g. up to 1408 x 1408 or 1024 x
 * 2048); a larger problem returns WORKSPACE with the sizes in the message.
 * All calls on one device share that device's array: calls that overlap in
 * time on one device (two streams, two threads) race and give wrong results;
 * calls in one stream order are safe, each overwrites what the last one
 * left. Stage-launch timing (gptq2d_stage_timing) is ignored. Errors:
 * INVALID_ARG, WORKSPACE, HIP. */
gptq2d_status gptq2d_round_noalloc(gptq2d_factors_t f, gptq2d_dtype dt, const void* X, int64_t ldx,
                                   int32_t* Z, int64_t ldz, void* Y, int64_t ldy, double* objective,
                                   int32_t* status_word, void* stream);

/* ---------------------------------------------------------------------------
 * Batched rounding: many independent problems (the layers of a model, Sec. 6)
 * in common launches. Stage k of every problem runs in one launch, so small
 * problems, which occupy a few compute units each, share the device instead
 * of running one after another.
 * ------------------------------------------------------------------------- */

/* Bytes of device workspace gptq2d_round_batched needs for the handles
 * f[0 .. count-1] (a host array; a handle may appear more than once). 0 if
 * count < 1, f is NULL or a handle is NULL. */
size_t gptq2d_round_batched_workspace_size(int count, const gptq2d_factors_t* f);

/* Enqueues the rounding of `count` problems, problem p exactly as
 * gptq2d_round(f[p], dt, X[p], ldx[p], Z[p], ldz[p], Y[p], ldy[p], ...) would
 * round it (the same kernels on the same data: identical Z, Y and objective).
 *   f, X, ldx, Z, ldz: host arrays of `count` entries; X[p] and Z[p] are device
 *       pointers (m_p x n_p, as for gptq2d_round); every problem has type dt.
 *   Y, ldy: host arrays of `count` entries, or both NULL (no corrected values);
 *       an entry Y[p] may be NULL.
 *   objective: NULL, or a device array of `count` doubles (problem p's
 *       objective in objective[p]).
 *   workspace: device memory of at least gptq2d_round_batched_workspace_size
 *       bytes for the same handles, 256-byte aligned, owned by the caller.
 *       Calls that overlap need distinct workspaces and outputs; the host
 *       arrays may be reused as soon as the call returns.
 * 1 <= count; handles may repeat (problems that share their bases). Errors:
 * INVALID_ARG, WORKSPACE, HIP. A non-finite X or an int32 overflow in any
 * problem is recorded in the workspace and reported by
 * gptq2d_round_batched_check. */
gptq2d_status gptq2d_round_batched(int count, const gptq2d_factors_t* f, gptq2d_dtype dt,
                                   const void* const* X, const int64_t* ldx, int32_t* const* Z,
                                   const int64_t* ldz, void* const* Y, const int64_t* ldy,
                                   double* objective, void* workspace, size_t ws_bytes,
                                   void* stream);

/* Synchronises `stream` and returns NONFINITE, OVERFLOW or TIMEOUT (in that
 * order of precedence) if any problem of the last gptq2d_round_batched that
 * used `workspace` met one, OK otherwise. The flags are the batch's, not a
 * problem's: to find the problem, round it on its own. */
gptq2d_status gptq2d_round_batched_check(const void* workspace, void* stream);

/* ---------------------------------------------------------------------------
 * Diagnostics
 * ------------------------------------------------------------------------- */

/* Static description of a status code. */
const char* gptq2d_status_string(gptq2d_status s);

/* Detail message of the last failing call on this thread ("" if none). */
const char* gptq2d_last_error(void);

/* Library version as 10000*major + 100*minor + patch. */
int gptq2d_version(void);

/* Launch timing of the sweep's stage kernel. With enable != 0, every later
 * gptq2d_round on f times each stage-kernel launch on the round's stream with
 * two HIP events that take the dispatch's own start and end time stamps (the
 * library creates them on first use and keeps them until
 * gptq2d_factors_destroy); enable = 0 stops recording.
 * Either call discards the pairs not yet read. Not for concurrent rounds on
 * one handle. Errors: INVALID_ARG. */
gptq2d_status gptq2d_stage_timing(gptq2d_factors_t f, int enable);

/* Waits for the last recorded pair and returns, over all launches bracketed
 * since the last read, the summed launch time in milliseconds (*total_ms) and
 * the number of launches (*launches); either pointer may be NULL. Resets the
 * record. Errors: INVALID_ARG, HIP. */
gptq2d_status gptq2d_stage_time(gptq2d_factors_t f, double* total_ms, int64_t* launches);

/* Host-only view of the deferred-feedback delivery plan of the sweep (the
 * lazy block update of Sec. 4.3 on 64 x 64 tiles), for inspection and tests;
 * touches no device. Tiles: MT = ceil(m/64) rows, NT = ceil(n/64) columns;
 * launch k (0 <= k < MT+NT-1) sweeps the tiles with I + J = k. Each task is
 * four int32 {dir | overwrite << 1 | (rows-1) << 2 | (cols-1) << 3,
 * first target tile row, first target tile column,
 * first source | (one past the last source) << 16}: it adds, to the block of
 * rows x cols target tiles (1 or 2 each), the product over source tiles s of
 * L[I][s] E[s][J] (dir 0, down buffer) or C[I][s] U[s][J] (dir 1, right
 * buffer). offsets (host, MT+NT entries, nullable) receives the first task
 * of every launch and the total; tasks (host, 4*cap int32, nullable) the
 * first cap tasks in launch order. g is the batch width in source tiles of
 * the far deliveries (g >= 1). Returns the task count, or -1 on a bad
 * argument. */
int64_t gptq2d_schedule_tasks(int m, int n, int g, int32_t* tasks, int64_t cap,
                              int32_t* offsets);

/* Host-only view of which tiles each launch of the sweep rounds (Fig. 1 at
 * the level of 64 x 64 tiles: the tiles of one tile anti-diagonal depend on
 * none of each other, Sec. 4.2); touches no device. Launch k sweeps tile rows
 * rows[2k] .. rows[2k+1] (host, 2*cap int32, nullable; filled for k < cap),
 * row I at tile column k - I. Returns the number of launches MT + NT - 1, or
 * -1 on a bad shape (1 <= m, n <= 65536) or a negative cap. */
int64_t gptq2d_schedule_sweeps(int m, int n, int32_t* rows, int64_t cap);

#ifdef __cplusplus
}
#endif

#endif /* GPTQ2D_H */
