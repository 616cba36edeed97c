/*
 * polyglot.h -- C ABI of the MI355X (gfx950) library for the minibatch SGD
 * step of the Polyglot window-ranking language model.
 *
 * Method.  Kulkarni, Al-Rfou, Perozzi, Skiena, "Exploring the power of GPU's
 * for training Polyglot language models" (arXiv:1404.1521).  The paper trains
 * the Polyglot model, a SENNA-like ranking language model (§1 Introduction),
 * with minibatch SGD (batch size discussion, §4.6), and finds that the
 * embedding-gradient update -- the "advanced indexing" increment that adds
 * row k of Y to row I[k] of W for every k (§4.2, Table 1:
 * GpuAdvancedIncSubtensor1) -- dominates training time; §4.3 replaces it
 * with a parallel kernel.  The paper does not write the model out; this
 * library implements the SENNA-style window ranker:
 *
 *   x     = concat(E[w_0] .. E[w_{win-1}])          K = win*d values
 *   x~    = x with block c = win/2 replaced by E[corrupt]
 *   s(x)  = w2 . tanh(W1 x + b1) + b2
 *   loss  = (1/B) sum_b max(0, 1 - s(x_b) + s(x~_b))
 *
 * and one SGD step P <- P - lr * dloss/dP over E, W1, b1, w2, b2, all
 * gradients taken at the pre-step parameters.  The hinge derivative at a
 * margin of exactly 0 is taken as 0.  A corrupt id equal to the true centre
 * is used as drawn (its gradient cancels).
 *
 * Conventions for every entry point.
 *   - All tensor arguments are DEVICE pointers (hipMalloc / torch CUDA
 *     tensors on the device the context was created on), C-contiguous,
 *     row-major, float32 or int32, owned by the caller.  The library never
 *     frees or retains them after the call returns.
 *   - Work is enqueued asynchronously on the context's HIP stream; the
 *     caller must synchronise that stream before reading results on the
 *     host or touching the buffers from another stream.
 *   - Return value: POLYGLOT_OK (0) or a negative POLYGLOT_E* code.  Errors
 *     that the host can detect (bad sizes, NULL pointers, non-finite lr,
 *     batch above the configured maximum) are returned before anything is
 *     enqueued.  Ids outside [0, V) are detected on the device: the step
 *     then modifies no parameter, writes NaN to its loss slot, and raises a
 *     sticky flag that polyglot_status() reports as POLYGLOT_EID.
 *   - A context is not thread-safe and must be used from one host thread
 *     and one stream at a time.
 *
 * Layouts (int32 ids, float32 values):
 *   E[V][d]  W1[H][win*d]  b1[H]  w2[H]  b2[1]
 *   windows[B][win] (centre at win/2)  corrupt[B]
 */
#ifndef POLYGLOT_H
#define POLYGLOT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define POLYGLOT_OK 0
#define POLYGLOT_EINVAL -1 /* bad dimension, even window, non-finite lr, bad mode */
#define POLYGLOT_ENULL -2  /* a required pointer is NULL */
#define POLYGLOT_EBATCH -3 /* B or N <= 0, or above the context's maximum */
#define POLYGLOT_EHIP -4   /* HIP runtime error; text in polyglot_last_error() */
#define POLYGLOT_EID -5    /* an id was outside [0, V) (reported by polyglot_status) */
#define POLYGLOT_ESTATE -6 /* call not valid in the context's current state */

/* How the embedding-gradient rows are added into the table (§4.3). */
#define POLYGLOT_SCATTER_SORTED 0 /* stable radix sort by row id, segmented sum: deterministic */
#define POLYGLOT_SCATTER_ATOMIC 1 /* one float atomic add per (entry, column): order-dependent rounding */

typedef struct polyglot_ctx polyglot_ctx;

typedef struct {
  int32_t V;            /* vocabulary rows of E, >= 1 */
  int32_t d;            /* embedding width, multiple of 16, 16..256; for H <= 64,
                           W1 (H x win*d floats) must also fit one workgroup's LDS */
  int32_t win;          /* window length, odd, 1..31 */
  int32_t H;            /* hidden units: 1..64, or a multiple of 64 up to 256 with d a
                           multiple of 64 (wide layers run as three separate
                           contractions: forward, dW1, per-entry gradient rows) */
  int32_t max_batch;    /* largest B accepted by train_step / score / gather */
  int32_t scatter_mode; /* POLYGLOT_SCATTER_SORTED or POLYGLOT_SCATTER_ATOMIC */
  int32_t max_scatter;  /* largest N accepted by polyglot_scatter_add (0: no workspace) */
  int32_t max_rows;     /* largest table row count for polyglot_scatter_add */
} polyglot_config;

/* Creates a context on the current HIP device.  `stream` is a hipStream_t
 * (NULL = the legacy default stream).  All workspace is allocated here, once,
 * sized for cfg->max_batch and cfg->max_scatter; no call below allocates.
 * On success *out receives the context; on error *out is left NULL. */
int polyglot_init(const polyglot_config* cfg, void* stream, polyglot_ctx** out);

/* Waits for the context's stream, frees its workspace and the context. */
int polyglot_destroy(polyglot_ctx* ctx);

/* Replaces the stream the context enqueues on (hipStream_t, NULL = default). */
int polyglot_set_stream(polyglot_ctx* ctx, void* stream);

/* One SGD step of the window-ranking model (model above; the embedding
 * update is the row scatter-add of §4.2/§4.3), in place on E, W1, b1, w2,
 * b2.  windows[B][win] and corrupt[B] are int32 ids in [0, V).  lr is the
 * SGD learning rate.  loss_dev, if not NULL, is a device float that
 * receives the mean hinge loss at the pre-step parameters (NaN if an id was
 * out of range).  1 <= B <= max_batch. */
int polyglot_train_step(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2, float* b2,
                        const int32_t* windows, const int32_t* corrupt, int32_t B, float lr,
                        float* loss_dev);

/* polyglot_train_step followed by a synchronisation: the step is enqueued on
 * the context's stream with its loss in a library-owned device slot, the
 * stream is synchronised, and the mean hinge loss (the quantity of the
 * model above, at the pre-step parameters) is written to *loss_host (host
 * memory, caller-owned).  Returns what polyglot_train_step returns for the
 * arguments (nothing is enqueued on such an error and *loss_host is left
 * unchanged); POLYGLOT_EHIP if the synchronisation fails; POLYGLOT_EID if a
 * device error word is raised once the step has run, in which case the step
 * changed no parameter and *loss_host is NaN.  The error words stay raised
 * (every later step is void) until polyglot_status() clears them. */
int polyglot_train_step_sync(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2,
                             float* b2, const int32_t* windows, const int32_t* corrupt,
                             int32_t B, float lr, float* loss_host);

/* S consecutive SGD steps, step s using windows + s*B*win and corrupt + s*B,
 * exactly as S calls of polyglot_train_step.  losses_dev[S] (device, may be
 * NULL) receives each step's loss.  The launches of the S steps are recorded
 * once into a HIP graph that the context caches (keyed on every argument)
 * and replays, which removes per-kernel host launch cost. */
int polyglot_train_steps(polyglot_ctx* ctx, float* E, float* W1, float* b1, float* w2,
                         float* b2, const int32_t* windows, const int32_t* corrupt, int32_t S,
                         int32_t B, float lr, float* losses_dev);

/* The score of the ranking model of §1 Introduction (the SENNA-like
 * network the paper trains), s(x) = w2 . tanh(W1 x + b1) + b2, of each of
 * the B windows: x = concat_j E[windows[b][j]].  windows[B][win] int32
 * (device), scores_dev[B] float32 (device, written).  A window holding an
 * out-of-range id scores NaN and raises the sticky flag.  1 <= B <= max_batch;
 * E and W1 16-byte aligned (else POLYGLOT_EINVAL). */
int polyglot_score(polyglot_ctx* ctx, const float* E, const float* W1, const float* b1,
                   const float* w2, const float* b2, const int32_t* windows, int32_t B,
                   float* scores_dev);

/* The window gather on its own: the input vector x of the §1 Introduction
 * model, the concatenation of the window's embedding rows, for every
 * window, X[B][win*d] = concat_j E[windows[b][j]], and the corrupted centre
 * rows Xc[B][d] = E[corrupt[b]] (bit-exact copies; a row with an
 * out-of-range id is written as NaN and raises the sticky flag).  All
 * pointers device; E, X and Xc 16-byte aligned; 1 <= B <= max_batch. */
int polyglot_gather(polyglot_ctx* ctx, const float* E, const int32_t* windows,
                    const int32_t* corrupt, int32_t B, float* X, float* Xc);

/* The advanced-indexing increment of §4.2/§4.3: for every k in [0, N),
 * table[idx[k]] += alpha * Y[k], where repeated indices accumulate.
 * table[rows][d], idx[N] int32 in [0, rows), Y[N][d].  mode selects the
 * sorted-segment or the atomic algorithm.  N <= max_scatter,
 * rows <= max_rows, d a multiple of 4 up to 256.  Out-of-range indices
 * leave the table untouched and raise the sticky flag. */
int polyglot_scatter_add(polyglot_ctx* ctx, float* table, int32_t rows, int32_t d,
                         const int32_t* idx, const float* Y, int32_t N, float alpha,
                         int32_t mode);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the sorted
 * mode of polyglot_scatter_add -- table[idx[k]] += alpha * Y[k] for every k in
 * [0, N), repeated indices accumulated in entry order, each touched row
 * written once -- with no context.  It allocates nothing: its sort buffers
 * live in a static device array of POLYGLOT_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends.
 *   table[rows][d], Y[N][d] float32 and idx[N] int32: device pointers owned by
 *     the caller; table and Y 16-byte aligned; d a multiple of 4 up to 256;
 *     1 <= rows <= POLYGLOT_NOALLOC_MAX_ROWS.
 *   1 <= N <= POLYGLOT_NOALLOC_MAX_N, else POLYGLOT_EBATCH.
 *   status_dev: device int32 (may be NULL), written on the device with
 *     POLYGLOT_OK, or POLYGLOT_EID when an index is outside [0, rows), in
 *     which case the call leaves the table untouched.  Nothing is sticky:
 *     every call starts clean.
 *   stream: hipStream_t the two launches go on (NULL = the default stream).
 * Returns POLYGLOT_OK once enqueued, POLYGLOT_ENULL, POLYGLOT_EBATCH,
 * POLYGLOT_EINVAL (rows, d, alignment, non-finite alpha) before anything is
 * enqueued, or POLYGLOT_EHIP.  All calls on one GPU share its scratch array:
 * calls that may overlap in time on one GPU (several streams or host
 * threads) race and must be serialised by the caller. */
#define POLYGLOT_NOALLOC_MAX_N 8192
#define POLYGLOT_NOALLOC_MAX_ROWS (1 << 26)
#define POLYGLOT_NOALLOC_SCRATCH_BYTES 66816
int polyglot_scatter_add_noalloc(float* table, int32_t rows, int32_t d, const int32_t* idx,
                                 const float* Y, int32_t N, float alpha, int32_t* status_dev,
                                 void* stream);

/* Storage formats and operations of polyglot_scatter_update. */
#define POLYGLOT_F32 0  /* IEEE binary32 */
#define POLYGLOT_BF16 1 /* bfloat16: the upper 16 bits of a binary32 */
#define POLYGLOT_F16 2  /* IEEE binary16 */
#define POLYGLOT_OP_INC 0 /* table[idx[k]] += alpha * Y[k] */
#define POLYGLOT_OP_SET 1 /* table[idx[k]] = Y[k]; alpha unused */

/* The general advanced-indexing op of §4.3 (the increment the paper
 * rewrites, in the library form it contributes: any table format, any
 * index vector, increment or assignment).
 *   table[rows][d] and Y[N][d]: device, row-major, both in storage format
 *     dtype; d in [1, 256]; aligned to their element size.
 *   idx[N]: device, int32 (idx_bytes 4) or int64 (idx_bytes 8), each in
 *     [0, rows); aligned to idx_bytes.
 *   op POLYGLOT_OP_INC: for every k, table[idx[k]] += alpha * Y[k];
 *     repeated indices accumulate.  Sorted mode adds each row's entries in
 *     float32 in entry order and rounds the row to its format once (round
 *     to nearest even).  Atomic mode: float32 tables only, one float atomic
 *     per element.
 *   op POLYGLOT_OP_SET: for every k in order, table[idx[k]] = Y[k]; for a
 *     repeated index the largest k wins (sorted mode only).
 * N <= max_scatter and rows <= max_rows of the context.  Float32 increments
 * take the same kernels as polyglot_scatter_add.  Faster forms, with the
 * same results: 16-bit increments whose rows are whole 4-byte words (d even,
 * table and Y 4-byte aligned) read and write two rows per word; assignments
 * copy rows in the widest words (up to 16 bytes) that divide a row and both
 * pointers' alignment.  The caller owns every
 * buffer; the call is asynchronous on the context stream.  Returns
 * POLYGLOT_EINVAL for a bad format, op, mode, width or alignment or an
 * unsupported mode combination, POLYGLOT_ENULL, POLYGLOT_EBATCH; an index
 * outside [0, rows) leaves the table untouched and raises the sticky flag
 * (POLYGLOT_EID from polyglot_status). */
int polyglot_scatter_update(polyglot_ctx* ctx, void* table, int32_t dtype, int32_t rows,
                            int32_t d, const void* idx, int32_t idx_bytes, const void* Y,
                            int32_t N, float alpha, int32_t op, int32_t mode);

/* The distinct values of the index vector I of the §4.2 increment
 * W[I[k]] += Y[k] in the last sorted-mode train step: the rows of E the step
 * updated (ids of the windows and the corrupt ids), ascending.  Synchronises
 * the stream.  ids_host: host array of cap ints (may be NULL with cap 0);
 * at most cap ids are written and the total to *count (host).
 * POLYGLOT_ESTATE if no sorted-mode step has run, or if a scatter-add has
 * reused the sort buffers since. */
int polyglot_touched_rows(polyglot_ctx* ctx, int32_t* ids_host, int32_t cap, int32_t* count);

/* Kernel ids reported by polyglot_kernel_times. */
#define POLYGLOT_K_FWDBWD 0   /* fused gather + forward + hinge + backward (+ sort start);
                                 wide layers: gather + forward + hinge + per-window dz */
#define POLYGLOT_K_SORT 1     /* entry sort launches of a step (large batches) or of
                                 polyglot_scatter_add */
#define POLYGLOT_K_UPDATE 2   /* embedding segmented update + dense SGD */
#define POLYGLOT_K_GATHER 3   /* polyglot_gather */
#define POLYGLOT_K_SCATTER 4  /* polyglot_scatter_add's table update (atomic mode: and the id
                                 check); its sort and fix-up count under SORT and SEGFIX */
#define POLYGLOT_K_SCORE 5    /* polyglot_score */
#define POLYGLOT_K_SEGFIX 6   /* rows whose sorted entries span several chunks */
#define POLYGLOT_K_WIDE_DW1 7 /* wide layers: dW1 partials over window slices */
#define POLYGLOT_K_WIDE_G 8   /* wide layers: per-entry embedding gradient rows */
#define POLYGLOT_NKERNELS 9

/* Per-kernel timing for measurement.  With enable != 0 every later kernel
 * launch of this context (outside graph capture) gets a start/stop event
 * pair that the HIP runtime binds to the kernel's own dispatch
 * (hipExtLaunchKernel), so the elapsed time is the kernel's execution, not
 * the host enqueue.  polyglot_kernel_times() synchronises the streams,
 * writes the summed elapsed milliseconds and the launch count of each kernel
 * id into ms[POLYGLOT_NKERNELS] and launches[POLYGLOT_NKERNELS] (host
 * arrays), and resets the sums.  An id with several launches in one call
 * (the sort: histogram and radix passes) sums all of them. */
int polyglot_set_timing(polyglot_ctx* ctx, int enable);
int polyglot_kernel_times(polyglot_ctx* ctx, double* ms, int32_t* launches);

/* Synchronises the stream and returns the sticky device error
 * (POLYGLOT_OK or POLYGLOT_EID), then clears it. */
int polyglot_status(polyglot_ctx* ctx);

/* Text of the last error recorded on this context ("" if none). */
const char* polyglot_last_error(const polyglot_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* POLYGLOT_H */
