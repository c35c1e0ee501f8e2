/*
 * agn.h -- C ABI of libagn, the MI355X (gfx950) implementation of the hot
 * path of Accumulated Gradient Normalization (AGN; Hermans, Spanakis and
 * Moeckel, ACML 2017).
 *
 * The library simulates n AGN workers and the parameter server on one GPU.
 * One call to agn_round() is one round of the method: every worker runs
 * lambda local mini-batch SGD steps on its own copy of a ReLU MLP with a
 * softmax cross-entropy output (Algorithm 1, inner loop), normalizes its
 * accumulated update by lambda (Algorithm 1, normalization step; Eq. 1),
 * and the commits are added to the central variable in the caller's order
 * (Eq. 2), each worker pulling the central variable right after its own
 * commit (Algorithm 1, final pull; the FIFO queue of Section 1).
 *
 * Conventions shared by every entry point:
 *   - Every function returns an int status: AGN_OK (0) or a negative code.
 *     No C++ exception crosses the ABI.  On error, agn_last_error() gives
 *     a message; the context's state is unchanged unless the code is
 *     AGN_EHIP, after which the context is poisoned (every later call
 *     returns AGN_ESTATE) and should be destroyed.
 *   - "DEVICE" pointers are HIP device pointers on the device that was
 *     current at agn_create(); "HOST" pointers are ordinary host memory.
 *     The caller owns every buffer it passes; the library keeps no pointer
 *     to caller memory beyond the call.
 *   - Work is enqueued on the context's stream (agn_set_stream; default:
 *     the null stream).  agn_round() returns without waiting; agn_central,
 *     agn_loss, agn_worker_params and agn_debug_batch_indices wait for the
 *     stream before returning.
 *   - A context is not thread-safe; use one context per host thread.
 *
 * Parameter layout seen by callers ("packed"): W_0, b_0, W_1, b_1, ...,
 * W_l row-major with shape [d_{l+1}][d_l], b_l of length d_{l+1};
 * P = sum_l (d_l * d_{l+1} + d_{l+1}) floats.
 */
#ifndef AGN_H
#define AGN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define AGN_OK 0
#define AGN_EINVAL (-1) /* bad argument, shape or commit order */
#define AGN_ENOMEM (-2) /* device or host allocation failed */
#define AGN_EHIP (-3)   /* HIP runtime or launch error; context poisoned */
#define AGN_ESTATE (-4) /* poisoned context, or call out of order */

/* arithmetic of the matrix products */
#define AGN_FP32 0 /* float32 operands, float32 accumulation */
#define AGN_BF16 1 /* bfloat16 operands (inputs, weight shadows, hidden
                      activations, output-side gradients), float32
                      accumulation, float32 master weights and central
                      variable */

#define AGN_MAX_LAYERS 16
#define AGN_MAX_WORKERS 256

typedef struct agn_ctx agn_ctx; /* opaque; owned by the library */

/* Shapes of the model (Section 4 runs the same MLP on every worker). */
typedef struct {
  int32_t num_layers;   /* L, 1 <= L <= AGN_MAX_LAYERS (weight layers)       */
  const int32_t* dims;  /* HOST, L+1 widths: dims[0] inputs, dims[L] = C >= 2
                           classes; every width >= 1                          */
  int32_t batch;        /* mini-batch size m >= 1 (Eq. 1)                     */
  int32_t dtype;        /* AGN_FP32 or AGN_BF16                               */
} agn_shapes;

/* Training data of one round; worker k owns rows [k*S, (k+1)*S),
 * S = floor(num_samples / n) (Section 1: n shards; Section 4: data equally
 * distributed over the workers). */
typedef struct {
  const void* x;        /* DEVICE, [num_samples][dims[0]] row-major: float32
                           (x_dtype 0) or bfloat16 bit patterns (x_dtype 1)  */
  const int32_t* y;     /* DEVICE, [num_samples] labels in [0, C).  Not
                           range-checked on the device: the caller
                           guarantees the range.                             */
  int64_t num_samples;  /* N >= n                                            */
  int32_t x_dtype;      /* 0 float32, 1 bfloat16; must be 1 iff the shapes'
                           dtype is AGN_BF16                                 */
} agn_data;

/* Create a context: validates every argument first (AGN_EINVAL, nothing
 * allocated), allocates all device state (no allocation happens later in
 * agn_round), draws the initial central variable from `seed` (He-normal
 * weights N(0, 2/d_in) from a SplitMix64 stream through Box-Muller, biases
 * zero) and gives every worker a copy of it (Algorithm 1, first pull).
 * n in [1, AGN_MAX_WORKERS]; lambda >= 1 local steps; eta finite learning
 * rate (constant: Section 4 applies no decay).  *out receives the context
 * (NULL on failure). */
int agn_create(const agn_shapes* shapes, int32_t n, int32_t lambda, float eta,
               uint64_t seed, agn_ctx** out);

/* Use `hip_stream` (a hipStream_t; NULL = null stream) for all later work. */
int agn_set_stream(agn_ctx* ctx, void* hip_stream);

/* Commit rule.  normalize = 1 (the default): each worker commits its
 * accumulated update divided by lambda (Eq. 1, Algorithm 1's normalization
 * step: AGN).  normalize = 0: it commits the accumulated update itself,
 * DOWNPOUR with local exploration (Section 2; the variant whose divergence
 * the normalization is introduced to prevent).  With lambda = 1 the two
 * rules coincide and are DOWNPOUR (Section 3, footnote to Eq. 1).
 * Only before the first round (the round's kernels are recorded once):
 * AGN_ESTATE afterwards, AGN_EINVAL for a value other than 0 or 1. */
int agn_set_normalization(agn_ctx* ctx, int32_t normalize);

/* Staleness-scaled commits (Section 4 compares AGN with DynSGD, which
 * scales each commit down by its staleness).  enable = 1: the j-th commit
 * of a round adds s_j * delta instead of delta, s_j = 1 / (tau_j + 1)
 * rounded to float32, tau_j = the number of commits applied since the
 * committing worker's last pull (agn_staleness).  The paper gives only the
 * effect (about 1 / (n - 1) at the expected staleness n - 1); the factor
 * 1 / (tau + 1) is this library's reading.  Combined with
 * agn_set_normalization(ctx, 0) the scaled delta is the accumulated update
 * (DynSGD-style commits of local work).  Default 0.  Only before the first
 * round: AGN_ESTATE afterwards, AGN_EINVAL for a value other than 0 or 1. */
int agn_set_staleness_scaling(agn_ctx* ctx, int32_t enable);

/* Staleness of the last round's commits, by commit position: out[j] = the
 * number of commits the server applied between the pull of the j-th
 * committing worker and its commit (Section 1: the FIFO queue; the expected
 * staleness with n workers is n - 1).  out: HOST, n int64.  AGN_ESTATE
 * before the first round.  Host bookkeeping; does not wait. */
int agn_staleness(agn_ctx* ctx, int64_t* out);

/* Local rule of the workers (Algorithm 1's gradient line, which names Adam
 * as an option).  AGN_OPT_SGD (the default): g = -eta * gradient.
 * AGN_OPT_ADAM (Kingma & Ba 2015): each worker keeps first and second
 * moment estimates m, v of its gradients (float32 per parameter, zero when
 * selected, kept across pulls as Algorithm 1's step counter is) and
 * g = -eta * mhat / (sqrt(vhat) + eps), mhat = m / (1 - beta1^t),
 * vhat = v / (1 - beta2^t) at the worker's local step t = r*lambda + i + 1.
 * Selecting Adam allocates the moment buffers (2 * n * P floats) and
 * zeroes them.  beta1, beta2 in [0, 1), eps > 0 finite (ignored for SGD).
 * Only before the first round: AGN_ESTATE afterwards, AGN_EINVAL for bad
 * values, AGN_ENOMEM if the buffers cannot be allocated. */
#define AGN_OPT_SGD 0
#define AGN_OPT_ADAM 1
int agn_set_optimizer(agn_ctx* ctx, int32_t optimizer, float beta1, float beta2, float eps);

/* Enqueue one AGN round.  commit_order: HOST, n entries, a permutation of
 * 0..n-1 (checked on the host; AGN_EINVAL leaves the state unchanged).
 * The j-th entry is the worker whose normalized delta is the j-th to be
 * added to the central variable (Eq. 2); that worker then pulls.  Worker k
 * at its local step t (counted from 0 over all rounds) uses the rows
 * k*S + ((t*m + j) mod S), j = 0..m-1 (FetchNextMiniBatch of Algorithm 1).
 * data->num_samples must be the same on every round of a context. */
int agn_round(agn_ctx* ctx, const agn_data* data, const int32_t* commit_order);

/* Copy the central variable into out (DEVICE, P floats, packed layout). */
int agn_central(agn_ctx* ctx, float* out);

/* Per-worker training loss of the last round: for worker k (indexed by
 * worker id, not commit position), the mean over its lambda steps of the
 * mini-batch mean softmax cross-entropy, each evaluated at the worker's
 * parameters before that step's update.  out: DEVICE, n floats.
 * AGN_ESTATE before the first round. */
int agn_loss(agn_ctx* ctx, float* out);

/* Result of agn_evaluate. */
typedef struct {
  double mean_loss;  /* mean over the rows of the softmax cross-entropy     */
  double accuracy;   /* correct / num_samples                               */
  int64_t correct;   /* rows whose predicted class equals the label         */
} agn_eval_result;

/* Evaluate the central variable on a labelled set: Section 4 follows the
 * training and validation accuracy of the central model over time (the
 * f(t) of Eq. 4).  data: the rows to evaluate, x and y as for agn_round
 * (num_samples >= 1, not split into shards, x_dtype as for agn_round).
 * For every row: the logits of the MLP at the central variable (the same
 * forward products as a training step; bfloat16 operands in AGN_BF16
 * contexts), the softmax cross-entropy logsumexp(z) - z_y and the
 * predicted class argmax z (the lowest index among equal maxima; a NaN
 * logit counts as larger than any number).
 *   row_loss: DEVICE, num_samples floats, or NULL.
 *   row_pred: DEVICE, num_samples int32, or NULL.
 *   out:      HOST, or NULL.  The mean loss is summed in float64 in a
 *             fixed order: repeated calls give identical results.
 * Rows go through the forward pass 8192 at a time in the evaluation's own
 * workspace, which the first call allocates (activations of 8192 rows, two
 * buffers of the widest hidden layer; AGN_ENOMEM if that fails) and no
 * round touches: a call between rounds changes nothing a round reads.  It
 * works before the first round (the initial model).  With out != NULL the
 * call waits for the stream; with out == NULL it returns after enqueueing. */
int agn_evaluate(agn_ctx* ctx, const agn_data* data, float* row_loss, int32_t* row_pred,
                 agn_eval_result* out);

/* Allocation-free variant of agn_evaluate, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, same results:
 * row_loss, row_pred and the correct count as agn_evaluate gives them; the
 * float64 mean loss may differ in its last bits when the rows are taken
 * in smaller groups (below).  It allocates nothing, on the device or the
 * host, and launches nothing but its kernels (no memset, no event).
 *
 * Its workspace is a file-scope device array of AGN_NOALLOC_SCRATCH_BYTES
 * (16 MiB) that every device the library runs on holds until the process
 * ends (its device address is looked up once per device by agn_create).
 * The rows go through the forward pass as many at a time as fit in it (a
 * multiple of 64, at most 8192): activations of the widest hidden layer
 * twice, the logits when the output layer is not fused (C > 32 or bf16),
 * and per-block partial sums.  AGN_EINVAL (nothing enqueued) when not even
 * 64 rows fit, i.e. a hidden layer wider than about 32,000 units (float32)
 * or 64,000 (bf16).  In AGN_BF16 contexts the bf16 operands of the central
 * variable are the copy the last commit wrote for its worker's pull, so no
 * conversion buffer is needed.
 *
 * Every call on one device shares that device's array and leaves its
 * contents behind (each call overwrites what it reads): calls that overlap
 * in time on one device -- from several contexts, streams or host threads
 * -- race and give wrong results; serialize them.  With out == NULL the
 * call returns after enqueueing (capturable); with out != NULL it waits for
 * the stream and copies the totals to the host. */
#define AGN_NOALLOC_SCRATCH_BYTES (16u << 20)
int agn_evaluate_noalloc(agn_ctx* ctx, const agn_data* data, float* row_loss, int32_t* row_pred,
                         agn_eval_result* out);

/* Temporal efficiency E(a, b) of Eq. 4 (Section 4): the area under
 * performance curve f_a over the area under f_b, both over [0, tm] with tm
 * the minimal shared training time, min(last time of a, last time of b).
 * A curve is n >= 2 samples (t_i, f_i), HOST arrays: t_0 = 0 < t_1 < ...,
 * all finite; between samples f is the straight line (trapezoid rule), and
 * the curve that runs longer is cut at tm on the line through the samples
 * around it.  *out = area_a / area_b (HOST).  AGN_EINVAL for a bad curve or
 * a zero area of b; the message is agn_last_error(NULL).  Host arithmetic
 * only: no context and no device work. */
int agn_temporal_efficiency(const double* t_a, const double* f_a, int64_t n_a, const double* t_b,
                            const double* f_b, int64_t n_b, double* out);

/* Number of parameters P (-1 for a NULL context). */
int64_t agn_num_params(const agn_ctx* ctx);

/* Message of the last error of ctx, or of the last failed agn_create when
 * ctx is NULL.  Never NULL; valid until the next call on the same ctx. */
const char* agn_last_error(const agn_ctx* ctx);

/* Free everything (waits for the stream first).  NULL is a no-op. */
void agn_destroy(agn_ctx* ctx);

/* ---- checkpoint / resume ---------------------------------------------- */

/* The complete state of a context between rounds, so that a context with
 * the same configuration continues the run exactly where it was saved
 * (Algorithm 1 keeps no other state across rounds): the central variable;
 * each worker's last pulled copy of it, from which its next round starts;
 * the round counter (the workers' local step counter t = round * lambda +
 * i, which picks the mini-batches); the commit bookkeeping behind the
 * staleness of each commit (commits applied so far, and per worker the
 * count at its last pull); the per-row losses of the last round (what
 * agn_loss reports); and, with Adam as the local rule, each worker's two
 * moment estimates.  The deltas of the last round are not part of it:
 * agn_debug_delta returns AGN_ESTATE until a round has run after
 * agn_set_state.
 *
 * Layout of the state (HOST memory, native byte order): a header (magic
 * "AGNSTATE", format version 1, the configuration: L, m, n, lambda, dtype,
 * optimizer, normalization, staleness scaling, dims, eta, Adam's beta1,
 * beta2, eps, P; the round counter, the commit counter, num_samples of the
 * rounds so far (-1: none), the worker that committed last); then n int64
 * pull counters, n int64 staleness values of the last round's commits, the
 * n * lambda * m float32 per-row losses; then float32 vectors of P
 * parameters in the packed layout of agn_central: the central variable,
 * the n pulled copies in worker order, and with Adam the n first-moment and
 * the n second-moment vectors. */

/* Size in bytes of the state of ctx (-1 for a NULL context). */
int64_t agn_state_bytes(const agn_ctx* ctx);

/* Write the state of ctx into out (HOST, exactly agn_state_bytes(ctx)
 * bytes, caller-owned).  Waits for the work enqueued on the context's
 * stream first.  AGN_EINVAL for a NULL out or another size. */
int agn_get_state(agn_ctx* ctx, void* out, int64_t bytes);

/* Replace the state of ctx by a state written by agn_get_state (HOST,
 * `bytes` bytes, read during the call only).  ctx must have the same
 * configuration as the context the state was taken from: layer widths, m,
 * n, lambda, eta, dtype, commit rule and staleness scaling, and the local
 * rule (select Adam with agn_set_optimizer before restoring an Adam state).
 * Everything is checked on the host before any device work: AGN_EINVAL
 * (state unchanged) for another size, magic, format version or
 * configuration, or inconsistent counters.  The bf16 copies of the pulled
 * copies (bf16 contexts) are rebuilt from the float32 ones, as the commit
 * writes them.  Returns after the copies have completed. */
int agn_set_state(agn_ctx* ctx, const void* in, int64_t bytes);

/* ---- test hooks (not on the timed path) ------------------------------- */

/* Before the first round only (AGN_ESTATE otherwise): set the central
 * variable and every worker's copy to `in` (DEVICE, P floats, packed). */
int agn_set_central(agn_ctx* ctx, const float* in);

/* Copy worker k's current parameters (its last pulled copy of the central
 * variable, the start of its next round) into out (DEVICE, P floats). */
int agn_worker_params(agn_ctx* ctx, int32_t worker, float* out);

/* Copy the delta worker k committed in the last round (Eq. 1: its
 * accumulated update divided by lambda; without normalization, see
 * agn_set_normalization, the accumulated update itself) into out (DEVICE,
 * P floats, packed).  AGN_ESTATE before the first round. */
int agn_debug_delta(agn_ctx* ctx, int32_t worker, float* out);

/* The m sample indices worker `worker` uses at local step `step_t`, for a
 * data set of `num_samples` rows: out (DEVICE, m int64). */
int agn_debug_batch_indices(agn_ctx* ctx, int32_t worker, int64_t step_t,
                            int64_t num_samples, int64_t* out);

/* ---- kernel timing ------------------------------------------------------ */

/* Kernel classes, in the order a local step launches them; each class is
 * one kernel (in float32 mode). */
#define AGN_K_FWD 0       /* forward products + bias + ReLU (and the logits
                             when the output layer is not fused)             */
#define AGN_K_OUTPUT 1    /* output layer: softmax cross-entropy, loss, output
                             gradient; with few classes also the logits and
                             the output layer's input gradient, fused        */
#define AGN_K_OUTPUT_DW 2 /* fused output layer only: its weight gradient
                             with the SGD update (float32 with at most 10
                             classes: carried by the AGN_K_DW_FIRST launch)  */
#define AGN_K_BWD 3       /* hidden layers l >= 1, one launch per layer: the
                             input-gradient product and the weight-gradient
                             product fused with the SGD update               */
#define AGN_K_DW_FIRST 4  /* first layer: weight-gradient product (rows
                             gathered from the data set) fused with the SGD
                             update (and the output layer's, see above)      */
#define AGN_K_COMMIT 5    /* normalize + commit + pull                       */
#define AGN_K_EVAL 6      /* agn_evaluate's forward products (not part of a
                             round)                                          */
#define AGN_K_NUM 7

/* Algorithmic work of one round attributed to a kernel class, as this
 * context launches it: flops = 2 * multiply-adds of the class's matrix
 * products; bytes = the memory traffic the class cannot avoid (for the
 * commit: central + n deltas read, n pulled copies + central written,
 * plus the bf16 copies of the pulls in bf16 mode;
 * for the classes with the update: the parameters they update read and
 * written once per local step, plus their bf16 shadow written in bf16
 * mode (and, for the hidden layers' backward launches, read by the input
 * gradient) and Adam's two moment estimates read and written; for the output
 * layer: its activations read and gradients written).  AGN_K_EVAL: the
 * work of the last agn_evaluate call instead (its rows' inputs and the
 * weights read once, the logits written once), zero before the first.
 * Work carried by another class's launch counts there (AGN_K_OUTPUT_DW).
 * HOST outputs. */
int agn_kernel_class_work(agn_ctx* ctx, int32_t kernel_class, double* flops,
                          double* bytes);

/* When enabled, every launch of the given class records a pair of HIP
 * events at its kernel's start and end (the dispatch records them, so the
 * time is the kernel's own), and rounds run their launches eagerly on the
 * context's stream instead of replaying the captured graph.  Enabling
 * resets the counters. */
int agn_set_kernel_timing(agn_ctx* ctx, int32_t kernel_class, int32_t enable);

/* Total milliseconds and number of launches of the class since timing was
 * enabled (waits for the stream). */
int agn_kernel_timing(agn_ctx* ctx, int32_t kernel_class, double* total_ms,
                      int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* AGN_H */
