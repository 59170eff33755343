/*
 * sats.h -- C ABI of the routed, threshold-sparsified gated-MLP library for
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (per token, independently):
 *
 *   route:  r = route_lut[token_id]      1 = base path, 0 = sparse path
 *           (the decision of the token-routing rule, Section 3.2, Eq. 13,
 *            precomputed per vocabulary id; a score below tau selects the
 *            sparse path, any other the base path)
 *   for each layer l = 0 .. n_layers-1, with h the layer input:
 *     a_j  = W_gate_T[l][j] . h  (a = h W_gate)        gated MLP, Eq. 1
 *     g    = SiLU(a) = a / (1 + exp(-a))                 Eq. 2
 *     keep = all columns                   if r == 1     (base MLP, Eq. 1)
 *            { j : |g_j| >= thresholds[l] } if r == 0    (CATS mask, Eq. 4-5)
 *     u_j  = W_up_T[l][j] . h              for j in keep  (x W_up, Eq. 1)
 *     y    = sum_{j in keep} g_j u_j W_down[l][j]         (Eq. 1)
 *     next h = rho(y / sqrt(mean(y^2) + 1e-6))    between layers
 *   out = rho(y of the last layer)
 *
 * rho rounds to the activation type (bf16: round to nearest even).  All
 * products and sums are float32.  The normalisation between layers is this
 * library's convention for chaining bare MLP layers (the paper places each
 * MLP inside a transformer block); a one-layer call is exactly Eq. 1 with the
 * Eq. 5 mask.
 *
 * Layouts (row-major, dense, no padding):
 *   x, out        [n_tokens][d]
 *   token_ids     [n_tokens]
 *   W_gate_T      [n_layers][d_ff][d]      W_gate transposed: row j = column j of W_gate
 *   W_up_T        [n_layers][d_ff][d]      W_up transposed: row j = column j of W_up
 *   W_down        [n_layers][d_ff][d]      row j = the output weights of neuron j
 * (every weight matrix holds one row of d weights per neuron: a linear
 * layer's weight as it is stored for W_gate and W_up, and its transpose for
 * W_down)
 *   thresholds    [n_layers]               float32, >= 0 or +inf
 *   route_lut     [vocab]                  uint8
 *
 * Ownership: every pointer is a DEVICE pointer owned by the caller and must
 * stay valid until the enqueued work has completed.  The library keeps no
 * pointer past that.  It owns a device workspace per (device, stream),
 * allocated on first use and grown when a larger shape arrives (a hipMalloc
 * on that call: call sats_reserve() first where allocation is not allowed).
 *
 * Errors: every call returns SATS_OK or a negative code synchronously, for
 * conditions the host can check (null pointers, shapes, overlap of out with
 * x other than exact equality, HIP launch failures).  The text of the last
 * error of the calling thread is returned by sats_last_error().  Execution
 * is asynchronous on `stream`; device-side faults surface at the caller's
 * next synchronisation.  n_tokens == 0 returns SATS_OK and enqueues nothing.
 *
 * Unchecked preconditions (device contents): 0 <= token_ids[i] < vocab;
 * thresholds not NaN and not negative; x and weights finite.
 *
 * Determinism: results do not depend on the run, on the batch a token is in
 * (for batches of one size class) or on the stream; every reduction has a
 * fixed order and no floating-point atomics are used.
 *
 * Concurrency: calls on different streams use different workspaces and may
 * overlap.  Calls on one stream are ordered by the stream.
 */
#ifndef SATS_H
#define SATS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t sats_bf16; /* raw bfloat16 bits */

enum {
  SATS_OK = 0,
  SATS_ERR_NULL = -1,      /* a required pointer is NULL                        */
  SATS_ERR_SHAPE = -2,     /* d < 1, d_ff < 1, n_layers < 1, n_tokens < 0, or too large */
  SATS_ERR_HIP = -3,       /* a HIP runtime call or kernel launch failed        */
  SATS_ERR_WORKSPACE = -4, /* workspace allocation failed                       */
  SATS_ERR_ARG = -5,       /* other invalid argument (partial overlap of out and x)        */
  SATS_ERR_DEVICE = -6     /* reported by sats_device_status: a device-side wait gave up  */
};

/*
 * Routed sparse forward (Section 3.2 routing over the Section 2 CATS-masked
 * gated MLP).  route_lut == NULL sends every token to the sparse path (the
 * static sparse model) and token_ids may then be NULL.  out may equal x
 * exactly (in-place); any other overlap is rejected.
 */
int sats_mlp_forward(const sats_bf16 *x, const int32_t *token_ids,
                     const sats_bf16 *W_gate_T, const sats_bf16 *W_up_T,
                     const sats_bf16 *W_down, const float *thresholds,
                     const uint8_t *route_lut, sats_bf16 *out,
                     int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers,
                     hipStream_t stream);

/*
 * Allocation-free variant of sats_mlp_forward, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, computation and results
 * as sats_mlp_forward (the same kernels), but the workspace is a fixed device
 * array of the library, SATS_NOALLOC_SCRATCH_BYTES (16 MiB) on each device
 * that runs it, held until the process ends, instead of a per-stream
 * allocation; the call allocates and frees nothing.  That covers single-token
 * calls at d <= 4096 and d_ff <= 16384 (any number of layers up to 64, bf16)
 * and small batches; a call whose workspace does not fit returns
 * SATS_ERR_WORKSPACE before any device work.  Every call on a device shares
 * that device's array and leaves its last contents there: each call first
 * clears the array's arrival counters with a small kernel (no memset), and
 * calls that overlap on one device (other streams or threads) race and must
 * not be issued.  sats_device_status also reports a bounded wait that gave up
 * in such a call.
 */
#define SATS_NOALLOC_SCRATCH_BYTES (16u << 20)
int sats_mlp_forward_noalloc(const sats_bf16 *x, const int32_t *token_ids,
                             const sats_bf16 *W_gate_T, const sats_bf16 *W_up_T,
                             const sats_bf16 *W_down, const float *thresholds,
                             const uint8_t *route_lut, sats_bf16 *out,
                             int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers,
                             hipStream_t stream);

/* Base path for every token: the unmasked gated MLP of Eq. 1, same layout. */
int sats_mlp_dense(const sats_bf16 *x, const sats_bf16 *W_gate_T,
                   const sats_bf16 *W_up_T, const sats_bf16 *W_down,
                   sats_bf16 *out, int64_t n_tokens, int64_t d, int64_t d_ff,
                   int64_t n_layers, hipStream_t stream);

/* float32 twins: x, weights and out are float32; rho rounds to float32. */
int sats_mlp_forward_f32(const float *x, const int32_t *token_ids,
                         const float *W_gate_T, const float *W_up_T,
                         const float *W_down, const float *thresholds,
                         const uint8_t *route_lut, float *out,
                         int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers,
                         hipStream_t stream);
int sats_mlp_dense_f32(const float *x, const float *W_gate_T, const float *W_up_T,
                       const float *W_down, float *out, int64_t n_tokens, int64_t d,
                       int64_t d_ff, int64_t n_layers, hipStream_t stream);

/*
 * Introspection for tests and measurement: the same computation as
 * sats_mlp_forward, plus extra stores.  Any of the extra outputs may be NULL.
 *   route_out     [n_tokens]                 decision used (1 base, 0 sparse)
 *   active_count  [n_layers][n_tokens]       |keep| of each token at each layer
 *   active_idx    [n_layers][n_tokens][d_ff] keep set, ascending, first
 *                                            active_count entries valid
 *   layer_in      [n_layers][n_tokens][d]    input h of each layer
 */
int sats_mlp_forward_inspect(const sats_bf16 *x, const int32_t *token_ids,
                             const sats_bf16 *W_gate_T, const sats_bf16 *W_up_T,
                             const sats_bf16 *W_down, const float *thresholds,
                             const uint8_t *route_lut, sats_bf16 *out,
                             int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers,
                             hipStream_t stream, uint8_t *route_out,
                             int32_t *active_count, int32_t *active_idx,
                             sats_bf16 *layer_in);
int sats_mlp_forward_inspect_f32(const float *x, const int32_t *token_ids,
                                 const float *W_gate_T, const float *W_up_T,
                                 const float *W_down, const float *thresholds,
                                 const uint8_t *route_lut, float *out,
                                 int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers,
                                 hipStream_t stream, uint8_t *route_out,
                                 int32_t *active_count, int32_t *active_idx,
                                 float *layer_in);

/*
 * LoRA-aware routed sparse forward (Section 5, the fine-tuned routed
 * models): sparse-path tokens run the base weights plus rank-r adapters on
 * the three projections,
 *   W_gate + scale A_gate B_gate,  W_up + scale A_up B_up,  W_down + scale A_down B_down,
 * and base-path tokens run the base weights alone (both paths share them, so
 * the adapters are not merged in).  The CATS threshold applies to
 * |SiLU(h (W_gate + scale A_gate B_gate))|.  Device arrays in the activation
 * type, stacked over n_layers like the weights, row-major:
 *   A_gate [d][rank], B_gate [rank][d_ff], A_up [d][rank],
 *   B_up_T [d_ff][rank] (B_up transposed, like W_up_T),
 *   A_down [d_ff][rank], B_down [rank][d].
 * The adapters run inside the same launches as the base computation: the up
 * adapter only for kept columns, the down adapter's first factor only over
 * kept rows.  rank is 8, 16, 32 or 64; the adapter arrays must be 16-byte
 * aligned.  Batches of two or more bf16 tokens whose shapes fit the matrix-core
 * path (d a multiple of 128 and at most 4096, d_ff a multiple of 64) run in
 * passes of up to 64 tokens with every row on the matrix cores: each row
 * applies its own route and keep rule, the gate and up adapter terms are
 * added in float32 before SiLU and the keep rule, z = p A_down is summed per
 * 64-column tile and scale z B_down is added with the output.  Otherwise the
 * shapes must fit the single-token path (d <= 4096, d and d_ff multiples of
 * 16 bytes' worth of elements) and tokens are processed one after another,
 * each on its own route.  Other arguments and the optional
 * inspection outputs as in sats_mlp_forward_inspect.  Errors: SATS_ERR_NULL
 * (a required array), SATS_ERR_SHAPE (rank or shape), SATS_ERR_ARG
 * (alignment, non-finite scale), and those of sats_mlp_forward.
 */
int sats_mlp_forward_lora(const sats_bf16 *x, const int32_t *token_ids, const sats_bf16 *W_gate_T,
                          const sats_bf16 *W_up_T, const sats_bf16 *W_down, const sats_bf16 *A_gate,
                          const sats_bf16 *B_gate, const sats_bf16 *A_up, const sats_bf16 *B_up_T,
                          const sats_bf16 *A_down, const sats_bf16 *B_down, int64_t rank, float scale,
                          const float *thresholds, const uint8_t *route_lut, sats_bf16 *out, int64_t n_tokens,
                          int64_t d, int64_t d_ff, int64_t n_layers, hipStream_t stream, uint8_t *route_out,
                          int32_t *active_count, int32_t *active_idx, sats_bf16 *layer_in);
int sats_mlp_forward_lora_f32(const float *x, const int32_t *token_ids, const float *W_gate_T, const float *W_up_T,
                              const float *W_down, const float *A_gate, const float *B_gate, const float *A_up,
                              const float *B_up_T, const float *A_down, const float *B_down, int64_t rank,
                              float scale, const float *thresholds, const uint8_t *route_lut, float *out,
                              int64_t n_tokens, int64_t d, int64_t d_ff, int64_t n_layers, hipStream_t stream,
                              uint8_t *route_out, int32_t *active_count, int32_t *active_idx, float *layer_in);

/*
 * Allocate the workspace of (current device, stream) for calls of up to
 * max_tokens tokens at this d, d_ff, n_layers and element size (2 = bf16,
 * 4 = f32), so that later calls of that size or smaller allocate nothing.
 */
int sats_reserve(int64_t max_tokens, int64_t d, int64_t d_ff, int64_t n_layers,
                 int elem_bytes, hipStream_t stream);

/*
 * Synchronise `stream` and report whether a kernel of this library on it
 * raised the device error flag since the last check (SATS_ERR_DEVICE; the
 * flag is cleared).  The single-token path's second reduction stage waits
 * for the other workgroups of its launch with a bounded wait that raises
 * the flag instead of hanging; the call also surfaces asynchronous HIP
 * errors of the stream.
 */
int sats_device_status(hipStream_t stream);

/*
 * SATS calibration (Section 3.1, Eq. 6-10): the offline step that produces
 * the per-layer thresholds the forward calls take.  Unlike the forward
 * calls, these take and return their small arrays in HOST memory, use
 * device buffers of their own (kept per device from call to call and grown
 * when a call needs more; calls are serialised; sats_release frees them),
 * and synchronise `stream` before returning, also when they fail.
 *
 * sats_calibration_curves -- one layer.  h [n][d] holds the layer's inputs
 * for n calibration rows (device, bf16; the base-path inputs in a stack),
 * W_gate_T, W_up_T, W_down [d_ff][d] each (device, bf16).  For
 * each level q_k of levels[n_levels] (host, ascending in [0, 1]) the
 * candidate threshold t_k is the Eq. 3 order statistic v_(ceil(q_k N)) of the
 * N = n d_ff post-gate magnitudes |SiLU(h W_gate)| (q_k = 0 gives t_k = 0;
 * q_k is taken to 1e-6), and
 *   err_out[k] = Err(t_k) = mean over rows of ||y - y_t|| / (||y|| + 1e-6)   (Eq. 6)
 *   sp_out[k]  = #{|g| < t_k} / N                      (the layer sparsity at t_k)
 * with y the dense MLP output of the row and y_t the output with the neurons
 * of |g| < t_k removed.  t_out, err_out, sp_out: host arrays [n_levels];
 * err_rows (device float [n][n_levels], or NULL) receives the per-row terms.
 * g and u accumulate in float32; p = g u enters the error product as two
 * bf16 terms (about 16 bits of p); the sums have a fixed order.
 * Shapes: d a multiple of 128 up to 4096, d_ff a multiple of 64.
 *
 * sats_calibrate_sats -- a stack.  The n_cal rows of x_cal (device bf16
 * [n_cal][d]) run through the base path of the n_layers-layer stack (the
 * forward calls' own inter-layer normalisation); every layer's curves are
 * measured on its inputs at the candidate levels 0, coarse_step,
 * 2 coarse_step, ... (Eq. 3 percentiles); for a budget b each layer takes
 * its largest candidate with Err <= b (Eq. 7), S(b) is the mean layer
 * sparsity (Eq. 9), and b* minimises |S(b) - s_tar| over every distinct
 * error value (Eq. 10; the smallest b on ties).  Then, per layer, levels
 * fine_step apart strictly between the two coarse levels adjacent to the
 * level of its choice (both sides of it) are added and b* is chosen again.  With guardrail != 0 (and n_layers > 1) the last
 * layer keeps its CATS threshold at level s_tar (its sparsity counts in S).
 * thresholds_out: host float [n_layers]; budget_out, realized_out: host
 * doubles (may be NULL) receiving b* and S(b*).
 */
int sats_calibration_curves(const sats_bf16 *h, const sats_bf16 *W_gate_T, const sats_bf16 *W_up_T,
                            const sats_bf16 *W_down, int64_t n, int64_t d, int64_t d_ff,
                            const double *levels, int64_t n_levels, float *t_out, double *err_out,
                            double *sp_out, float *err_rows, hipStream_t stream);
int sats_calibrate_sats(const sats_bf16 *x_cal, int64_t n_cal, const sats_bf16 *W_gate_T,
                        const sats_bf16 *W_up_T, const sats_bf16 *W_down, int64_t d, int64_t d_ff,
                        int64_t n_layers, double s_tar, double coarse_step, double fine_step,
                        int guardrail, float *thresholds_out, double *budget_out,
                        double *realized_out, hipStream_t stream);

/*
 * Routing-table construction (Section 3.2, Eq. 11-14), the offline step that
 * produces route_lut.  token_ids [n_tokens] with loss_base and loss_sparse
 * [n_tokens] (device, float32: the next-token cross-entropy of each
 * occurrence of the routing corpus on the base and the sparse path) give
 * each id x the score s(x) = mean over its occurrences of
 * d = max(0, loss_sparse - loss_base) (Eq. 11-12; d taken in float32 and
 * rounded to a multiple of 2^-32, so that the per-id sums are exact;
 * s = +inf for an id without occurrences).  heldout_ids [n_heldout] (device)
 * calibrate the threshold: tau* minimises |R(tau) - r_tar| over the distinct
 * finite scores of the held-out ids and +inf (Eq. 14; the smallest on ties),
 * R(tau) being the fraction of held-out occurrences whose id scores below
 * tau.  route_lut [vocab] (device) receives 0 (sparse path) where
 * s(x) < tau*, else 1 (base path) -- the table the forward calls take.
 * scores [vocab] (device double, or NULL) receives s; tau_out and
 * realized_out (host, or NULL) receive tau* and R(tau*); the selection of
 * tau* runs on the device.  Synchronises the stream; its device buffers are
 * kept per device from call to call (calls are serialised; sats_release
 * frees them).  On an error route_lut is left as it was.  Errors:
 * SATS_ERR_NULL, SATS_ERR_SHAPE,
 * SATS_ERR_ARG (r_tar outside [0, 1], an id outside [0, vocab), a loss
 * difference NaN or >= 2^31).  The per-id sums of d must stay below 2^32.
 */
int sats_route_table(const float *loss_base, const float *loss_sparse, const int32_t *token_ids, int64_t n_tokens,
                     const int32_t *heldout_ids, int64_t n_heldout, int64_t vocab, double r_tar,
                     uint8_t *route_lut, double *scores, double *tau_out, double *realized_out, hipStream_t stream);

/*
 * Execution options: which kernels the forward calls made afterwards on the
 * calling thread run.  Every field's default, 0, is the library's own
 * choice; sats_set_options(NULL) restores the defaults.  Meant for tests
 * and measurement (results of every choice agree with the definition above
 * within the stated tolerances); nothing else changes the kernels a call
 * takes.  Errors: SATS_ERR_ARG for a value outside its range.
 *   batch_path      SATS_BATCH_AUTO, or for batches of 2 or more bf16 tokens:
 *                   SATS_BATCH_MFMA     every token on the matrix cores, each
 *                                       with its own route and keep rule;
 *                   SATS_BATCH_SPLIT    the base-path group on the matrix
 *                                       cores, the sparse group on the
 *                                       compacted kernels;
 *                   SATS_BATCH_COMPACT  every token on the compacted kernels
 *                                       (gate, then up and down over the
 *                                       union of kept rows of each 4-token
 *                                       tile, with a per-row token mask).
 *   single_token    SATS_SINGLE_AUTO: one-token calls on the single-token
 *                   kernels where the shape fits them; SATS_SINGLE_OFF: on
 *                   the batch kernels.
 *   dec_block_cols  single-token layer launch: gate columns per workgroup,
 *                   one partial of y each (1 .. 64; 0 = d_ff over the
 *                   compute units, at least 8).
 *   lora_per_token  1: LoRA batches token after token on the single-token
 *                   kernels instead of the matrix-core passes.
 */
enum { SATS_BATCH_AUTO = 0, SATS_BATCH_MFMA = 1, SATS_BATCH_SPLIT = 2, SATS_BATCH_COMPACT = 3 };
enum { SATS_SINGLE_AUTO = 0, SATS_SINGLE_OFF = 1 };
typedef struct {
  int batch_path;
  int single_token;
  int dec_block_cols;
  int lora_per_token;
} sats_options;
int sats_set_options(const sats_options *opt);

/*
 * The kernels a forward call (without adapters) of this shape would run
 * under the calling thread's options, answered on the host without device
 * work: *path receives SATS_PATH_SINGLE_TOKEN, SATS_PATH_BATCH_MFMA,
 * SATS_PATH_BATCH_SPLIT or SATS_PATH_BATCH_COMPACT (for the first pass of
 * up to 64 tokens; 0 for n_tokens == 0).  elem_bytes: 2 (bf16) or 4
 * (float32); aligned16: whether x, out and the weights are 16-byte aligned;
 * n_cus: compute units of the device (0: the current device's).  Errors:
 * SATS_ERR_NULL, SATS_ERR_SHAPE and SATS_ERR_ARG as for the forward calls.
 */
enum { SATS_PATH_SINGLE_TOKEN = 1, SATS_PATH_BATCH_MFMA = 2, SATS_PATH_BATCH_SPLIT = 3,
       SATS_PATH_BATCH_COMPACT = 4 };
int sats_query_path(int64_t n_tokens, int64_t d, int64_t d_ff, int elem_bytes, int aligned16, int n_cus,
                    int *path);

/* Free every workspace of the calling process, and the kept buffers of the
 * routing-table construction and of the calibration (synchronises each
 * device). */
int sats_release(void);

/* Thread-local text of the last error returned on this thread ("" if none). */
const char *sats_last_error(void);

/*
 * Kernel timing for measurement.  sats_timing_begin(kind, capacity) arms
 * HIP-event pairs around the next `capacity` launches of one kernel kind
 * (SATS_K_*), recorded on the stream the kernel is launched on.
 * sats_timing_end(kind, &total_ms, &count) waits for the recorded events,
 * returns the summed duration and the number of launches timed, and disarms.
 * SATS_K_ROUTE_ACCUM times the per-chunk pass over the routing split
 * (route_part_kernel; for vocabularies past 2^22 ids the atomic form,
 * route_accum_kernel), SATS_K_ROUTE_MERGE the merge of its entries.
 */
enum { SATS_K_GATE = 0, SATS_K_UP = 1, SATS_K_DOWN = 2, SATS_K_INSPECT = 3, SATS_K_DENSE = 4,
       SATS_K_DEC_LAYER = 5, SATS_K_DEC_LORA_V = 6, SATS_K_CAL_ERR = 7, SATS_K_CAL_GATEUP = 8,
       SATS_K_ROUTE_ACCUM = 9, SATS_K_LORA_V = 10, SATS_K_DEC_REDUCE = 11, SATS_K_DENSE_DOWN = 12,
       SATS_K_DEC_REDUCE_LORA = 13, SATS_K_ROUTE_MERGE = 14, SATS_K_COUNT = 15 };
int sats_timing_begin(int kind, int capacity);
int sats_timing_end(int kind, double *total_ms, int64_t *count);
const char *sats_kernel_name(int kind);

#ifdef __cplusplus
}
#endif

#endif /* SATS_H */
