/*
 * libcats -- CATS (Contextually-Aware Thresholding for Sparsity) gated-MLP
 * hot path for AMD Instinct MI355X (gfx950).
 *
 * The operations follow Lee et al., "CATS: Contextually-Aware Thresholding
 * for Sparsity in Large Language Models" (COLM 2024):
 *   Section 3, Eq. 1   Gated-MLP(x) = (SiLU(x W_gate) * (x W_up)) W_down,
 *                      x in R^{b x d}, W_gate, W_up in R^{d x m},
 *                      W_down in R^{m x d}
 *   Section 3, Eq. 2   SiLU(z) = z / (1 + e^{-z})
 *   Section 4.1, Eq. 3 cutoff t = min{t' : F(t') >= k}, F the empirical CDF
 *                      of the absolute gate activations of one MLP block
 *   Section 4.2, Eq. 4-5  CATS_t keeps an activation when |.| >= t
 *   Section 4.3 and Appendix D  kernel algorithms "MLP using CATS"
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Plain C ABI.  Every pointer argument is caller-owned; the library never
 *    frees or keeps a pointer after returning.  "dev" marks device memory,
 *    "host" host memory.  `stream` is a hipStream_t (NULL = the default
 *    stream of the current device); every device pointer must belong to the
 *    current device.
 *  - The forward, dense, pack and rmsnorm calls only enqueue work on
 *    `stream` (no host synchronisation, no allocation).  Outputs are valid
 *    once the stream reaches that point.  The two calibration calls
 *    synchronise `stream` because they return t on the host.
 *  - Arguments are validated on the host before any HIP call; a rejected
 *    call returns its status and touches nothing.  HIP failures return
 *    CATS_ERR_HIP.  cats_last_error() gives a message for the last failure
 *    on the calling thread.  No call aborts or throws.
 *  - Debugging: with the environment variable CATS_SYNC_CHECK set (to
 *    anything but "" or "0"), every enqueue-only call synchronises `stream`
 *    after its launches and returns CATS_ERR_HIP for an asynchronous failure
 *    (a kernel fault, a launch error), naming the call that caused it.  Not
 *    applied to a stream under graph capture.
 *  - Scratch memory comes from a caller-provided workspace `ws` of
 *    `ws_bytes` bytes (256-byte aligned, device), sized with
 *    cats_workspace_bytes().  Calls that run concurrently need separate
 *    workspaces.  A workspace needs no clearing: it may hold anything when
 *    a call starts (leftovers of other calls or entry points included);
 *    the arrival counters some kernels keep there are tagged per call.
 *  - x, y, residual, thresholds and calibration inputs are fp32.  Weights
 *    are CATS_F32 or CATS_BF16; all arithmetic accumulates in fp32.
 *  - Weight layout is neuron-major: W_gate^T and W_up^T are stored [m x d]
 *    (row j holds neuron j's d input weights contiguously, the paper's
 *    "column-major W_up"), W_down is [m x d] row-major as in Eq. 1.  Use
 *    cats_pack_weights to produce W^T from the math layout [d x m].
 */
#ifndef CATS_H
#define CATS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CATS_VERSION 1

typedef enum {
  CATS_OK = 0,
  CATS_ERR_NULL = 1,          /* a required pointer is NULL */
  CATS_ERR_SHAPE = 2,         /* d, m, B or N out of the supported range */
  CATS_ERR_RANGE = 3,         /* sparsity or t outside its domain */
  CATS_ERR_DTYPE = 4,         /* unknown weight dtype */
  CATS_ERR_ALIGN = 5,         /* a pointer misses its required alignment */
  CATS_ERR_WORKSPACE = 6,     /* workspace NULL or too small */
  CATS_ERR_HIP = 7,           /* a HIP runtime call failed */
  CATS_ERR_UNIMPLEMENTED = 8  /* combination the library does not implement */
} cats_status;

typedef enum { CATS_F32 = 0, CATS_BF16 = 1 } cats_dtype;

/* Supported sizes.  d must be a positive multiple of 8 (16-byte vector
 * loads of bf16 rows); 1 <= m <= CATS_MAX_M; batch rows 1..CATS_MAX_BATCH. */
#define CATS_MAX_D_BF16 8192
#define CATS_MAX_M 65536
#define CATS_MAX_D_F32 4096
#define CATS_MAX_BATCH 16
/* Layers of one cats_stack_forward call. */
#define CATS_MAX_LAYERS 1024
/* Each weight matrix (m * d elements) is addressed with 32-bit offsets and
 * may span at most 1 GiB. */
#define CATS_MAX_MATRIX_BYTES (1ull << 30)

/* One gated-MLP block (Eq. 1) in neuron-major layout.  Plain data: the
 * struct and the weights stay owned by the caller. */
typedef struct {
  int32_t d;              /* hidden size */
  int32_t m;              /* intermediate size (number of neurons) */
  int32_t wdtype;         /* cats_dtype of all three matrices */
  const void* w_gate_t;   /* dev [m x d], row j = W_gate[:, j] */
  const void* w_up_t;     /* dev [m x d], row j = W_up[:, j] */
  const void* w_down;     /* dev [m x d], row j = W_down[j, :] */
} cats_layer;

/* Optional per-row outputs of cats_mlp_forward; any member may be NULL.
 * For batch row b, in ascending neuron order:
 *   active_idx[b*m + q]  index of the q-th neuron kept by CATS_t (Eq. 5)
 *   active_cnt[b]        number of kept neurons
 *   active_v[b*m + q]    its activation v = SiLU(x W_gate[:, j]) (Eq. 2)
 *   active_h[b*m + q]    v * (x W_up[:, j]), the x1 of the CATS kernel
 *                        algorithm (Section 4.3), before W_down
 * Entries past active_cnt[b] are left untouched.  All dev, int32 / fp32. */
typedef struct {
  int32_t* active_idx;
  int32_t* active_cnt;
  float* active_v;
  float* active_h;
} cats_forward_aux;

/* Library version (CATS_VERSION). */
int32_t cats_version(void);

/* Static description of a status code; never NULL. */
const char* cats_status_string(cats_status s);

/* Message for the last failed call on this thread ("" if none). */
const char* cats_last_error(void);

/* Workspace bytes needed by any call on a block of size d x m with up to
 * `max_batch` rows per forward, dense or stack call and up to `max_calib_values`
 * calibration activations (N * m) per calibration call (0 if calibration
 * is not used).  Pure host arithmetic, no HIP call.  Returns 0 for
 * arguments outside the supported range. */
size_t cats_workspace_bytes(int32_t d, int32_t m, int32_t max_batch, int64_t max_calib_values);

/* Transpose a row-major [rows x cols] matrix into [cols x rows]
 * (w_t[c*rows + r] = w[r*cols + c]), bit for bit.  Used to turn the math
 * layout W_gate, W_up [d x m] of Eq. 1 into the neuron-major [m x d]
 * the kernels stream (Section 4.3 stores W_up this way so that a masked
 * neuron's weights are one contiguous row).  dev w, dev w_t, no overlap. */
cats_status cats_pack_weights(const void* w, void* w_t, int32_t rows, int32_t cols,
                              int32_t dtype, void* stream);

/* Calibration activations (Section 4.1): for N vectors x_n (dev [N x d],
 * fp32) writes acts[n*m + j] = |SiLU(x_n . W_gate[:, j])| (dev [N x m]).
 * fp32 accumulation; with bf16 weights the products run on the matrix
 * cores with x split into two bf16 parts (16 of its 24 significand bits,
 * each product exact), so a dot product differs from an fp32 one by about
 * 2^-16 of its absolute terms.  Enqueue only. */
cats_status cats_calib_activations(const cats_layer* layer, const float* x, int32_t N,
                                   float* acts, void* stream);

/* Cutoff threshold from activations (Eq. 3): with n values a (dev, fp32;
 * the absolute value is taken inside) returns in *t_out (host) the r-th
 * smallest |a|, r = ceil(k*n - 1e-6) clamped to [1, n], which is
 * min{t' : F(t') >= k} for the empirical CDF F.  k = sparsity in [0, 1];
 * k = 0 gives t = 0 without touching the device.  Selection is exact (a
 * radix select on the fp32 bit patterns).  Synchronises `stream`. */
cats_status cats_threshold_from_acts(const float* acts, int64_t n, double sparsity,
                                     void* ws, size_t ws_bytes, void* stream, float* t_out);

/* Per-block cutoff calibration (Section 4.1, Eq. 3): activations of the N
 * calibration vectors (dev [N x d], fp32) through the gate, pooled over
 * all N*m values, then cats_threshold_from_acts.  *t_out is host.
 * Synchronises `stream`.  Needs max_calib_values >= N*m in the workspace. */
cats_status cats_calibrate_threshold(const cats_layer* layer, const float* calib_x, int32_t N,
                                     double sparsity, void* ws, size_t ws_bytes, void* stream,
                                     float* t_out);

/* CATS MLP forward (Eq. 1 with the CATS_t activation of Eq. 5; the
 * "MLP using CATS" algorithm of Section 4.3):
 *   v = SiLU(x W_gate); Mask = |v| >= t; x1 = (x W_up[Mask]) * v[Mask];
 *   y = residual + x1 W_down[Mask]
 * for B rows x (dev [B x d]); y (dev [B x d]); residual dev [B x d] or
 * NULL.  t >= 0 (t = +inf masks everything, y = residual or 0); each row
 * has its own Mask, and the rows of W_up / W_down read are the union of
 * the rows' masks.  Only the active rows of W_up and W_down are read.
 * aux may be NULL.  y must not alias x.  Enqueue only. */
cats_status cats_mlp_forward(const cats_layer* layer, const float* x, int32_t B, float t,
                             const float* residual, float* y, const cats_forward_aux* aux,
                             void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the CATS
 * forward above with the same arguments, semantics and kernels, minus the
 * workspace.  Its scratch memory is a fixed array of
 * CATS_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends; the call itself allocates nothing.  Blocks and
 * batches whose cats_workspace_bytes(d, m, B, 0) exceeds that size are
 * rejected with CATS_ERR_WORKSPACE before any device work (the batch-1
 * forward fits up to d = 8192 with m = 28672; 4 rows at d = 4096,
 * m = 11008).  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (other streams, other threads) race and must be
 * serialised by the caller.  Enqueue only. */
#define CATS_NOALLOC_SCRATCH_BYTES (32u << 20)
cats_status cats_mlp_forward_noalloc(const cats_layer* layer, const float* x, int32_t B, float t,
                                     const float* residual, float* y, const cats_forward_aux* aux,
                                     void* stream);

/* Dense gated MLP (Eq. 1, every neuron kept): the comparison baseline
 * ("Dense" of Section 5.3).  Same arguments and layouts as the forward. */
cats_status cats_mlp_dense(const cats_layer* layer, const float* x, int32_t B,
                           const float* residual, float* y, void* ws, size_t ws_bytes,
                           void* stream);

/* Residual stack of CATS MLP blocks: the MLP half of a decoder's decode
 * step, with the attention sub-layers left out (the paper sparsifies only
 * the MLP blocks, Section 4; norms and residuals are outside its formulas,
 * Appendix B).  For l = 0 .. L-1:
 *   x_{l+1} = x_l + MLP_l(RMSNorm(x_l))
 * with unit-gain RMSNorm of epsilon eps (computed inside the fused kernel)
 * and MLP_l the CATS forward of layers[l] at threshold t[l] (host array of
 * L values, each >= 0), or the dense MLP for every layer when t is NULL.
 *   layers   host array of L blocks (1 <= L <= CATS_MAX_LAYERS), one d for
 *            all; m may differ per layer
 *   x0       dev [B x d] fp32, the residual stream entering layer 0
 *   x_out    dev [B x d] fp32, receives x_L; must not overlap x0 or ws
 *   x_all    dev [(L+1) x B x d] fp32 or NULL; receives every x_l
 *            (x_all[0] = x0)
 *   aux      host array of L cats_forward_aux (layer l's outputs for its
 *            MLP, as in cats_mlp_forward) or NULL; needs t
 * Workspace: cats_workspace_bytes(d, the largest m, B, 0).  Enqueue only;
 * two launches per layer on `stream`. */
cats_status cats_stack_forward(const cats_layer* layers, int32_t L, const float* t,
                               const float* x0, int32_t B, float eps, float* x_out,
                               float* x_all, const cats_forward_aux* aux, void* ws,
                               size_t ws_bytes, void* stream);

/* Per-token top-k variant of the forward (the appendix comparing target and
 * actual sparsity suggests enforcing the target sparsity per layer at
 * inference as future work): row b keeps the neurons with
 * |v_bj| >= t_b, where t_b is the r-th smallest of its own m values |v_b.|,
 * r = ceil(sparsity * m - 1e-6) clamped to [1, m] (Eq. 3 over one token);
 * sparsity = 0 keeps every neuron.  Each row keeps at least m - r + 1
 * neurons (ties at t_b are kept).  Three steps on `stream`: the gate
 * activations of all rows, an exact per-row radix select (for a single row
 * of up to 16384 neurons done by the gate kernel's last block), and the
 * fused forward reading those activations (W_gate is read once).  Arguments as
 * cats_mlp_forward; t_out: dev [B] fp32 receiving t_b, or NULL.  Rows are
 * processed in passes of at most 8 (the vector-ALU kernel).  Workspace:
 * cats_topk_workspace_bytes(d, m, B).  Enqueue only. */
size_t cats_topk_workspace_bytes(int32_t d, int32_t m, int32_t max_batch);
cats_status cats_mlp_forward_topk(const cats_layer* layer, const float* x, int32_t B,
                                  double sparsity, const float* residual, float* y,
                                  const cats_forward_aux* aux, void* ws, size_t ws_bytes,
                                  void* stream, float* t_out);

/* The forward in the paper's own kernel structure (Section 4.3 and
 * Appendix D), for the ablation of how the up and down kernels find their
 * rows.  Four launches on `stream` per pass of at most 8 rows: the gate
 * activations v = SiLU(x W_gate) to memory, an up-projection kernel writing
 * h = v * (x W_up) on the active neurons to memory, a down-projection kernel
 * into per-block partial sums, and their fixed-order sum (+ residual).
 *   mode CATS_UNFUSED_MASK:  the up and down kernels visit every neuron and
 *        load a row only under the mask |v_j| >= t (the algorithm without
 *        atomic operations); a masked row is never read;
 *   mode CATS_UNFUSED_INDEX: the gate pass also writes each block's
 *        ascending list of the neurons active in some row (compacted without
 *        atomics), and the up and down kernels visit only those.
 * Both compute exactly what cats_mlp_forward computes (same t semantics,
 * fp32 accumulation); the fused forward is the product path, this entry
 * point exists to measure the paper's structure.  Arguments as
 * cats_mlp_forward (no aux outputs).  Workspace:
 * cats_unfused_workspace_bytes(d, m, B).  Enqueue only. */
#define CATS_UNFUSED_MASK 0
#define CATS_UNFUSED_INDEX 1
size_t cats_unfused_workspace_bytes(int32_t d, int32_t m, int32_t max_batch);
cats_status cats_mlp_forward_unfused(const cats_layer* layer, const float* x, int32_t B, float t,
                                     int32_t mode, const float* residual, float* y, void* ws,
                                     size_t ws_bytes, void* stream);

/* CATS on the input of a linear layer.  Appendix B wraps each attention
 * block's input in CATS_t, so its query / key / value projections take a
 * sparse input:
 *   y_b = residual_b + CATS_t(x_b) W,   CATS_t(z) = z where |z| >= t, else 0
 * (Eq. 4, ties kept).  Only the rows of W of the channels some batch row
 * keeps are read (the union over rows; each row keeps its own channels).
 *   w        dev [d x n] row-major, row i = input channel i (bf16 only:
 *            CATS_F32 returns CATS_ERR_UNIMPLEMENTED); 1 <= d <= CATS_MAX_M,
 *            n a positive multiple of 8, d * n * 2 <= CATS_MAX_MATRIX_BYTES
 *   x        dev [B x d] fp32, 1 <= B <= CATS_MAX_BATCH
 *   residual dev [B x n] or NULL;  y dev [B x n] (must not alias x)
 *   aux      per row, ascending: active_idx [B x d] kept channels,
 *            active_cnt [B], active_v = active_h [B x d] their values; or NULL
 * t >= 0; t = 0 keeps every channel (the dense product).  Workspace:
 * cats_sparse_input_workspace_bytes(d, n, B).  Enqueue only; may be captured
 * in a graph (the cross-block sum's counters carry a tag the host draws per
 * call, and the last block of each column tile returns its counter to zero
 * under that tag, so replays of one captured call and eager calls mix). */
size_t cats_sparse_input_workspace_bytes(int32_t d, int32_t n, int32_t max_batch);
cats_status cats_sparse_input_gemv(const void* w, int32_t d, int32_t n, int32_t wdtype,
                                   const float* x, int32_t B, float t, const float* residual,
                                   float* y, const cats_forward_aux* aux, void* ws,
                                   size_t ws_bytes, void* stream);

/* Per-block cutoffs of a stack (Eq. 3 for every block, Section 4.1): the
 * N calibration vectors (dev [N x d] fp32, the residual stream entering
 * layer 0) are propagated through the stack densely, as the thresholds
 * are set on the unsparsified model, and block l's threshold is calibrated
 * on what it sees, RMSNorm(x_l) with epsilon eps:
 *   t_out[l] = cats_calibrate_threshold(layer l, RMSNorm(x_l), sparsity)
 *   x_{l+1}  = x_l + dense MLP_l(RMSNorm(x_l))
 * t_out is a host array of L floats.  k = 0 gives t = 0 for every layer
 * without touching the device.  Workspace:
 * cats_calibrate_stack_workspace_bytes(d, largest m, N).  Synchronises
 * `stream` (once per layer).  Offline. */
size_t cats_calibrate_stack_workspace_bytes(int32_t d, int32_t max_m, int32_t N);
cats_status cats_calibrate_stack(const cats_layer* layers, int32_t L, const float* calib_x,
                                 int32_t N, double sparsity, float eps, void* ws,
                                 size_t ws_bytes, void* stream, float* t_out);

/* RMSNorm with unit gain, xn = x / sqrt(mean(x^2) + eps), rows of d fp32
 * (dev [B x d]); the normalisation in front of each MLP block of a
 * decoder stack (the paper leaves norms out of its formulas, Appendix B).
 * B >= 1, any d >= 1, eps >= 0.  Enqueue only. */
cats_status cats_rmsnorm(const float* x, float* xn, int32_t B, int32_t d, float eps,
                         void* stream);

/* Attainable read bandwidth (a measurement aid; nothing of the method):
 * streams `bytes` of device memory at `buf` (16-byte aligned, a positive
 * multiple of 16, at most 1 GiB) with the 16-byte non-temporal loads the
 * weight kernels use, from `blocks` (1..65536) workgroups of 256 threads,
 * each lane keeping `inflight` (4, 8 or 16) loads of a step outstanding.
 * runs = 0: a step's loads of all waves lie side by side (wave w reads the
 * w-th KB of each 1 KB x waves stripe); runs = 1: each wave reads its own
 * run of `inflight` KB.  `sink` is a device u32 array of `blocks` entries
 * that the kernel may write (contents meaningless).  Enqueue only; the
 * launch is timed under the name "stream_read" by cats_timer_*. */
cats_status cats_stream_read(const void* buf, size_t bytes, int32_t blocks, int32_t inflight, int32_t runs,
                             uint32_t* sink, void* stream);

/* Per-kernel timing.  While enabled, every kernel the library launches is
 * bracketed by HIP events recorded on its launch stream.  cats_timer_get
 * waits for the pending events and returns, for kernel name i, the number
 * of launches and their summed duration in ms.  Not for use under graph
 * capture. */
cats_status cats_timer_enable(int32_t on);
cats_status cats_timer_reset(void);
int32_t cats_timer_count(void);
cats_status cats_timer_get(int32_t i, const char** name, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* CATS_H */
