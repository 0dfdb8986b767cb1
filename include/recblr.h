/*
 * recblr.h - C ABI of librecblr.so, the MI355X (gfx950) BD-LRU scan library.
 *
 * The behavior-dependent linear recurrent unit of RecBLR ("Behavior-Dependent
 * Linear Recurrent Units for Efficient Sequential Recommendation", CIKM 2024,
 * arXiv 2406.12580), section 3.2:
 *
 *     r_t = sigmoid(W_r x_t + b_r)            recurrence gate
 *     i_t = sigmoid(W_i x_t + b_i)            input gate
 *     alpha_t = exp(-softplus(Lambda) * r_t)
 *     beta_t  = sqrt(1 - alpha_t^2) * i_t
 *     h_t     = alpha_t * h_{t-1} + beta_t * x_t        (eq:linrnn)
 *
 * computed for every channel (b, d) of a [B, L, D] batch of behavior
 * sequences.  Section 3.3 evaluates the recurrence as a parallel scan with the
 * associative operator (a2, b2) . (a1, b1) = (a2 a1, a2 b1 + b2); the library
 * does the same on the GPU with a chunked scan, and its results equal the
 * sequential recurrence up to floating-point rounding order.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are dense and row-major: [B][L][D] with D fastest, [B][D], [D],
 *    and gate weights [D][D] stored [out][in], so z[d] = sum_k W[d][k] x[k] + b[d].
 *  - Tensor pointers are DEVICE pointers (hipMalloc'ed or equivalent) and must
 *    be aligned to their element size.  `io` selects the element type of
 *    the sequence tensors: RECBLR_F32 (float) or RECBLR_BF16 (bfloat16, stored
 *    as its 16-bit pattern).  Lambda, h0, hT, dh0, dLambda, h_prev, h_next and
 *    the weight gradients are always float.  Gate weights and biases use `io`.
 *  - All arithmetic is fp32; recurrent state and carries are fp32; bf16 outputs
 *    are rounded to nearest even.
 *  - h0 == NULL means a zero initial state (the paper's c_1 = beta'_1).
 *    Optional outputs (hT, dh0) may be NULL.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *    enqueues work on it and returns; results are valid once the stream has
 *    been synchronised.  The library never synchronises, never allocates and
 *    keeps no state between calls, so concurrent calls on different streams
 *    with disjoint buffers are safe.
 *  - `ws`/`ws_bytes`: caller-owned device scratch of at least
 *    recblr_workspace_size(...) bytes, 256-byte aligned (NULL is accepted when
 *    that size is 0).  Its contents need no initialisation and are garbage
 *    after the call, with one exception: where recblr_bdlru_scan_forward or
 *    recblr_bdlru_scan_backward (and their _timed variants) take a nonzero
 *    workspace, the uint32 at byte offset 4 of ws is a status word that the
 *    call sets to 0 and that becomes nonzero only if a workgroup's bounded
 *    wait for another workgroup's state ran out (the affected outputs are
 *    then NaN): it tells such a NaN apart from one that came with the inputs.
 *    The waits are bounded for safety; tiles are handed out in an order that
 *    lets every wait end, so the word stays 0 in normal operation.  Two calls
 *    in flight at once must not share a workspace.
 *  - Validation happens on the host, before anything is enqueued; a call that
 *    returns an error has enqueued nothing.  Output buffers must not overlap
 *    inputs or each other (recblr_bdlru_scan_step and recblr_bdlru_step allow
 *    h_next == h_prev exactly).  B == 0 or D == 0 is a no-op; L == 0 writes only
 *    hT := h0 (forward) and dh0 := dhT, dLambda := 0 (backward).
 *  - NaN and Inf inputs propagate; they are not checked.  Results are
 *    deterministic: the same inputs give bitwise identical outputs.
 */
#ifndef RECBLR_H_
#define RECBLR_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
enum {
    RECBLR_OK = 0,
    RECBLR_ERR_INVALID_ARGUMENT = -1, /* NULL/misaligned/overlapping pointer, negative size */
    RECBLR_ERR_UNSUPPORTED = -2,      /* unknown dtype or op, size beyond the supported range */
    RECBLR_ERR_WORKSPACE = -3,        /* ws NULL, too small or not 256-byte aligned */
    RECBLR_ERR_HIP = -4,              /* a kernel launch failed (hipGetLastError) */
    RECBLR_ERR_SCRATCH = -5           /* recblr_bdlru_scan_backward_noalloc: the problem needs
                                         more scratch than the static device buffer holds */
};

/* Element type of the sequence tensors. */
enum { RECBLR_F32 = 0, RECBLR_BF16 = 1 };

/* Operations, for recblr_workspace_size. */
enum {
    RECBLR_OP_SCAN_FORWARD = 0,
    RECBLR_OP_SCAN_BACKWARD = 1,
    RECBLR_OP_FORWARD = 2,
    RECBLR_OP_BACKWARD = 3,
    RECBLR_OP_STEP = 4,
    RECBLR_OP_GATED_FORWARD = 5,
    RECBLR_OP_GATED_BACKWARD = 6,
    RECBLR_OP_SCAN_BACKWARD_METHOD = 7
};

/* Human-readable name of a status code (static string, never NULL). */
const char* recblr_status_string(int status);

/* Bytes of workspace `op` needs for this problem; 0 means none (ws may be NULL).
 * For RECBLR_OP_STEP, L is ignored.  Returns 0 for invalid arguments too, which
 * the entry point then reports. */
size_t recblr_workspace_size(int op, int64_t B, int64_t L, int64_t D, int io);

/*
 * Gated scan forward from given gate pre-activations (section 3.2 with
 * z_r = W_r x + b_r and z_i = W_i x + b_i already computed).  This is the
 * hot path: the gate activation is fused into the scan's loads.
 *   x, z_r, z_i : [B][L][D] io        inputs
 *   lambda      : [D] float           decay parameter Lambda
 *   h0          : [B][D] float|NULL   initial state
 *   h           : [B][L][D] io        output, h_t for every step
 *   hT          : [B][D] float|NULL   output, final state h_L (kept in fp32)
 */
int recblr_bdlru_scan_forward(const void* x, const void* z_r, const void* z_i,
                              const float* lambda, const float* h0, void* h, float* hT,
                              int64_t B, int64_t L, int64_t D, int io, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * Backward of recblr_bdlru_scan_forward: the exact adjoint of the recurrence
 * of eq:linrnn and of the gate equations of section 3.2 (the paper states no
 * backward pass; see the derivation in scan_bwd.hip).
 *   h    : [B][L][D] io    the forward output (saved activations)
 *   dh   : [B][L][D] io    dLoss/dh_t for every step
 *   dhT  : [B][D] float|NULL  dLoss/dh_L of the final-state output
 * Outputs:
 *   dx   : [B][L][D] io    dLoss/dx through beta'_t = beta_t x_t only (the
 *                          z inputs are independent here)
 *   dz_r, dz_i : [B][L][D] io
 *   dlambda    : [D] float  summed over b and t in a fixed order (fp64 final stage)
 *   dh0        : [B][D] float|NULL
 */
int recblr_bdlru_scan_backward(const void* x, const void* z_r, const void* z_i,
                               const float* lambda, const float* h0, const void* h,
                               const void* dh, const float* dhT, void* dx, void* dz_r,
                               void* dz_i, float* dlambda, float* dh0, int64_t B, int64_t L,
                               int64_t D, int io, void* ws, size_t ws_bytes, void* stream);

/*
 * Measurement variants of the two scans above: the same work, arguments and
 * errors, plus two caller-created HIP events (hipEvent_t; either may be NULL)
 * that take the start and end times of the scan kernel itself: the kernel is
 * launched with hipExtLaunchKernelGGL, which stamps the events from the
 * kernel's dispatch.  The look-back state reset before it and, in the
 * backward, the dLambda reduction after it fall outside the pair, so the time
 * between the events is that one kernel's duration.  The events are set only
 * when the scan kernel is launched (not for B, D or L = 0); a validation error
 * sets neither.  A launch with events still idles the stream for about 5 us on
 * each side of the kernel on MI355X, so a loop timed for throughput should
 * call the plain entry points.
 */
int recblr_bdlru_scan_forward_timed(const void* x, const void* z_r, const void* z_i,
                                    const float* lambda, const float* h0, void* h, float* hT,
                                    int64_t B, int64_t L, int64_t D, int io, void* ws,
                                    size_t ws_bytes, void* stream, void* ev_begin,
                                    void* ev_end);
int recblr_bdlru_scan_backward_timed(const void* x, const void* z_r, const void* z_i,
                                     const float* lambda, const float* h0, const void* h,
                                     const void* dh, const float* dhT, void* dx, void* dz_r,
                                     void* dz_i, float* dlambda, float* dh0, int64_t B,
                                     int64_t L, int64_t D, int io, void* ws, size_t ws_bytes,
                                     void* stream, void* ev_begin, void* ev_end);

/*
 * recblr_bdlru_scan_backward for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same work, arguments, results and errors, with no
 * workspace argument.  The scratch of its kernels (look-back state words and
 * ticket, per-tile dLambda partials) is a static device array of 16 MiB
 * inside the library, one per GPU, held until the process ends; the call
 * allocates and frees nothing.  The array's address on the current device is
 * looked up on the first call on that device, so make one call before
 * capturing a graph.  The kernels clear what must start at zero themselves,
 * so nothing carries over between calls; but every call on one GPU uses the
 * same array, so calls that may overlap on one GPU (two streams, two threads)
 * race and must be serialised by the caller.  Problems whose scratch
 * (recblr_workspace_size(RECBLR_OP_SCAN_BACKWARD, ...)) exceeds 16 MiB are
 * rejected with RECBLR_ERR_SCRATCH before anything is enqueued; this covers,
 * e.g., B*L*D = 2^26 at L = 2048, D = 128 (fp32) and L = 16384, D = 256 (bf16).
 * The stream must belong to the current device.
 */
int recblr_bdlru_scan_backward_noalloc(const void* x, const void* z_r, const void* z_i,
                                       const float* lambda, const float* h0, const void* h,
                                       const void* dh, const float* dhT, void* dx, void* dz_r,
                                       void* dz_i, float* dlambda, float* dh0, int64_t B,
                                       int64_t L, int64_t D, int io, void* stream);

/*
 * One recurrent step for inference (eq:linrnn applied once; the paper's
 * low-cost recurrent inference):  h_next = alpha(z_r) h_prev + beta(z_r, z_i) x.
 *   x, z_r, z_i : [B][D] io;  h_prev, h_next : [B][D] float (h_next may == h_prev)
 */
int recblr_bdlru_scan_step(const void* x, const void* z_r, const void* z_i,
                           const float* lambda, const float* h_prev, float* h_next, int64_t B,
                           int64_t D, int io, void* stream);

/*
 * Full forward with the gate projections (section 3.2): z_r = x W_r^T + b_r and
 * z_i = x W_i^T + b_i on the matrix cores, then the gated scan.
 *   W_r, W_i : [D][D] io;  b_r, b_i : [D] io or NULL (zero bias)
 * Other arguments as recblr_bdlru_scan_forward.  Supports 1 <= D <= 1024.
 */
int recblr_bdlru_forward(const void* x, const void* W_r, const void* b_r, const void* W_i,
                         const void* b_i, const float* lambda, const float* h0, void* h,
                         float* hT, int64_t B, int64_t L, int64_t D, int io, void* ws,
                         size_t ws_bytes, void* stream);

/*
 * Full backward: scan backward, then the projection backward
 *   dx += dz_r W_r + dz_i W_i,  dW = sum_rows dz^T x,  db = sum_rows dz.
 *   dx : [B][L][D] io, the TOTAL gradient with respect to x
 *   dW_r, dW_i : [D][D] float;  db_r, db_i : [D] float;  dlambda : [D] float
 *   dh0 : [B][D] float|NULL
 */
int recblr_bdlru_backward(const void* x, const void* W_r, const void* b_r, const void* W_i,
                          const void* b_i, const float* lambda, const float* h0, const void* h,
                          const void* dh, const float* dhT, void* dx, float* dW_r, float* db_r,
                          float* dW_i, float* db_i, float* dlambda, float* dh0, int64_t B,
                          int64_t L, int64_t D, int io, void* ws, size_t ws_bytes,
                          void* stream);

/* Full single step: projections of x_t, then one recurrent step
 * (section 3.2 gates, eq:linrnn), z kept on chip.
 *   x : [B][D] io;  h_prev, h_next : [B][D] float (h_next may == h_prev)
 * For bf16 I/O with D in {64, 128, 192, 256} (x, W_r, W_i 16-byte aligned)
 * persistent workgroups keep W_r and W_i in registers and the workspace is
 * not touched; other cases use the workspace of
 * recblr_workspace_size(RECBLR_OP_STEP, ...). */
int recblr_bdlru_step(const void* x, const void* W_r, const void* b_r, const void* W_i,
                      const void* b_i, const float* lambda, const float* h_prev, float* h_next,
                      int64_t B, int64_t D, int io, void* ws, size_t ws_bytes, void* stream);

/*
 * Gated recurrent layer core (Algorithm alg:gated_recurrent):
 *   x'_t = SiLU(conv_b + sum_{j<K} conv_w[d][j] hx_{t-j})   causal, depthwise
 *   h    = BD-LRU(x') with z = x' W^T + b                  (as recblr_bdlru_forward)
 *   y_t  = h_t * SiLU(hz_t)
 * The kernel size is not stated in the paper; 1 <= K <= 4, and hx before step
 * 0 counts as zero.  The linear layers around this core in the same
 * algorithm (the input projections to hx and hz, the output projection) are
 * plain GEMMs outside the library.
 *   hx, hz, y : [B][L][D] io;  h : [B][L][D] io or NULL (the BD-LRU output,
 *   kept for a backward);  conv_w : [D][K] float;  conv_b : [D] float or NULL;
 *   W_r, b_r, W_i, b_i, lambda, h0, hT : as recblr_bdlru_forward.
 * Workspace: recblr_workspace_size(RECBLR_OP_GATED_FORWARD, ...).  Where the
 * weights-resident fused forward applies (D = 128 fp32 or bf16, D = 256 bf16,
 * 16-byte aligned hx and weights) one kernel does the three lines: x' is
 * formed on load from hx rows staged in LDS, z on the matrix cores, and y is
 * stored directly (neither x', z nor h needs to reach memory).  Elsewhere x'
 * is formed by one streaming kernel first.
 * Errors: UNSUPPORTED for K outside 1..4 or D > 1024; otherwise as
 * recblr_bdlru_forward.
 */
int recblr_gated_forward(const void* hx, const void* hz, const float* conv_w,
                         const float* conv_b, int K, const void* W_r, const void* b_r,
                         const void* W_i, const void* b_i, const float* lambda, const float* h0,
                         void* y, void* h, float* hT, int64_t B, int64_t L, int64_t D, int io,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * Backward of recblr_gated_forward.  The paper gives no backward pass; this is
 * the exact chain rule through the core of Algorithm alg:gated_recurrent:
 *   dh    = dy (x) SiLU(hz)                     (dhT adds on the final state)
 *   dhz   = dy (x) h (x) SiLU'(hz)
 *   dx', dW_r, db_r, dW_i, db_i, dlambda, dh0   as recblr_bdlru_backward at x'
 *   dc    = dx' (x) SiLU'(c),  c the conv output (x' = SiLU(c))
 *   dhx_t = sum_{j<K, t+j<L} conv_w[d][j] dc_{t+j}
 *   dconv_w[d][j] = sum_{b, t>=j} dc_t hx_{t-j},  dconv_b[d] = sum_{b,t} dc_t
 *   hx, hz, conv_w, conv_b, K, W_*, b_*, lambda, h0 : the forward's inputs
 *   h    : [B][L][D] io   the forward's BD-LRU output (its `h` argument)
 *   dy   : [B][L][D] io   dLoss/dy;  dhT : [B][D] float|NULL  dLoss/dh_L
 * Outputs: dhx, dhz : [B][L][D] io;  dconv_w : [D][K] float;  dconv_b : [D]
 *   float|NULL;  dW_*, db_*, dlambda, dh0 : as recblr_bdlru_backward.  Every
 *   sum over b and t is taken in a fixed order, so results are bitwise
 *   repeatable.
 * Workspace: recblr_workspace_size(RECBLR_OP_GATED_BACKWARD, ...).  x' is
 * formed again from hx (one streaming kernel) rather than kept by the forward.
 * Errors: as recblr_gated_forward; outputs overlapping inputs or each other
 * give INVALID_ARGUMENT.
 */
int recblr_gated_backward(const void* hx, const void* hz, const float* conv_w,
                          const float* conv_b, int K, const void* W_r, const void* b_r,
                          const void* W_i, const void* b_i, const float* lambda, const float* h0,
                          const void* h, const void* dy, const float* dhT, void* dhx, void* dhz,
                          float* dconv_w, float* dconv_b, float* dW_r, float* db_r, float* dW_i,
                          float* db_i, float* dlambda, float* dh0, int64_t B, int64_t L,
                          int64_t D, int io, void* ws, size_t ws_bytes, void* stream);

/*
 * Full RecBLR model: one training step of the paper's model (sections 2 and
 * 3.1), as a model-level harness around the BD-LRU path:
 *   H = LayerNorm(Dropout(E[ids]))                      (eq:layernorm; no positions)
 *   `layers` times (behaviour-modelling layer):
 *     H1 = LayerNorm(H + Dropout(GRL(H)))  GRL: Algorithm alg:gated_recurrent with
 *          Hx, Hz = H Wx^T + bx, H Wz^T + bz (D -> E*D), the gated layer core of
 *          recblr_gated_forward (h0 = 0), output projection Wo (E*D -> D)
 *     H  = LayerNorm(H1 + Dropout(PFFN(H1)))
 *          PFFN = SiLU(H1 W1^T + b1) W2^T + b2 (eq. PFFN)
 *   logits = h_T E^T over the V items (h_T: each row's last step);
 *   loss = mean over rows of the cross entropy of softmax(logits) with targets.
 * Readings (the paper leaves them open): residual + LayerNorm after each
 * sub-layer, dropout on the embedding and on each sub-layer's output before
 * its residual sum (section 3.1 lists dropout without placing it), the cross
 * entropy of the next item at the last step.  Positions holding the padding
 * id (recblr_model_step_opts) enter as the zero vector: left padding with
 * zeros (section 3.3).  The linear layers of the behaviour-modelling layers run on
 * this library's matrix-core kernels (fp32 products for the forward and the
 * data gradients; bias, SiLU and its derivative fused in); the prediction
 * layer's products are rocBLAS fp32 GEMMs; all other steps run in this
 * library's kernels.
 *
 * Parameters are one flat float buffer, each tensor starting at a multiple of
 * 64 floats (recblr_model_param_offsets), weights [out][in], in this order:
 *   E [V][D], emb_ln_g [D], emb_ln_b [D], then per layer
 *   Wx [ED][D], bx [ED], Wz [ED][D], bz [ED], conv_w [ED][K], conv_b [ED],
 *   Wr [ED][ED], br [ED], Wi [ED][ED], bi [ED], lambda [ED], Wo [D][ED], bo [D],
 *   ln1_g [D], ln1_b [D], W1 [4D][D], b1 [4D], W2 [D][4D], b2 [D], ln2_g [D],
 *   ln2_b [D]                                               (ED = E * D)
 */
typedef struct {
    int64_t B;      /* rows (sequences) per batch */
    int64_t T;      /* steps per sequence */
    int64_t D;      /* embedding dimension: 64, 128 or 256 */
    int64_t E;      /* expansion factor of the gated recurrent layer, E * D <= 1024 */
    int64_t V;      /* items */
    int64_t layers; /* behaviour-modelling layers, 1..64 */
    int K;          /* conv taps, 1..4 */
    float ln_eps;   /* LayerNorm epsilon, >= 0 */
} recblr_model_dims;

/* Number of floats of the flat parameter (and gradient) buffer; 0 for
 * unsupported dimensions. */
size_t recblr_model_param_count(const recblr_model_dims* m);
/* Writes the offset (in floats) of each tensor, in the order above, to
 * offsets[0 .. n) and returns the number of tensors (3 + 21 * layers); -1 for
 * unsupported dimensions. */
int64_t recblr_model_param_offsets(const recblr_model_dims* m, int64_t* offsets, int64_t n);
/* Workspace bytes of recblr_model_train_step (saved activations of every
 * layer, backward scratch, the sort of the item ids); 0 if unsupported. */
size_t recblr_model_workspace_size(const recblr_model_dims* m);

/*
 * Per-step options of recblr_model_train_step (NULL: no dropout, no padding).
 *
 * Dropout is inverted dropout with drop probability `dropout`: an element is
 * kept or zeroed and kept elements are scaled by 1 / (1 - dropout) (float).
 * Its masks come from Philox4x64-10 (Salmon, Moraes, Dror and Shaw, SC 2011),
 * so any implementation can draw them: element e (row-major over [B][T][D])
 * of dropout site s (0 the embedding, 1 + 2l layer l's gated recurrent
 * output, 2 + 2l layer l's PFFN output) takes the 32-bit word e mod 8 (the
 * low half of each 64-bit output word first) of Philox4x64-10 at counter
 * (floor(e / 8), s, 0, 0) under key (seed, offset), and is dropped when that
 * word is below floor(dropout * 2^32).  The backward uses the same masks.
 * A caller that wants new masks each step changes offset (e.g. the step count).
 *
 * pad_id marks left padding: a position holding it enters as the zero vector
 * (its lookup sends no gradient to E) and is otherwise processed like any
 * other position; the prediction softmax still runs over all V ids.
 */
typedef struct {
    float dropout;   /* drop probability, 0 <= dropout < 1; 0 turns dropout off */
    int32_t pad_id;  /* padding id in [0, V), or -1 for none */
    uint64_t seed;   /* Philox key, word 0 */
    uint64_t offset; /* Philox key, word 1 */
} recblr_model_step_opts;

/* rocBLAS handle for the model step's prediction-layer GEMMs: created and
 * destroyed by the caller (creation allocates rocBLAS' own state; the step
 * itself allocates nothing).  A handle serves one stream at a time. */
int recblr_blas_create(void** handle);
int recblr_blas_destroy(void* handle);

/*
 * Forward and backward of one batch:
 *   opts : dropout and padding (may be NULL: neither);
 *   params : flat float parameters (256-byte aligned);  ids : [B][T] int32 item
 *   ids;  targets : [B] int32 next items;  grads : flat float, the layout of
 *   params (padding zero);  loss : one float.
 * Every sum over rows is taken in a fixed order (double), so loss and
 * gradients repeat bitwise for a given rocBLAS handle, GPU and opts.  An id
 * or target outside [0, V) makes the loss NaN (nothing is read out of bounds).
 * Errors: INVALID_ARGUMENT for a NULL pointer or misaligned buffer or
 * overlapping outputs, a dropout outside [0, 1) or a pad_id outside
 * [-1, V); UNSUPPORTED for dimensions outside the ranges above; WORKSPACE;
 * HIP for a failed launch or GEMM.
 */
int recblr_model_train_step(const recblr_model_dims* m, const recblr_model_step_opts* opts,
                            const float* params, const int32_t* ids, const int32_t* targets,
                            float* grads, float* loss, void* ws, size_t ws_bytes, void* blas,
                            void* stream);

/*
 * Adam (Kingma and Ba, Algorithm 1) over n floats, in place: step is the
 * 1-based update count; m1, m2 the moment buffers (zero before step 1).
 */
int recblr_adam_update(float* params, const float* grads, float* m1, float* m2, int64_t n,
                       int64_t step, float lr, float beta1, float beta2, float eps, void* stream);

/*
 * Scan algorithms of the efficiency ablation (section 4, Table tab:efficiency;
 * the two-tree scan of section 3.3, figure fig:scan): the gated scan forward
 * from a zero initial state by one of
 *   RECBLR_SCAN_CHUNKED  the production kernels (recblr_bdlru_scan_forward;
 *                        workspace as for RECBLR_OP_SCAN_FORWARD);
 *   RECBLR_SCAN_SERIAL   one wave per 64 channels walks the whole sequence,
 *                        no parallelism along it (no workspace);
 *   RECBLR_SCAN_TREE     up-sweep / down-sweep over the power of two >= L,
 *                        the leading positions padded with the identity,
 *                        i.e. left zero padding applied inside the scan
 *                        (embedding padding); L <= 4096 (no workspace).
 * Sequence padding is the caller's: pass inputs already left-padded to the
 * power of two.  Arguments as recblr_bdlru_scan_forward (h0 = 0, no hT).
 * Errors: INVALID_ARGUMENT for an unknown method; UNSUPPORTED for a tree
 * scan longer than 4096 steps.
 */
enum { RECBLR_SCAN_CHUNKED = 0, RECBLR_SCAN_SERIAL = 1, RECBLR_SCAN_TREE = 2 };
int recblr_scan_forward_method(int method, const void* x, const void* z_r, const void* z_i,
                               const float* lambda, void* h, int64_t B, int64_t L, int64_t D,
                               int io, void* ws, size_t ws_bytes, void* stream);

/*
 * Backward of the same scan algorithms, for the training side of the
 * ablation (the table times training epochs): dx, dz_r, dz_i and dLambda of
 * the gated scan from h0 = 0 (no dL/dh_T, no dh0), given the forward output
 * h and dh = dL/dh, by one of
 *   RECBLR_SCAN_CHUNKED  the production kernels (recblr_bdlru_scan_backward);
 *   RECBLR_SCAN_SERIAL   one thread per channel walks the sequence from
 *                        t = L - 1 down (one wave per 64 channels);
 *   RECBLR_SCAN_TREE     the two-tree scan of section 3.3 on the reversed
 *                        sequence of pairs (alpha_{t+1}, dL/dh_t), padded at
 *                        its end with the identity (embedding padding seen
 *                        from the other end); L <= 4096.
 * The adjoint delta_t = dL/dh_t + alpha_{t+1} delta_{t+1} is derived (the
 * paper gives the forward only); the gradient formulas are those of
 * recblr_bdlru_scan_backward.  Arguments as recblr_bdlru_scan_backward
 * without h0, dhT and dh0; bf16 I/O takes bf16 z and writes bf16 dz.
 * Workspace: recblr_workspace_size(RECBLR_OP_SCAN_BACKWARD_METHOD, ...) covers
 * every method.  dLambda sums are in a fixed order (deterministic).
 * Errors: as recblr_scan_forward_method.
 */
int recblr_scan_backward_method(int method, const void* x, const void* z_r, const void* z_i,
                                const float* lambda, const void* h, const void* dh, void* dx,
                                void* dz_r, void* dz_i, float* dlambda, int64_t B, int64_t L,
                                int64_t D, int io, void* ws, size_t ws_bytes, void* stream);

/*
 * Raw first-order recurrence h_t = a_t h_{t-1} + u_t (eq:linrnn with the
 * coefficients given directly), float only.  Same kernel as the gated scan
 * with the gate stage removed; used to check the scan against closed forms.
 *   a, u, h : [B][L][D] float;  h0, hT : [B][D] float|NULL
 */
int recblr_linear_scan_forward(const float* a, const float* u, const float* h0, float* h,
                               float* hT, int64_t B, int64_t L, int64_t D, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RECBLR_H_ */
