/*
 * layup.h -- C ABI of the LayUp layer-wise backward -> update -> gossip-mix
 * step on one AMD Instinct MI355X (gfx950).
 *
 * What the library computes (LayUp, Algorithm 1, one worker):
 *   forward pass, loss;  then for every layer ("unit") from the output back to
 *   the input: that layer's backward pass (dX and dW GEMMs), the local
 *   optimizer update of that layer as soon as its gradient exists (section
 *   3.2, layer-wise updates; Algorithm 1 "Local Update"), and the weighted
 *   average of the updated layer with a peer replica's copy of the same layer
 *   (Algorithm 1 "Peer Update", push-sum weights of section 3.1):
 *       p <- (1 - alpha) * p + alpha * q.
 *   The peer copy q is a device buffer supplied by the caller (it stands in for
 *   the gossip message of the multi-device system).  The update of layer u runs
 *   on a second HIP stream and overlaps the backward of layer u-1 (the paper's
 *   overlap of communication/update with computation, figure 1).
 *
 * Conventions
 *   - Every pointer named "device" is HIP device memory owned by the caller.
 *     The library never allocates or frees device memory; it owns only the
 *     context, HIP events and host-side tables.
 *   - Streams are hipStream_t values passed as void*.  NULL means the
 *     context's compute stream (or the default stream where no context is
 *     involved).
 *   - Calls only enqueue work; they return before the GPU finishes.  Argument
 *     errors are detected synchronously and nothing is enqueued then.
 *     Asynchronous device faults surface at layup_synchronize or at the next
 *     HIP call.
 *   - A context is not thread-safe: one host thread per context.
 *   - bf16 buffers are uint16_t bit patterns of bfloat16 values.
 *   - Every function returns a layup_status; the text of the last error of a
 *     context is returned by layup_last_error (context-free calls report
 *     through layup_global_error).  No C++ exception crosses this ABI.
 */
#ifndef LAYUP_H
#define LAYUP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct layup_ctx layup_ctx;

typedef enum {
  LAYUP_OK = 0,
  LAYUP_ERR_INVALID_ARG = 1, /* null pointer, out-of-range index or value */
  LAYUP_ERR_SHAPE = 2,       /* dimensions inconsistent or unsupported */
  LAYUP_ERR_ALIGN = 3,       /* pointer or leading dimension misaligned */
  LAYUP_ERR_DTYPE = 4,       /* unsupported precision / model combination */
  LAYUP_ERR_STATE = 5,       /* call out of order (e.g. backward before forward) */
  LAYUP_ERR_HIP = 6          /* a HIP runtime call failed; see the error text */
} layup_status;

typedef enum { LAYUP_SGD_MOMENTUM = 0, LAYUP_ADAMW = 1 } layup_optim;

/* Optimizer hyperparameters of the local update (Algorithm 1 "Local Update",
 * realised as the optimizers of the experiments, LibTorch semantics):
 *   SGD momentum: g' = g + wd*p (decayed tensors only); m = momentum*m + g';
 *                 p = p - lr*m.
 *   AdamW:        p *= 1 - lr*wd (decayed tensors only);
 *                 m = b1*m + (1-b1)*g;  v = b2*v + (1-b2)*g^2;
 *                 p -= lr/(1-b1^t) * m / (sqrt(v)/sqrt(1-b2^t) + eps).
 * step is t >= 1 (AdamW bias correction; unused by SGD). */
typedef struct {
  int32_t kind; /* layup_optim */
  float lr, momentum, weight_decay, beta1, beta2, eps;
  int64_t step;
} layup_hparams;

/* How the locally updated layer p1 meets the peer copy q (Algorithm 1 "Peer
 * Update", weights alpha = w_sender / (w_sender + w_receiver) of section 3.1):
 *   LAYUP_MIX_PULL: p <- (1 - alpha) p1 + alpha q; q is read only.  The worker
 *                   plays the receiver for the peer's copy q after its own
 *                   local update (one worker with a resident peer buffer).
 *   LAYUP_MIX_PUSH: p <- p1 and q <- (1 - alpha) q + alpha p1, as Algorithm 1
 *                   writes it: the sender keeps its update and overwrites the
 *                   receiving replica's layer (replicas resident on one GPU). */
typedef enum { LAYUP_MIX_PULL = 0, LAYUP_MIX_PUSH = 1 } layup_mix_mode;

/* One tensor of a layer for the fused update+mix.  All pointers are device
 * pointers, 16-byte aligned (bf16 copies 8-byte aligned).
 * param/state0/state1/param_bf16 are updated in place; grad is read only;
 * peer is read only in pull mode and mixed in place in push mode; param must
 * alias neither grad nor peer.  state0 is the momentum (SGD) or first moment m
 * (AdamW); state1 the second moment v (AdamW; ignored for SGD).  param_bf16 is
 * an optional bfloat16 copy rewritten from the new float32 param; peer_bf16
 * (push mode only, nullable) the same for the peer.  decay selects weight
 * decay for this tensor. */
typedef struct {
  float* param;
  const float* grad;
  float* state0;
  float* state1;
  float* peer;
  uint16_t* param_bf16;
  uint16_t* peer_bf16;
  int64_t numel;
  int32_t decay;
  int32_t reserved;
} layup_tensor;

/* ---------------------------------------------------------------- models */

typedef enum {
  LAYUP_MODEL_MLP_F32 = 0,  /* ReLU MLP, float32 everywhere, softmax CE */
  LAYUP_MODEL_GPT_BF16 = 1  /* GPT-2 decoder: bf16 GEMM operands and
                               activations, float32 master weights */
} layup_model;

#define LAYUP_MAX_MLP_LAYERS 8

/* Model description.  MLP: n_mlp_layers linear layers with
 * mlp_dims[0] -> mlp_dims[1] -> ... -> mlp_dims[n_mlp_layers] and ReLU between
 * them; batch rows per step.  GPT: n_layer blocks of width d_model, n_head
 * heads, MLP width d_ff, sequence length seq, batch sequences, logical
 * vocabulary vocab (the output head is tied with the token embedding).
 * n_peers is the number of resident peer replicas (>= 1). */
typedef struct {
  int32_t model;
  int32_t n_mlp_layers;
  int32_t mlp_dims[LAYUP_MAX_MLP_LAYERS + 1];
  int32_t n_layer, d_model, n_head, d_ff, seq, vocab;
  int32_t batch;
  int32_t n_peers;
} layup_config;

/* Where one parameter tensor lives inside the flat parameter buffer.  All
 * flat buffers (params, grads, state0, state1, every peer replica) share this
 * layout.  Tensors are grouped by unit; within a unit decayed tensors come
 * first.  Offsets are multiples of 64 elements.  rows x cols is the logical
 * shape (cols = 1 for vectors); the token embedding is stored with
 * padded_rows rows (vocabulary rounded up to a multiple of 64), the padding
 * rows must be zero in params and peers and are never updated. */
typedef struct {
  char name[32];
  int64_t offset;
  int64_t numel;       /* logical elements (rows * cols) */
  int32_t rows, cols, padded_rows;
  int32_t unit;
  int32_t decay;
  int32_t reserved;
} layup_tensor_info;

layup_status layup_param_layout(const layup_config* cfg, int32_t* n_tensors, int32_t* n_units,
                                int64_t* total_elems);
layup_status layup_tensor_layout(const layup_config* cfg, int32_t index, layup_tensor_info* out);

/* Caller-owned device buffers of a model (all in the flat layout above).
 * peers holds n_peers replicas back to back (n_peers * total_elems floats).
 * params_bf16 is required for GPT (the GEMMs read weights from it) and
 * ignored for the MLP.  v is required for AdamW.  trace (nullable) receives
 * (step, unit) int32 pairs, one per unit update, in the order the updates
 * run; trace_counter (device int32, required with trace) counts appended
 * pairs and is never reset by the library. */
typedef struct {
  float* params;
  float* grads;
  float* m;
  float* v;
  const float* peers;
  uint16_t* params_bf16;
  int32_t* trace;
  int32_t* trace_counter;
  int32_t trace_capacity; /* pairs */
  int32_t reserved;
} layup_buffers;

/* Bytes of device workspace (activations saved by the forward, gradient
 * scratch, split-K partials) the model needs; 256-byte alignment. */
layup_status layup_workspace_size(const layup_config* cfg, size_t* bytes);

/* Create a context.  workspace: device, >= layup_workspace_size bytes,
 * 256-byte aligned.  compute_stream runs forward and backward;
 * update_stream runs the per-unit update+mix (may equal compute_stream,
 * which serialises the two).  Streams must be default priority. */
layup_status layup_init(layup_ctx** out, const layup_config* cfg, const layup_buffers* bufs,
                        void* workspace, size_t workspace_bytes, void* compute_stream,
                        void* update_stream);
void layup_destroy(layup_ctx* ctx);
const char* layup_last_error(const layup_ctx* ctx);
const char* layup_global_error(void);
layup_status layup_synchronize(layup_ctx* ctx);

/* Rewrite params_bf16 from params for every unit (call after the caller
 * changes params outside the library).  Enqueued on the compute stream. */
layup_status layup_refresh_shadow(layup_ctx* ctx);

/* Forward pass and loss (Algorithm 1 "Forward pass"), followed by the
 * gradient of the mean loss with respect to the logits.
 *   GPT: tokens device int32 [batch, seq+1]; inputs are tokens[:, :seq],
 *        targets tokens[:, 1:].  x must be NULL.
 *   MLP: tokens device int32 [batch] class labels; x device float32
 *        [batch, mlp_dims[0]].
 * loss_out: device float32 scalar (nullable).  Enqueued on the compute
 * stream (with a separate update stream, half of the batch and the token
 * sort on that stream).  Valid only once the previous step's updates are
 * done (the library orders this itself through the streams).  tokens and x
 * are read asynchronously: the caller keeps them allocated and unchanged
 * until the step's work on both streams is done (the compute stream's join
 * at the end of layup_step_ex, or layup_synchronize). */
layup_status layup_forward(layup_ctx* ctx, const int32_t* tokens, const float* x, float* loss_out);

/* Backward pass of one unit (Algorithm 1 "Backward pass at layer l"):
 * writes the unit's parameter gradients into grads and the gradient with
 * respect to the unit's input into the workspace, then records the unit's
 * "gradient ready" event (Algorithm 1 "Notify").  Units must be called in
 * reverse order n_units-1 ... 0 after layup_forward. */
layup_status layup_layer_backward(layup_ctx* ctx, int32_t unit);

/* Update+mix of one unit of the model (Algorithm 1 "Local Update" and "Peer
 * Update") on the update stream, after the unit's gradient-ready event.
 * peer_slot selects the resident peer replica.  disagreement (device float,
 * nullable) receives sum((p_updated - q)^2) over the unit, taken before the
 * mix.  Appends (step, unit) to the trace. */
layup_status layup_unit_update_mix(layup_ctx* ctx, int32_t unit, const layup_hparams* hp,
                                   float alpha, int32_t peer_slot, float* disagreement);

/* Fused update+mix of arbitrary tensors (one layer of any model), single pass,
 * HBM bound: reads p, g, m, (v), q once and writes p, m, (v), (p_bf16) once,
 * and in push mode also q and (q_bf16).  mix_mode is a layup_mix_mode.
 * ctx may be NULL; stream NULL = the context's update stream (or the default
 * stream without a context).  disagreement (device float, nullable, needs a
 * context) receives sum((p_updated - q)^2) summed over the tensors, taken
 * before the mix (appendix, model disagreement).  n_tensors >= 1; a tensor
 * with numel 0 is skipped and its pointers are not used (they may be NULL);
 * with every tensor empty the disagreement is 0. */
layup_status layup_layer_update_mix(layup_ctx* ctx, const layup_tensor* tensors, int32_t n_tensors,
                                    const layup_hparams* hp, float alpha, int32_t mix_mode,
                                    float* disagreement, void* stream);

/* layup_layer_update_mix without a context, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same kernels and results, with the
 * disagreement output (device float, nullable) allowed.  Its per-workgroup
 * partial sums live in a fixed array of the library in device memory
 * (16384 floats = 64 KiB per GPU, kept until the process ends).  The
 * update+mix grid is capped at that many workgroups (larger tensors are
 * walked in a grid-stride loop), so tensors of any size fit; with a
 * disagreement output a call takes at most 16 tensors (one launch), more are
 * refused with LAYUP_ERR_INVALID_ARG.  Nothing is allocated or freed.  Every
 * call on one GPU shares that GPU's array: calls with a disagreement output
 * that overlap on one GPU (different streams, or different host threads)
 * race and may report wrong sums; their tensor updates are unaffected.
 * Each call writes every partial it reads, so nothing needs clearing
 * between calls.  stream NULL = the default stream.  Errors are reported
 * through layup_global_error. */
layup_status layup_layer_update_mix_static(const layup_tensor* tensors, int32_t n_tensors,
                                           const layup_hparams* hp, float alpha, int32_t mix_mode,
                                           float* disagreement, void* stream);

/* Update+mix of several units whose gradients are all ready (Algorithm 1's
 * updater taking the layers in backward order: "Local Update" and "Peer
 * Update" of each), in as few passes as possible.  tensors are listed unit by
 * unit in the order the units are visited (output side first); units[i]
 * (host array) is tensor i's unit id, 0 <= id < 2^30, and a unit's tensors
 * are adjacent (a unit id that reappears after another unit is
 * LAYUP_ERR_INVALID_ARG).  When every non-empty tensor sits at the same place
 * in the param, grad, state and peer buffers (the same byte distance from
 * param to grad, state0, state1 and peer for each tensor, bf16 copies at the
 * param's element offset: a flat layout such as layup_tensor_layout's) and
 * the tensors span fewer than 2^31 elements, up to 192 tensors of whole units
 * go in one launch, their chunks numbered unit by unit in list order;
 * otherwise each unit is its own launch (as layup_layer_update_mix).  The
 * result is the same either way.  trace (device, nullable; trace_counter
 * required with it) receives one (trace_step, unit) pair per unit in list
 * order.  No disagreement output.  stream NULL = the default stream; no
 * context; errors through layup_global_error.  Tensor rules as
 * layup_tensor. */
layup_status layup_units_update_mix(const layup_tensor* tensors, const int32_t* units, int32_t n_tensors,
                                    const layup_hparams* hp, float alpha, int32_t mix_mode, int32_t* trace,
                                    int32_t* trace_counter, int32_t trace_capacity, int32_t trace_step,
                                    void* stream);

/* Push-mode update of one unit of the model (Algorithm 1 "Local Update",
 * "Communication" and "Peer Update" as written): the worker's own layer gets
 * the local update, then the receiving replica's copy of the layer becomes
 * (1 - alpha) q + alpha p_updated.  peer_params (device float, flat layout of
 * this model's configuration) is the receiving replica's parameter buffer,
 * mixed in place; peer_params_bf16 (nullable) its bfloat16 copy, rewritten
 * for the mixed elements.  The receiver must not run a step of its own
 * concurrently.  Otherwise as layup_unit_update_mix. */
layup_status layup_unit_update_push(layup_ctx* ctx, int32_t unit, const layup_hparams* hp, float alpha,
                                    float* peer_params, uint16_t* peer_params_bf16,
                                    float* disagreement);

/* When the unit updates run relative to the backward pass.
 *   LAYUP_SCHEDULE_LAYERWISE:      update+mix of unit u as soon as its
 *                                  gradient exists (section 3.2, LayUp),
 *                                  overlapping the backward of unit u-1.
 *   LAYUP_SCHEDULE_AFTER_BACKWARD: all units' update+mix after the whole
 *                                  backward pass (the GoSGD-style schedule
 *                                  the paper compares against).
 * On one worker both produce the same numbers (no unit's backward reads a
 * unit updated before it); they differ in when each update lands. */
typedef enum {
  LAYUP_SCHEDULE_LAYERWISE = 0,
  LAYUP_SCHEDULE_AFTER_BACKWARD = 1,
  /* layer-wise, with each GPT block's weight matrices updated and mixed by
   * their own dW GEMM (its epilogue, or its split-K sum) right after the
   * block's dX GEMMs have read them: the matrices' gradients are never
   * written to HBM (grads keeps stale values for them); the block's vectors
   * and the embedding / final-LayerNorm units take the update+mix kernel as
   * in the layer-wise schedule.  GPT model, pull form, no disagreement. */
  LAYUP_SCHEDULE_FUSED_DW = 2
} layup_schedule;

/* Arguments of layup_step_ex. */
typedef struct {
  const int32_t* tokens;        /* as layup_forward */
  const float* x;               /* as layup_forward */
  const layup_hparams* hp;
  float alpha;                  /* mixing weight of the peer side */
  int32_t schedule;             /* layup_schedule */
  int32_t mix_mode;             /* layup_mix_mode */
  int32_t peer_slot;            /* pull: resident peer replica */
  float* push_params;           /* push: receiving replica's params (device) */
  uint16_t* push_params_bf16;   /* push: its bfloat16 copy (nullable) */
  float* loss_out;              /* device float scalar, nullable */
  float* disagreement;          /* device float [n_units], nullable */
} layup_step_args;

/* One whole step: forward, then for u = n_units-1 ... 0
 * layup_layer_backward(u) on the compute stream and the unit's update+mix on
 * the update stream, scheduled as args->schedule says, then the compute
 * stream waits for the update stream (join).  Records the per-unit timeline
 * read by layup_unit_timeline. */
layup_status layup_step_ex(layup_ctx* ctx, const layup_step_args* args);

/* layup_step_ex with the layer-wise schedule and pull mode. */
layup_status layup_step(layup_ctx* ctx, const int32_t* tokens, const float* x,
                        const layup_hparams* hp, float alpha, int32_t peer_slot, float* loss_out,
                        float* disagreement /* device [n_units] or NULL */);

/* Timeline of the last completed step of the context (waits for it), in
 * milliseconds from the start of the step's forward pass, from HIP events:
 * forward_ms (host float, nullable) when the forward pass and loss gradient
 * ended; for every unit, ready_ms when its gradient was ready (end of its
 * backward on the compute stream) and applied_ms when its update+mix had
 * been applied (end of the launch on the update stream).  applied - ready is
 * the delay with which the unit's update lands, the drift that section 3.2
 * counts per layer; the last ready time minus forward_ms is the backward
 * time.  ready_ms and applied_ms are host arrays of n_units floats.
 * LAYUP_ERR_STATE if no whole step has run. */
layup_status layup_unit_timeline(layup_ctx* ctx, float* forward_ms, float* ready_ms, float* applied_ms);

/* GEMM timing of the path: with enable != 0, every later backward of a GPT
 * block brackets each of its linear layers' dX and dW GEMMs (and their
 * split-K sums) with HIP events on the compute stream; enabling or disabling
 * waits for the context and resets the counters.  layup_gemm_timing_read
 * waits for the context and returns the summed GEMM time in milliseconds,
 * the number of timed GEMMs and their algorithmic FLOPs (2 M N K each).  The
 * brackets include each launch's dispatch (a few microseconds per GEMM) and
 * the events slow the step; leave timing off when timing steps. */
layup_status layup_gemm_timing(layup_ctx* ctx, int32_t enable);
layup_status layup_gemm_timing_read(layup_ctx* ctx, float* total_ms, int32_t* launches, double* flops);

/* ------------------------------------------------------------- push-sum */

/* Push-sum weights of the workers (section 3.1): each starts at 1/M; a sender
 * halves its weight when it sends (Algorithm 1, start of the updater's
 * round); the receiver mixes the incoming layers with
 * alpha = w_sender / (w_sender + w_receiver); after the round the receiver's
 * weight grows by the sender's.  Host arithmetic in double on the caller's
 * array w[n_workers]; sum(w) is unchanged by a send followed by its receive.
 *   send:    w[sender] /= 2; *alpha_out = w[sender] / (w[sender] + w[receiver])
 *   receive: w[receiver] += w[sender]
 * Errors: null pointers, n_workers < 2, indices out of range, sender ==
 * receiver, non-positive or non-finite weights (LAYUP_ERR_INVALID_ARG, text
 * in layup_global_error). */
layup_status layup_push_sum_send(double* w, int32_t n_workers, int32_t sender, int32_t receiver,
                                 float* alpha_out);
layup_status layup_push_sum_receive(double* w, int32_t n_workers, int32_t sender, int32_t receiver);

/* Saved forward activation of the context, for inspection (device pointer
 * into the workspace).  which: 0 = block input x (f32), 1 = LN1 out (bf16),
 * 2 = qkv (bf16), 3 = attention probabilities (bf16, [B][H][T][T]; stored
 * only when the head width is not 32, 64 or 128), 4 = attention output
 * (bf16), 5 = residual after attention (f32), 6 = LN2 out (bf16), 7 = MLP
 * pre-activation (bf16), 8 = GELU out (bf16), 9 = final LN out (bf16),
 * 10 = logit gradient (bf16), 11 = final residual (f32), 12 = base-2
 * log-sum-exp of each query's scaled causal scores (f32, [B][H][T]; fused
 * attention, head width 32, 64 or 128, only), 13 = float32 gradient of the
 * loss with respect to the input of the unit whose backward ran last, i.e.
 * the output gradient the next unit's backward consumes ([batch*seq,
 * d_model]; Algorithm 1 "Backward pass at layer l" hands it down; valid
 * after layup_layer_backward of a unit >= 1 and until the next backward or
 * forward, LAYUP_ERR_STATE otherwise).  layer is the block index for 0..8
 * and 12.  dtype_out: 0 = f32, 1 = bf16.  Asking for an activation the
 * configuration does not store is LAYUP_ERR_INVALID_ARG. */
layup_status layup_activation(layup_ctx* ctx, int32_t which, int32_t layer, const void** ptr,
                              int64_t* numel, int32_t* dtype_out);

/* ------------------------------------------------------------- raw GEMM */

/* C = op(A) op(B) (+ bias[n]) with float32 accumulation, batched.
 *   a_kmajor = 1: A element (m,k) at A[m*lda + k]   (rows of A contiguous in k)
 *   a_kmajor = 0: A element (m,k) at A[k*lda + m]
 *   b_kmajor = 1: B element (k,n) at B[n*ldb + k]
 *   b_kmajor = 0: B element (k,n) at B[k*ldb + n]
 *   C element (m,n) at C[m*ldc + n]; c_f32 = 1 stores float32, 0 bfloat16
 *   (round to nearest even).
 * Batch z in [0, batch) offsets each operand by (z / inner)*s_outer +
 * (z % inner)*s_inner elements (inner >= 1).  The dX GEMM of a linear layer
 * is a_kmajor=1, b_kmajor=0; the dW GEMM a_kmajor=0, b_kmajor=0; the forward
 * a_kmajor=1, b_kmajor=1.  Contiguous dimensions and leading dimensions must
 * be multiples of 8 elements and pointers 16-byte aligned.  The float32 path
 * (layup_gemm_f32, not batched) has the same layout rules with float operands
 * and no alignment requirement; it always writes float32.  M = 0 or N = 0 is
 * a no-op; K = 0 writes C = bias (or 0).  Operands that are not read (A with
 * M = 0 or K = 0, B with N = 0 or K = 0) may be NULL. */
typedef struct {
  int32_t a_kmajor, b_kmajor;
  int64_t M, N, K;
  const void* A;
  int64_t lda;
  const void* B;
  int64_t ldb;
  void* C;
  int64_t ldc;
  int32_t c_f32;
  int32_t batch;
  int32_t inner;
  int32_t reserved;
  const float* bias;
  int64_t a_outer, a_inner, b_outer, b_inner, c_outer, c_inner;
  void* workspace;        /* device, optional: float32 split-K partials
                             (batch 1 only; split-K is chosen only when the
                             partials fit).  Either way the result is
                             deterministic; with and without a workspace the
                             summation order, and so the rounding, differ. */
  size_t workspace_bytes;
  float* a_rowsum;        /* device, optional (bf16 path, a_kmajor = 0, batch
                             1): a_rowsum[m] = sum over k of A(m, k) in
                             float32, accumulated by the same kernel from
                             the A operand it multiplies -- for the dW GEMM
                             of a linear layer (A = dY^T) the bias gradient
                             db = column sums of dY (Algorithm 1, backward
                             pass).  With split-K the workspace also holds
                             one float per row per split. */
} layup_gemm_desc;

layup_status layup_gemm_bf16(const layup_gemm_desc* d, void* stream);
layup_status layup_gemm_f32(const layup_gemm_desc* d, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LAYUP_H */
