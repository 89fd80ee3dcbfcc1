/*
 * tgp.h -- C ABI of an MI355X (gfx950) micro-batch pipeline stage with
 * checkpointing: the GPipe method of torchgpipe (Kim et al., arXiv
 * 2004.09910) taken at the scale of one GPU.
 *
 * The network is a sequence of black-box, referentially transparent layers
 * (Sec. 3) cut into n contiguous partitions f^1..f^n (Sec. 2).  A mini-batch
 * of B samples is split into m micro-batches of b = B/m samples.  The four
 * entry points the method is built from are
 *
 *   tgp_stage_forward            task F_{i,j}   (eq. (F_ij); Sec. 2.1 checkpointing)
 *   tgp_stage_backward_recompute F'_{i,j} then B_{i,j}  (eq. (B_ij); Sec. 2.1)
 *   tgp_grad_accumulate          g^j += g_i^j   (Sec. 2, sum of g_i^j over i)
 *   tgp_pipeline_step            all tasks in deterministic clock-cycle order
 *                                (Algorithm 1, Sec. 3.2.1) and its reverse
 *
 * Conventions for every call
 *   - Tensors are NHWC.  Activations, activation gradients and weights are
 *     bfloat16 (raw 16-bit storage) for TGP_BF16 nets and float32 for
 *     TGP_FP32 nets.  Biases, weight-gradient accumulators and the loss are
 *     float32 in both.  Weights are KRSC: [cout][kh][kw][cin] for 3x3 and 1x1
 *     convolutions, [c][3][3] for depthwise.
 *   - Device pointers are plain device addresses owned by the caller.  The
 *     library never allocates device memory: the caller sizes a workspace with
 *     tgp_plan and binds it with tgp_bind_workspace.  Pointers must stay
 *     valid for as long as the calls that use them may run.
 *   - Alignment (kernels use 16-byte vector accesses along the channel
 *     dimension): whole tensors -- weights, biases and accumulators given to
 *     tgp_bind_params, and x, target and y_out of tgp_pipeline_step -- must
 *     start at a multiple of 16 bytes, loss_dev at a multiple of 4.  The
 *     micro-batch slices given to the stage calls (x_in, y_out, dy_out,
 *     dx_in and their paired forms) must start at a multiple of the largest
 *     power of two up to 16 that divides the tensor's channel row (channels x
 *     element size): 16 bytes for every tensor of 8 or more bf16 (4 or more
 *     fp32) channels in multiples of 8 (4).  Violations return TGP_EINVAL.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls enqueue work and return without synchronising; kernel faults
 *     surface at the caller's next synchronisation.
 *   - All argument and state checks run on the host before anything is
 *     enqueued.  A call that returns an error has enqueued nothing, except
 *     TGP_EHIP, which reports a failed launch (tgp_last_error names it).
 *   - A tgp_net is not thread safe.  Results are deterministic: every
 *     reduction has a fixed order, no kernel uses floating-point atomics, and
 *     kernel choice and launch shape depend only on tensor shapes.
 */
#ifndef TGP_H
#define TGP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tgp_net tgp_net;

typedef enum {
  TGP_OK = 0,
  TGP_EINVAL = 1,       /* bad argument (shape, index, NULL pointer, mismatch) */
  TGP_ESTATE = 2,       /* call out of the order the method requires */
  TGP_ENOSPACE = 3,     /* bound workspace smaller than tgp_plan asked for */
  TGP_EHIP = 4,         /* a HIP launch failed */
  TGP_EUNSUPPORTED = 5  /* layer/dtype combination not built */
} tgp_status;

typedef enum { TGP_BF16 = 0, TGP_FP32 = 1 } tgp_dtype;

/* Checkpoint policy (Sec. 2.1): ALWAYS checkpoints every micro-batch,
 * EXCEPT_LAST skips F'_{m,j} (the last micro-batch keeps its activations),
 * NEVER stores all activations.  EXCEPT_LAST with m = 1 is NEVER. */
typedef enum { TGP_CKPT_ALWAYS = 0, TGP_CKPT_EXCEPT_LAST = 1, TGP_CKPT_NEVER = 2 } tgp_ckpt;

typedef enum { TGP_CONV3X3 = 0, TGP_CONV1X1 = 1, TGP_DWCONV3X3 = 2 } tgp_kind;

/* Input transform applied before a layer's convolution:
 * MAXPOOL2: 2x2 stride-2 max-pool of the previous output (argmax ties go to
 *           the first element in row-major window order);
 * UPCAT2:   channel concat [nearest 2x upsample of the previous output,
 *           skip tensor `pop_id`] (Sec. 3.3 skip connections). */
typedef enum { TGP_PRO_NONE = 0, TGP_PRO_MAXPOOL2 = 1, TGP_PRO_UPCAT2 = 2 } tgp_prologue;

/* One layer: y = act(conv(prologue(x)) + b), act = ReLU if relu != 0.
 * Convolutions are cross-correlations, stride 1, zero padding 1 (3x3) or 0
 * (1x1).  stash_id >= 0 stashes the output as skip `stash_id` for a later
 * UPCAT2 layer (Sec. 3.3); pop_id names the skip an UPCAT2 layer consumes. */
typedef struct {
  int32_t kind;      /* tgp_kind */
  int32_t cin;       /* channels after the prologue */
  int32_t cout;
  int32_t relu;      /* 0/1 */
  int32_t bias;      /* 0/1 */
  int32_t prologue;  /* tgp_prologue */
  int32_t stash_id;  /* -1 or 0..63 */
  int32_t pop_id;    /* -1 or 0..63 (UPCAT2 only) */
} tgp_layer;

/* Schedule-trace opcodes (tgp_schedule_trace). */
enum { TGP_OP_FORWARD = 0, TGP_OP_RECOMPUTE = 1, TGP_OP_BACKWARD = 2,
       TGP_OP_ACCUMULATE = 3, TGP_OP_LOSS = 4 };

/* Creates a network description (host memory only; no device work).
 * `layers` is copied.  in_c/H/W describe one sample of the network input.
 * Errors: EINVAL for inconsistent channels or sizes, odd sizes under a pool,
 * an UPCAT2 whose skip is missing or of the wrong size, n_layers < 1;
 * EUNSUPPORTED for a kind/dtype the library does not build. */
tgp_status tgp_net_create(const tgp_layer* layers, int n_layers, int in_c, int H, int W,
                          int dtype, tgp_net** out);
void tgp_net_destroy(tgp_net* net);

/* Forward FLOPs of one sample through layer `layer` (2 per multiply-add). */
tgp_status tgp_layer_flops(const tgp_net* net, int layer, int64_t* flops);

/* Partition into n contiguous parts (Sec. 2: f = f^n o ... o f^1).
 * balance[j] = number of layers of partition j+1 (sum = n_layers, each >= 1).
 * balance == NULL picks the split that minimises the largest per-partition
 * forward FLOP count (exact dynamic programme); among such splits, the one
 * with the smallest sum of squared partition costs; then the earliest cut
 * points (Sec. 3: a partition with small pairwise resource discrepancy).
 * A later tgp_plan is required. */
tgp_status tgp_set_partition(tgp_net* net, int n, const int* balance);
tgp_status tgp_get_partition(const tgp_net* net, int* n, int* balance /* >= n entries */);

/* The same split rule as a pure function of per-layer costs: cost[L], n
 * parts; writes balance[n].  Host only. */
tgp_status tgp_balance_minmax(const int64_t* cost, int L, int n, int* balance);

/* Time-based balance (Sec. 3: partitions balanced on per-layer costs that
 * are measured by running the layers, rather than on an estimate).
 *
 * tgp_layer_times_plan plans the network as n_layers one-layer partitions
 * for one micro-batch of b samples (m = 1) under checkpoint mode `mode`,
 * keeping the current partition aside, and writes the workspace size the
 * timing needs to *bytes (the plan's workspace plus four activation buffers:
 * a layer's input, output, output gradient and input gradient).
 *
 * tgp_layer_times binds ws (device, 256-byte aligned, at least *bytes,
 * caller-owned; zeroed here, so timings see zero data), then for each layer
 * l runs F (and F' when `mode` checkpoints), B and the accumulation of
 * partition l + 1 once to warm up and `iters` times timed with HIP events on
 * `stream`, and writes the mean microseconds of those three calls to
 * us[n_layers].  Layer 0 skips its input gradient, as in tgp_pipeline_step.
 * Every layer's parameters must be bound; the accumulators are overwritten.
 * It synchronizes `stream`, then restores the partition kept aside and
 * leaves no plan (call tgp_plan again).  ESTATE without a timing plan;
 * ENOSPACE / EINVAL from the workspace binding keep the timing plan.
 *
 * tgp_balance_by_time runs tgp_layer_times and then sets the partition that
 * tgp_balance_minmax picks for the measured times (in whole nanoseconds)
 * into n parts; writes it to balance[n], and the times to us (if not NULL).
 * A later tgp_plan is required. */
tgp_status tgp_layer_times_plan(tgp_net* net, int b, int mode, size_t* bytes);
tgp_status tgp_layer_times(tgp_net* net, void* ws, size_t bytes, int iters, float* us,
                           void* stream);
tgp_status tgp_balance_by_time(tgp_net* net, void* ws, size_t bytes, int iters, int n,
                               int* balance, float* us /* NULL or n_layers entries */,
                               void* stream);

/* Binds layer parameters (device pointers, caller-owned):
 * w: weights (net dtype, KRSC); b: float32 bias (NULL iff the layer has no
 * bias); dw_acc, db_acc: float32 gradient accumulators g^j, same layouts
 * (db_acc NULL iff no bias).  Every layer must be bound before any step. */
tgp_status tgp_bind_params(tgp_net* net, int layer, const void* w, const float* b,
                           float* dw_acc, float* db_acc);

/* Concurrency lanes (1..TGP_MAX_LANES, default 1; invalidates the plan, so
 * call before tgp_plan).  The workspace holds one copy per lane of every
 * buffer a task uses only while it runs (activations of checkpointed
 * passes, transformed weights, temporaries); micro-batch i uses lane
 * (i - 1) % lanes.  With more than one lane, each micro-batch also gets its
 * own slot for g_i^j.  Tasks of different lanes may then run concurrently
 * on different streams (micro-batches have no dependency on each other,
 * which is what lets Sec. 3.2.3 give each micro-batch its own stream),
 * provided the caller keeps each lane's tasks in order on one stream (or
 * orders them with events), runs tgp_grad_accumulate(j, i) after B_{i,j}
 * and after tgp_grad_accumulate(j, i + 1) (one accumulation stream that
 * waits for each B_{i,j} does both, and keeps the sum over i in its order,
 * so results stay bit-identical), and makes B_{i,j} wait for whatever
 * produced its dy_out.  With one stream every lane count gives the same
 * results as lanes = 1. */
#define TGP_MAX_LANES 16
tgp_status tgp_set_lanes(tgp_net* net, int lanes);

/* Fixes the mini-batch size B, the micro-batch count m (B % m == 0) and the
 * checkpoint policy for the following calls, and returns the workspace size
 * in bytes.  Resets the per-task state.  Requires a partition. */
tgp_status tgp_plan(tgp_net* net, int B, int m, int ckpt_mode, size_t* workspace_bytes);

/* Binds caller-owned device memory of at least the planned size (ENOSPACE
 * otherwise).  Base address must be 256-byte aligned. */
tgp_status tgp_bind_workspace(tgp_net* net, void* dev, size_t bytes);

/* Device address of micro-batch i's (1-based) slot of skip `stash_id`
 * (grad = 0) or of the gradient flowing back into it (grad = 1); NHWC,
 * b x H x W x C of the stashing layer, net dtype.  Stage runs read exported
 * skips here and write the upstream gradients of exported skips here before
 * tgp_stage_backward_recompute.  Requires a bound workspace. */
tgp_status tgp_stash_ptr(tgp_net* net, int i, int stash_id, int grad, void** p);

/* Task F_{i,j} (eq. (F_ij)), 1-based i in 1..m and j in 1..n, for
 * micro-batch i: runs partition j's layers on x_in (b x H x W x C of the
 * partition input) and writes its output to y_out.  Skips popped here are
 * read from their stash slots; skips stashed here are written to theirs.
 * checkpoint = 1 keeps only x_in (and the popped skips) for the backward
 * (Sec. 2.1); checkpoint = 0 keeps every activation in the workspace.  The
 * flag must equal the planned policy's decision for i (EINVAL otherwise).
 * x_in and y_out must stay untouched until B_{i,j} has run.
 * ESTATE if F_{i,j} already ran in this step. */
tgp_status tgp_stage_forward(tgp_net* net, int j, int i, int checkpoint, const void* x_in,
                             void* y_out, void* stream);

/* F'_{i,j} (when F_{i,j} was checkpointed: the forward rerun from the saved
 * input with the same kernels, so bit-identical) followed by B_{i,j} (eq.
 * (B_ij)): dy_out is the gradient of the partition output (shape of y_out);
 * writes dx_in, the gradient of the partition input, unless dx_in is NULL
 * (then the first layer's data gradient is skipped).  Gradients of skips
 * popped here go to their gradient slots; skips stashed here add the
 * gradient found in theirs.  The weight gradient g_i^j is left for
 * tgp_grad_accumulate, as partial sums over pixel ranges in the workspace.
 * Order (Sec. 2.1): for a given j, i = m, m-1, .., 1, each after F_{i,j}
 * and after B_{i+1,j}; with one shared gradient slot (one lane, or a plan
 * without per-micro-batch slots) also after tgp_grad_accumulate(j, i+1);
 * ESTATE otherwise.  The accumulations still run in the order i = m..1. */
tgp_status tgp_stage_backward_recompute(tgp_net* net, int j, int i, const void* dy_out,
                                        void* dx_in, void* stream);

/* Two tasks at once (Sec. 3.2.3: micro-batches are independent).
 * tgp_stage_forward2 runs F_{i0,j} and F_{i1,j}, and
 * tgp_stage_backward_recompute2 runs F'_{i0,j} + B_{i0,j} and F'_{i1,j} +
 * B_{i1,j} with i1 = i0 - 1, layer by layer, each convolution and weight
 * gradient as one launch over both micro-batches where its kernel takes two
 * tensors.  Each micro-batch's arguments, checks and results are those of
 * the single-task call (bit-identical values); the two must be on different
 * lanes, and the backward pair needs two or more lanes (per-micro-batch
 * gradient slots), so B_{i1,j} may run before the accumulation of i0;
 * tgp_grad_accumulate still runs in the order i = m..1.  dx0 and dx1 are
 * both NULL or both set. */
tgp_status tgp_stage_forward2(tgp_net* net, int j, int i0, int i1, int checkpoint0,
                              int checkpoint1, const void* x0, const void* x1, void* y0,
                              void* y1, void* stream);
tgp_status tgp_stage_backward_recompute2(tgp_net* net, int j, int i0, int i1, const void* dy0,
                                         const void* dy1, void* dx0, void* dx1, void* stream);

/* The same for a group of count (1..16) tasks: tgp_stage_forward_n runs
 * F_{i,j} for i = i0, i0 + 1, .., i0 + count - 1 (checkpoint[k], x_in[k]
 * and y_out[k] belong to micro-batch i0 + k), and
 * tgp_stage_backward_recompute_n runs F'_{i,j} + B_{i,j} for i = i0, i0 - 1,
 * .., i0 - count + 1 (dy_out[k] and dx_in[k] belong to micro-batch i0 - k),
 * each layer's convolutions as one launch over the whole group where the
 * kernel takes that many tensors, else as launches of two and one.  Each
 * micro-batch's arguments, checks and results are those of the single-task
 * call (bit-identical values).  The group's micro-batches must be on
 * different lanes: count <= lanes (EINVAL otherwise); a backward group of
 * two or more needs per-micro-batch gradient slots (two or more lanes).
 * dx_in[k] are all NULL or all set.  The arrays hold count entries. */
tgp_status tgp_stage_forward_n(tgp_net* net, int j, int i0, int count, const int* checkpoint,
                               const void* const* x_in, void* const* y_out, void* stream);
tgp_status tgp_stage_backward_recompute_n(tgp_net* net, int j, int i0, int count,
                                          const void* const* dy_out, void* const* dx_in,
                                          void* stream);

/* g^j (+)= g_i^j into the bound float32 accumulators of partition j's layers
 * (Sec. 2: the gradient is the sum of g_i^j over i); the partial sums B_{i,j}
 * left are added up here, in an order fixed by the shapes.  overwrite must be 1
 * exactly for i = m (the first backward of a step), else 0.  Requires
 * B_{i,j} and, for i < m, the accumulation of i + 1; ESTATE otherwise. */
tgp_status tgp_grad_accumulate(tgp_net* net, int j, int i, int overwrite, void* stream);

/* The accumulations of count (1..16) micro-batches i0, i0 - 1, ..,
 * i0 - count + 1, in that order, as one launch where their pending sums lie
 * at one stride from each other (else one launch per micro-batch): the same
 * values as count tgp_grad_accumulate calls, each g_i^j added to g^j in
 * turn (Sec. 2).  overwrite must be 1 exactly for i0 = m.  Requires B_{i,j}
 * of every micro-batch of the group and, for i0 < m, the accumulation of
 * i0 + 1 (ESTATE otherwise); EINVAL for a count or a range outside 1..m. */
tgp_status tgp_grad_accumulate_n(tgp_net* net, int j, int i0, int count, int overwrite,
                                 void* stream);

/* One training step over the whole network: scatter x (B samples) into m
 * micro-batches; forward clocks k = 1..m+n-1 running F_{i,j} for i+j-1 = k
 * with j ascending (Algorithm 1); MSE loss sum (y-t)^2 / numel(target) of
 * each micro-batch's final output against its slice of `target`, with no
 * 1/2 factor; backward clocks k = m+n-1..1 with j descending, each task
 * F'_{i,j} (if checkpointed) + B_{i,j} + grad accumulate.  Writes the loss
 * (float32) to *loss_dev and the network output to y_out (may be NULL).
 * B, m, n and ckpt_mode must match tgp_plan and tgp_set_partition.
 * With more than one lane (tgp_set_lanes) the step forks from `stream`
 * onto library-owned streams (default priority), micro-batch i's tasks on
 * lane (i - 1) % lanes and the accumulations, in schedule order, on one
 * more stream that waits for each B_{i,j}, and joins back into `stream`
 * before the loss; the results are bit-identical to one lane.  The streams
 * are created on first use (on the current device) and destroyed with the
 * net; the fork and join are events, so the step can be captured into a
 * HIP graph from `stream`.  If a task fails (TGP_EHIP) the step is
 * abandoned: the lanes are still joined into `stream`, every task returns to
 * its idle state, and the next tgp_pipeline_step (or stage call) starts a
 * fresh step; the work already enqueued still runs and the outputs and
 * accumulators hold partial results. */
tgp_status tgp_pipeline_step(tgp_net* net, const void* x, const void* target, int B, int m,
                             int n, int ckpt_mode, float* loss_dev, void* y_out, void* stream);

/* tgp_pipeline_step without a bound workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The step runs exactly as
 * tgp_pipeline_step (same kernels, bit-identical results) with the library's
 * own static device array of TGP_STATIC_SCRATCH_BYTES as its workspace; it
 * calls no hipMalloc, hipFree or other allocating routine.  The caller still
 * passes x, target, loss_dev and y_out (same meaning, layout and ownership
 * as tgp_pipeline_step) and must have called tgp_plan; a workspace bound
 * with tgp_bind_workspace is left bound and unused by this call.  Each
 * device holds its own copy of the array from the first call on it until
 * the process ends; every call on one device shares that copy and leaves
 * its contents behind, so calls that may run at the same time on one device
 * (other streams, other threads, other nets) race and must be serialised by
 * the caller.  Nothing in the array needs to start at zero.
 * Errors: ENOSPACE when the plan's workspace exceeds TGP_STATIC_SCRATCH_BYTES;
 * EINVAL with more than one lane (lane streams would have to be created);
 * EUNSUPPORTED on a device index of TGP_STATIC_MAX_DEVICES or more; all
 * errors of tgp_pipeline_step otherwise. */
#define TGP_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
#define TGP_STATIC_MAX_DEVICES 64
tgp_status tgp_pipeline_step_static(tgp_net* net, const void* x, const void* target, int B,
                                    int m, int n, int ckpt_mode, float* loss_dev, void* y_out,
                                    void* stream);

/* Host-only: the (op, i, j) sequence tgp_pipeline_step issues for (m, n,
 * ckpt_mode), as 3 int32 per op in `ops` (capacity `cap` ops); *count gets
 * the number of ops.  EINVAL if cap is too small (count still set). */
tgp_status tgp_schedule_trace(int m, int n, int ckpt_mode, int32_t* ops, int cap, int* count);

/* Measurement hooks (outside the method).  While enabled on the calling
 * thread, each kernel launch is bracketed by two HIP events on its stream.
 * tgp_profile_read waits for the recorded events, returns one entry per
 * kernel (launch count, summed duration in ms, and the algorithmic FLOPs and
 * HBM bytes the launcher attributes to those launches) and clears the record.
 * EINVAL if cap is too small (count still set). */
typedef struct {
  char name[96];
  int64_t launches;
  double ms;
  double flops;
  double bytes;
} tgp_kernel_stat;
tgp_status tgp_profile_enable(int enable);
tgp_status tgp_profile_read(tgp_kernel_stat* out, int cap, int* count);
/* Drops the recorded events without reading them. */
tgp_status tgp_profile_clear(void);

/* Kernel-selection overrides, for testing and tuning only (process-wide,
 * not synchronised: set them while no other thread launches work).  Each
 * returns the previous value.
 *
 * tgp_debug_set_fwd_variant(v) forces the kernel family and tile
 * configuration of every bf16 convolution launch that goes through the
 * forward-convolution path (forward, recompute and data gradient): 0 is the
 * automatic per-shape plan; 1..7 row-stage tiles; 100..102 per-tap tiles;
 * 201..207 persistent row-stage tiles; 300 the 16x16x32 row-tiled kernel
 * (301 + i its configuration i); 400 the nine-tap whole-row kernel (401 + i
 * its configuration i).  A forced choice that does not fit a shape falls
 * back to the per-tap kernel.
 *
 * tgp_debug_set_rowtile_mask(m) enables kernel families in the automatic
 * plan: bit 0 the row-tiled kernel for forward calls, bit 1 for data-gradient
 * calls, bit 2 the row-blocked weight gradient, bit 3 the nine-tap whole-row
 * kernel (default: bits 0-3 set); bit 4 restricts the nine-tap kernel to
 * its four-wave layouts (by default it picks among four- and eight-wave
 * ones), bit 5 makes the row-blocked weight gradient use its four-wave
 * layout at every width, bit 6 keeps it at one filter row per work item
 * (by default launches of several micro-batches of four or more samples at
 * widths 96, 48 and 24 take all three filter rows per item, with the values
 * of the four-wave layout). */
int tgp_debug_set_fwd_variant(int v);
int tgp_debug_set_rowtile_mask(int m);

/* Launch-failure injection, for tests of the error path only (per calling
 * thread).  tgp_debug_fail_launch(n) with n >= 1 makes the n-th kernel launch
 * from now on fail as a rejected launch would: that launch and every later
 * one of the same library call are skipped (nothing reaches the device) and
 * the call returns TGP_EHIP with tgp_last_error naming the operation.  n = 0
 * disarms.  Returns the launches that were left before the previous setting
 * would have fired (0 if disarmed). */
int tgp_debug_fail_launch(int n);

/* Message of the last failed call on this thread ("" if none). */
const char* tgp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TGP_H */
