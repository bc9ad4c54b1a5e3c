/*
 * swapnet.h -- C ABI of the block-swapped inference engine for MI355X (gfx950).
 *
 * The engine runs a network whose weights do not fit a device-memory budget.
 * It follows the problem statement of the SwapNet paper (Sec. 3, "Basic
 * Idea"): given a budget b for a model of size s > b, the model is cut into
 * ordered blocks of layers that are brought into memory and executed one by
 * one.  On this hardware a swap-in is one DMA (hipMemcpyAsync) per slab from
 * a pinned host image that already holds the device layout (the analogue of
 * the paper's copy-free dispatch, Sec. 4.2.2), into a budget-sized HBM arena
 * carved once at create time; parameters are bound by pointer into the arena
 * (assembly by reference, Sec. 5.2); swap-out is write-back free (Sec. 4.1):
 * a slab's range is reused as soon as its compute has finished.  The next
 * slab is loaded on a copy stream while the current one computes (the m = 2
 * parallel blocks of Sec. 6.2.2), ordered by hipEvents.
 *
 * Lifecycle:  sn_create -> sn_add_block (1..n times) -> sn_plan -> sn_infer*
 *             -> sn_destroy.
 *
 * Errors: every call returns SN_OK (0) or a negative sn_status; nothing
 * aborts.  sn_last_error(ctx) returns a description of the last failure on
 * that context (sn_last_error(NULL): last failure of sn_create on this
 * thread).  A context is not thread-safe; distinct contexts are independent.
 *
 * Numerics: fp16 weights and activations, fp32 accumulation; bias, residual,
 * ReLU, SwiGLU, softmax, RMSNorm and RoPE evaluated in fp32; each kernel
 * output rounded once to fp16 (logits stay fp32).  Kernels are deterministic
 * and the reduction order of every output depends only on the layer, never
 * on how the layer was split into slabs, so a swapped run is bit-identical
 * to an all-resident run of the same network.
 */
#ifndef SWAPNET_H
#define SWAPNET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SN_API_VERSION 1

typedef struct sn_ctx sn_ctx;

/* Status codes (negative = failure). */
enum sn_status {
    SN_OK = 0,
    SN_E_INVALID = -1,      /* malformed argument or layer descriptor          */
    SN_E_STATE = -2,        /* call not allowed in the context's current state */
    SN_E_INFEASIBLE = -3,   /* no slab partition satisfies the pair constraint */
    SN_E_NOMEM = -4,        /* host or device allocation failed                */
    SN_E_HIP = -5,          /* a HIP runtime call failed (text in last_error)  */
    SN_E_UNSUPPORTED = -6   /* operation not available (e.g. host-only context)*/
};

/* Layer operators.  Activations live in "slots" (device buffers outside the
 * budget).  Image networks keep activations as H x W x C_pad (channels
 * innermost, C_pad = C rounded up to 8, padding channels zero); token
 * networks keep [tokens][C].  Canonical weight layouts below are what the
 * caller passes to sn_add_block; the engine repacks them once, at plan time,
 * into the device layout held in the pinned image. */
enum sn_op {
    SN_OP_CONV2D = 1,           /* w [c_out][c_in][k][k], bias [c_out] (fp16).
                                   Cross-correlation, zero padding, stride,
                                   dilation; + bias (+ slot res) (ReLU)        */
    SN_OP_LINEAR = 2,           /* w [c_out][c_in], optional bias [c_out].
                                   y = W x + b (+ res) (ReLU).  SN_FLAG_SWIGLU:
                                   w is [2F][c_in] = [W1; W3] stacked and the
                                   output (F = c_out) is silu(W1 x) * (W3 x)  */
    SN_OP_MAXPOOL = 3,          /* k x k window, stride, pad (never selected)  */
    SN_OP_GAVGPOOL = 4,         /* mean over H x W -> [C]                      */
    SN_OP_UPSAMPLE_BILINEAR = 5,/* integer factor `scale`, half-pixel centres,
                                   edge-clamped (align_corners = false)        */
    SN_OP_EMBED = 6,            /* table [c_out = vocab][c_in = d]; rows are
                                   gathered by token id, never streamed       */
    SN_OP_RMSNORM = 7,          /* gain [c_in]: v / sqrt(mean(v^2)+eps) * g    */
    SN_OP_ATTENTION = 8         /* src = [T][3d] (q|k|v); RoPE (rotate-half,
                                   theta), append k, v to the KV cache of
                                   kv_layer, causal softmax(q k^T/sqrt(hd)) v;
                                   head_dim a power of two in [8, 512]
                                   (else SN_E_UNSUPPORTED at sn_add_block)     */
};

/* Layer flags. */
enum sn_flag {
    SN_FLAG_RELU = 1,           /* ReLU after bias/residual                    */
    SN_FLAG_FLATTEN_CHW = 2,    /* linear over an H x W x C activation whose
                                   canonical weight columns are in (C,H,W)
                                   order (framework flatten order)             */
    SN_FLAG_SWIGLU = 4,         /* see SN_OP_LINEAR                            */
    SN_FLAG_OUT_F32 = 8,        /* output stored as fp32 (logits)              */
    SN_FLAG_LAST_ROW = 16       /* token linear applied to the last row only   */
};

typedef struct sn_layer {
    int32_t op;                 /* enum sn_op                                  */
    int32_t src, res, dst;      /* activation slots; res = -1 for none.  The
                                   network input is slot `src` of layer 0; the
                                   output is slot `dst` of the last layer     */
    int32_t c_in, c_out;        /* channels / features                         */
    int32_t h_in, w_in;         /* input spatial size (image layers)          */
    int32_t k, stride, pad, dilation;   /* conv / pool window                  */
    int32_t scale;              /* upsample factor                             */
    int32_t heads, head_dim;    /* attention                                   */
    int32_t kv_layer;           /* attention: index of this layer's KV cache  */
    int32_t max_tokens;         /* embed: tokens per call (activation rows)    */
    int32_t max_seq;            /* attention: KV cache capacity (positions)    */
    int32_t flags;              /* enum sn_flag                                */
    float eps, theta;           /* rmsnorm epsilon, RoPE base                  */
    int64_t w_off, w_bytes;     /* canonical weight (or gain / table) tensor,
                                   byte offset and size in the block buffer;
                                   w_bytes = 0 if the layer has none          */
    int64_t b_off, b_bytes;     /* canonical bias; b_bytes = 0 if none        */
} sn_layer;

/* Create a context whose weight arena is `budget_bytes` of HBM, allocated
 * here, once (no allocation happens per swap).  Also creates the copy and
 * compute streams.  Returns NULL on failure (reason: sn_last_error(NULL)). */
sn_ctx *sn_create(size_t budget_bytes);

/* Context flags for sn_create_ex. */
enum sn_create_flag {
    SN_CREATE_HOST_ONLY = 1     /* no device calls at all: planning and
                                   prepacking only, for inspection; the infer
                                   calls return SN_E_UNSUPPORTED              */
};
sn_ctx *sn_create_ex(size_t budget_bytes, int flags);

/* Register one block: `n_layers` descriptors (copied) and the block's
 * weights in canonical layout (`weights`, `weight_bytes` bytes, copied; the
 * caller may free both on return).  Blocks run in the order added.  A block
 * is the user's partition unit (the paper's block, Sec. 3); the planner may
 * split it further but never merges blocks.
 * Errors: SN_E_INVALID (bad descriptor or out-of-range offsets),
 * SN_E_STATE (after sn_plan). */
int sn_add_block(sn_ctx *ctx, const sn_layer *layers, int n_layers,
                 const void *weights, size_t weight_bytes);

/* Plan and prepare: lower blocks to slabs so that every two consecutive
 * slabs fit the budget together (the pair constraint s_i + s_{i+1} <= b of
 * Sec. 6.2.2, Eq. 3, with the reserved share delta = 0 because activations
 * live outside the budget); split a block at layer boundaries, then a layer
 * by output channels, when needed; place slabs alternately at the two ends of
 * the arena; build the pinned host image in device layout, slab after slab;
 * allocate activations (and the KV cache) outside the budget.  If the whole
 * image fits the budget it is uploaded once here and every inference runs
 * all-resident.  Errors: SN_E_INFEASIBLE, SN_E_NOMEM, SN_E_HIP, SN_E_STATE. */
int sn_plan(sn_ctx *ctx);

/* Re-plan a planned context in place for a new budget (`budget_bytes`; 0 =
 * keep the budget) and the current options (SN_OPT_PARTITION,
 * SN_OPT_MAX_SLAB, SN_OPT_SPLIT_BUDGET if it was set, else the new budget,
 * and the delay model), without registering the network again: Sec. 6
 * re-forms blocks from the layers extracted at registration.  The layers'
 * device-layout tensors are gathered from the pinned image and written to a
 * new image in the new slab order; activations, the KV cache and the token
 * position are kept, so a token network continues where it was.  A budget
 * above the arena's allocation allocates a larger arena.  Waits for earlier
 * inferences first.  Errors: SN_E_STATE (before sn_plan), SN_E_INVALID,
 * SN_E_INFEASIBLE and SN_E_NOMEM leave the context as it was; SN_E_HIP
 * after the old plan was released leaves it unusable (only sn_destroy and
 * the introspection calls remain). */
int sn_replan(sn_ctx *ctx, size_t budget_bytes);

/* Budgets of n models sharing `total` bytes of device memory (Sec. 6,
 * Eq. 1).  If the demands need[i] (bytes) fit, out[i] = need[i].  Otherwise
 *   out[i] = need[i] / sum(need) * (1 - 1/n) * total
 *          + PS[i] / sum(PS) * (1/n) * total,   PS[i] = urgency[i] *
 *            latency_s[i] / need[i]
 * (equal shares of the second part if every PS is 0), each rounded down to
 * a multiple of 256 bytes.  Host only; no context.  Errors: SN_E_INVALID
 * (n <= 0, NULL, need <= 0, negative or non-finite latency or urgency). */
int sn_split_budget(int n, const int64_t *need, const double *latency_s, const double *urgency,
                    int64_t total, int64_t *out);

/* Options (set before sn_plan unless noted; SN_OPT_SPLIT_BUDGET,
 * SN_OPT_MAX_SLAB and SN_OPT_PARTITION may also be set later and take
 * effect at the next sn_replan). */
enum sn_option {
    SN_OPT_SPLIT_BUDGET = 1,    /* budget used for slab lowering (default: the
                                   arena budget).  With an arena >= image and
                                   a smaller split budget the run is resident
                                   but has the slabs of the swapped plan      */
    SN_OPT_TIMING = 2,          /* 1: record per-slab DMA / compute events;
                                   2: also one event pair per layer piece
                                   (adds launch overhead; for profiling only).
                                   May be set after plan                      */
    SN_OPT_MAX_SLAB = 3,        /* cap on slab bytes (0 = none)               */
    SN_OPT_SWAPIN = 5,          /* how a slab is swapped in.  2 (default):
                                   hipMemcpyAsync (SDMA engine) issued by the
                                   context's copy thread once the compute it
                                   must follow has finished, so the calling
                                   thread never blocks; 1: the same DMA issued
                                   by the calling thread with a stream-event
                                   dependency (the runtime then blocks the
                                   caller until the dependency is met); 0: a
                                   copy kernel on the copy stream reads the
                                   pinned image through its device mapping
                                   (uses compute units, never blocks)         */
    SN_OPT_SWAPIN_BLOCKS = 6,   /* workgroups of the swap-in copy kernel
                                   (default 32)                               */
    SN_OPT_COPY_STREAMS = 7,    /* DMA queues used by the copy thread: 1
                                   (default) a single queue; 2 alternates
                                   consecutive slabs between two queues so
                                   that one queue's per-copy start-up overlaps
                                   the other's transfer (the two then share
                                   the link, which delays each slab)          */
    SN_OPT_PARTITION = 8,       /* 0 (default): slabs follow the user blocks,
                                   split only where the pair constraint
                                   (Eq. 3) requires; 1: the layers of all
                                   blocks are re-cut into n = ceil(2 s / B)
                                   slabs of about s / n bytes each (Sec. 6:
                                   m = 2 parallel blocks of equal share),
                                   cutting layers by output channels where a
                                   slab boundary falls inside one; fewer,
                                   larger DMAs at small budgets; 2: the
                                   partition with the least predicted time
                                   per inference under the context's delay
                                   model (sn_cost_model; Sec. 6, Eq. 4),
                                   searched over slab counts around
                                   ceil(2 s / B) and cut points at layer
                                   boundaries or inside large layers, with
                                   partitions 0 and 1 as candidates too      */
    SN_OPT_SYNC = 9,            /* copy-thread mode (SN_OPT_SWAPIN 2): how
                                   the copy and compute streams order each
                                   other.  2 (default): each swap-in is a
                                   ROCr SDMA copy (hsa_amd_memory_async_copy)
                                   with a completion signal per slab, and a
                                   one-wave gate kernel ahead of the slab's
                                   kernels polls that signal (bounded wait:
                                   after 2 s plus 1 s per GB of image it
                                   flags an error that the next call
                                   reports as SN_E_HIP); "slab
                                   computed" as in 0.  Runs with per-slab
                                   timing (SN_OPT_TIMING) and contexts with
                                   an image file use mode 0's ordering.
                                   0: hipEvents for "slab loaded" and a
                                   one-thread kernel that bumps a mapped
                                   counter for "slab computed"; 1: stream
                                   writes / waits of 64-bit values in mapped
                                   memory (hipStreamWriteValue64 /
                                   hipStreamWaitValue64) for both.  May be
                                   set after plan, between inferences         */
    SN_OPT_NAIVE = 10,          /* measurement only: flags of sn_naive_flag;
                                   0 (default) = the engine as described.  Any
                                   other value runs a swapped plan slab after
                                   slab on the compute stream (no overlap, no
                                   graphs, no copy thread).  May be set after
                                   plan, between inferences                   */
    SN_OPT_CONV_KERNEL = 11,    /* measurement only: 0 (default) chooses each
                                   convolution's kernel from the layer shape;
                                   k > 0 uses kernel variant k - 1
                                   (sn_kernel_name) for every layer of that
                                   variant's kind (1x1 / token GEMM, taps
                                   with Cin_p % 64 == 0, or general).  Set
                                   before sn_plan (or before sn_replan)       */
    SN_OPT_GATE_LIMIT_US = 12,  /* failure tests only: bound of each gate
                                   kernel's wait (SN_OPT_SYNC 2) in
                                   microseconds; 0 (default) = 2 s plus 1 s
                                   per GB of image.  A gate that runs out
                                   lets its slab's kernels start before the
                                   slab has landed (their output is then
                                   undefined) and the next call reports
                                   SN_E_HIP.  May be set after plan,
                                   between inferences                         */
    SN_OPT_GRAPH = 4            /* 1 (default): the kernels of each slab of an
                                   image network are captured once per
                                   (input, output) buffer pair into one HIP
                                   graph per slab and replayed; the swap-in
                                   DMAs and events stay on the streams.  0:
                                   launch kernel by kernel.  Not used while
                                   SN_OPT_TIMING is on, nor for token nets    */
};
int sn_set_option(sn_ctx *ctx, int option, int64_t value);

/* SN_OPT_NAIVE flags: the redundant memory operations the paper removes
 * (Sec. 4.2: a swap-in that allocates and copies through a staging path;
 * Sec. 5.2: assembly that copies parameters into a model), put back one by
 * one to measure what each costs on this hardware. */
enum sn_naive_flag {
    SN_NAIVE_SEQUENTIAL = 1,    /* swap-in then compute, slab after slab      */
    SN_NAIVE_ALLOC = 2,         /* hipMalloc per swap-in, hipFree after the
                                   slab's compute (instead of the arena)      */
    SN_NAIVE_PAGEABLE = 4,      /* copy from pageable host memory (a malloc'd
                                   copy of the image) with hipMemcpy          */
    SN_NAIVE_COPY_ASSEMBLY = 8  /* copy every parameter tensor, one
                                   hipMemcpyAsync each, into a second device
                                   allocation and bind the kernels to that    */
};

/* Delay model of a swapped run (Sec. 5: input, execution and output delays
 * of a block, each linear in the block's bytes, parameter depth or FLOPs,
 * with device-dependent coefficients).  For this engine, in seconds:
 *   swap-in of a slab    t_in  = alpha * bytes + beta   (one DMA per slab;
 *                                 binding parameters by pointer costs the
 *                                 device nothing, so the paper's depth term
 *                                 becomes a per-DMA term);
 *   execution of a slab  t_ex  = slab_ex + sum of its pieces, a piece being
 *                                 a layer or an output-channel slice of one:
 *                                 layer time T = layer_ex[l] if given (>= 0),
 *                                 else gamma * FLOPs + kappa; a slice of
 *                                 u of U units takes kappa + (T - kappa) u/U;
 *   swap-out             t_out = 0 (no write-back; the range is reused).
 * A swap-in starts `gate` after the compute it waits for has finished (and
 * after the previous DMA); a slab's compute starts `wake` after its swap-in
 * has finished (and after the previous slab's compute).  The predicted time
 * of a plan replays this schedule for inferences issued back to back. */
typedef struct sn_cost_model {
    double alpha;               /* s per byte swapped in                      */
    double beta;                /* s per swap-in DMA                          */
    double gamma;               /* s per FLOP (layers without layer_ex)       */
    double kappa;               /* s per layer launch (ditto)                 */
    double gate;                /* s, compute end -> waiting DMA start        */
    double wake;                /* s, DMA end -> waiting compute start        */
    double slab_ex;             /* s per slab on the compute stream           */
    const float *layer_ex;      /* n_layers measured layer times (s; < 0 =
                                   not measured), or NULL                     */
    int32_t n_layers;           /* 0, or the number of layers added           */
} sn_cost_model;

/* Replace the context's delay model (defaults: coefficients measured on one
 * MI355X, no per-layer times).  Any state; the partition (SN_OPT_PARTITION
 * 2) is chosen at sn_plan from the model set by then, so per-layer times must
 * be given after the last sn_add_block.  The context copies layer_ex.
 * Errors: SN_E_INVALID (negative or non-finite coefficient, layer count
 * mismatch). */
int sn_set_cost_model(sn_ctx *ctx, const sn_cost_model *model);

/* Read the context's delay model.  If `layer_ex` is not NULL it must hold
 * `n_layers` = the number of layers added; it receives the per-layer times
 * (-1: not measured) and out->layer_ex points to it; else out->layer_ex is
 * NULL and out->n_layers 0. */
int sn_get_cost_model(const sn_ctx *ctx, sn_cost_model *out, float *layer_ex, int n_layers);

/* Measure the delay model of this planned context on its device and keep it
 * (what sn_get_cost_model then returns; gamma and kappa are kept):
 *  - alpha, beta: X = min(image, budget) bytes of the image copied into the
 *    arena as one DMA and as 16 DMAs with an event after each (beta = the
 *    extra time per DMA, alpha = the rest per byte; best of `reps`); with
 *    SN_OPT_SYNC 2 (no image file) the same copies are then issued as the
 *    engine issues them, through ROCr with a completion signal, timed on
 *    the host from the first issue to the last completion, and kept;
 *  - layer_ex: per-piece events (timing level 2), median of `reps`
 *    inferences; for image networks then scaled, slab by slab, to the time
 *    of the slab's captured graph replayed without swap-ins, so that they
 *    include the per-slab overhead (slab_ex is then 0);
 *  - swapped plans: wake from per-slab events (timing level 1); with
 *    SN_OPT_SYNC 2 instead what a gate kernel on a completed copy's signal
 *    adds ahead of the next kernel (two gates against one); gate fitted (in
 *    [0, 1 ms]) so that the model's time per inference equals the measured
 *    one for 8 inferences issued back to back.
 * The inferences run on the staging buffers (image networks, zero input) or
 * with token id 0 at the current position, which is not advanced (token
 * networks: the KV entry at that position is overwritten; needs position <
 * max_seq).  A resident arena holds the image at the same offsets, so it
 * keeps its weights.  Synchronous; waits for earlier inferences first.  reps
 * in [1, 64].  Errors: SN_E_STATE, SN_E_UNSUPPORTED (host-only),
 * SN_E_INVALID, SN_E_HIP. */
int sn_calibrate(sn_ctx *ctx, int reps);

/* Choose the partition by measurement: calibrate the delay model on the
 * current plan (as sn_calibrate), then plan the context in place
 * (sn_replan) with each of SN_OPT_PARTITION 0, 1 and 2 (the last searched
 * under the fresh model; with SN_OPT_SYNC 2 searched twice, under the model
 * measured on the ROCr path and under the one measured with events), time
 * 8 inferences issued back to back for each (best of max(1, reps / 2)
 * rounds) and keep the fastest plan and its model; SN_OPT_PARTITION is
 * left at the chosen value.  `times_s` (NULL or 3 doubles) receives the
 * measured seconds per inference of partitions 0, 1, 2 (the faster of the
 * two searches for 2; 0: infeasible).  A
 * resident plan is left as it is.  Runs inferences as sn_calibrate does.
 * Errors: as sn_calibrate and sn_replan. */
int sn_tune(sn_ctx *ctx, int reps, double *times_s);

/* Predicted time of the planned context under its delay model: one
 * inference from an idle start (`latency_s`) and the steady-state time per
 * inference when inferences are issued back to back (`period_s`).  Host
 * only (also for host-only contexts).  Errors: SN_E_STATE before sn_plan. */
int sn_predict(const sn_ctx *ctx, double *latency_s, double *period_s);

/* Image networks.  `input` is the fp16 input in canonical C x H x W order;
 * `output` receives the last layer's output (C x H x W fp16 for spatial
 * outputs, [c_out] for linear outputs, fp32 if SN_FLAG_OUT_F32).  Host
 * pointers; synchronous. */
int sn_infer(sn_ctx *ctx, const void *input, void *output);

/* As sn_infer with device pointers; the work is ordered after prior work on
 * `hip_stream` (a hipStream_t; NULL = the context's compute stream) and the
 * output is ready when that stream reaches the point of return.  No host
 * synchronisation. */
int sn_infer_dev(sn_ctx *ctx, const void *d_input, void *d_output, void *hip_stream);

/* Token networks (first layer SN_OP_EMBED).  Runs `n_ids` tokens (host
 * int32 ids) at positions pos..pos+n_ids-1, appending to the KV cache, and
 * writes the fp32 logits of the last token to `logits` (host, c_out floats).
 * Synchronous. */
int sn_infer_tokens(sn_ctx *ctx, const int32_t *ids, int n_ids, float *logits);

/* Clear the token position (the KV cache is overwritten from position 0). */
int sn_reset(sn_ctx *ctx);

typedef struct sn_stats {
    int64_t budget_bytes;       /* arena size                                  */
    int64_t image_bytes;        /* pinned image (sum of slab bytes)            */
    int64_t arena_high_water;   /* highest arena byte used by the placement    */
    int64_t streamed_bytes;     /* weight bytes DMA'd per inference (0 when
                                   resident)                                   */
    int64_t activation_bytes;   /* device bytes outside the budget:           */
    int64_t kv_bytes;           /*   activations, KV cache,                   */
    int64_t table_bytes;        /*   host-side tables (plan, bindings)        */
    int32_t n_slabs, n_pieces, n_layers, resident;
    int64_t n_infers;
    double last_ms;             /* last inference, host wall clock (ms)       */
    int64_t input_bytes;        /* bytes sn_infer reads from `input` (0 for
                                   token networks)                             */
    int64_t output_bytes;       /* bytes sn_infer / sn_infer_tokens write to
                                   `output` / `logits`                         */
    int64_t host_weight_bytes;  /* host memory holding weights: the pinned
                                   image, or with an image file attached, the
                                   two staging slots                           */
    int32_t file_backed;        /* 1: swap-ins read the image file            */
    int32_t direct_io;          /* 1: that file is read with O_DIRECT (no page
                                   cache); 0: the file system refused it      */
    double read_ms;             /* copy thread's time in file reads since the
                                   file was attached (ms)                      */
} sn_stats;
int sn_get_stats(const sn_ctx *ctx, sn_stats *out);

typedef struct sn_slab_info {
    int64_t image_off;          /* byte offset in the pinned image            */
    int64_t arena_off;          /* byte offset in the arena                   */
    int64_t bytes;              /* slab bytes (tensors 256-byte aligned)      */
    int32_t first_piece, n_pieces;
    float t_in_ms, t_ex_ms;     /* last inference's DMA and compute time of
                                   this slab (SN_OPT_TIMING), else 0          */
    float t_in_start_ms, t_ex_start_ms; /* start times from inference start   */
    int32_t wait_slab;          /* this slab's swap-in waits for the compute of
                                   this earlier slab (-1: none), whose arena
                                   range it overwrites                         */
    int32_t wrap_slab;          /* wait_slab == -1 only: the swap-in of the
                                   next inference waits for this inference's
                                   compute of this later slab, the last one
                                   overlapping its range (-1: none; with
                                   wait_slab == -1 too, no other slab shares
                                   the range and the swap-in waits for
                                   nothing)                                    */
} sn_slab_info;
int sn_get_slab(const sn_ctx *ctx, int i, sn_slab_info *out);

typedef struct sn_piece_info {
    int32_t layer;              /* global layer index                          */
    int32_t c0, c1;             /* output channels [c0, c1) of that layer     */
    int32_t kernel;             /* kernel variant chosen for the layer        */
    int64_t w_off, b_off;       /* offsets in the slab (-1 if none)           */
    int64_t w_bytes, b_bytes;
    float t_ms;                 /* last inference's duration (timing level 2) */
    int32_t ksplit;             /* K splits of the layer's convolution (1: none) */
    float t_main_ms;            /* of t_ms, the main kernel alone (a split-K
                                   convolution's reduction kernel excluded)    */
} sn_piece_info;
int sn_get_piece(const sn_ctx *ctx, int j, sn_piece_info *out);

/* Name of a kernel variant id (as reported in sn_piece_info.kernel), or "?". */
const char *sn_kernel_name(int kernel);

/* Pinned host image (after sn_plan): pointer and size, for inspection.
 * SN_E_STATE once an image file is attached (the image is in the file). */
int sn_get_image(const sn_ctx *ctx, const void **ptr, size_t *bytes);

/* Storage tier: direct block fetch (Sec. 4.2.1).  The paper keeps the
 * blocks in external storage and swaps a block in with direct I/O (no page
 * cache, no second copy in memory).  sn_save_image writes the planned image
 * (device layout, the slabs of this plan) to `path`: a header, then each
 * slab at a 4 KiB-aligned offset, padded to 4 KiB, so that one O_DIRECT read
 * fetches a slab.  Any context (host-only too) after sn_plan.  Errors:
 * SN_E_STATE (not planned, or the image is already in a file),
 * SN_E_INVALID (path NULL or not writable). */
int sn_save_image(sn_ctx *ctx, const char *path);

/* Swap in from the image file written by sn_save_image for this plan: the
 * file is opened with O_DIRECT (buffered if the file system refuses it;
 * sn_stats.direct_io), every slab is read back once and compared with the
 * in-memory image, then the pinned image is released and host memory keeps
 * two pinned staging slots of the largest slab (sn_stats.host_weight_bytes).
 * Per inference the copy thread reads each slab into a free slot (the next
 * slab is read while the current one is DMA'd and computed; after the last
 * slab, the first slab of the next inference) and DMAs it into the arena.
 * Results are bit-identical to the in-memory image.  Afterwards sn_replan,
 * sn_tune, sn_calibrate, sn_get_image, SN_OPT_NAIVE and swap-in modes other
 * than 2 return SN_E_STATE.  Errors: SN_E_STATE (not planned, resident
 * plan, swap-in mode != 2 or naive flags set, already attached),
 * SN_E_UNSUPPORTED (host-only context), SN_E_INVALID (path missing, not an
 * image of this plan, content differs), SN_E_NOMEM, SN_E_HIP. */
int sn_attach_image_file(sn_ctx *ctx, const char *path);

const char *sn_last_error(const sn_ctx *ctx);

/* Release everything (NULL-safe).  Waits for outstanding work first. */
void sn_destroy(sn_ctx *ctx);

#ifdef __cplusplus
}
#endif
#endif /* SWAPNET_H */
