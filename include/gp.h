/*
 * gp.h -- C ABI of one GPipe pipeline partition on one MI355X (gfx950).
 *
 * GPipe (Huang et al., "GPipe: Easy Scaling with Micro-Batch Pipeline
 * Parallelism") splits a network given as a sequence of L layers into K cells
 * of consecutive layers, one per accelerator (Section 2.1).  Every mini-batch
 * of N examples is divided into M equal micro-batches (Section 2.2).  Each
 * partition runs its composite forward function F_k on every micro-batch,
 * keeping only the activations at its boundary (re-materialisation, Section
 * 2.3); in the backward pass it recomputes F_k and runs B_k.  Gradients of
 * all M micro-batches are accumulated and applied in one synchronous update
 * at the end of the mini-batch (Section 2.2).
 *
 * This library is one partition's share of that work: a stack of pre-LN
 * Transformer layers (the layer kind the paper trains in Sections 3 and 5),
 * driven micro-batch by micro-batch.  All compute runs in HIP kernels on the
 * caller's stream.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every function returns gp_status; none aborts or throws.  On failure a
 *    thread-local message is available from gp_last_error().
 *  - Argument and call-order errors are detected on the host before anything
 *    is enqueued, and leave the partition unchanged.
 *  - Device pointers are plain HIP device addresses of contiguous row-major
 *    buffers owned by the caller; the library never frees them.  The library
 *    owns its parameters, gradient accumulators, stash and workspaces, which it
 *    allocates in gp_partition_configure and frees in gp_partition_destroy;
 *    nothing is allocated on the per-micro-batch path.
 *  - "Partition dtype" (gp_config.dtype) is the element type of boundary
 *    tensors: float32 (GP_F32) or bfloat16 (GP_BF16, bf16 GEMM operands with
 *    fp32 accumulation; the residual stream, LayerNorm statistics, softmax,
 *    losses and gradient accumulators stay fp32).
 *  - Calls on one partition are not thread-safe; use one partition per host
 *    thread.  Work is ordered by the stream passed in; device faults surface
 *    as GP_ERR_HIP at the next call that synchronises.
 *  - Forward and backward calls may be given different streams (see
 *    gp_forward_microbatch and gp_backward_microbatch_remat); the library
 *    orders what they share.  The caller orders its own data: the inputs a
 *    call reads, and the outputs it wrote on another stream.
 */
#ifndef GP_H
#define GP_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A HIP stream handle (the same type as hipStream_t); NULL is the default stream. */
typedef struct ihipStream_t* gp_stream;

typedef struct gp_partition gp_partition; /* opaque, library-owned */

typedef enum {
    GP_OK = 0,
    GP_ERR_INVALID_ARG = 1, /* bad size, NULL required pointer, mini-batch not M equal parts */
    GP_ERR_STATE = 2,       /* call out of the forward/backward/step order */
    GP_ERR_OOM = 3,         /* device allocation failed (configure) */
    GP_ERR_HIP = 4,         /* a HIP runtime call failed */
    GP_ERR_NONFINITE = 5,   /* check_finite found a non-finite gradient; update skipped */
    GP_ERR_UNSUPPORTED = 6  /* valid request outside what the kernels implement */
} gp_status;

typedef enum { GP_F32 = 0, GP_BF16 = 1 } gp_dtype;

/* Layer kind of every layer in the partition. */
typedef enum {
    GP_ENCODER = 0,      /* x1 = x + SelfAttn(LN1 x) Wo + bo;  y = x1 + FFN(LN2 x1) */
    GP_DECODER_CROSS = 1 /* causal self-attention, cross-attention to a memory, FFN */
} gp_layer_kind;

/* What ends the partition's forward pass (Section 2.2: the last partition
 * owns the loss; every other partition receives dL/dy from its successor). */
typedef enum {
    GP_LOSS_NONE = 0,   /* boundary partition: dL/dy arrives in gp_backward_microbatch_remat */
    GP_LOSS_MSE = 1,    /* sum (y - target)^2 / (N S D) over the mini-batch */
    GP_LOSS_XENT_LS = 2 /* final LayerNorm, [D, V] projection, label-smoothed cross-entropy / (N S) */
} gp_loss;

/* The one synchronous update of gp_accumulate_and_step.  The paper counts 12
 * bytes per parameter because it trains with RMSProp (Table 1 caption):
 * the parameter, its gradient and the running mean square. */
typedef enum {
    GP_OPT_SGD = 0,    /* W <- W - lr G */
    GP_OPT_RMSPROP = 1 /* ms <- rho ms + (1 - rho) G^2;  W <- W - lr G / sqrt(ms + eps);  ms starts at 0 */
} gp_optimizer;

typedef struct {
    int seq_len;             /* S, tokens per sequence */
    int seqs_per_microbatch; /* n = N / M sequences in each micro-batch */
    int num_microbatches;    /* M */
    int dtype;               /* gp_dtype */
    int kind;                /* gp_layer_kind */
    int mem_seq_len;         /* decoder: memory length S_mem; else 0 */
    int loss;                /* gp_loss */
    int vocab;               /* GP_LOSS_XENT_LS: V; else 0 */
    float label_smoothing;   /* GP_LOSS_XENT_LS: eps, target q = (1-eps) onehot + eps / V */
    float ln_eps;            /* LayerNorm epsilon inside the square root (e.g. 1e-5) */
    int check_finite;        /* nonzero: gp_accumulate_and_step checks G and syncs */
    int keep_activations;    /* 0: re-materialise each micro-batch's forward inside its backward
                                (Section 2.3); 1: keep every micro-batch's intermediates from its
                                forward instead (no recompute; activation memory O(N L) rather than
                                O(N + L N / M)), the stored-activation baseline */
    int optimizer;           /* gp_optimizer */
    float rms_decay;         /* GP_OPT_RMSPROP: rho in [0, 1) */
    float rms_eps;           /* GP_OPT_RMSPROP: eps > 0, inside the square root */
    float logit_clip;        /* GP_LOSS_XENT_LS: c > 0 clips every logit to [-c, c] before the softmax
                                (Section 5 bounds the magnitude of the softmax pre-activations for
                                trainability); the gradient passes where |z| <= c.  0 = off */
} gp_config;

/* Parameter tensors.  Matrices are logical [in, out] (y = x W + b); attention
 * head h owns columns [h d_h, (h+1) d_h) of Wq/Wk/Wv and rows of Wo. */
typedef enum {
    GP_P_LN1_G = 0, GP_P_LN1_B, GP_P_WQ, GP_P_BQ, GP_P_WK, GP_P_BK, GP_P_WV, GP_P_BV,
    GP_P_WO, GP_P_BO, GP_P_LN2_G, GP_P_LN2_B, GP_P_W1, GP_P_B1, GP_P_W2, GP_P_B2,
    /* decoder layers: cross-attention (LN2 precedes it) and LN3 before the FFN */
    GP_P_XWQ, GP_P_XBQ, GP_P_XWK, GP_P_XBK, GP_P_XWV, GP_P_XBV, GP_P_XWO, GP_P_XBO,
    GP_P_LN3_G, GP_P_LN3_B,
    /* loss head (layer index -1): final LayerNorm and vocabulary projection */
    GP_P_LNF_G, GP_P_LNF_B, GP_P_WOUT, GP_P_BOUT,
    GP_P_COUNT
} gp_param_id;

/*
 * Create a partition of `layers` Transformer layers of width d_model, FFN
 * width d_ff and `heads` attention heads (Section 2.1: a cell p_k of
 * consecutive layers).  Touches no device.  *out receives the handle.
 * GP_ERR_INVALID_ARG: a size <= 0, d_model % heads != 0, out == NULL.
 */
gp_status gp_partition_create(int layers, int d_model, int d_ff, int heads, gp_partition** out);

/*
 * Fix the micro-batch geometry and allocate every device buffer on the
 * current HIP device: fp32 master parameters (initialised to 0; LayerNorm
 * gains to 1), their bf16 (or fp32) working copies, fp32 gradient
 * accumulators, the boundary stash of M micro-batches and the
 * re-materialisation workspace of one micro-batch (Section 2.3: activation
 * memory O(N + L/K * N/M)).  Once per partition.
 * GP_ERR_INVALID_ARG: non-positive sizes, unknown enums, missing vocab.
 * GP_ERR_UNSUPPORTED: bf16 attention needs d_model / heads == 64 and
 *   seq_len, mem_seq_len multiples of 32 and <= 256.
 * GP_ERR_STATE: configured already.  GP_ERR_OOM / GP_ERR_HIP on device failure.
 */
gp_status gp_partition_configure(gp_partition* p, const gp_config* cfg);

/* Free everything the partition owns (synchronises the device first).  NULL is a no-op. */
gp_status gp_partition_destroy(gp_partition* p);

/*
 * Copy one parameter tensor between host fp32 memory and the partition.
 * `layer` is 0..layers-1, or -1 for the head parameters; `count` must equal
 * the tensor's element count (logical [in, out] row-major for matrices).
 * gp_set_param also refreshes the working copies.  gp_get_param reads the
 * fp32 master; gp_get_grad reads the fp32 accumulator, which after the last
 * backward micro-batch holds the mini-batch gradient sum_m dL_m/dw.
 * These calls synchronise the device.
 * GP_ERR_INVALID_ARG: bad layer, id not present in this layer kind, count.
 * GP_ERR_STATE: not configured, or gp_set_param between the first forward
 *   and the step of a mini-batch (Section 2.2: all micro-batches of a
 *   mini-batch see the same parameters).
 */
gp_status gp_set_param(gp_partition* p, int layer, int id, const float* host, size_t count);
gp_status gp_get_param(gp_partition* p, int layer, int id, float* host, size_t count);
gp_status gp_get_grad(gp_partition* p, int layer, int id, float* host, size_t count);

/* Bytes held in device memory for parameters (masters, working copies and,
 * with RMSProp, the running mean squares), gradient accumulators, the
 * boundary stash, and all workspaces.  Any pointer
 * may be NULL.  Requires a configured partition. */
gp_status gp_partition_memory(gp_partition* p, size_t* params, size_t* grads, size_t* stash,
                              size_t* workspace);

/* The byte counts gp_partition_memory would report for a partition of these
 * sizes configured with *cfg (Section 2.3: with re-materialisation the
 * stash holds the N boundary inputs and the workspace one micro-batch's
 * intermediates, O(N + L N / M); with keep_activations every micro-batch's,
 * O(N L)), computed on the host without touching a device.  The schedule
 * settings read from the environment at configure apply here too.
 * GP_ERR_INVALID_ARG / GP_ERR_UNSUPPORTED: as gp_partition_create and
 * gp_partition_configure. */
gp_status gp_memory_plan(int layers, int d_model, int d_ff, int heads, const gp_config* cfg, size_t* params,
                         size_t* grads, size_t* stash, size_t* workspace);

/*
 * GPipe's partitioning algorithm (Sections 2.1-2.2): split `layers` layers,
 * layer i with cost estimate costs[i] (host array, finite, >= 0), into
 * `cells` cells of consecutive layers whose summed costs C_k have the least
 * variance, (1/K) sum_k (C_k - mean)^2.  Exact (a dynamic program over the
 * prefix sums, O(cells layers^2) host time); among equal optima the one with
 * the smallest cuts.  first_layer (host, `cells` ints) receives the index of
 * each cell's first layer (first_layer[0] = 0); variance (nullable) the
 * least variance.  Host code only: no device is touched.
 * GP_ERR_INVALID_ARG: NULL costs or first_layer, not 1 <= cells <= layers,
 *   a negative or non-finite cost.
 */
gp_status gp_plan_cells(const double* costs, int layers, int cells, int* first_layer, double* variance);

/* Number of trainable parameters (layers plus head). */
gp_status gp_param_count(gp_partition* p, size_t* count);

/*
 * Forward pass of micro-batch `mb` (Sections 2.2-2.3).  Micro-batches are
 * taken in order mb = 0, 1, ..., M-1 within a mini-batch.
 *   x   : device [n, S, D] in the partition dtype, the micro-batch's boundary
 *         input.  It is copied into the library's stash, so the caller may
 *         reuse the buffer once the stream has passed this call.
 *   mem : decoder: device [n, S_mem, D] partition dtype, also stashed; else NULL.
 *   y   : device [n, S, D] partition dtype, the partition output F_k(x);
 *         may be NULL (loss partitions need not emit it).
 * Every intermediate of the layers is discarded; only the stash is kept.
 * Streams: consecutive micro-batches' forwards may be issued on two streams
 * and then run side by side.  The library keeps two first-pass workspaces,
 * for even and odd mb, and orders each forward after the previous one in its
 * workspace and after the last gp_accumulate_and_step (the weights it reads),
 * and the mini-batch's first backward after all M forwards, whatever streams
 * they ran on.  y is written on the call's stream; a consumer on another
 * stream waits for that stream.  Under stream capture only waits within the
 * same capture are made.
 * GP_ERR_STATE: not configured, mb out of order, or backward already begun.
 * GP_ERR_INVALID_ARG: x (or mem for the decoder) NULL, mb out of range.
 */
gp_status gp_forward_microbatch(gp_partition* p, int mb, const void* x, const void* mem, void* y,
                                gp_stream stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * forward pass as gp_forward_microbatch, same arguments, same results bit
 * for bit, with no allocation of any kind.  The split-K partial tiles of its
 * GEMMs go to a static device array of the library (32 MiB, one per device,
 * held until the process ends) instead of the partition's workspace; it does
 * not start the early recompute of the last micro-batch (that backward then
 * recomputes on its own stream).  Every call on a device shares the array:
 * calls that overlap on one device (two streams, two host threads) race; on
 * one partition each of these calls waits for the previous forward in both
 * first-pass workspaces, so they never overlap each other.
 * GP_ERR_UNSUPPORTED: the partition's forward needs more split-K scratch
 *   than the array holds (the message states both sizes).
 * GP_ERR_HIP: the array has no address on this device.
 * Otherwise as gp_forward_microbatch.
 */
gp_status gp_forward_microbatch_noalloc(gp_partition* p, int mb, const void* x, const void* mem, void* y,
                                        gp_stream stream);

/*
 * Backward pass of micro-batch `mb` with re-materialisation (Section 2.3):
 * the layers' forward is recomputed from the stashed boundary input, keeping
 * this micro-batch's intermediates only, then back-propagated in reverse
 * layer order.  Parameter gradients are added in place into the fp32
 * accumulators (the first backward micro-batch of a mini-batch overwrites
 * them); the LayerNorm gain and shift gradients are summed over the
 * micro-batches in the library's own buffers and written to the
 * accumulators by the last backward micro-batch (mb = 0), so every gradient
 * is complete once all M backwards have run.  Micro-batches are taken in
 * order mb = M-1, ..., 0, after all M forwards.
 *   dy_or_target : GP_LOSS_NONE:   device [n, S, D] partition dtype, dL/dy;
 *                  GP_LOSS_MSE:    device [n, S, D] partition dtype, targets;
 *                  GP_LOSS_XENT_LS: device int32 [n, S] labels in [0, V).
 *   dx   : device [n, S, D] partition dtype, dL/dx for the previous
 *          partition; may be NULL.
 *   dmem : decoder: device [n, S_mem, D] partition dtype, dL/dmem summed over
 *          the layers; may be NULL.  Else must be NULL.
 * Streams: each backward call is ordered after the previous one, and the
 * update after the last, whatever streams they were given, except that where
 * a recompute unit is a pair of micro-batches (at most 2048 rows each,
 * recompute-ahead and the weight-gradient stream on), the pair's two calls
 * issued on two streams run side by side: the odd member's in a second set of
 * scratch buffers, the even member's following it (its loss head after the
 * odd member's, each layer's LayerNorm gradient sums after the odd member's
 * layer, so every result, the loss included, equals the one-stream result bit
 * for bit).
 * GP_ERR_STATE: forwards incomplete, or mb out of order.
 * GP_ERR_INVALID_ARG: dy_or_target NULL, mb out of range.
 */
gp_status gp_backward_microbatch_remat(gp_partition* p, int mb, const void* dy_or_target, void* dx,
                                       void* dmem, gp_stream stream);

/*
 * A non-blocking HIP stream of default priority on the current device, for a
 * caller that issues micro-batches on a second stream (a helper, not a step
 * of the method).  HIP maps streams onto a small pool of hardware queues
 * (GPU_MAX_HW_QUEUES); two busy streams on one queue run one after the other,
 * and a wait issued on one holds the other back.  A framework's stream pool
 * spreads many streams over the queues, so a second stream taken from it may
 * share a queue with one of the library's; a stream created here, once per
 * process, does not as long as the process keeps no more busy streams than
 * there are queues.  Destroy it with gp_stream_destroy once no work on it is
 * pending.
 * GP_ERR_INVALID_ARG: out (or stream) NULL.  GP_ERR_HIP: the runtime failed.
 */
gp_status gp_stream_create(gp_stream* out);
gp_status gp_stream_destroy(gp_stream stream);

/*
 * The one synchronous update at the end of the mini-batch (Section 2.2):
 * W <- W - lr * G on the fp32 masters (G = the accumulated, undivided sum of
 * the micro-batch gradients; losses are normalised by the whole mini-batch),
 * then the working copies are refreshed (fp32 -> bf16 round-to-nearest-even).
 * G keeps its value until the next mini-batch's first backward overwrites it.
 *   loss_out : if non-NULL, receives the mini-batch loss (0 for GP_LOSS_NONE)
 *              and the call synchronises the stream.
 * With check_finite set the call synchronises, and if any gradient is
 * non-finite the update is skipped and GP_ERR_NONFINITE returned.
 * GP_LOSS_XENT_LS: a label outside [0, V) is read as class 0 on the device
 * and flagged; the next call that synchronises (loss_out non-NULL or
 * check_finite) then skips the update and returns GP_ERR_INVALID_ARG.
 * GP_ERR_STATE: not all M backward micro-batches done.
 */
gp_status gp_accumulate_and_step(gp_partition* p, float lr, double* loss_out, gp_stream stream);

/*
 * Launch timers (instrumentation; not part of the method).  Each library
 * launch belongs to one role: a linear layer's forward ("FWD", Y = X W + b),
 * input-gradient ("DX", dX = dY W^T) or weight-gradient ("DW", G_W += X^T dY
 * with the bias gradient fused) GEMM, including its split-K reduction when
 * one is used; an attention forward or backward; a LayerNorm forward or
 * backward.  While a role is selected, every launch of that role is
 * bracketed by two HIP events recorded on the stream the launch is enqueued
 * on, and the role's algorithmic work is added up: GEMM 2 M N K FLOPs;
 * attention 4 n H Sq Sk dh FLOPs forward and twice that backward (halved
 * when causal; the recomputed scores are not counted); bytes = each operand
 * read once and each output written once.
 */
typedef enum {
    GP_K_NONE = 0,
    GP_K_QKV_FWD, GP_K_QKV_DX, GP_K_QKV_DW,
    GP_K_O_FWD, GP_K_O_DX, GP_K_O_DW,
    GP_K_FFN1_FWD, GP_K_FFN1_DX, GP_K_FFN1_DW,
    GP_K_FFN2_FWD, GP_K_FFN2_DX, GP_K_FFN2_DW,
    GP_K_XQ_FWD, GP_K_XQ_DX, GP_K_XQ_DW,
    GP_K_XKV_FWD, GP_K_XKV_DX, GP_K_XKV_DW,
    GP_K_XO_FWD, GP_K_XO_DX, GP_K_XO_DW,
    GP_K_HEAD_FWD, GP_K_HEAD_DX, GP_K_HEAD_DW,
    GP_K_ATTN_FWD, GP_K_ATTN_BWD, GP_K_XATTN_FWD, GP_K_XATTN_BWD,
    GP_K_LN_FWD, GP_K_LN_BWD,
    GP_K_COUNT
} gp_kernel_role;

/* Select the timed role: one gp_kernel_role, GP_K_NONE to stop timing, or
 * GP_K_COUNT to time every role (brackets every launch; for finding the
 * dominant role, not for throughput runs).  Recorded launches are kept.
 * GP_ERR_INVALID_ARG: role out of range. */
gp_status gp_timer_select(gp_partition* p, int role);

/* Time one launch in `every` of the selected role(s): launches 0, every,
 * 2 every, ... since the last reset are bracketed, the others run without
 * events (default 1: every launch).  Keeps the events' own cost out of most
 * launches of a timed region; the recorded totals then cover the sampled
 * launches only.  GP_ERR_INVALID_ARG: NULL partition or every < 1. */
gp_status gp_timer_sample(gp_partition* p, int every);

/* Totals of one role over the launches recorded since the last reset: summed
 * event-to-event milliseconds, launch count, algorithmic FLOPs and bytes.
 * Waits for the role's last recorded event.  Any output pointer may be NULL. */
gp_status gp_timer_read(gp_partition* p, int role, double* ms, long* launches, double* flops, double* bytes);

/* Forget every recorded launch (the events are kept for reuse). */
gp_status gp_timer_reset(gp_partition* p);

/* Instrumentation (re-materialisation check, Section 2.3: the backward
 * recomputes the same F_k): write the partition output F_k(x_mb) as
 * re-materialised inside the most recent gp_backward_microbatch_remat call of
 * this mini-batch (micro-batch mb), rounded to the partition dtype, into the
 * caller's device buffer y [n, S, D].  Enqueued on `stream`, which must be the
 * stream that backward call was given; valid until the next backward or step
 * call, after which that recompute's workspace may be reused.  Recomputing
 * with the kernels and launch shapes of the first pass, it equals the y that
 * gp_forward_microbatch emitted for mb bit for bit.
 * GP_ERR_INVALID_ARG: p or y NULL.  GP_ERR_STATE: not configured, or no
 * backward micro-batch has run since the last step. */
gp_status gp_recomputed_output(gp_partition* p, void* y, gp_stream stream);

/* Instrumentation: the sustained bf16 MFMA rate of the current device, the
 * reference for "fraction of the measured MFMA peak".  Runs a register-only
 * loop of v_mfma_f32_32x32x16_bf16 (pseudo-random operands, 8 independent
 * accumulators per wave, two 4-wave workgroups per CU) on `stream` (a
 * hipStream_t; NULL = the null stream), waits for it, and stores the best of
 * three timed runs (after a warm-up run) in *tflops, in TFLOP/s.  Allocates a
 * small output buffer with hipMalloc and frees it with hipFree (so it must not
 * be called under stream capture).
 * GP_ERR_INVALID_ARG: tflops is NULL; GP_ERR_HIP: a launch or event failed. */
gp_status gp_mfma_peak(void* stream, double* tflops);

/* Message of the calling thread's last failure (library-owned, valid until the
 * thread's next failing call); "" if none. */
const char* gp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GP_H */
