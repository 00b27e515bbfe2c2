/*
 * erase.h -- C ABI of the MI355X detached-block training step (ERASE).
 *
 * The operation (paper, Section 2): a network is cut into B blocks by
 * stop-gradients, z_b = f_b(sg[z_{b-1}]; theta_b) (Eq. 1).  Every block has a
 * local head and loss l_b; the objective is L = sum_b lambda_b l_b (Eq. 2), so
 * the gradient of block b needs only block b's forward and local loss.  ERASE
 * (Section 2.2) launches block b's backward as soon as its forward and loss
 * finish, on a second stream whose events enforce the remaining dependencies,
 * so it overlaps the forward of block b+1.  One call of erase_step() enqueues
 * one such training step: for each block the forward, local sigmoid-BCE head
 * and loss gradient, the weight/input gradients and an Adam update.
 *
 * Conventions shared by every entry point:
 *  - Every function returns erase_status; nothing throws across the ABI.
 *  - "device" pointers are HIP device allocations on the device that is
 *    current when erase_init() runs; "host" pointers are ordinary memory.
 *  - Streams are passed as `void*` holding a hipStream_t.  All streams must
 *    be distinct, non-null, created by the caller with default priority and
 *    belong to the current device.  The library never destroys them.
 *  - The caller owns all device memory (parameters, Adam moments, gradients,
 *    workspace, inputs, labels, losses).  The library owns only the context,
 *    its events and its HIP graphs, and never frees caller memory.  After
 *    erase_init() it allocates no device memory.
 *  - A context is not thread-safe; use one context per host thread.
 *  - Arguments are validated on the host before anything is enqueued: an
 *    invalid call returns an error and enqueues nothing.  Errors raised by
 *    the device (HIP launch failures, a non-finite loss) surface at
 *    erase_sync() and are sticky: every later call returns ERASE_ERR_STATE
 *    until erase_destroy().
 */
#ifndef ERASE_H_
#define ERASE_H_

#include <stddef.h>
#include <stdint.h>

/* The entry points below are the only symbols the library exports (it is
 * built with hidden visibility). */
#define ERASE_API __attribute__((visibility("default")))

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque training-step context: created by erase_init(), owned by the
 * library, released by erase_destroy(). */
typedef struct erase_ctx erase_ctx;

typedef enum {
  ERASE_OK = 0,
  ERASE_ERR_INVALID_ARG = -1,  /* null pointer, bad enum, bad hyper-parameter, misaligned pointer */
  ERASE_ERR_SHAPE = -2,        /* dimensions that do not chain or are out of range               */
  ERASE_ERR_UNSUPPORTED = -3,  /* a well-formed request this library does not implement          */
  ERASE_ERR_WORKSPACE = -4,    /* workspace null, misaligned (256 B) or smaller than required    */
  ERASE_ERR_HIP = -5,          /* a HIP runtime call failed                                       */
  ERASE_ERR_STATE = -6,        /* context already failed, or call out of order                    */
  ERASE_ERR_NONFINITE = -7     /* a block loss was NaN or infinite                                */
} erase_status;

/* Storage type of inputs, weights used by the GEMMs and activations.
 * ERASE_BF16: bf16 GEMM operands and stored activations/activation-gradients,
 * fp32 accumulation; master parameters, Adam moments, gradients, logits and
 * losses stay fp32.  ERASE_F32: everything fp32. */
typedef enum { ERASE_F32 = 0, ERASE_BF16 = 1 } erase_dtype;

/* Layer kinds of a block body (paper: f_b of Eq. 1; the CTR subarchitectures
 * of Section 3.2 are dense MLPs, DCNv2 cross layers are the other common
 * dense block of CTR models).
 *   LINEAR_RELU: a_l = max(a_{l-1} W^T + b, 0),      W[out,in], b[out]
 *   CROSS:       a_l = a_0 * (a_{l-1} W^T + b) + a_{l-1}, in == out == width
 *                of the block input a_0; cross layers must precede every
 *                LINEAR_RELU layer of the block. */
typedef enum { ERASE_LAYER_LINEAR_RELU = 0, ERASE_LAYER_CROSS = 1 } erase_layer_kind;

/* Local objective of a block: s = z w + c (head Linear(last->1)),
 * l_b = mean_i [max(s_i,0) - s_i y_i + log(1 + exp(-|s_i|))]. */
typedef enum { ERASE_LOSS_BCE = 0 } erase_loss_kind;

/* Input of a block: the shared input x (independent detached
 * subarchitectures), or sg[z_{b-1}], the previous block's output (Eq. 1). */
typedef enum { ERASE_IN_X = 0, ERASE_IN_PREV = 1 } erase_input_src;

/* Schedules of one step.  All of them run the identical kernels on identical
 * inputs and produce bit-identical results.
 *   SERIAL:        everything on the forward stream: forward+loss of blocks
 *                  1..B, then backward of blocks B..1, then Adam of 1..B
 *                  (a block whose first-layer weight gradient carries its
 *                  Adam update runs all of its Adam in that launch, at the
 *                  end of its backward).
 *   OVERLAP:       ERASE early backward: forward+loss of block b on the
 *                  forward stream, then block b's backward and Adam on the
 *                  backward stream after an event, overlapping block b+1's
 *                  forward; the step ends with the forward stream joined on
 *                  the backward stream.
 *   SERIAL_GRAPH / OVERLAP_GRAPH: the same sequences captured once into a HIP
 *                  graph (per distinct x/labels/losses pointers and step
 *                  parity) and replayed.
 *   PIPELINE:      the OVERLAP order without the end-of-step join: block
 *                  b's next forward waits only for its own previous backward
 *                  (and, in a chain, for block b+1's), so one step's last
 *                  backwards overlap the next step's first forwards.  Work
 *                  enqueued on the forward stream after a PIPELINE step is
 *                  not ordered after that step's backward; call erase_sync()
 *                  before reading parameters.  Any other schedule, and
 *                  erase_sync(), joins the outstanding backward first.
 *   OVERLAP_ADAM_END: early backward as in OVERLAP, but the parameter
 *                  updates wait for the end of the step: after every
 *                  backward has finished, the forward stream runs Adam of
 *                  blocks 1..B (gradients are produced early, the optimizer
 *                  steps once per step, as in Section 2.2).
 *   UNDETACHED:    the conventional baseline the paper compares against
 *                  (Section 3): the same network and objective without the
 *                  stop-gradient at the cuts.  A block reading the previous
 *                  block's output sends the gradient at its input back into
 *                  that block, so the gradients differ from the detached
 *                  schedules for chains (identical for blocks on the shared
 *                  input).  Every forward, then one backward from the last
 *                  block to the first, then Adam, all on the forward stream.
 *                  ERASE_ERR_UNSUPPORTED unless each chained block starts,
 *                  and the block it reads ends, with a linear+ReLU layer.
 *   UNDETACHED_GRAPH: UNDETACHED captured as a HIP graph and replayed (the
 *                  conventional step without per-launch host cost, the
 *                  control of OVERLAP_GRAPH); same results as UNDETACHED. */
typedef enum {
  ERASE_SCHED_SERIAL = 0,
  ERASE_SCHED_OVERLAP = 1,
  ERASE_SCHED_SERIAL_GRAPH = 2,
  ERASE_SCHED_OVERLAP_GRAPH = 3,
  ERASE_SCHED_PIPELINE = 4,
  ERASE_SCHED_OVERLAP_ADAM_END = 5,
  ERASE_SCHED_UNDETACHED = 6,
  ERASE_SCHED_UNDETACHED_GRAPH = 7
} erase_schedule;

typedef struct {
  int32_t kind;     /* erase_layer_kind */
  int32_t in_dim;   /* >= 1 */
  int32_t out_dim;  /* >= 1, <= 65536 */
} erase_layer_spec;

typedef struct {
  int32_t input_src;                /* erase_input_src; block 0 must read x */
  int32_t n_layers;                 /* 1..16; the last layer must be LINEAR_RELU */
  const erase_layer_spec* layers;   /* host, [n_layers] */
  int32_t loss;                     /* erase_loss_kind */
  float lambda;                     /* weight of l_b in Eq. 2 (finite) */
} erase_block_spec;

typedef struct {
  int32_t n_blocks;                 /* 1..64 */
  const erase_block_spec* blocks;   /* host, [n_blocks] */
  int32_t batch;                    /* M, 1..2^24 */
  int32_t in_dim;                   /* width of x, >= 1 */
  int32_t x_ld;                     /* row pitch of x in elements, >= in_dim, multiple of 16 bytes */
  int32_t dtype;                    /* erase_dtype */
  float lr, beta1, beta2, eps;      /* Adam (bias-corrected, eps outside the sqrt); lr >= 0,
                                       0 <= beta < 1, eps >= 0 */
  int32_t x_in_place;               /* 0: every step copies x into a zero-padded buffer of the
                                       workspace.  1: the GEMMs read x where it is; the caller
                                       guarantees that x's row tails [in_dim, x_ld) are zero, and
                                       x_ld and batch must be multiples of 128 (ERASE_ERR_SHAPE) */
} erase_config;

/* Per-block fp32 device buffers, each of erase_param_count() elements, in
 * this flat order: for every layer W[out][in] (row-major) then b[out]; then
 * the head weight w[last] and bias c[1] (torch nn.Linear order).
 * param/m/v are read and updated in place; grad (may be NULL) receives the
 * step's gradient of L = sum lambda_b l_b. */
typedef struct {
  float* param;
  float* m;
  float* v;
  float* grad;
} erase_block_buffers;

/* Number of fp32 parameters of block `block`.  Host only; no HIP call. */
ERASE_API erase_status erase_param_count(const erase_config* cfg, int32_t block, int64_t* count);

/* Bytes of device workspace erase_init() needs for `cfg` (activations in both
 * row- and feature-major layouts, activation gradients, GEMM copies of the
 * weights, split-reduction partials, counters).  Host only; no HIP call. */
ERASE_API erase_status erase_workspace_bytes(const erase_config* cfg, size_t* bytes);

/* Validate `cfg`, carve `workspace` (device, 256-byte aligned, ws_bytes >=
 * erase_workspace_bytes) and create the context with its events.  Enqueues on
 * s_fwd the derivation of the GEMM weight copies from the current parameters
 * and resets the step counter to 0; does not synchronize.  `bufs` is a host
 * array of n_blocks entries whose device buffers must stay valid for the
 * context's life.  The config is copied; `cfg` may be freed afterwards. */
ERASE_API erase_status erase_init(const erase_config* cfg, const erase_block_buffers* bufs,
                        void* workspace, size_t ws_bytes, void* s_fwd, void* s_bwd,
                        erase_ctx** ctx_out);

/* erase_init() with `n_bwd` backward streams (1..8, distinct, none equal to
 * s_fwd; `s_bwd` is a host array).  In the overlapped schedules block b's
 * backward and Adam run on s_bwd[b % n_bwd], so the backwards of different
 * blocks may also overlap one another (the paper's CTR model used four side
 * streams, Section 3.2).  erase_init() is this call with n_bwd = 1. */
ERASE_API erase_status erase_init_streams(const erase_config* cfg, const erase_block_buffers* bufs,
                                void* workspace, size_t ws_bytes, void* s_fwd, void* const* s_bwd,
                                int32_t n_bwd, erase_ctx** ctx_out);

/* Enqueue one training step (Section 2.2) and return without waiting.
 *   x:      device, [batch][x_ld] of dtype, 16-byte aligned, rows' tails
 *           beyond in_dim are ignored;
 *   labels: device fp32 [batch], values in {0,1};
 *   losses: device fp32 [n_blocks], receives the unweighted l_b.
 * x, labels and losses must stay unmodified and valid until erase_sync().
 * The step increments the device step counter before its Adam updates. */
ERASE_API erase_status erase_step(erase_ctx* ctx, const void* x, const float* labels, int32_t schedule,
                        float* losses);

/* Wait for all enqueued work of the context, then report deferred errors
 * (HIP errors, non-finite loss: ERASE_ERR_NONFINITE, sticky). */
ERASE_API erase_status erase_sync(erase_ctx* ctx);

/* Read / overwrite the device step counter t (Adam bias correction uses t+1
 * at the next step).  Both synchronize the forward stream.  Used for
 * checkpoint/resume together with the caller-owned param/m/v buffers. */
ERASE_API erase_status erase_get_step(erase_ctx* ctx, int64_t* t);
ERASE_API erase_status erase_set_step(erase_ctx* ctx, int64_t t);

/* Re-derive the GEMM weight copies after the caller changed `param` (e.g. a
 * checkpoint load).  Enqueued on s_fwd. */
ERASE_API erase_status erase_refresh_weights(erase_ctx* ctx);

/* Per-launch kernel timing, for measurement.  When enabled, non-graph
 * schedules bracket every kernel launch with timing events on the launch's
 * own stream (graph schedules return ERASE_ERR_UNSUPPORTED while enabled).
 * erase_read_timing() fills up to `cap` records of the last completed step
 * (call after erase_sync()) and sets *n to the number of records: record 0
 * is an empty event pair on the forward stream (kind 7; its length is the
 * cost of the timing itself), then one record per launch in enqueue order. */
typedef struct {
  int32_t kind;      /* 0 prologue, 1 forward GEMM, 2 head+loss, 3 weight-grad GEMM,
                        4 input-grad GEMM, 5 Adam, 6 input- and weight-grad GEMMs of one
                        layer in one launch, 7 empty interval (no kernel), 8 last
                        forward GEMM of a block with the head+loss in its epilogue
                        (used when the last layer is linear+ReLU and at most 128
                        wide in bf16, 64 in fp32; kind 2 does not appear then),
                        9 forward GEMM with two k-groups per workgroup (bf16
                        forward launches of at most one workgroup per CU),
                        10 weight-grad GEMM of a block's first layer with two
                        k-groups and that layer's Adam update in its epilogue
                        (kind 5 then updates the block's other parameters),
                        11 the launch of kind 10 that also runs the Adam
                        update of the block's other parameters in extra
                        workgroups (used whenever a block's Adam directly
                        follows its backward: every schedule but
                        OVERLAP_ADAM_END; no kind 5 for the block then) */
  int32_t block;     /* block index, -1 for the step prologue */
  int32_t layer;     /* layer index within the block, -1 if none */
  int32_t stream;    /* 0 forward stream, 1 + k backward stream k */
  float start_ms;    /* relative to the step's first event on the forward stream */
  float end_ms;
  int32_t tile_m;    /* GEMM workgroup tile rows (0 for non-GEMM kernels) */
  int32_t tile_n;    /* GEMM workgroup tile columns */
  int32_t split;     /* GEMM contraction slices */
  int32_t grid;      /* workgroups launched */
  double flops;      /* algorithmic floating-point operations of the launch */
  double bytes;      /* algorithmic HBM bytes of the launch */
} erase_kernel_time;

ERASE_API erase_status erase_set_timing(erase_ctx* ctx, int32_t enable);
ERASE_API erase_status erase_read_timing(erase_ctx* ctx, erase_kernel_time* out, int32_t cap, int32_t* n);

/* Host dispatch of the ERASE schedules (Section 2.2: blocking dispatch on
 * the main thread vs non-blocking dispatch on a thread pool).
 *   ERASE_DISPATCH_CALLER (default): erase_step() enqueues every launch and
 *       event on the calling thread.
 *   ERASE_DISPATCH_WORKER: for OVERLAP, OVERLAP_ADAM_END and PIPELINE, a
 *       host thread owned by the context enqueues each block's backward,
 *       Adam and backward-stream events while the calling thread goes on
 *       with the next block's forward.  erase_step() may return before the
 *       worker has enqueued the step's backward work; the next
 *       erase_step() orders itself against it, and erase_sync() (like every
 *       other call) first waits for it.  HIP errors on the worker surface at
 *       the next call.  Graph schedules, the serial schedules and timed
 *       steps (erase_set_timing) always dispatch on the caller.
 * Results are bit-identical in both modes; the order in which the two
 * streams' launches reach the device is not fixed in worker mode.  The
 * thread is started on the first switch to ERASE_DISPATCH_WORKER (the
 * calling thread's current device must be the context's) and joined by
 * erase_destroy().  ERASE_ERR_INVALID_ARG for an unknown mode. */
typedef enum { ERASE_DISPATCH_CALLER = 0, ERASE_DISPATCH_WORKER = 1 } erase_dispatch;
ERASE_API erase_status erase_set_dispatch(erase_ctx* ctx, int32_t mode);

/* Embedding-bag input stage of the CTR workload.  The paper feeds its CTR
 * model (Section 3.2) an input embedding x (Section 2.1) without describing
 * it; this is the synthetic CTR input recipe of the benchmark workload, on
 * the device:
 *   x[m][j]                   = log1p(dense[m][j])                 j < n_dense
 *   x[m][n_dense + t*dim + d] = sum over i in bag (t, m) of tables[t][indices[i]][d]
 *   x[m][k]                   = 0        n_dense + n_tables*dim <= k < x_ld
 * Bag (t, m) is indices[offsets[t*(batch+1) + m] .. offsets[t*(batch+1) + m + 1]).
 * Each bag is summed in fp32 in index order, then rounded (to nearest even)
 * to x's dtype; log1p is evaluated in fp32.
 * Device pointers: dense fp32 [batch][n_dense] (NULL when n_dense = 0),
 * offsets int64 [n_tables][batch+1], indices int32 [nnz] (NULL when
 * nnz = 0), tables fp32 [n_tables][rows][dim] (16-byte aligned), x
 * [batch][x_ld] of dtype (16-byte aligned, x_ld*esz a multiple of 16
 * bytes), status int32 [1] or NULL.  The caller owns all of them.
 * Invalid offsets (not 0 <= begin <= end <= nnz) or indices (outside
 * [0, rows)) read nothing and contribute zero; they set *status = 1, which
 * the library never clears.  Enqueued on `stream` (a HIP stream handle,
 * NULL for the default stream); returns without waiting.
 * ERASE_ERR_INVALID_ARG (null or misaligned pointer) / ERASE_ERR_SHAPE
 * (batch 1..2^24, n_dense 0..4096, n_tables 1..4096 with n_tables*batch <
 * 2^31, dim a multiple of 4 in 4..256, rows 1..2^31-1, nnz 0..2^31-1,
 * x_ld >= n_dense + n_tables*dim) before anything is enqueued;
 * ERASE_ERR_HIP if the launch fails. */
typedef struct {
  int32_t batch;
  int32_t n_dense;
  int32_t n_tables;
  int32_t dim;
  int64_t rows;
  int64_t nnz;
  int32_t dtype;  /* erase_dtype of x */
  int64_t x_ld;
} erase_bag_config;

ERASE_API erase_status erase_embed_bags(const erase_bag_config* cfg, const float* dense, const int64_t* offsets,
                              const int32_t* indices, const float* tables, void* x, int32_t* status,
                              void* stream);

/* Backward of the embedding-bag stage: the gradient of the tables given the
 * gradient dx at x (the part of a model the paper leaves to the usual
 * end-of-step backward, Section 2.2, when it trains its tables from the
 * gradient every block sends into the shared input; under this library's
 * detached reading no block sends one):
 *   table_grad[t][r][d] = sum over the entries i of the bags of table t with
 *                         indices[i] == r of dx[m(i)][n_dense + t*dim + d]
 * where m(i) is the bag (row of x) holding entry i.  Each row's entries are
 * summed in fp32 in a fixed order of increasing entry index: rows of at most
 * 64 entries by the lane groups of one wave (G = dim/4 rounded up to a
 * power of two lanes each; entry k to group k mod 64/G, each group in order,
 * the groups then added by a fixed butterfly); rows of 65..1024 entries by
 * the lane groups of a 256-thread workgroup and rows of 1025..16384 entries
 * by those of a 1024-thread one (entry k to group k mod threads/G, the
 * groups' partial rows then added in group order); larger rows
 * in increasing entry order (by repeated selection: correct but slow).  The
 * result does not depend on scheduling; rows no entry selects are zero.
 * Bags must not overlap (each entry belongs to at most one bag; entries of
 * no bag are ignored).
 * Device pointers: offsets, indices as for erase_embed_bags; dx [batch][x_ld]
 * of dtype (16-byte aligned); table_grad fp32 [n_tables][rows][dim]
 * (16-byte aligned, fully written); scratch of
 * erase_embed_bags_backward_scratch_bytes() bytes (16-byte aligned, any
 * contents; the call clears what it needs); status as for erase_embed_bags
 * (invalid offsets or ids set it to 1).  Eleven launches on `stream`, no wait.
 * ERASE_ERR_SHAPE also when n_tables * rows >= 2^31; ERASE_ERR_WORKSPACE for
 * a missing, misaligned or small scratch. */
ERASE_API erase_status erase_embed_bags_backward_scratch_bytes(const erase_bag_config* cfg, size_t* bytes);
ERASE_API erase_status erase_embed_bags_backward(const erase_bag_config* cfg, const int64_t* offsets, const int32_t* indices,
                                       const void* dx, float* table_grad, void* scratch, size_t scratch_bytes,
                                       int32_t* status, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc):
 * erase_embed_bags_backward() with the library's own scratch instead of a
 * caller's.  Same arguments, results and errors otherwise.  The scratch is
 * one static device array of ERASE_BAG_SCRATCH_MAX bytes per GPU, created
 * with the library's code on that GPU and held until the process ends; its
 * device address is looked up on the first call on each device.  Shapes
 * whose erase_embed_bags_backward_scratch_bytes() exceeds it return
 * ERASE_ERR_WORKSPACE before anything is enqueued (the 26 x 100000-row,
 * 4096-row-batch CTR shape needs about 48 MB).  Allocates nothing: no
 * hipMalloc, hipFree or allocating library call.  Every call on one GPU
 * shares that GPU's array (the launches clear what they need first): calls
 * that overlap on one GPU -- unordered streams, or several host threads --
 * race; order them on one stream. */
#define ERASE_BAG_SCRATCH_MAX ((size_t)64 << 20)
ERASE_API erase_status erase_embed_bags_backward_noalloc(const erase_bag_config* cfg, const int64_t* offsets,
                                                         const int32_t* indices, const void* dx, float* table_grad,
                                                         int32_t* status, void* stream);

/* Destroy the context: waits for its dispatch thread and streams, frees
 * events and graphs.  Never frees caller memory.  NULL is accepted. */
ERASE_API erase_status erase_destroy(erase_ctx* ctx);

/* Static description of a status code. */
ERASE_API const char* erase_status_str(int32_t status);

/* Last error message recorded on the context ("" if none). */
ERASE_API const char* erase_last_error(erase_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* ERASE_H_ */
