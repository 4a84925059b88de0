/*
 * ppipe.h -- C ABI of the MI355X partition-forward library.
 *
 * A pipeline partition is the contiguous range of fused layers [begin, end)
 * of a CNN, "layers i to j (exclusive)" in the paper's MILP inputs (Appendix
 * A.1, table of inputs, C_ldbij and X_ldbij).  The library runs that range at
 * a batch size b on one GPU (the batched inference each GPU of a pool
 * performs, Sec. 2 and Sec. 3) and measures the per-layer latency table
 * L_kbi and feature-map sizes S_i that the planner consumes (Sec. 3 "Inputs",
 * Sec. 5.1 offline phase, Sec. 5.2: partition latency is the sum of its
 * constituent latencies).
 *
 * Conventions shared by every call:
 *  - Activations are NHWC, densely packed, in the partition's storage dtype.
 *  - Host parameter arrays are fp32; weights use the OIHW layout of the
 *    framework that defined the model ([out][in] for fully connected layers,
 *    whose input index follows the (c, h, w) flattening of the producer's
 *    output).  The library repacks them at create time.
 *  - A "layer" is fused: a convolution carries its batch norm, bias,
 *    residual add and activation.  Layer indices are global to the model.
 *  - Failing calls return NULL or a negative status and leave a message for
 *    ppipe_last_error() in the calling thread.  No call aborts the process.
 *  - A handle is not thread-safe; distinct handles are independent.
 */
#ifndef PPIPE_H
#define PPIPE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { PPIPE_F32 = 0, PPIPE_F16 = 1, PPIPE_BF16 = 2 } ppipe_dtype;

typedef enum {
    PPIPE_OP_CONV = 0,           /* k x k convolution, groups 1 or depthwise (groups = c_in = c_out) */
    PPIPE_OP_MAXPOOL = 1,        /* k x k window, stride, padding that never wins the max */
    PPIPE_OP_AVGPOOL_GLOBAL = 2, /* mean over H x W, output 1 x 1 */
    PPIPE_OP_FC = 3,             /* y = act(W x + b) on the flattened input */
    PPIPE_OP_FC_SOFTMAX = 4      /* p = softmax(W x + b), fp32 output; must be the range's last layer */
} ppipe_op;

typedef enum { PPIPE_ACT_NONE = 0, PPIPE_ACT_RELU = 1, PPIPE_ACT_RELU6 = 2 } ppipe_act;

typedef enum {
    PPIPE_OK = 0,
    PPIPE_E_INVALID = -1,        /* bad argument, shape or batch */
    PPIPE_E_SPLIT = -2,          /* a tensor other than layer begin-1's output crosses the boundary */
    PPIPE_E_UNSUPPORTED = -3,    /* layer shape outside what the kernels implement */
    PPIPE_E_NOMEM = -4,          /* device allocation failed */
    PPIPE_E_HIP = -5             /* HIP runtime error (launch, event, stream, graph) */
} ppipe_status;

/* One fused layer.  Host pointers belong to the caller and are read only
 * during ppipe_partition_create; they may be NULL for layers outside the
 * created range.  For CONV with batch norm, all four bn_* arrays are given
 * (length c_out) and the layer computes
 *     act( (conv(x) + bias - mean) / sqrt(var + bn_eps) * gamma + beta + res ),
 * else act(conv(x) + bias + res); bias may be NULL (zero). */
typedef struct {
    int32_t op;          /* ppipe_op */
    int32_t src;         /* producer layer index, -1 = model input */
    int32_t res_src;     /* layer whose output is added before act, -1 = none (CONV only) */
    int32_t c_in;        /* input channels; for FC the flattened input length */
    int32_t c_out;
    int32_t k;           /* square window (CONV, MAXPOOL) */
    int32_t stride;
    int32_t pad;
    int32_t groups;      /* 1, or c_in (== c_out) for depthwise */
    int32_t act;         /* ppipe_act */
    const float* weight; /* CONV [c_out][c_in/groups][k][k]; FC [c_out][c_in] */
    const float* bias;   /* [c_out] or NULL */
    const float* bn_gamma;
    const float* bn_beta;
    const float* bn_mean;
    const float* bn_var;
    float bn_eps;
    const char* name;    /* NUL-terminated layer name (copied at create), or NULL: "layer<i>" */
} ppipe_layer_desc;

/* The whole model (all layers from 0), so shapes can be derived for any
 * range.  Input is in_c x in_h x in_w per image. */
typedef struct {
    int32_t n_layers;
    const ppipe_layer_desc* layers;
    int32_t in_c, in_h, in_w;
    int32_t max_batch;   /* largest batch run() accepts; <= 0 selects 64 */
} ppipe_model_desc;

typedef struct ppipe_partition ppipe_partition;

typedef struct {
    int32_t layer_begin, layer_end;  /* the range [begin, end) */
    int32_t dtype;                   /* ppipe_dtype of activations and weights */
    int32_t max_batch;
    int32_t in_c, in_h, in_w;        /* per-image input of the range (NHWC) */
    int32_t out_c, out_h, out_w;     /* per-image output of the range */
    int32_t out_dtype;               /* PPIPE_F32 when the range ends with FC_SOFTMAX */
    int64_t in_bytes_per_image, out_bytes_per_image;
    int64_t weight_bytes;            /* device bytes of packed weights, scales and biases */
    int64_t workspace_bytes;         /* device bytes of activation and split-K buffers */
    int32_t tuned;                   /* 1 when created with a planner override
                                        (ppipe_partition_create_tuned), else 0 */
    int32_t cus;                     /* compute units the kernel grids were planned for:
                                        the device's, or one CU share's
                                        (ppipe_partition_create_on_share) */
} ppipe_partition_info_t;

typedef struct {
    int32_t index;                   /* global layer index */
    int32_t op;                      /* ppipe_op */
    int32_t out_c, out_h, out_w;
    int32_t kernel_count;            /* launches this layer issues at the queried batch */
    int64_t out_bytes_b1;            /* S_i: output feature-map bytes at batch 1 */
    double flops_b1;                 /* algorithmic FLOPs at batch 1 (2 per multiply-add) */
    double act_bytes_b1;             /* input + output (+ residual) activation bytes at batch 1 */
    double param_bytes;              /* weight bytes in dtype + fp32 scale/bias, once per run */
    char kernel[96];                 /* kernel configuration chosen at the queried batch;
                                        ends in " paired=J" when the layer runs in one
                                        launch with layer J */
    char name[64];                   /* the layer's name from its description */
    int32_t forced;                  /* 1 when a tuning override chose this layer's
                                        kernel at the queried batch */
} ppipe_layer_info_t;

typedef struct {
    int32_t layer;                   /* global layer index */
    int32_t launch;                  /* 0-based launch number within the layer */
    char kernel[96];                 /* kernel configuration */
    double flops;                    /* algorithmic FLOPs attributed to this launch */
    double bytes;                    /* algorithmic HBM bytes attributed to this launch */
    float mean_us, median_us, min_us;
} ppipe_kernel_record;

/* Build a partition of layers [layer_begin, layer_end) of desc in dtype.
 * Validates the range and every layer shape, folds batch norm into fp32
 * per-channel scale and bias, repacks weights to the kernels' layout in
 * dtype, and allocates device weights plus activation and split-K buffers
 * sized for desc->max_batch.  Returns NULL on error (PPIPE_E_SPLIT when a
 * layer in the range reads a tensor produced before layer_begin other than
 * layer_begin-1's output, or a layer after the range reads one produced
 * inside it other than layer_end-1's output).  Uses the current HIP device. */
ppipe_partition* ppipe_partition_create(const ppipe_model_desc* desc,
                                        int32_t layer_begin, int32_t layer_end,
                                        int32_t dtype);

/* Planner overrides, for kernel tests and tuning sweeps only.  A
 * partition created with overrides runs the configurations they name
 * instead of the planner's choices; ppipe_partition_info reports `tuned`
 * and ppipe_layer_info `forced` for every layer the overrides changed, so a
 * latency table taken on such a handle says so.  Zero fields (gemm_cfg -1)
 * leave the planner's choice. */
typedef struct {
    int32_t gemm_cfg;      /* -1, or a GEMM configuration id forced on every eligible layer */
    int32_t gemm_waves;    /* waves per block of a forced skinny configuration (4, 8, 16) */
    int32_t gemm_splits;   /* K splits of a forced LDS-staged configuration (1..64) */
    int32_t no_pointwise;  /* nonzero: never plan the streaming 1x1 kernel */
    int32_t no_stem;       /* nonzero: never plan the stem kernel */
    int32_t stream_grid;   /* > 0: blocks along the pixels of the streaming 1x1 and stem kernels */
    int32_t no_pair;       /* nonzero: never run paired layers as one launch */
    int32_t dw_outputs;    /* 0, or 2 / 4 outputs per thread of stride-1 depthwise layers */
} ppipe_tuning;

/* ppipe_partition_create with planner overrides (NULL: none, the same as
 * ppipe_partition_create).  PPIPE_E_INVALID for a field out of range. */
ppipe_partition* ppipe_partition_create_tuned(const ppipe_model_desc* desc,
                                              int32_t layer_begin, int32_t layer_end,
                                              int32_t dtype, const ppipe_tuning* tuning);

/* ppipe_partition_create for a handle that will run on the streams of one of
 * `parts` CU shares (ppipe_stream_create_cu_share(i, parts, ...), a virtual
 * GPU of 1/parts, Sec. 5.3): the planner sizes every kernel grid for the
 * compute units of one share instead of the whole device, as the paper
 * profiles each virtual-GPU size on its own.  Outputs stay within the
 * stated tolerances of the oracle; they can differ in the last bits from a
 * handle planned for the whole device (other tiles, other K splits).
 * parts = 1 is ppipe_partition_create.  NULL with PPIPE_E_INVALID for parts
 * outside 1..8. */
ppipe_partition* ppipe_partition_create_on_share(const ppipe_model_desc* desc,
                                                 int32_t layer_begin, int32_t layer_end,
                                                 int32_t dtype, int32_t parts);

/* Forward pass of the range at batch size `batch` (1..max_batch).
 * in:  device pointer, [batch][in_h][in_w][in_c] in dtype (caller-owned).
 * out: device pointer, [batch][out_h][out_w][out_c] in out_dtype (caller-owned);
 *      [batch][classes] fp32 probabilities when the range ends with FC_SOFTMAX.
 * stream: a hipStream_t (NULL = default stream).  Asynchronous: enqueues work
 * on the stream and returns; no host synchronisation, no allocation.  If a
 * graph for (batch, in, out) was captured with ppipe_partition_capture it is
 * replayed, otherwise the kernels are launched directly.  A GEMM layer and
 * a later GEMM layer that read the same tensor (a residual stage's first
 * convolution and its downsample projection) go out as one launch when both
 * are planned on the same tile configuration without a K split; timed and
 * profiled runs keep one launch sequence per layer.  Concurrent runs of
 * one handle on different streams race on its buffers. */
int ppipe_partition_run(ppipe_partition* h, int32_t batch, const void* in,
                        void* out, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, allocation-free serving loops, harnesses that forbid hipMalloc):
 * ppipe_partition_run with the kernels' scratch memory -- split-K partial
 * sums, the fp32 logits of a final FC + softmax and the channel-padded input
 * of a stem -- taken from a fixed device array of PPIPE_STATIC_SCRATCH_BYTES
 * that the library holds on every device it runs on (from the first create
 * on that device until the process ends), instead of the handle's
 * workspace.  Intermediate activations stay in the handle's buffers, which
 * create allocated.  Launches directly (a graph captured for the handle is
 * not replayed); allocates nothing, no host synchronisation.  Same arguments
 * and layouts as ppipe_partition_run and bit-identical output.  Returns
 * PPIPE_E_INVALID, launching nothing, when the handle at `batch` needs more
 * scratch than PPIPE_STATIC_SCRATCH_BYTES, PPIPE_E_HIP when the array's
 * address could not be resolved on the handle's device.  Every call on one
 * device shares that device's array and leaves its contents behind: calls
 * whose work overlaps in time on one device (different streams, threads or
 * handles) race on it. */
#define PPIPE_STATIC_SCRATCH_BYTES ((int64_t)64 << 20)
int ppipe_partition_run_static_scratch(ppipe_partition* h, int32_t batch, const void* in,
                                       void* out, void* stream);

/* Record the launches run() would issue for (batch, in, out) into a HIP
 * graph (host-side work only; allocates graph objects).  Later runs with the
 * same triple replay it.  Returns a status. */
int ppipe_partition_capture(ppipe_partition* h, int32_t batch, const void* in,
                            void* out);

/* Per-layer latency table, in sequence: for each batch_sizes[j], `warmup`
 * untimed runs, then `reps` runs of the range in layer order on a private
 * stream, each layer's first kernel launch recording a HIP event before it
 * and its last launch one after it (events recorded by the launches
 * themselves, nothing between the kernels); out_us[i * n_batches + j] =
 * median microseconds of layer begin + i over the runs.  out_partition_us[j]
 * = median over three trials of the whole range replayed `reps` times back
 * to back as one captured HIP graph (per replay).  Either output may be NULL.
 * Allocates its own input and output buffers, synchronises internally.
 * Returns a status. */
int ppipe_profile_layers(ppipe_partition* h, const int32_t* batch_sizes,
                         int32_t n_batches, int32_t warmup, int32_t reps,
                         float* out_us, float* out_partition_us);

/* Per-launch timing at one batch: like ppipe_profile_layers but with events
 * around every kernel launch.  Writes up to `capacity` records, sets *count
 * to the number of launches per run.  Returns a status. */
int ppipe_profile_kernels(ppipe_partition* h, int32_t batch, int32_t warmup,
                          int32_t reps, ppipe_kernel_record* records,
                          int32_t capacity, int32_t* count);

/* Partition-boundary quantisation (Implementation section: fp32 feature
 * maps cross a partition boundary as fp16, halving the transfer).  Converts
 * n elements of `in` (in_dtype) into `out` (out_dtype) on `stream`,
 * asynchronously, on the current HIP device.  Narrowing rounds to nearest
 * even, overflows to +-inf, keeps subnormals and NaN; widening is exact.
 * in / out: device pointers, caller-owned, not overlapping, NHWC order
 * unchanged.  Returns a status (PPIPE_E_INVALID for a bad dtype, n < 0 or a
 * null buffer with n > 0). */
int ppipe_cast(const void* in, int32_t in_dtype, void* out, int32_t out_dtype, int64_t n,
               void* stream);

/* Virtual GPUs (Sec. 5.3: a physical GPU split into 1/1, 1/2, 1/3 or 1/4
 * shares; the paper uses MPS).  Creates a stream, at default priority, on
 * the current device whose kernels run only on share `part` of `parts`
 * near-equal shares of the compute units (CU i of the device's mask
 * numbering, which goes round-robin over the XCDs, belongs to share
 * (i / 8) mod parts, so every share keeps CUs on every XCD).  *stream receives a hipStream_t; release it
 * with ppipe_stream_destroy.  Runs of different handles on the streams of
 * different shares proceed side by side.  Returns a status. */
int ppipe_stream_create_cu_share(int32_t part, int32_t parts, void** stream);
int ppipe_stream_destroy(void* stream);

/* ---- pre-partitioning (host only, no device needed) ---- */

/* Valid partition boundaries of a model: ok[p] (p = 0 .. n_layers) is 1 when
 * a partition may start at layer p, i.e. every layer p, p+1, ... reads only
 * layer p-1 or later (one feature map crosses the boundary, the problem
 * statement's Y_bj); ok[0] = ok[n_layers] = 1.  `ok` holds n_layers + 1
 * entries, caller-owned.  Returns a status. */
int ppipe_split_points(const ppipe_model_desc* desc, int32_t* ok);

/* DNN pre-partitioning (Sec. 5.2): from the first layer on, consecutive
 * layers are grouped until the group's summed latency is as close as
 * possible to 1/n_blocks of the whole model's; repeated until the last
 * layer.  Groups end only at valid boundaries (split_ok as returned by
 * ppipe_split_points); of equally close ends the earlier one is taken.
 * layer_us: n_layers latencies (>= 0).  block_begin receives the first layer
 * of every block and, after them, n_layers (capacity n_layers + 1); *n_out
 * the number of blocks (close to n_blocks, not always equal).  Returns a
 * status. */
int ppipe_prepartition(const double* layer_us, const int32_t* split_ok, int32_t n_layers,
                       int32_t n_blocks, int32_t* block_begin, int32_t* n_out);

/* ---- resource-reservation adaptive batching (host only, no device) ----
 *
 * The request scheduler of Sec. 5.4 (Alg. 1 and Alg. 2 of the appendix).
 * A cluster has GPUs on nodes; each node has one uplink and one downlink
 * shared by its GPUs.  A pooled pipeline is a chain of stages (partitions);
 * each stage is a pool of GPUs that all hold that partition.  The scheduler
 * keeps, for every GPU, uplink and downlink, the time intervals reserved on
 * it, and for each decision
 *  1. probes every pipeline at its unified batch size and takes the one
 *     whose path waits least for its resources (sum over the path's
 *     transfers and inferences of slot start - earliest possible start);
 *  2. probes that pipeline from its unified batch size down to 1 and takes
 *     the first size whose completion meets the oldest queued request's
 *     deadline;
 *  3. drops the oldest request if no size does; waits if fewer requests are
 *     queued than that size (until the queued requests would just still
 *     meet the oldest deadline); otherwise reserves the probed intervals
 *     and dispatches that many requests from the head of the queue.
 * A probe walks the stages in order and, in each pool, takes the GPU that
 * completes the stage earliest (first such GPU in pool order): the transfer
 * into a stage needs the previous GPU's uplink and this GPU's downlink free
 * together for the transfer latency, then this GPU free for the inference
 * latency, each at the earliest such time (earliest slot).  Two slips of the
 * printed pseudocode are read as the prose states them: the drop test is on
 * the chosen batch size, and what is reserved is the chosen batch's probe.
 * Times are microseconds on any common clock.  A handle is not thread-safe.
 */
#define PPIPE_MAX_STAGES 16

typedef struct {
    int32_t n_stages;              /* 1 .. PPIPE_MAX_STAGES */
    const int32_t* stage_n_gpus;   /* [n_stages], each >= 1 */
    const int32_t* stage_gpus;     /* GPU ids of stage 0's pool, then stage 1's, ... */
    int32_t max_bs;                /* latency tables cover batch 1 .. max_bs */
    int32_t unified_bs;            /* the plan's batch size for this pipeline, <= max_bs */
    const double* infer_us;        /* [n_stages][max_bs]: stage s at batch b -> [s][b-1] */
    const double* net_us;          /* [n_stages][max_bs]: transfer into stage s (row 0 unused) */
} ppipe_pipeline_desc;

typedef enum {
    PPIPE_DECISION_IDLE = 0,       /* queue empty */
    PPIPE_DECISION_DISPATCH = 1,   /* bs requests from first_id on leave on `path` */
    PPIPE_DECISION_DROP = 2,       /* request first_id cannot meet its deadline */
    PPIPE_DECISION_WAIT = 3        /* call again at wake_us or at the next arrival */
} ppipe_decision_kind;

typedef struct {
    int32_t kind;                  /* ppipe_decision_kind */
    int32_t pipeline;              /* chosen pipeline (-1 when idle) */
    int32_t bs;                    /* dispatched / awaited batch size; 1 for a drop */
    int32_t probes;                /* probes this decision made */
    int64_t first_id;              /* id of the first dispatched or the dropped request */
    double start_us;               /* dispatch: first stage's inference start */
    double finish_us;              /* dispatch: last stage's inference end */
    double deadline_us;            /* dispatch: the oldest dispatched request's deadline */
    double wake_us;                /* wait: when the queued requests must go (else +inf) */
    int32_t path[PPIPE_MAX_STAGES];/* dispatch: GPU of each stage */
} ppipe_decision;

typedef struct {
    int64_t requests, dispatched, dropped;
    int64_t late;                  /* dispatched requests finishing after their deadline */
    int64_t batches, decisions, probes;
    int64_t dispatch_probes;       /* probes made by the decisions that dispatched */
    double decision_us;            /* host wall time of every decision */
    double dispatch_us;            /* host wall time of the decisions that dispatched */
    double max_finish_us;
} ppipe_sim_stats;

typedef struct ppipe_batcher ppipe_batcher;

/* Builds a scheduler over n_gpus GPUs; gpu_node[g] is GPU g's node (NULL:
 * one node per GPU).  Copies every table; the caller keeps its arrays.
 * Returns NULL on a bad description (status PPIPE_E_INVALID). */
ppipe_batcher* ppipe_batcher_create(int32_t n_gpus, const int32_t* gpu_node,
                                    int32_t n_pipelines, const ppipe_pipeline_desc* pipelines);
void ppipe_batcher_destroy(ppipe_batcher* b);

/* Queues a request; arrivals must be non-decreasing.  Returns a status. */
int ppipe_batcher_submit(ppipe_batcher* b, int64_t id, double arrival_us, double deadline_us);

/* One decision at time now_us.  deadline_wake != 0 marks a call at the
 * wake_us of a previous WAIT: the queued requests go now, so the batch size
 * is capped at the queue length.  A DISPATCH or DROP changes the state;
 * call again until IDLE or WAIT.  Returns a status. */
int ppipe_batcher_step(ppipe_batcher* b, double now_us, int32_t deadline_wake,
                       ppipe_decision* d);

/* Probe without reserving: completion time, waiting time and path (n_stages
 * entries, may be NULL) of a batch of bs (1 .. max_bs) on `pipeline` at
 * now_us.  Returns a status. */
int ppipe_batcher_probe(ppipe_batcher* b, int32_t pipeline, int32_t bs, double now_us,
                        double* finish_us, double* wait_us, int32_t* path);

/* Invariant check: *overlaps = pairs of overlapping reservations on any
 * resource (0 for a correct scheduler), *intervals = reservations held. */
int ppipe_batcher_check(const ppipe_batcher* b, int64_t* overlaps, int64_t* intervals);

/* Event-driven run over n requests arriving at arrivals_us (sorted), each
 * with deadline arrival + slo_us and id = its index: a decision round at
 * every arrival (steps until IDLE or WAIT) and at every pending wake-up.
 * Continues on the handle's state.  Fills *stats; writes up to
 * log_capacity non-idle decisions to log (may be NULL) and their number to
 * *log_count (may be NULL).  Returns a status. */
int ppipe_batcher_simulate(ppipe_batcher* b, const double* arrivals_us, int64_t n,
                           double slo_us, ppipe_sim_stats* stats, ppipe_decision* log,
                           int64_t log_capacity, int64_t* log_count);

/* Isolated-cold per-launch timing at one batch: before each of `reps`
 * repetitions of a launch, a sweep reads `sweep_bytes` of a private buffer
 * (>= 32 MiB; 512 MiB or more evicts L2 and the 256 MB memory-side cache), so
 * the launch finds its weights and activations in HBM only; the launch then
 * records a pair of HIP events around its kernel.  Records as in
 * ppipe_profile_kernels (mean, median, min over the repetitions).
 * Allocates its own buffers, synchronises internally.  Returns a status. */
int ppipe_profile_kernels_cold(ppipe_partition* h, int32_t batch, int32_t reps,
                               int64_t sweep_bytes, ppipe_kernel_record* records,
                               int32_t capacity, int32_t* count);

/* Launch timing.  Prepares (batch, in, out) for ppipe_partition_run_timed:
 * every kernel launch of a timed run records a pair of HIP events around
 * the kernel itself (hipExtLaunchKernel), on the run's stream, with no
 * packets between the kernels.  Timed runs launch directly: events recorded
 * inside a replayed graph cannot be timed on ROCm.  Allocates the events;
 * replaces an earlier set-up of the handle.  Returns a status. */
int ppipe_timing_setup(ppipe_partition* h, int32_t batch, const void* in, void* out);

/* One run of the set-up (batch, in, out) on `stream` with its launch events.
 * Asynchronous; each run overwrites the previous run's event times.
 * Returns a status (PPIPE_E_INVALID without a set-up). */
int ppipe_partition_run_timed(ppipe_partition* h, void* stream);

/* Durations of the launches of the most recent timed run, in launch order,
 * as records like ppipe_profile_kernels' with mean = median = min = that
 * run's duration.  Waits for the run's last event.  Writes up to `capacity`
 * records and sets *count to the launches per run.  Returns a status. */
int ppipe_timing_read(ppipe_partition* h, ppipe_kernel_record* records, int32_t capacity,
                      int32_t* count);

int ppipe_partition_info(const ppipe_partition* h, ppipe_partition_info_t* info);

/* Static description of global layer `index` (begin <= index < end) with the
 * kernel choice and launch count at `batch`. */
int ppipe_layer_info(const ppipe_partition* h, int32_t index, int32_t batch,
                     ppipe_layer_info_t* info);

/* Free every device and host resource of the handle.  NULL is a no-op.  The
 * caller must ensure no run() on the handle is still executing. */
void ppipe_partition_destroy(ppipe_partition* h);

/* Message of the last failing call in this thread ("" if none). */
const char* ppipe_last_error(void);

/* ppipe_status of the last failing call in this thread (0 if none); the way
 * to tell why ppipe_partition_create returned NULL. */
int32_t ppipe_last_status(void);

#ifdef __cplusplus
}
#endif

#endif /* PPIPE_H */
