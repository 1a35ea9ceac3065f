/*
 * lpp.h -- C ABI of liblpp.so, the MI355X (gfx950) implementation of the
 * per-node step of LPP-SGD (locally-partitioned asynchronous parallel SGD;
 * Chatterjee, Kungurtsev, Alistarh, "Scaling the Wild: Decentralizing
 * Hogwild!-style Shared-memory SGD", arXiv 2203.06638).
 *
 * The paper's problem statement (Sec. 2 and Sec. 3) in this library's terms:
 *   - a model is an ordered list of parameter tensors, flattened into one
 *     vector x of d floats and cut into blocks x_1..x_P of successive tensors;
 *     block 0 is the whole vector (Sec. 3, "Block partitions", eq.
 *     (partition));
 *   - K model replicas x^q live in the same HBM (the paper's workers q, one per
 *     GPU, stand in here as co-resident replicas);
 *   - each replica has P updaters (the paper's U updater processes u^q; here:
 *     "workers", one HIP stream each) and one averager (a^q);
 *   - an updater reads-and-increments the replica's counter C^q, snapshots
 *     x^q, computes the minibatch gradient with respect to one block only
 *     (partial backpropagation: it stops at that block), and subtracts
 *     lr * direction from that block of x^q in place without locks (Alg. 1,
 *     updater loop);
 *   - the averager snapshots the replicas, averages them, and adds
 *     (average - own snapshot) to each replica in place, again without
 *     locks (Alg. 1, averaging loop).
 *
 * Conventions
 *   - Every function returns an int status (enum lpp_status); nothing throws
 *     across the ABI.  lpp_last_error() returns a message for the calling
 *     thread's last failure.
 *   - "device" pointers are HIP device addresses (e.g. torch CUDA tensors'
 *     data_ptr()); "host" pointers are ordinary CPU memory.
 *   - Flat parameter vectors are float32 in the model's canonical order: the
 *     layers' parameter tensors in layer order, each flattened in its natural
 *     layout: conv W[cout][cin][k][k] then bias[cout]; batch-norm gamma[c]
 *     then beta[c]; linear W[out][in] then bias[out].
 *   - worker w in [0, K*P) belongs to replica q = w / P; its default block is
 *     w % P + 1 (the paper's rank(u^q), Sec. 3 "Block Selection Rule").  Any
 *     worker may run any partition; the selection rule is caller policy.
 */
#ifndef LPP_H
#define LPP_H

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lpp_ctx lpp_ctx; /* opaque; owns all device state it allocates */

enum lpp_status {
    LPP_OK = 0,
    LPP_EINVAL = -1,       /* bad argument or model description             */
    LPP_ENOMEM = -2,       /* device or host allocation failed              */
    LPP_EHIP = -3,         /* a HIP runtime call failed                     */
    LPP_ESTATE = -4,       /* call not valid in the context's current state */
    LPP_EUNSUPPORTED = -5  /* valid request the library does not implement  */
};

enum lpp_op {
    LPP_CONV = 0,    /* cross-correlation, zero padding; params W (+bias)     */
    LPP_BN = 1,      /* training-mode batch norm over (N,H,W); gamma, beta    */
    LPP_RELU = 2,
    LPP_ADD = 3,     /* elementwise sum of in0 and in1                        */
    LPP_MAXPOOL = 4, /* k x k window, stride, pad; padding never wins         */
    LPP_GAP = 5,     /* mean over H x W                                       */
    LPP_LINEAR = 6,  /* y = x W^T + b on the flattened input; params W, b     */
    LPP_CONCAT = 7   /* channels of in0 followed by channels of in1 (same H, W) */
};

enum lpp_dtype { LPP_FP32 = 0, LPP_BF16 = 1 };
/* Sequential: lpp_step and lpp_average wait for their work; batch-norm sums
 * are merged across workgroups in a fixed order, so repeated runs are
 * bitwise identical.  Async: calls return at once (Alg. 1's lock-free
 * updaters); batch-norm sums are merged by fp64 atomic adds, whose order
 * varies, so runs agree to rounding but not bit for bit. */
enum lpp_mode { LPP_SEQUENTIAL = 0, LPP_ASYNC = 1 };

typedef struct {
    int op;          /* enum lpp_op                                              */
    int in0, in1;    /* producer layer indices (< this layer); -1 = image batch  */
    int cin, cout;   /* conv/linear channels; bn: cout = channels                */
    int k, stride, pad; /* conv and maxpool geometry                             */
    int bias;        /* conv/linear: 1 if the layer has a bias vector            */
    int block;       /* 1..P for a layer that owns parameters, else ignored      */
} lpp_layer;

typedef struct {
    int n_layers;
    const lpp_layer* layers; /* host; the last layer's output are the logits   */
    int in_c, in_h, in_w;    /* image shape                                    */
    int n_classes;
    int batch;               /* images per step                                */
    int dtype;               /* enum lpp_dtype: LPP_BF16 = bf16 activations and
                                MFMA operands, fp32 accumulation and fp32
                                master parameters                              */
    float momentum;          /* heavy-ball momentum, 0 = plain SGD             */
    float weight_decay;      /* coupled L2 (g + wd*x), block-restricted        */
    float bn_eps;
} lpp_model_desc;

typedef struct {
    int mode;                     /* enum lpp_mode                              */
    void* const* worker_streams;  /* host array of K*P hipStream_t, or NULL: the
                                     library creates its own streams (default
                                     priority)                                  */
    void* avg_stream;             /* hipStream_t or NULL (library-created)      */
    int unfused;                  /* 0: fused kernels (default); 1: one kernel
                                     sequence per layer, every layer output kept
                                     (for lpp_get_activation on any layer)     */
    int no_graphs;                /* 0: each (worker, partition) step is captured
                                     once into a HIP graph and replayed
                                     (default); 1: kernels launched one by one.
                                     Steps run with a kernel timer enabled are
                                     always launched one by one.               */
} lpp_options;

typedef struct {
    const float* images; /* device, NCHW float32 [batch][in_c][in_h][in_w]       */
    const int* labels;   /* device, int32 [batch], 0 <= y < n_classes            */
    int n;               /* must equal the model's batch                         */
} lpp_batch;

/* Host-side summary of a model description (no GPU needed). */
typedef struct {
    long d;                  /* number of parameters                            */
    int P;                   /* number of blocks                                */
    long block_lo[65];       /* [lo, hi) of block i in x, i = 0..P (0 = whole)  */
    long block_hi[65];
    double fwd_flops;        /* forward multiply-add flops per step (2 per MAC) */
    double bwd_flops[65];    /* truncated-backward flops for partition i        */
} lpp_model_info;

/*
 * Validates a model description and summarises it without touching the GPU:
 * d, the block ranges (Sec. 3, eq. (partition)) and the flops of the
 * forward pass and of the truncated backward pass of each partition.
 * Blocks must be contiguous runs of layers in parameter order numbered
 * 1..P without gaps.  The last layer (a linear layer or a global pool) has
 * n_classes outputs: the logits.  Channel counts are multiples of 4 (of 8 for
 * bf16 convs), except the output of a 1x1, stride-1, unpadded fp32 conv,
 * which may then feed only ReLU, pooling or linear layers.  Returns
 * LPP_EINVAL for an invalid description, LPP_EUNSUPPORTED for a valid one
 * outside these limits.
 */
int lpp_describe(const lpp_model_desc* desc, int P, lpp_model_info* out);

/*
 * Creates a context: K replicas of the model (paper: Q workers, Sec. 2), each
 * with P workers and a shared iteration counter C^q = 0 (Sec. 2), on the
 * current HIP device.  Allocates replicas (fp32, K*d), per-worker snapshot,
 * momentum, gradient and activation workspaces.  Replicas start at zero: set
 * them with lpp_set_params.  opt may be NULL (sequential mode, library
 * streams).  On failure *out is NULL and nothing stays allocated.
 */
int lpp_init(const lpp_model_desc* desc, int K, int P, const lpp_options* opt, lpp_ctx** out);

/*
 * One updater iteration of worker `worker` (Alg. 1, updater loop):
 *   1. s = read&inc(C^q) on the host (q = worker / P);
 *   2. snapshot v = x^q (lock-free copy of all d entries, into the worker's
 *      own buffer and kernel layouts);
 *   3. full forward pass at v on `batch`, mean softmax cross-entropy;
 *   4. backward pass truncated at block `partition`: gradients of
 *      activations only down to the first layer of that block, parameter
 *      gradients only inside it (partial backpropagation, Sec. 3 "Discussion
 *      on the Rule"); partition 0 is the whole model;
 *   5. lock-free in-place update of that block of x^q:
 *      m = momentum*m + g + wd*x;  x -= lr*m   (m: the worker's own buffer;
 *      with momentum == 0 and wd == 0 this is x -= lr*g, Alg. 1).
 * All device work is enqueued on the worker's stream.  Sequential mode waits
 * for it before returning; async mode returns at once (the batch buffers
 * must stay valid until lpp_sync).  0 <= partition <= P; lr finite;
 * batch->n == desc->batch.  The same worker must not be entered from two
 * host threads at once; different workers may.
 */
int lpp_step(lpp_ctx* ctx, int worker, const lpp_batch* batch, int partition, float lr);

/*
 * One averaging round over the listed replicas (Alg. 1, averaging loop with
 * the all-reduce over peers done in HBM): per entry e, v_k = x_k[e] for each
 * listed k, vbar = (sum of v_k in list order) / n, x_k[e] += vbar - v_k,
 * re-reading x_k[e] (past the compute unit's cache) just before the write,
 * so a concurrent block update written back between the two reads is kept.
 * One that lands after the re-read, or is not yet visible to the averaging
 * kernel, is overwritten: a lost update, as lock-free updates permit.
 * replicas == NULL with n_replicas == 0 means all K in order.  Runs on the
 * averaging stream, concurrently with steps in async mode.
 */
int lpp_average(lpp_ctx* ctx, const int* replicas, int n_replicas);

/* Host <-> device copies of a replica's parameters (canonical fp32 layout,
 * d floats).  replica -1 in set_params writes all replicas.  Both wait for
 * all outstanding work of the context first. */
int lpp_set_params(lpp_ctx* ctx, int replica, const float* host, long d);
int lpp_get_params(lpp_ctx* ctx, int replica, float* host, long d);

/* The gradient of the worker's last step (canonical layout, d floats; zero
 * outside the stepped block), its momentum buffer, its loss and its logits
 * ([batch][n_classes]).  Wait for outstanding work first. */
int lpp_get_grad(lpp_ctx* ctx, int worker, float* host, long d);
int lpp_get_momentum(lpp_ctx* ctx, int worker, float* host, long d);
int lpp_set_momentum(lpp_ctx* ctx, int worker, const float* host, long d);
int lpp_get_loss(lpp_ctx* ctx, int worker, float* loss);
int lpp_get_logits(lpp_ctx* ctx, int worker, float* host, long n);

/* Forward activation of `layer` from the worker's last step, as float32 NCHW
 * [batch][c][h][w] (n floats).  For checking a run layer by layer; with
 * fused kernels only the outputs of convolutions and of each fused group are
 * kept (LPP_ESTATE otherwise). */
int lpp_get_activation(lpp_ctx* ctx, int worker, int layer, float* host, long n);

/* Gradient of the loss with respect to the output of `layer` from the
 * worker's last step, float32 NCHW (n floats).  LPP_ESTATE if that step's
 * truncated backward pass did not reach the layer. */
int lpp_get_activation_grad(lpp_ctx* ctx, int worker, int layer, float* host, long n);

long lpp_num_params(const lpp_ctx* ctx);
int lpp_block_range(const lpp_ctx* ctx, int i, long* lo, long* hi);
/* Current value of replica q's shared iteration counter C^q (Sec. 2). */
long lpp_counter(const lpp_ctx* ctx, int replica);

/* Waits for all work of every worker stream and the averaging stream. */
int lpp_sync(lpp_ctx* ctx);
int lpp_destroy(lpp_ctx* ctx);
const char* lpp_last_error(void);

/*
 * Kernel timing.  lpp_timer_enable(ctx, name) times every launch of the
 * kernel family `name` (e.g. "conv_fwd", "conv_wgrad", "sgd_update",
 * "average"): HIP events recorded in the dispatch packets of the family's
 * kernels themselves (start with the first kernel of a launch, stop with the
 * last), so each interval is the kernels' execution on the GPU without the
 * stream's dispatch gaps.  lpp_timer_read returns the summed event time
 * (ms), the number of launches and the summed algorithmic work of those
 * launches (flops for convolutions, bytes for the streaming kernels).  name
 * NULL disables timing.  Reading waits for all outstanding work.
 */
int lpp_timer_enable(lpp_ctx* ctx, const char* name);
int lpp_timer_read(lpp_ctx* ctx, double* ms, long* launches, double* work);

/*
 * Step tracing: the orders of the paper's delay model (Sec. 5 "snapshot
 * order", "update order", "iteration order"; their definitions in the
 * appendix) observed on the device.  lpp_trace_enable(ctx, capacity)
 * allocates logs for `capacity` steps and `capacity` averaging rounds
 * (capacity 0 frees them and stops tracing); while it is on, every
 * lpp_step brackets its snapshot and its block update with timestamp
 * kernels and every lpp_average brackets its averaging kernel (timestamps of
 * the device's constant-rate clock, lpp_trace_clock_khz ticks per ms; a
 * timestamp kernel runs in stream order between its neighbours, so the
 * intervals contain the bracketed kernels).  Traced steps replay graphs of
 * their own; untraced steps are unchanged.  Steps and rounds beyond the
 * capacity run untraced.  lpp_trace_read waits for all work and copies the
 * records in issue order (NULL arrays: counts only); LPP_ESTATE when
 * tracing is off, LPP_EINVAL when an array is too small.
 */
typedef struct {
    int worker, replica, partition;
    long counter;               /* C^q the step read (its snapshot order)    */
    unsigned long long t[4];    /* before the snapshot, after it, before the
                                   block update, after it                    */
} lpp_trace_step;
typedef struct {
    long index;                 /* averaging round j (the iteration order)   */
    int n_replicas;
    long counter_min;           /* smallest replica counter when issued      */
    unsigned long long t[2];    /* before and after the averaging kernel     */
} lpp_trace_avg;
int lpp_trace_enable(lpp_ctx* ctx, long capacity);
int lpp_trace_read(lpp_ctx* ctx, lpp_trace_step* steps, long max_steps, long* n_steps, lpp_trace_avg* avgs,
                   long max_avgs, long* n_avgs);
long lpp_trace_clock_khz(const lpp_ctx* ctx);

/*
 * Stand-alone launches of the two streaming kernels on caller buffers, for
 * bandwidth measurement at arbitrary sizes.  All pointers are device
 * pointers; stream may be NULL (default stream).  No allocation.
 *   lpp_kernel_sgd_update: for e in [0, n): m[e] = mu*m[e] + g[e] + wd*x[e];
 *     x[e] -= lr*m[e]   (m NULL: x[e] -= lr*(g[e] + wd*x[e]))
 *   lpp_kernel_average: replicas[k] (device pointers, host array of n_rep),
 *     each of n floats, averaged in place as in lpp_average.
 */
int lpp_kernel_sgd_update(float* x, float* m, const float* g, long n, float lr, float mu, float wd, void* stream);
int lpp_kernel_average(float* const* replicas, int n_rep, long n, void* stream);

/*
 * Stand-alone snapshot (Alg. 1, updater: "collect a snapshot" of the shared
 * model), the kernel lpp_step runs first, on caller buffers.  A parameter
 * vector x of d floats (device) holds conv weight tensors, each described by
 * an lpp_snap_conv; the snapshot writes
 *   - every conv weight W[cout][cin][kh][kw] (canonical, at x + src) into
 *     wbuf in the two layouts the conv kernels read: the forward layout
 *     W_f[cout][kh][kw][cin_p] at element dst_f (input channels cin..cin_p-1
 *     are never written: keep them zero) and the data-gradient layout
 *     W_d[cin][kh][kw][cout] at element dst_d, as float32 (dtype LPP_FP32)
 *     or as bf16 rounded to nearest even (LPP_BF16: wbuf holds 16-bit
 *     elements);
 *   - every other entry of x into v[e] (device, d floats); v's conv weight
 *     entries are not written.
 * Algorithmic traffic: 4 + 2 x (4 or 2) bytes per conv weight, 8 per other
 * entry.  Descriptors are sorted by src with disjoint weight ranges inside
 * [0, d); cout and cin_p are multiples of 4 (8 for bf16), cin <= cin_p;
 * dst_f and dst_d are multiples of 4 (8 for bf16) and both layouts lie
 * inside wbuf's wbuf_elems elements, else LPP_EINVAL before anything is
 * launched.
 *
 * lpp_snapshot_plan_create validates the list and builds the kernel's work
 * table (host array of convs, copied; it allocates the table in device
 * memory: at most 2 n_convs + 1 entries of 72 bytes).  lpp_kernel_snapshot
 * enqueues the snapshot on `stream` (hipStream_t, NULL = default stream)
 * and returns at once; x, v and wbuf must stay valid until it has run.  A
 * plan may be used from several threads; destroy it after its last
 * snapshot has run.
 */
typedef struct {
    long src;          /* index of the tensor's first element in x              */
    int cout, cin;     /* output / input channels                              */
    int cin_p;         /* input channels stored per W_f row                    */
    int kh, kw;        /* filter height and width                              */
    long dst_f, dst_d; /* element offsets of W_f and W_d in wbuf               */
} lpp_snap_conv;
typedef struct lpp_snap_plan lpp_snap_plan;
int lpp_snapshot_plan_create(const lpp_snap_conv* convs, int n_convs, long d, int dtype, long wbuf_elems,
                             lpp_snap_plan** out);
int lpp_kernel_snapshot(const lpp_snap_plan* plan, const float* x, float* v, void* wbuf, void* stream);
int lpp_snapshot_plan_destroy(lpp_snap_plan* plan);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * snapshot as lpp_kernel_snapshot, same arguments and results, without a
 * plan.  Its work table goes into a fixed array in the library's device
 * memory (one per GPU, 257 entries of 72 bytes, held until the process
 * ends), so it calls no allocating routine.  At most 128 convs per call
 * (LPP_EINVAL beyond, and for any list lpp_snapshot_plan_create rejects).
 * The call copies the table (hipMemcpyAsync on `stream`), launches the
 * snapshot and waits for the stream before it returns.  Every call on one
 * GPU shares that GPU's table: calls that overlap on one GPU (from several
 * host threads) race and must not be made.
 */
int lpp_kernel_snapshot_noalloc(const lpp_snap_conv* convs, int n_convs, long d, int dtype, long wbuf_elems,
                                const float* x, float* v, void* wbuf, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LPP_H */
