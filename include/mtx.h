/*
 * mtx.h -- C ABI of the MI355X (gfx950) library for one rank's step of synchronous
 * data-parallel SGD, after "User-transparent Distributed TensorFlow" (arXiv 1704.04560).
 *
 * The paper's method (Sec. III-A, III-D, III-E): every replica holds identical weights
 * (Broadcast operator, Sec. III-D.1), computes the gradient of its own shard of the batch, the
 * replicas' gradients are averaged by an all-reduce issued layer by layer in a fixed order
 * (MPI_Allreduce operator, Sec. III-D.2; Sec. II-B uses the reduction "for averaging
 * gradients"), and the optimizer step follows, so that the result equals sequential SGD
 * (Sec. III-D.2, III-E).  The user's training loop stays unchanged (Sec. I problem statement,
 * Sec. III-D, Fig. 3): here one mtx_train_step call on the whole batch hides the R replicas.
 *
 * On one GPU the R replicas are R shards of the batch processed against one shared weight
 * copy; their gradients land in R separate buffers and are averaged on the device (the local
 * half of the all-reduce), fused with the momentum update.
 *
 * Conventions for every call:
 *   - Tensor pointers are DEVICE pointers unless the name ends in _host.  The caller owns all
 *     device memory and the stream; the library never allocates device memory.  A model
 *     handle owns only host-side metadata.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued asynchronously;
 *     only the calls documented as synchronous wait for the stream.
 *   - Every call returns an mtx_status.  Arguments are validated before anything is enqueued;
 *     an invalid argument returns MTX_EINVAL (or MTX_EUNSUPPORTED) and changes nothing.  A HIP
 *     launch or copy failure returns MTX_EHIP.  mtx_last_error() gives a message for the last
 *     non-OK status of the calling thread.
 *   - Floating-point tensors are fp32 unless stated.  Layouts are logical, row-major:
 *     activations NCHW; fully connected weights W[out][in]; convolution weights
 *     W[out][in/groups][k][k]; the input of a fully connected layer that follows a
 *     convolution or pooling layer is the (c, h, w) flattening of that layer's output.
 *   - The flat parameter vector holds the layers in forward order, each layer's W followed by
 *     its bias b (the paper's ordered list of per-layer reductions, Sec. III-D.2).
 *   - A model handle must not be used from two threads, or on two streams, at once.
 */
#ifndef MTX_H
#define MTX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MTX_OK = 0,
    MTX_EINVAL = -1,       /* invalid argument (null pointer, bad size, misaligned pointer) */
    MTX_ENOMEM = -2,       /* host allocation failed, or a caller buffer is too small */
    MTX_EHIP = -3,         /* a HIP runtime call failed */
    MTX_EUNSUPPORTED = -4, /* a valid network the library does not implement */
    MTX_ENONFINITE = -5    /* the non-finite check found a non-finite gradient average */
} mtx_status;

typedef enum { MTX_F32 = 0, MTX_BF16 = 1 } mtx_dtype;

typedef enum {
    MTX_FC = 0,
    MTX_CONV = 1,
    MTX_MAXPOOL = 2,
    MTX_BN = 3,
    MTX_ADD = 4,
    MTX_ADDP = 5
} mtx_kind;

/* One layer (Sec. I and Fig. 1: fully connected and convolution layers; pooling between
 * convolutions; Table II's ResNet-50 adds batch normalisation and residual additions).
 *   MTX_FC:      out = number of outputs; relu = apply max(0, .) to the output.
 *   MTX_CONV:    out = output channels, k x k kernel, stride >= 1, zero padding pad >= 0,
 *                groups >= 1 dividing both channel counts; relu as above.
 *   MTX_MAXPOOL: k x k window (k <= 16), stride >= 1, no padding ("valid" windows); out,
 *                pad, groups and relu must be 0 (groups may also be 1).
 *   MTX_BN:      batch normalisation with the statistics of each replica's shard (mean and
 *                biased variance over its samples and positions, eps = 1e-3):
 *                y = gamma (x - mean) / sqrt(var + eps) + beta; parameters gamma[c] (in the
 *                place of W, initialised to 1) and beta[c] (in the place of b, 0); relu as
 *                above; out may be 0 or the channel count, k, pad 0.  With per-shard statistics
 *                the average of the shard gradients is not the full-batch gradient.
 *   MTX_ADD:     residual addition y = x + (output of layer k), k an earlier layer other than
 *                the previous one, with the same output shape; a layer is added at most once;
 *                relu as above; no parameters.
 *   MTX_ADDP:    residual addition through a projection shortcut (the downsampling blocks of
 *                ResNet-50, Table II): y = x + P, P = W * a_k + b, a 1x1 convolution of the
 *                given stride (pad 0, groups 1) of the output a_k of an earlier layer k other
 *                than the previous one, mapping it to this layer's shape; out = the channel
 *                count of x; parameters W[out][channels of a_k] and b[out], Glorot-initialised
 *                as a convolution's.  P is a stored output (bf16 in MTX_BF16 mode) before the
 *                addition; a layer is the source of at most one addition; relu as above.
 * The last layer must be MTX_FC without ReLU; its outputs are the class scores of a softmax
 * cross-entropy loss. */
typedef struct {
    int kind, out, k, stride, pad, groups, relu;
} mtx_layer;

typedef struct {
    int in_c, in_h, in_w;     /* per-sample input shape */
    int n_layers;
    const mtx_layer* layers;  /* read during mtx_model_sizes / mtx_init_model only */
    int compute;              /* mtx_dtype: MTX_F32, or MTX_BF16 = bfloat16 operands with fp32
                                 accumulation and fp32 master weights */
} mtx_model_desc;

typedef struct {
    size_t n_params;         /* P: length of the flat parameter vector */
    size_t grad_stride;      /* elements between the R shard gradient buffers (>= P) */
    size_t workspace_bytes;  /* device workspace mtx_init_model needs */
} mtx_sizes;

/* Device buffers of a model, all owned by the caller and 256-byte aligned:
 *   w        [P]                  fp32 master weights (updated in place by mtx_train_step)
 *   v        [P]                  fp32 momentum velocity (updated in place)
 *   grads    [R][grad_stride]     per-shard gradients, written by every mtx_train_step
 *   grad_avg [P]                  averaged gradient, written by every mtx_train_step
 *   workspace, workspace_bytes    scratch for activations, decisions and partial sums
 * The buffers must not overlap and must stay valid until mtx_free_model. */
typedef struct {
    float* w;
    float* v;
    float* grads;
    float* grad_avg;
    void* workspace;
    size_t workspace_bytes;
} mtx_buffers;

typedef struct mtx_model mtx_model;

/* Sizes for a network trained on R shards of shard_batch samples each (global batch
 * B = R * shard_batch; strong scaling, Sec. IV-B).  Host only, enqueues nothing. */
int mtx_model_sizes(const mtx_model_desc* desc, int R, int shard_batch, mtx_sizes* out);

/* Create a model handle bound to `bufs`, and initialise the replicas identically (the
 * Broadcast operator of Sec. III-D.1 -- on one GPU the R replicas share one weight vector):
 * every weight tensor W is drawn Glorot-uniform U(-a, a), a = sqrt(6 / (fan_in + fan_out))
 * (fully connected: fan_in = in, fan_out = out; convolution: fan_in = in/groups * k * k,
 * fan_out = out * k * k), from the counter-based generator
 *   h = SplitMix64 first output for state (seed XOR ((layer_index << 32) | element_index)),
 *   u = (h >> 40) / 2^24,  value = (float)(a * (2u - 1)) evaluated in double,
 * every bias is 0 and the velocity v is 0.  The copies are enqueued on `stream`; the call
 * synchronises with `stream` before it returns.  On success *out receives the handle. */
int mtx_init_model(const mtx_model_desc* desc, int R, int shard_batch, uint64_t seed,
                   const mtx_buffers* bufs, void* stream, mtx_model** out);

/* The same model creation for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops that must not call hipMalloc, harnesses that forbid it): the
 * model's workspace is a static array of 64 MiB that the library holds on every device it runs
 * on until the process ends, instead of a caller buffer.  bufs->workspace must be NULL and
 * bufs->workspace_bytes 0; w, v, grads and grad_avg come from the caller as for mtx_init_model.
 * A network whose workspace (mtx_model_sizes) exceeds 64 MiB returns MTX_ENOMEM, one with more
 * than 16 weight layouts to prepare MTX_EUNSUPPORTED.  Neither this call nor the steps of the
 * model allocate device memory.  All static models on one device share the one array: every
 * mtx_train_step of such a model first re-writes what it needs there (its preparation jobs, the
 * zeroed loss counter and padded input), so their steps may alternate, but steps of two static
 * models that overlap in time on one device race, and mtx_get_layer_output /
 * mtx_get_pool_argmax return the outputs of the last static step on the device. */
int mtx_init_model_static(const mtx_model_desc* desc, int R, int shard_batch, uint64_t seed,
                          const mtx_buffers* bufs, void* stream, mtx_model** out);

/* One synchronous data-parallel SGD step on the whole batch (Sec. III-D.2, III-E):
 *   x [B][in_c][in_h][in_w] fp32 images, labels [B] int32 in [0, num_classes); shard r is
 *   rows r*shard_batch .. (r+1)*shard_batch-1.
 *   For each shard: forward pass, softmax cross-entropy loss averaged over the shard, and the
 *   gradient of that loss into grads[r] (layer order, W then b).  Then
 *     grad_avg = (1/R) sum_r grads[r];  v = momentum*v + grad_avg;  w = w - lr*v
 *   (momentum == 0: w = w - lr*grad_avg and v is neither read nor written).
 *   loss_out (device, nullable) receives the mean loss over the batch, fp32 [1].
 * With MTX_BF16 compute, x, the weights, every hidden layer's output and every data gradient
 * are rounded to bfloat16 (round to nearest even); sums, logits, weight gradients, the average
 * and the update are fp32.  An out-of-range label gives that sample a NaN loss.  x must be
 * 16-byte aligned (it is read with 16-byte loads), labels and loss_out 4-byte aligned.
 * Asynchronous; results are deterministic run to run. */
int mtx_train_step(mtx_model* m, const float* x, const int32_t* labels, float lr,
                   float momentum, float* loss_out, void* stream);

/* avg[i] = (1/R) sum_{r<R} grads[r*ld + i] for i < n: the averaging of replica gradients
 * (Sec. II-B, III-D.2) over R buffers held on this GPU.  Requires R >= 1, n >= 1, ld >= n;
 * avg must not overlap grads.  Asynchronous. */
int mtx_average_grads(const float* grads, int R, size_t n, size_t ld, float* avg, void* stream);

/* The average above fused with the optimizer step (Sec. III-D.2, III-E; momentum method of
 * Sec. I in TensorFlow 1.0 form):
 *   g = (1/R) sum_r grads[r*ld + i];  v = momentum*v + g;  w = w - lr*v
 * momentum == 0 gives plain SGD, w = w - lr*g, and then v may be NULL (it is not touched).
 * avg_out (nullable) receives g.  w, v, avg_out must not overlap grads or each other.
 * Asynchronous. */
int mtx_sgd_update(float* w, float* v, const float* grads, int R, size_t n, size_t ld,
                   float lr, float momentum, float* avg_out, void* stream);

/* The average above followed by Adam, one of the update rules Sec. I lists among the
 * improvements to gradient descent that TensorFlow offers; the paper gives no formula, so the
 * rule is Algorithm 1 of the work it cites (Kingma and Ba), at step number `step` (>= 1):
 *   g = (1/R) sum_r grads[r*ld + i];  m = beta1*m + (1-beta1)*g;  v = beta2*v + (1-beta2)*g^2;
 *   w = w - lr * (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * g is summed in double and rounded to float once (the step divides by about |g|, so the
 * average's rounding must not be amplified where it nearly cancels).  w, m, v [n] fp32 are
 * updated in place (m = v = 0 before the first step); avg_out (nullable) receives g.  Requires 0 <= beta1, beta2 < 1, eps >= 0, finite lr; w, m, v, avg_out and grads
 * must not overlap.  Asynchronous. */
int mtx_adam_update(float* w, float* m, float* v, const float* grads, int R, size_t n,
                    size_t ld, float lr, float beta1, float beta2, float eps, long long step,
                    float* avg_out, void* stream);

/* The average followed by AdaGrad (diagonal form of the work Sec. I cites, Duchi, Hazan and
 * Singer):  g = (1/R) sum_r grads[r*ld + i];  acc = acc + g^2;  w = w - lr * g / (sqrt(acc) + eps)
 * g is summed in double and rounded once, as for Adam.  w, acc [n] fp32 are updated in place
 * (acc holds its initial value before the first step);
 * avg_out (nullable) receives g.  Requires eps >= 0 and finite lr; buffers must not overlap.
 * Asynchronous. */
int mtx_adagrad_update(float* w, float* acc, const float* grads, int R, size_t n, size_t ld,
                       float lr, float eps, float* avg_out, void* stream);

/* Copy the weights (and, if v_host != NULL, the velocity) to host memory [P], in the flat
 * logical layout.  Synchronous (waits for the model's last stream). */
int mtx_get_params(const mtx_model* m, float* w_host, float* v_host);

/* Overwrite the weights (and, if v_host != NULL, the velocity) from host memory [P].
 * Synchronous.  Used for checkpoint restore and for tests that inject parameters. */
int mtx_set_params(mtx_model* m, const float* w_host, const float* v_host);

/* Introspection of the last mtx_train_step, synchronous:
 * mtx_get_layer_output copies layer `layer`'s stored output for the whole batch
 * [B][c][h][w] (after bias and ReLU, or the pooled values) into host memory as fp32; `n` is
 * the capacity of dst in elements and must be at least the output size.
 * mtx_get_pool_argmax copies a max-pool layer's window decisions [B][c][oh][ow] (index
 * u*k + v of the first maximal element) into host memory. */
int mtx_get_layer_output(const mtx_model* m, int layer, float* dst_host, size_t n);
int mtx_get_pool_argmax(const mtx_model* m, int layer, uint8_t* dst_host, size_t n);

/* Graph replay (execution option; default off: on MI355X direct launches of the step measured
 * faster than replaying it from a graph).  With it on, mtx_train_step records its kernel sequence
 * into a HIP graph on a private stream and replays it on the caller's stream for as long as
 * (x, labels, lr, momentum, loss_out) stay the same; other arguments trigger a new capture, and
 * after three captures in a row the model stays on direct launches.  Steps run directly, without
 * a graph, while kernel timing is on or when the caller's stream is itself being captured.  The
 * results do not depend on this option.  enable = 0 switches it off (and frees the graph). */
int mtx_set_graph_replay(mtx_model* m, int enable);

/* Overlap (execution option; default on when a step's matrix work is at least 50 GFLOP, where
 * it measured faster, off for smaller steps).  The data gradients of a step form a chain from the
 * last layer to the first; each layer's weight gradient needs only that layer's output
 * gradient and input.  With overlap on, mtx_train_step runs the weight gradients on a second
 * stream of the model, forked from the caller's stream after each output gradient is written
 * and joined back before the average + update, so they run beside the chain.  The results do
 * not depend on this option.  Steps run on the caller's stream alone while kernel timing is
 * on.  enable = 0 switches it off. */
int mtx_set_overlap(mtx_model* m, int enable);

/* Non-finite check (option, default off; for training loops that must not let an overflow
 * into the weights).  With it on, mtx_train_step averages the R shard gradients into grad_avg
 * first and flags any average that is not finite (Inf or NaN), then applies the momentum rule
 * from grad_avg only if nothing was flagged (the same values as without the check), waits for
 * the step (a synchronisation of the caller's stream) and returns MTX_ENONFINITE when the update
 * was skipped: w and v are then unchanged, grads and grad_avg hold the step's values.  The check
 * needs the momentum rule and a caller's stream that is not being captured (MTX_EUNSUPPORTED
 * otherwise); the fused and layer-wise updates are not used while it is on.  Returns MTX_EINVAL
 * for a NULL model. */
int mtx_set_nonfinite_check(mtx_model* m, int enable);

/* Fused average + update of large fully connected layers (execution option, default on).  With
 * the momentum rule (not Adam or AdaGrad) and without the layer-wise option, a fully connected
 * layer of at least 2^20 parameters whose weight gradient has at least 512 output tiles of
 * 128 x 128 and an unsplit reduction computes each output tile for all R shards in one block,
 * writes the R shard
 * rows as before, and averages and updates that tile's parameters (w, v, grad_avg) in the same
 * launch, as Sec. III-D.2 reduces and updates one layer at a time; the average + update at the
 * end of the step then covers only the other parameters.  Each element's arithmetic and order
 * are those of mtx_sgd_update (the R stored fp32 values added in ascending r, divided by R, then
 * the momentum rule), so the results are bit-identical either way.  enable = 0 switches it off.
 * Returns MTX_EINVAL for a NULL model. */
int mtx_set_fused_update(mtx_model* m, int enable);

/* Layer-wise average + update (execution option, default off; Sec. III-D.2 reduces the
 * gradients one layer at a time, in layer order).  With it on, mtx_train_step averages and
 * updates each layer's parameters (its W and b slice of w, v, grad_avg) on a third stream of the
 * model as soon as that layer's R shard gradients are written, beside the rest of the backward
 * pass, instead of once over all P parameters at the end; the step still returns after every
 * layer's update (the caller's stream waits for them).  Each element's arithmetic is the same,
 * so the results are bit-identical either way.  Measured on MI355X it was not faster: the
 * bandwidth-bound updates slowed the concurrent backward kernels by as much as they overlapped.
 * Ignored while kernel timing is on.  Returns MTX_EINVAL for a NULL model. */
int mtx_set_layerwise_update(mtx_model* m, int enable);

/* Update rule that mtx_train_step applies after the average of the R shard gradients.
 * MTX_OPT_MOMENTUM (the default): the momentum rule above, with the lr and momentum arguments
 * of each mtx_train_step.  MTX_OPT_ADAM and MTX_OPT_ADAGRAD: the rules of mtx_adam_update and
 * mtx_adagrad_update (the other update rules Sec. I names), with the lr argument of each step
 * and the momentum argument ignored:
 *   Adam: first moment in the model's v buffer, second moment in s2 (device, P floats, 16-byte
 *         aligned, owned by the caller, which zeroes it before the first step, as v = 0 after
 *         mtx_init_model); beta1, beta2 in [0, 1), eps >= 0; the step number t counts the
 *         mtx_train_step calls since this call (1 for the first).
 *   AdaGrad: accumulator in the model's v buffer (its content is the initial accumulator;
 *         mtx_set_params sets it); eps >= 0; beta1, beta2 and s2 unused.
 * mtx_get_params / mtx_set_params read and write v as that state.  A step with Adam is never
 * replayed from a graph (its bias correction changes every step).  Returns MTX_EINVAL for an
 * unknown kind, invalid hyperparameters, or an s2 that overlaps the model's buffers. */
typedef enum { MTX_OPT_MOMENTUM = 0, MTX_OPT_ADAM = 1, MTX_OPT_ADAGRAD = 2 } mtx_optimizer;
int mtx_set_optimizer(mtx_model* m, int kind, float beta1, float beta2, float eps, float* s2);

/* Kernel timing of mtx_train_step (measurement support; not part of the method).
 * mtx_set_timing(m, 1) makes every later mtx_train_step record a HIP event pair on its stream
 * around each kernel launch; mtx_set_timing(m, 0) stops it.  mtx_get_timing waits for the
 * recorded events and fills up to `capacity` entries, one per launch site of the step, in launch
 * order; *count receives the number of sites.  reset != 0 clears the accumulated times.
 * Launch-site names: "prep_w" (weight layouts), "prep_x" (input layout), "fwd", "pool_fwd",
 * "bn_fwd", "add_fwd", "softmax_xent" (with the loss mean), "wgrad" (weight and bias gradient),
 * "dgrad", "pool_bwd", "bn_bwd", "add_bwd", "skip_add", "avg_update" (a residual addition right
 * after a batch normalisation is computed in that layer's "bn_fwd_apply" and has no "add_fwd"
 * of its own; "add_bwd" runs only where the previous layer's gradient is not the addition's
 * own buffer; "skip_add" adds a shortcut's share into its source's gradient); "fwd_direct" and
 * "wgrad_direct" for a first convolution of one input channel and a 3x3, 5x5 or 7x7 window
 * (at most 32 outputs), which runs on direct kernels instead of the matrix kernels; the second
 * kernel of an operation is a site of its own: "<site>_reduce" (the second pass of a split
 * reduction), "dgrad_col2im", "bn_fwd_finalize" / "bn_bwd_finalize" (per-channel statistics
 * from the partial sums) and "bn_fwd_apply" / "bn_bwd_apply" (the elementwise pass after the
 * batch statistics).  Timing adds one event pair per kernel;
 * use it for measurement runs. */
typedef struct {
    char name[32];
    int layer;        /* layer index, or -1 for a kernel that is not tied to one layer */
    int launches;     /* number of timed launches */
    double total_ms;  /* sum of the launches' durations */
} mtx_kernel_time;

int mtx_set_timing(mtx_model* m, int enable);
int mtx_get_timing(mtx_model* m, mtx_kernel_time* out, int capacity, int* count, int reset);

/* Matrix-core launches of the last enqueued mtx_train_step (introspection for tests and
 * measurement; not part of the method).  One entry per launch of the tiled MFMA kernel, in
 * launch order: the launch site (as in mtx_get_timing: "fwd", "dgrad", "wgrad", "wgrad_update"),
 * the layer, the output tile (rows x columns of the GEMM C[p][q] = sum_k P[p][k] Q[q][k]), the
 * reduction tile, the number of reduction splits (> 1: a second kernel adds the fp32 partial
 * sums), and flags: 1 = interleaved scheduling order, 2 = an operand loaded straight into LDS,
 * 4 = the weight gradient fused with the average + update (mtx_set_fused_update).  Host only, does
 * not synchronise; fills up to `capacity` entries and sets *count to the number of launches. */
typedef struct {
    char site[32];
    int layer;
    int tile_rows, tile_cols, k_tile;
    int splits;
    int flags;
} mtx_launch_info;

int mtx_get_launches(const mtx_model* m, mtx_launch_info* out, int capacity, int* count);

/* Free the host handle (device buffers stay with the caller).  NULL is allowed. */
void mtx_free_model(mtx_model* m);

/* Message for the calling thread's last non-OK status ("" if none). */
const char* mtx_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MTX_H */
