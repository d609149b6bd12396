/*
 * gcpsl.h -- C ABI of the GCPSL hot path on one MI355X (gfx950).
 *
 * GCPSL (Kohankhaki, Rentschler, Schmeink, "Concurrent Split Learning Through
 * Stable Client Clustering") assigns K stable clients to C fixed clusters
 * (Alg. 1), runs one GPSL workload with batch B per cluster (Sec. IV-B,
 * Alg. 2) and periodically fuses the client and server segments of the
 * cluster replicas with sample-count weights (Eq. 5).  This library runs all
 * C cluster workloads side by side on one GPU: every kernel is batched over
 * the replica index.
 *
 * Conventions shared by every call:
 *   - Return value: GCPSL_OK (0) or a negative GCPSL_E* code.  On error,
 *     gcpsl_last_error() returns a thread-local message describing it.  No
 *     call aborts, throws or prints.
 *   - Device memory is owned by the caller.  The library never allocates
 *     device memory: it works in the caller's buffers and in one caller-owned
 *     workspace of gcpsl_workspace_bytes() bytes.  Device pointers passed to
 *     gcpsl_create must stay valid until gcpsl_destroy.
 *   - Device work is enqueued on the caller's HIP stream (hipStream_t passed
 *     as void*; NULL is the default stream) and returns without waiting.
 *     Argument and state errors are reported synchronously, before any work
 *     is enqueued.  A failed kernel launch returns GCPSL_EHIP.
 *   - A context is not thread-safe: calls on one context must not overlap.
 *
 * Layouts: activations are NHWC.  Parameters of one replica form one flat
 * fp32 vector of P entries: for every conv / linear layer in order, its weight
 * then its bias; conv weights are [cout][3][3][cin], linear weights
 * [cout][cin].  The client segment's parameters come first (P_client entries).
 */
#ifndef GCPSL_H
#define GCPSL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GCPSL_OK 0
#define GCPSL_EINVAL (-1)       /* bad argument: sizes, null pointers, rule   */
#define GCPSL_ESTATE (-2)       /* call out of order (e.g. step not sampled) */
#define GCPSL_EHIP (-3)         /* HIP runtime or launch error               */
#define GCPSL_EUNSUPPORTED (-4) /* valid request outside what is implemented */

/* Assignment rules of Alg. 1 (Sec. IV-A). */
#define GCPSL_RULE_RANDOM 0   /* permute, then round-robin                   */
#define GCPSL_RULE_SIZE 1     /* size-balanced: lightest allowed cluster     */
#define GCPSL_RULE_LABEL_L1 2 /* greedy label-histogram L1 placement         */
#define GCPSL_RULE_LABEL_JSD 3 /* Eq. 4 move search: size + JSD objective     */

/* Compute precisions. */
#define GCPSL_F32 0  /* fp32 activations and weights                        */
#define GCPSL_BF16 1 /* bf16 activations and weights, fp32 master weights   */

/* Round schedules (Sec. III-A, Sec. IV-D). */
#define GCPSL_SCHED_LOCKSTEP 0 /* every cluster takes one local round per step  */
#define GCPSL_SCHED_EPOCH 1    /* epoch barrier: a cluster takes floor(n_n/B)
                                  rounds per system epoch, then waits          */

/* Categories of the logical application payload (gcpsl_payload, Sec. V-E). */
#define GCPSL_PAYLOAD_ACTIVATIONS 0  /* cut activations and labels, client -> server */
#define GCPSL_PAYLOAD_CUT_GRADS 1    /* cut gradients, server -> client             */
#define GCPSL_PAYLOAD_CLIENT_GRADS 2 /* active clients' client-segment gradients    */
#define GCPSL_PAYLOAD_CLIENT_MODEL 3 /* averaged client segment to every replica    */
#define GCPSL_PAYLOAD_FUSION 4       /* fusion: states up, fused state down         */
#define GCPSL_PAYLOAD_COUNT 5

/* Layer kinds of the split CNN. */
#define GCPSL_CONV3X3 1 /* 3x3, stride 1, zero pad 1, bias, ReLU            */
#define GCPSL_MAXPOOL2 2 /* 2x2 max pool, stride 2                           */
#define GCPSL_AVGPOOL 3  /* global average pool                              */
#define GCPSL_LINEAR 4   /* fully connected layer producing the logits       */
#define GCPSL_BATCHNORM 5 /* batch norm of the conv before it, then ReLU     */
#define GCPSL_GROUPNORM 6 /* group norm of the conv before it, then ReLU     */
#define GCPSL_BLOCK 7     /* ResNet basic block (Sec. V-A), see below        */

/* Layer flags. */
#define GCPSL_RESIDUAL 1 /* conv output is ReLU(conv(x) + b + x); cin == cout */
#define GCPSL_STRIDE2 2  /* GCPSL_BLOCK: stride 2 (first conv, shortcut)     */

typedef struct gcpsl_layer {
  int32_t kind;   /* GCPSL_CONV3X3 ... GCPSL_BLOCK                        */
  int32_t cin;    /* input channels (conv, linear, norm, block); ignored for pools */
  int32_t cout;   /* output channels (conv, linear, block; norm: = cin)    */
  int32_t flags;  /* GCPSL_RESIDUAL (conv), GCPSL_STRIDE2 (block) or 0     */
  int32_t groups; /* GCPSL_GROUPNORM, GCPSL_BLOCK: groups (dividing the
                     channels; block: 0 = batch norm); else 0              */
} gcpsl_layer;

/*
 * Supported model shapes: layer 0 is a conv; every max pool follows a conv,
 * norm or block layer and sees an even H and W; the last two layers are
 * GCPSL_AVGPOOL then GCPSL_LINEAR (cout = L), optionally preceded by one max
 * pool; conv channel counts are either 3 (the image layer) or multiples of 8;
 * at most 48 weight-copy jobs (two per conv: 24 convs, a block counting its
 * two or three).  Other shapes return GCPSL_EUNSUPPORTED.
 *
 * GCPSL_BLOCK, the basic block of the paper's ResNet-18 (Sec. V-A): y =
 * ReLU(norm2(conv2(ReLU(norm1(conv1(x))))) + shortcut(x)), conv1 3x3 with
 * the block's stride (1, or 2 with GCPSL_STRIDE2; pad 1), conv2 3x3 stride 1,
 * shortcut = x when stride 1 and cin == cout, else norm(conv 1x1 with the
 * stride, no pad) (no ReLU on that norm); every norm is batch norm (groups
 * 0) or group norm with `groups` groups, applied as for GCPSL_BATCHNORM /
 * GCPSL_GROUPNORM below.  cin, cout multiples of 8; a block follows a conv
 * with ReLU, a norm or a block.  Its parameters, in the parameter vector:
 * conv1 weight [cout][3][3][cin] and bias, norm1 gamma and beta, conv2
 * weight [cout][3][3][cout] and bias, norm2 gamma and beta, then (with a
 * projection) the 1x1 weight [cout][1][1][cin] and bias, its norm's gamma
 * and beta.  With batch norm its running statistics (norm1, norm2, the
 * projection's) follow in norm_state in that order.
 *
 * Normalisation layers (Sec. IV-B: GroupNorm in the client segment,
 * BatchNorm in the server segment) follow a conv without GCPSL_RESIDUAL; that
 * conv then stores its raw output z and the norm layer applies
 * u = gamma_c (z - mean) / sqrt(var + 1e-5) + beta_c and ReLU, with mean and
 * biased var per channel over (batch, H, W) (batch norm) or per example over
 * (H, W, the channels of a group) (group norm).  gamma and beta are the
 * layer's weight and bias in the parameter vector (initial values 1 and 0).
 * Each round also updates the replica's batch-norm running statistics
 * (momentum 0.1: mean <- 0.9 mean + 0.1 batch mean, var <- 0.9 var + 0.1
 * unbiased batch variance; counter + 1) in norm_state.
 */
typedef struct gcpsl_desc {
  int32_t K;          /* clients (Sec. III-A), 1..65536                     */
  int32_t C;          /* clusters = concurrent replicas, 1..1024            */
  int32_t B;          /* examples per cluster batch (Eq. 3), >= 1           */
  int32_t L;          /* classes                                            */
  int32_t H, W, Cin;  /* image shape (NHWC)                                 */
  int32_t dtype;      /* GCPSL_F32 or GCPSL_BF16                            */
  int64_t n_examples; /* |D|                                                */
  int32_t n_layers;   /* entries of `layers`                                */
  int32_t cut;        /* client segment = layers[0, cut)                    */
  const gcpsl_layer *layers; /* host, copied at create                      */
  float lr;           /* SGD learning rate                                  */
  float momentum;     /* SGD momentum mu: v <- mu v + g, theta -= lr v      */
  float weight_decay; /* L2 term wd >= 0 (Sec. V-A): the update uses
                         g + wd theta in place of the gradient g           */
  int32_t nesterov;   /* 1: Nesterov term (Sec. V-A), theta -= lr (g + mu v)
                         with the new v; 0: theta -= lr v                   */
  float label_smoothing; /* eps in [0, 1) (Sec. V-A): the cross-entropy
                         target is (1 - eps) onehot(y) + eps / L            */
  uint64_t seed;      /* sampler seed                                       */
  int64_t max_steps;  /* rows of the participation table (steps recorded)   */
  int32_t max_window; /* largest nsteps accepted by gcpsl_sample, >= 1      */
  int32_t schedule;   /* GCPSL_SCHED_LOCKSTEP or GCPSL_SCHED_EPOCH          */
  const int32_t *client_of_example; /* host [n_examples], in [0, K)         */
  const int32_t *cluster_of_client; /* host [K], in [0, C) (Alg. 1 output)  */
  const float *images;   /* device [n_examples][H][W][Cin] fp32             */
  const int32_t *labels; /* device [n_examples], in [0, L)                  */
  float *theta;          /* device [C][P] fp32 masters, in/out              */
  float *momentum_buf;   /* device [C][P] fp32 momentum, in/out             */
  float *norm_state;     /* device [C][S] fp32 batch-norm running statistics
                            (per batch-norm layer in order: running mean[ch],
                            running variance[ch], counter), in/out; NULL if
                            the model has no batch norm (S = 0)             */
  void *workspace;       /* device, >= gcpsl_workspace_bytes(), 256-aligned */
  size_t workspace_bytes;
} gcpsl_desc;

typedef struct gcpsl_ctx gcpsl_ctx;

/* Parameter counts of one replica: P (total) and P_client (entries of the
 * client segment, which come first).  Host only.  EINVAL / EUNSUPPORTED on a
 * bad model description. */
int gcpsl_param_count(const gcpsl_desc *d, int64_t *P, int64_t *P_client);

/* Entries S of one replica's normalisation state (norm_state).  Host only. */
int gcpsl_state_count(const gcpsl_desc *d, int64_t *S);

/* Workspace size in bytes for this description.  Host only. */
int gcpsl_workspace_bytes(const gcpsl_desc *d, size_t *bytes);

/*
 * Static client clustering, Alg. 1 (Sec. IV-A).  Host only, no device work.
 *   rule RANDOM:   Fisher-Yates permutation of the clients (SplitMix64 stream
 *                  seeded with seed + 0x41535349474E, bounded draws by
 *                  Lemire's multiply-shift with rejection), then client
 *                  perm[i] -> cluster i mod C.  counts/hist may be NULL.
 *   rule SIZE:     clients in (count desc, id asc) order, each to the allowed
 *                  cluster (fewer than ceil(K/C) clients) with the smallest
 *                  summed count, ties to the lower index.  Needs counts.
 *   rule LABEL_L1: same order; each client with samples goes to the allowed
 *                  cluster whose label histogram after placement has the
 *                  smallest L1 distance between normalised histograms and
 *                  the global one (exact integer comparison), ties to the
 *                  smaller summed count, then the lower index; a client with
 *                  no samples goes to the allowed cluster with the fewest
 *                  clients.  Needs counts and hist.
 *   rule LABEL_JSD: the paper's label-aware rule (Eq. 4, Alg. 1): start from
 *                  the SIZE assignment, then repeatedly apply the single-client
 *                  move with the lowest J = sum_n |w_n - |D|/C| / |D| +
 *                  sum_n (w_n/|D|) JSD(p_n, p) (nats) while it lowers J, at
 *                  most 4K moves; a move keeps the source at >= floor(K/C) - s
 *                  and the destination at <= ceil(K/C) + s clients,
 *                  s = max(1, K/(4C)); first strict minimum in (client,
 *                  destination) order.  Needs counts and hist with at least
 *                  one sample.
 * counts: host [K] int64 sample counts; hist: host [K][L] int64 class
 * histograms (row k sums to counts[k]); cluster_of_client: host [K] output,
 * caller-owned.  EINVAL on K < 1, C < 1, C > K, unknown rule, missing
 * metadata or negative counts.
 */
int gcpsl_assign(int32_t K, int32_t C, int32_t rule, uint64_t seed, const int64_t *counts,
                 const int64_t *hist, int32_t L, int32_t *cluster_of_client);

/*
 * Create a context: validates the description, builds each cluster's example
 * list (ascending global id) and its fusion weight n_n = |D_{C_n}| (Eq. 5),
 * reads the labels back to count the data set's examples per class (the
 * global distribution of the batch deviation, Sec. V-E), and uploads these
 * into the workspace (synchronous copies).  Replicas are not
 * initialised here: the caller fills theta with C equal copies (Alg. 2,
 * "initialize all split-model replicas equally") and zeroes momentum_buf.
 * EINVAL if any cluster holds fewer than B examples, on null pointers,
 * out-of-range ids or labels or a too-small workspace; EUNSUPPORTED on an
 * unsupported model shape or L > 4096; EHIP on a failed copy.
 */
int gcpsl_create(const gcpsl_desc *d, gcpsl_ctx **out);

/*
 * gcpsl_create for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same context, whose workspace is a static device array of the library
 * (GCPSL_STATIC_WORKSPACE_BYTES per device, held from the library's load
 * until the process ends) instead of d->workspace, which is ignored (may be
 * NULL).  Allocates no device memory.  The caller still owns images, labels,
 * theta, momentum_buf and norm_state.  Every later call works on the
 * returned context as on any other.
 * One such context per device at a time: the array is shared by every call
 * on that device and keeps the previous context's contents (the tables that
 * must start at zero are cleared here), so a second one would race with the
 * first; it is refused with ESTATE until gcpsl_destroy releases the first.
 * EINVAL when gcpsl_workspace_bytes of the description exceeds
 * GCPSL_STATIC_WORKSPACE_BYTES; otherwise the errors of gcpsl_create.
 */
#define GCPSL_STATIC_WORKSPACE_BYTES (32u << 20)
int gcpsl_create_static(const gcpsl_desc *d, gcpsl_ctx **out);

/*
 * Steps.  A step is one slot of the round schedule.
 *   LOCKSTEP: at step s every cluster takes its local round s.
 *   EPOCH (the system epoch of Sec. III-A and Eq. 6 of Sec. IV-D): with
 *     r_n = floor(n_n / B) rounds of cluster n per epoch and R = max_n r_n
 *     slots per system epoch, step s = m R + t is slot t of system epoch m;
 *     cluster n takes its local round m r_n + t when t < r_n and otherwise
 *     waits at the fusion barrier: no batch, no update, no participating
 *     client.  The caller fuses (gcpsl_fuse) after slot R - 1 of each epoch.
 *
 * Cluster-local global sampling (Eq. 1, Eq. 3) for steps
 * [step, step + nsteps), with the gather of the sampled images and labels.
 * Cluster n draws its batch at local round s from its own pooled examples:
 * epoch e = s / S_n, S_n = floor(n_n / B), takes positions [tB, (t+1)B),
 * t = s mod S_n, of a keyed Feistel permutation of [0, n_n) (key from
 * seed, n, e); so every batch has exactly B distinct examples of the cluster.
 * Also records |A_{n,t}| (clients supplying >= 1 example, Sec. III-A; 0 for
 * a waiting cluster) for each sampled step below max_steps.
 * idx_out: device [nsteps][C][B] int32 global example ids (-1 for a waiting
 * cluster), or NULL.
 * The gathered inputs stay staged until the next gcpsl_sample call; each
 * staged step can then be run once or more by gcpsl_step.
 * EINVAL: step < 0, nsteps < 1 or > max_window.
 */
int gcpsl_sample(gcpsl_ctx *ctx, int64_t step, int32_t nsteps, int32_t *idx_out, void *stream);

/*
 * One local round of every cluster that takes one at this step (all clusters
 * under LOCKSTEP; Alg. 2 inner loop): client-segment
 * forward to the cut, server-segment forward, softmax cross-entropy (mean
 * over B), server backward, cut-gradient hand-off (same buffer on one GPU),
 * client backward, and the SGD update of both segments of every replica
 * (v <- mu v + g; theta <- theta - lr v).  The client gradient is that of
 * the batch-mean loss, which is the b_k/B-weighted average of the active
 * clients' gradients (Sec. III-B).
 * loss_out: device [C] fp32, the forward loss of each cluster before the
 * update, or NULL.  ESTATE if `step` is not among the staged steps.
 */
int gcpsl_step(gcpsl_ctx *ctx, int64_t step, float *loss_out, void *stream);

/*
 * The local round of one cluster only, exactly as gcpsl_step computes it for
 * that cluster (same kernels, same arithmetic, bit-identical results): the
 * clusters of a step may run one after another instead of side by side,
 * which is the sequential execution that Eq. 6 compares with the concurrent
 * one.  loss_out: device [C] (only entry `replica` is written) or NULL.
 * EINVAL if replica is outside [0, C) or the cluster waits at this step;
 * ESTATE if `step` is not staged.
 */
int gcpsl_step_replica(gcpsl_ctx *ctx, int64_t step, int32_t replica, float *loss_out, void *stream);

/*
 * Rounds of the epoch schedule: rounds host [C] receives r_n = floor(n_n / B)
 * and slots the system-epoch length R = max_n r_n (Eq. 6).  Host only; valid
 * under either schedule.
 */
int gcpsl_epoch_rounds(gcpsl_ctx *ctx, int64_t *rounds, int64_t *slots);

/*
 * Fusion and broadcast, Eq. 5 (Sec. IV-C): theta_bar = sum_n (n_n / W)
 * theta_n over both segments, accumulated in fp64 in cluster order, divided
 * once by W = sum_n n_n and rounded once to fp32, then written to every
 * replica.  The server normalisation state (norm_state) is fused the same way
 * (Sec. IV-B, IV-C).  Momentum is not touched (optimizer state stays local).
 */
int gcpsl_fuse(gcpsl_ctx *ctx, void *stream);

/*
 * The fusion of gcpsl_fuse in two halves (Eq. 5, Sec. IV-C), for a run whose
 * replicas are spread over several devices: every device reduces its own
 * replicas, the caller sums the devices' partials (e.g. an all-reduce), and
 * every device divides by the global W and broadcasts to its replicas.
 *   gcpsl_fuse_partial:  partial[p] = sum_n n_n theta_n[p] over this
 *     context's replicas, in fp64, in cluster order; entries [0, P) are the
 *     parameters, [P, P + S) the normalisation state (S = gcpsl_state_count).
 *   gcpsl_fuse_finalise: theta_n[p] = fp32(partial[p] / W) (one division, one
 *     rounding to nearest even) for every replica n, and the same for the
 *     normalisation state.  W is the sum of n_n over every replica of the run
 *     (on one device: the sum of gcpsl_cluster_sizes).
 * partial: device [P + S] fp64, 8-byte aligned, caller-owned (written by
 * partial, read by finalise).  On one device, partial then finalise with that
 * device's W gives gcpsl_fuse's result bit for bit.  Asynchronous on stream;
 * EINVAL on a null or misaligned partial or W outside [1, 2^53]; EHIP on a
 * failed launch.
 */
int gcpsl_fuse_partial(gcpsl_ctx *ctx, double *partial, void *stream);
int gcpsl_fuse_finalise(gcpsl_ctx *ctx, const double *partial, int64_t W, void *stream);

/*
 * The same sample-weighted fusion (Eq. 5, Sec. IV-C) on caller-owned
 * replicas, without a context: theta_bar[p] = (sum_n weights[n] theta[n][p])
 * / W, W = sum_n weights[n], accumulated in fp64 in replica order, rounded
 * once to fp32 and written to all C rows.
 * theta: device [C][P] fp32, row n = replica n, 4-byte aligned, in/out,
 * caller-owned; weights: host [C] int64 in [0, 2^29] with W > 0 (e.g. the
 * replicas' example counts n_n), read before the call returns; 1 <= C <= 64
 * (the weights travel in the kernel arguments); P >= 1.  Each product is
 * exact in fp64, and for identical replicas so is each partial sum (W <=
 * 2^29), so identical replicas come back unchanged.  Asynchronous on stream;
 * EINVAL on a bad argument, EHIP on a failed launch.  The form a benchmark
 * times at arbitrary sizes.
 */
int gcpsl_fuse_replicas(float *theta, int32_t C, int64_t P, const int64_t *weights, void *stream);

/*
 * Direct data participation (Sec. V-E): over the recorded horizon
 * [0, T_h), T_h = 1 + the largest step run by gcpsl_step (capped at
 * max_steps), active_slots = sum_t sum_n |A_{n,t}| and total_slots = K T_h;
 * participation = active / total.  per_step: host [T_h][C] int32 or NULL
 * (caller-owned, at least max_steps * C entries).  Synchronises the device.
 */
int gcpsl_participation(gcpsl_ctx *ctx, int64_t *active_slots, int64_t *total_slots,
                        int32_t *per_step);

/*
 * Batch deviation (Sec. V-E): the l1 distance sum_c |h_c / B - g_c / |D||
 * between a batch's class distribution (h_c of its B examples in class c)
 * and the data set's (g_c of |D|), recorded by gcpsl_sample for every batch,
 * as the exact integer numerator sum_c |h_c |D| - B g_c| over the common
 * denominator denom = B |D|.  Over the recorded horizon [0, T_h) (as for
 * gcpsl_participation): sum_num = the numerators summed over every batch
 * drawn, batches = their number (waiting clusters draw none), so the mean
 * deviation is sum_num / (batches denom).  per_step: host [T_h][C] int64
 * numerators, -1 where a cluster drew no batch, or NULL (caller-owned, at
 * least max_steps * C entries).  Synchronises the device.
 */
int gcpsl_batch_deviation(gcpsl_ctx *ctx, int64_t *sum_num, int64_t *batches, int64_t *denom,
                          int64_t *per_step);

/*
 * Logical application payload (Sec. V-E): bytes of the tensors handed between
 * application endpoints over the recorded horizon [0, T_h) and the fusions
 * so far, by category (bytes: host [GCPSL_PAYLOAD_COUNT] int64, caller-owned):
 *   ACTIVATIONS  per local round, B cut activations (the client segment's
 *                output, in the compute precision) and B int32 labels;
 *   CUT_GRADS    per local round, B cut gradients (same size);
 *   CLIENT_GRADS per local round, |A_{n,t}| client-segment gradients
 *                (P_client fp32 entries each, Sec. III-B averaging);
 *   CLIENT_MODEL per local round, the averaged client segment to each of
 *                the cluster's |C_n| client replicas (P_client fp32 each);
 *   FUSION       per fusion, every replica's P + S fp32 entries up and the
 *                fused state down (gcpsl_fuse_partial counts the first half,
 *                gcpsl_fuse_finalise the second).
 * A cluster waiting at the epoch barrier adds nothing.  Synchronises.
 */
int gcpsl_payload(gcpsl_ctx *ctx, int64_t *bytes);

/* Host copy of the per-cluster example counts n_n: sizes host [C] int64. */
int gcpsl_cluster_sizes(gcpsl_ctx *ctx, int64_t *sizes);

/*
 * Device view of a named workspace tensor, for inspection by tests.  Names:
 * "x" (staged inputs [max_window][C][B][H][W][Cx]; Cx = Cin when Cin is a
 * multiple of 8 (bf16) / 4 (fp32), otherwise the image layer's im2col rows:
 * Cx = 9 Cin rounded up to that multiple, column (r, s, c) = pixel
 * (h + r - 1, w + s - 1) channel c, zero outside the image and in the padding),
 * "idx", "y"
 * ([max_window][C][B] int32), "hits" ([max_steps][C] int32, |A_{n,t}| of
 * every sampled step), "act<i>" (output of layer i, [C][B][...]),
 * "gpre<i>" (gradient w.r.t. conv layer i's pre-activation), "gin<i>"
 * (gradient w.r.t. the input of conv layer i when layer i-1 is a max pool),
 * "route<j>" (routing codes of max-pool layer j, [C][B][H/2][W/2][channels]
 * uint8: the row-major window position 0..3 of the first maximum, 4 where
 * the maximum is not positive and no gradient passes), "dh" ([C][B][channels]
 * fp32 gradient of the pooled feature), "grad" ([C][P] fp32 last gradient).
 * A bf16 conv whose ReLU output feeds a stored 2 x 2 max pool and then
 * another conv (the 32 x 32, 32 -> 64 image-side layer) keeps only the pool's
 * output and "route<j>": its "act<i>" and "gpre<i>" are not stored (its
 * gradient is "gin<j+1>" routed through the codes).  A bf16 head conv whose
 * max pool and mean are fused into it keeps "route<j>" of that pool and its
 * "gpre<i>", not its "act<i>".  dtype receives
 * GCPSL_F32, GCPSL_BF16, -1 for int32 or -2 for uint8.  EINVAL on an unknown
 * or unstored name.
 */
int gcpsl_tensor(gcpsl_ctx *ctx, const char *name, void **ptr, int64_t *numel, int32_t *dtype);

/*
 * Per-kernel timing, for measurement.  gcpsl_timing(ctx, 1) makes every later
 * kernel launch of this context record a hipEvent before and after it on the
 * caller's stream (the stream the kernel runs on); 0 turns it off (default).
 * gcpsl_timing_read synchronises the device, aggregates the recorded launches
 * by kernel instantiation and clears the record.  Each entry holds the summed
 * event time and the summed algorithmic work of its launches: FLOPs of the
 * contraction (2 M N K for a conv pass) and the minimum HBM bytes the launch
 * must move (each operand read once, each result written once).  out: host
 * array of cap entries (caller-owned); n receives the number of distinct
 * kernels (entries beyond cap are dropped).
 */
typedef struct gcpsl_kernel_stat {
  char name[64];    /* kernel instantiation, e.g. "conv_fwd<bf16,128x128,vec>" */
  int64_t launches; /* launches aggregated                                    */
  double ms;        /* summed event time in milliseconds                      */
  double flops;     /* summed algorithmic FLOPs                               */
  double bytes;     /* summed algorithmic HBM bytes                           */
} gcpsl_kernel_stat;

int gcpsl_timing(gcpsl_ctx *ctx, int32_t on);
int gcpsl_timing_read(gcpsl_ctx *ctx, gcpsl_kernel_stat *out, int32_t cap, int32_t *n);

/* Release the context (host metadata only; device memory is the caller's;
 * a context of gcpsl_create_static releases its device's static workspace). */
void gcpsl_destroy(gcpsl_ctx *ctx);

/* Thread-local description of the last error, "" if none. */
const char *gcpsl_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GCPSL_H */
