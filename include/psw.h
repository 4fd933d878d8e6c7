/*
 * psw.h -- C ABI of libpsw: pipelined CNN training with stale weights on
 * AMD Instinct MI355X (gfx950).
 *
 * Method: Zhang & Abdelrahman, "Pipelined Training with Stale Weights of
 * Deep Convolutional Neural Networks" (arXiv 1912.12675).  Sec. 2 states
 * layered backpropagation (x^(l) from x^(l-1) and W^(l); delta^(l-1) from
 * delta^(l); dE/dW^(l) from x^(l-1) and delta^(l); update after all
 * gradients).  Sec. 3 inserts pipeline register pairs after layers p_1..p_K
 * (the Pipeline Placement Vector) so that forward stage FS_i computes with
 * weights that are several updates old ("degree of staleness").  Sec. 4
 * switches from pipelined to non-pipelined training after n_p iterations.
 * App. A/B fix SGD with momentum 0.9 and a per-stage learning rate (Table 7).
 *
 * Conventions shared by every entry point
 *  - Every pointer argument is a DEVICE pointer unless its comment says
 *    "host".  The caller owns all device memory; the library never
 *    allocates device memory.
 *  - Activations are float32 NCHW (the only layout); conv weights are
 *    KCRS [K_out][C_in][R][S]; FC weights are [out][in]; all contiguous.
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).
 *    Every call only enqueues work on that stream; nothing synchronises the
 *    host.  Faults inside kernels surface at the caller's next sync.
 *  - `prec`: PSW_FP32, or PSW_BF16 = both operands of every conv/FC product
 *    rounded to bfloat16 (round to nearest even) with fp32 accumulation;
 *    all other arithmetic and all storage stay fp32.
 *  - Return value: PSW_OK (0) or a negative PSW_ERR_* code.  Nothing is
 *    enqueued when argument validation fails.  psw_last_error() returns a
 *    thread-local description of the last failure on the calling thread.
 *  - Workspaces: entry points that need scratch device memory take
 *    (ws, ws_bytes) and report the size they need through a *_ws_bytes
 *    query; a too-small workspace is PSW_ERR_WORKSPACE.
 */
#ifndef PSW_H
#define PSW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    PSW_OK = 0,
    PSW_ERR_NULL = -1,        /* a required pointer is NULL */
    PSW_ERR_SHAPE = -2,       /* inconsistent or out-of-range sizes */
    PSW_ERR_UNSUPPORTED = -3, /* valid request the library does not implement */
    PSW_ERR_STALENESS = -4,   /* staleness < 0 or >= ring depth */
    PSW_ERR_STEP_ORDER = -5,  /* stage_step t is not the expected next step */
    PSW_ERR_WORKSPACE = -6,   /* workspace / arena too small */
    PSW_ERR_HIP = -7,         /* the HIP runtime reported an error */
    PSW_ERR_STATE = -8        /* object not ready (e.g. net not bound) */
};

enum { PSW_FP32 = 0, PSW_BF16 = 1 };

/* Thread-local message of the last failing call on this thread ("" if none). */
const char *psw_last_error(void);
/* Library version string. */
const char *psw_version(void);

/* ------------------------------------------------------------------------ */
/* Per-layer operations (Sec. 2, layered backpropagation).                  */
/* ------------------------------------------------------------------------ */

/* Convolution forward (Sec. 2: x^(l) from x^(l-1) and W^(l)):
 *   y[n,k,p,q] = bias[k] + sum_{c,r,s} w[k,c,r,s] x[n,c,p*stride+r-pad,q*stride+s-pad]
 *   followed by max(0,.) when relu != 0.  Zero padding.
 * x: [n,c,h,w]; w: [k,c,r,s]; bias: [k] or NULL; y: [n,k,p,q] with
 * p = (h+2pad-r)/stride+1, q likewise.  y must not overlap x. */
int psw_conv_fwd(int n, int c, int h, int w, int k, int r, int s, int stride, int pad,
                 const float *x, const float *wt, const float *bias, int relu, float *y, int prec,
                 void *stream);

/* Convolution backward-data (Sec. 2: delta^(l-1) from delta^(l) and W):
 * the adjoint of the forward map (without bias/ReLU; mask dy first with
 * psw_relu_mask when the forward applied ReLU).
 *   dx[n,c,ih,iw] (+)= sum over (k,r,s,p,q) with ih=p*stride+r-pad, iw=q*stride+s-pad
 *                      of dy[n,k,p,q] w[k,c,r,s]
 * Overwrites dx when accumulate == 0, adds into it otherwise. */
int psw_conv_bwd_data(int n, int c, int h, int w, int k, int r, int s, int stride, int pad,
                      const float *wt, const float *dy, float *dx, int accumulate, int prec,
                      void *stream);

/* Workspace bytes psw_conv_bwd_weight needs for this shape and precision. */
size_t psw_conv_bwd_weight_ws_bytes(int n, int c, int h, int w, int k, int r, int s, int stride,
                                    int pad, int prec);

/* Convolution backward-weight (Sec. 2: dE/dW^(l) from x^(l-1) and delta^(l)):
 *   dw[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] x[n,c,p*stride+r-pad,q*stride+s-pad]
 *   dbias[k]    = sum_{n,p,q} dy[n,k,p,q]        (skipped when dbias == NULL)
 * Overwrites dw / dbias.  The reduction over n*p*q is split across
 * workgroups and the partial sums are added in a fixed order, so the result
 * is bit-reproducible. */
int psw_conv_bwd_weight(int n, int c, int h, int w, int k, int r, int s, int stride, int pad,
                        const float *x, const float *dy, float *dw, float *dbias, int prec, void *ws,
                        size_t ws_bytes, void *stream);

/* Allocation-free psw_conv_bwd_weight, for callers that cannot allocate
 * device memory or pass a workspace (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc).  Same arguments and
 * results (bit for bit) without (ws, ws_bytes): the split partial sums live
 * in a static device array of PSW_NOALLOC_SCRATCH_BYTES that the library
 * holds on every GPU it runs on until the process ends; its address is
 * resolved on the first call on each device (the calling thread's current
 * device, to which `stream` must belong).  No call allocates or frees
 * device memory.  A shape whose workspace (psw_conv_bwd_weight_ws_bytes)
 * exceeds the array is rejected with PSW_ERR_WORKSPACE, nothing enqueued.
 * All calls on one GPU share the array and every call overwrites it before
 * reading it: calls that can overlap on one GPU (on different streams, or
 * from different threads) race and must be ordered by the caller. */
#define PSW_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int psw_conv_bwd_weight_noalloc(int n, int c, int h, int w, int k, int r, int s, int stride, int pad,
                                const float *x, const float *dy, float *dw, float *dbias, int prec,
                                void *stream);

/* Workspace bytes of the batch-norm entry points for [n,c,h,w]. */
size_t psw_bn_ws_bytes(int n, int c, int h, int w);

/* Batch norm in training mode, optional residual add, optional ReLU (the
 * normalisation the paper's VGG and ResNet training uses, App. A/B):
 *   mean_c, var_c over n*h*w (biased);  xhat = (y-mean)/sqrt(var+eps)
 *   z = gamma*xhat + beta [+ sc(res)];  z = max(z,0) if relu
 * sc(res): identity when res is [n,c,h,w]; otherwise the CIFAR-ResNet
 * "option A" shortcut: res [n,rc,rh,rw] with rh = h*k, rw = w*k, rc <= c,
 * subsampled at even positions and zero-padded by (c-rc)/2 channels on each
 * side.  res may be NULL (rc, rh, rw ignored).
 * save_mean / save_invstd [c] receive the batch statistics for the
 * backward pass.  run_mean / run_var [c] (both NULL or both set) are
 * updated as r = (1-momentum) r + momentum * stat, unbiased variance. */
int psw_bn_relu_fwd(int n, int c, int h, int w, const float *y, const float *gamma,
                    const float *beta, const float *res, int rc, int rh, int rw, int relu, float eps,
                    float momentum, float *z, float *save_mean, float *save_invstd, float *run_mean,
                    float *run_var, void *ws, size_t ws_bytes, void *stream);

/* Backward of psw_bn_relu_fwd.  g = dz * [z > 0] (relu) or dz;
 *   dbeta = sum g;  dgamma = sum g*xhat;
 *   dy = gamma*invstd*(g - dbeta/M - xhat*dgamma/M)   (overwrites dy)
 *   dres (+)= sc^T(g)  (when dres != NULL; accumulate per res_accumulate)
 * gamma is whichever version the caller passes: the stale-weight schedule
 * passes the current weights (the backward stage reads the single, already
 * updated copy, Sec. 3).  y is the BN input saved by the forward pass. */
int psw_bn_relu_bwd(int n, int c, int h, int w, const float *dz, const float *z, const float *y,
                    const float *gamma, const float *save_mean, const float *save_invstd, int relu,
                    float *dy, float *dgamma, float *dbeta, float *dres, int rc, int rh, int rw,
                    int res_accumulate, void *ws, size_t ws_bytes, void *stream);

enum { PSW_POOL_MAX = 0, PSW_POOL_GAVG = 1 };

/* Pooling forward.  PSW_POOL_MAX: k x k window, step `stride`, no padding,
 * floor mode; argmax [n,c,p,q] receives the flat in-plane index (ih*w+iw)
 * of the first maximum in row-major window order.  Only non-overlapping
 * windows (k == stride) are supported.  PSW_POOL_GAVG: global average,
 * y [n,c] (k, stride, argmax ignored). */
int psw_pool_fwd(int kind, int n, int c, int h, int w, int k, int stride, const float *x, float *y,
                 int32_t *argmax, void *stream);

/* Pooling backward: MAX routes dy to the saved argmax; GAVG spreads dy/(h*w)
 * over the plane.  dx [n,c,h,w] overwritten (accumulate == 0) or added to. */
int psw_pool_bwd(int kind, int n, int c, int h, int w, int k, int stride, const float *dy,
                 const int32_t *argmax, float *dx, int accumulate, void *stream);

/* Fully connected forward: y[n,o] = b[o] + sum_i x[n,i] w[o,i], then
 * max(0,.) if relu.  x [n,in], w [out,in], b [out] or NULL, y [n,out]. */
int psw_fc_fwd(int n, int in, int out, const float *x, const float *wt, const float *b, int relu,
               float *y, int prec, void *stream);

size_t psw_fc_bwd_ws_bytes(int n, int in, int out);

/* Fully connected backward (dy already masked for a ReLU output):
 *   dx[n,i] (+)= sum_o dy[n,o] w[o,i]   (dx may be NULL)
 *   dw[o,i]  = sum_n dy[n,o] x[n,i];  db[o] = sum_n dy[n,o] (db may be NULL) */
int psw_fc_bwd(int n, int in, int out, const float *x, const float *wt, const float *dy, float *dx,
               int dx_accumulate, float *dw, float *db, int prec, void *ws, size_t ws_bytes,
               void *stream);

/* ReLU backward in place: g[i] = 0 where z[i] <= 0 (z = the ReLU output). */
int psw_relu_mask(int64_t count, const float *z, float *g, void *stream);

/* Softmax cross-entropy, mean over the mini-batch (the training error e of
 * Sec. 2):  loss = (1/n) sum_i [logsumexp(logits_i) - logits_i[label_i]],
 * dlogits = (softmax - onehot)/n.  loss: one device float.  labels [n] in
 * [0, classes) (not checked on the device). */
int psw_softmax_xent(int n, int classes, const float *logits, const int32_t *labels, float *loss,
                     float *dlogits, void *stream);

/* SGD with momentum (App. A/B):  d = g + wd*w_in;  v = mom*v + d;
 *   w_out = w_in - lr*(nesterov ? d + mom*v : v).
 * w_out may equal w_in (in-place); otherwise the ranges must not overlap. */
int psw_sgd_momentum_step(int64_t count, const float *w_in, float *w_out, float *v, const float *g,
                          float lr, float mom, float wd, int nesterov, void *stream);

/* Dropout (App. A: VGG-16 trains with dropout), inverted:
 *   out[j] (+)= keep(j) ? in[j] * 2^24 / (2^24 - p24) : 0
 * over count floats (accumulate != 0 adds to out).  The mask is a function of
 * (seed, op, t, j) only: element j is kept iff the top 24 bits of word j % 4
 * of Philox4x32-10 (Salmon et al., SC 2011) with counter (j / 4, op,
 * t mod 2^32, t / 2^32) and key (seed mod 2^32, seed / 2^32) are >= p24, so
 * drop probability = p24 / 2^24 (0 < p24 < 2^24) and the backward pass of a
 * mini-batch is the same call on the gradients with the same (seed, op, t).
 * count / 4 must fit in 32 bits; t >= 0.  in and out may be the same array
 * when accumulate == 0. */
int psw_dropout(int64_t count, const float *in, float *out, int accumulate, int p24, uint64_t seed,
                int32_t op, int64_t t, void *stream);

/* ------------------------------------------------------------------------ */
/* Networks and the stale-weight stage scheduler (Sec. 3, Sec. 4).          */
/* ------------------------------------------------------------------------ */

/* One operation of a network; tensor 0 is the mini-batch, operation i
 * writes tensor i+1.  kind: PSW_OP_*.  in0: input tensor id; in1: residual
 * tensor id of a batch norm (-1 none).  cin/cout: channels (features for
 * FC); k, stride, pad: conv / max-pool geometry; for PSW_OP_DROPOUT k is the
 * drop threshold p24 of psw_dropout, and the mask of step t is that of
 * psw_dropout with op = the operation's index and the net's dropout seed
 * (psw_net_set_dropout_seed).  flags: PSW_F_BIAS, PSW_F_RELU.  Parameters of a stage are packed, in operation order, as
 * conv (weight, bias), bn (gamma, beta), fc (weight, bias). */
typedef struct {
    int32_t kind, in0, in1, cin, cout, k, stride, pad, flags;
} psw_layer;

enum { PSW_OP_CONV = 1, PSW_OP_BN = 2, PSW_OP_MAXPOOL = 3, PSW_OP_GAVG = 4, PSW_OP_FC = 5, PSW_OP_DROPOUT = 6 };
enum { PSW_F_BIAS = 1, PSW_F_RELU = 2 };

typedef struct psw_net psw_net;

/* Build a network plan (host only; no device work, no HIP call).
 * layers[n_layers]; the input batch is [batch, c0, h0, w0]; the last
 * operation produces the logits.  stage_end[n_stages]: one past the last
 * operation of each stage (the PPV of Sec. 3 expressed in operations;
 * stage_end[n_stages-1] == n_layers).  ring_depth[s] >= 1: number of weight
 * versions stage s keeps resident (max staleness it will be asked for + 1).
 * *out receives the new object (free with psw_net_destroy). */
int psw_net_create(const psw_layer *layers, int n_layers, int batch, int c0, int h0, int w0,
                   const int32_t *stage_end, int n_stages, const int32_t *ring_depth, int prec,
                   psw_net **out);

void psw_net_destroy(psw_net *net);

/* Sizes the caller must allocate before psw_net_bind (host outputs):
 * stage_params[s] = parameters of stage s; ring_floats = sum_s
 * ring_depth[s]*stage_params[s]; n_params = sum_s stage_params[s];
 * bn_channels = running-statistic entries (sum of BN channels);
 * arena_bytes = activations, gradients and workspaces of one step. */
int psw_net_sizes(const psw_net *net, int64_t *stage_params, int64_t *ring_floats,
                  int64_t *n_params, int64_t *bn_channels, int64_t *arena_bytes);

/* Attach device memory.  ring [ring_floats]: stage-major, then version slot,
 * then that stage's packed parameters; the caller writes W^(0) into slot 0
 * of every stage (see psw_net_slot) before step 0.  momentum, grad
 * [n_params] (stage-major; momentum must start at zero).  run_mean,
 * run_var [bn_channels] (may be NULL).  arena [arena_bytes] (>= 256-byte
 * aligned). */
int psw_net_bind(psw_net *net, float *ring, float *momentum, float *grad, float *run_mean,
                 float *run_var, void *arena, size_t arena_bytes);

/* One training step of mini-batch t under the stale-weight schedule.
 * For every stage s, with d_s = staleness[s] (host array, 0 <= d_s <
 * ring_depth[s]):
 *   the forward pass reads weight version r_s = max(0, t - d_s) (Sec. 3:
 *     FS_i computes with weights several updates old; pipeline fill clamps
 *     at version 0),
 *   the backward pass computes weight gradients from the activations that
 *     forward pass saved and data gradients with the current version t
 *     (one weight copy per partition, no stashing),
 *   the update writes version t+1 = SGD(version t, grad) with rate lr[s]
 *     (host array; per-stage rates as in Table 7).
 * All stages d_s = 0 is plain mini-batch SGD (Sec. 2); switching every
 * d_s to 0 at t = n_p is the hybrid schedule of Sec. 4.
 * t must equal the previous call's t + 1 (0 for the first call, or the value
 * set by psw_net_set_step), else PSW_ERR_STEP_ORDER.
 * x [batch,c0,h0,w0] and labels [batch] are device buffers; loss_out is one
 * device float; versions_out (host, [n_stages], may be NULL) receives r_s.
 * Streams: the forward pass and the data-gradient chain run on `stream`;
 * the weight gradients and each stage's update (issued as soon as the
 * backward pass is done with that stage) run on a stream of the library,
 * joined back into `stream` before the call returns, so all work of the
 * step is ordered before whatever the caller enqueues next on `stream`. */
int psw_stage_step(psw_net *net, int64_t t, const int32_t *staleness, const float *lr, float mom,
                   float wd, int nesterov, const float *x, const int32_t *labels, float *loss_out,
                   int32_t *versions_out, void *stream);

/* Pipelined execution of steps t0 .. t0+n_steps-1 (Sec. 3 mapped onto one
 * GPU): the result is exactly that of n_steps psw_stage_step calls with
 * the same arguments (same kernels, same order within every dependency),
 * but the forward pass of mini-batch t+1 runs on a library stream
 * concurrently with the backward pass of mini-batch t wherever the
 * stale-weight schedule allows it: stage s's forward pass of step t only
 * waits for the update that wrote its version t - d_s, so with d_s >= 1 it
 * overlaps the backward pass of step t-1 (with every d_s = 0 nothing
 * overlaps, as in plain SGD).  The step sets (activations, saved
 * statistics, gradients) rotate between the net's arena and one or two more
 * sets bound with psw_net_bind_pipeline: psw_net_pipeline_bytes gives the
 * size of one set; `bytes` covering two sets gives three step sets, so the
 * forward pass of step t waits for the weight stream to finish step t-3
 * instead of t-2.
 * staleness and lr: host arrays [n_steps][n_stages].  x: device array of
 * n_batches mini-batches [n_batches][batch,c0,h0,w0]; step t0+i uses batch
 * i mod n_batches (labels likewise [n_batches][batch]); every batch must
 * stay unchanged until the call's work on `stream` is complete.  losses:
 * device [n_steps].  versions_out: host [n_steps][n_stages] or NULL.  All
 * work is joined into `stream` before the call returns. */
int psw_net_pipeline_bytes(const psw_net *net, int64_t *bytes);
int psw_net_bind_pipeline(psw_net *net, void *step_set, size_t bytes);
int psw_pipeline_run(psw_net *net, int64_t t0, int n_steps, const int32_t *staleness, const float *lr,
                     float mom, float wd, int nesterov, const float *x, const int32_t *labels,
                     int n_batches, float *losses, int32_t *versions_out, void *stream);

/* The same pipelined steps captured once into a HIP graph and replayed:
 * psw_pipeline_capture records (does not run) n_steps steps from the net's
 * next step t0 with psw_pipeline_run's arguments; every psw_graph_launch
 * then runs the next n_steps steps on `stream` (net at step t0 + k*n_steps
 * or any step congruent to t0 modulo the period; else PSW_ERR_STEP_ORDER),
 * with the captured staleness, lr, batches (relative to the launch) and
 * losses buffer.  n_steps must be a multiple of the period
 * lcm(ring_depth[s], number of step sets) after which ring slots and step
 * sets repeat, and no captured step may clamp its version at 0 (run the
 * pipeline fill eagerly).  Nets with dropout are rejected
 * (PSW_ERR_UNSUPPORTED): their masks depend on the step, which a replay
 * would not advance.
 * The captured pointers must stay valid until psw_graph_destroy.  Graph
 * launches skip the host-side cost of issuing ~10^2 kernels and events per
 * step, which otherwise bounds small networks. */
typedef struct psw_graph psw_graph;
int psw_pipeline_capture(psw_net *net, int n_steps, const int32_t *staleness, const float *lr, float mom,
                         float wd, int nesterov, const float *x, const int32_t *labels, int n_batches,
                         float *losses, psw_graph **out);
int psw_graph_launch(psw_graph *g, void *stream);
int psw_graph_destroy(psw_graph *g);

/* Set the next expected step (resume from a checkpoint whose ring holds
 * versions t-ring_depth+1 .. t in their slots v mod ring_depth). */
int psw_net_set_step(psw_net *net, int64_t t);

/* Device pointer (through *params) of stage `stage`'s weight version
 * `version`, which must be resident: next_t - ring_depth < version <= next_t
 * (any version <= next_t while next_t < ring_depth).  Slot = version mod
 * ring_depth. */
int psw_net_slot(const psw_net *net, int stage, int64_t version, float **params);

/* Read-back of the step set psw_stage_step uses (for tests and inspection):
 * *ptr receives the device address of tensor `tensor` (1..n_layers; tensor
 * i+1 is operation i's output) and *count (may be NULL) its element count.
 * grad == 0: the value the last psw_stage_step's forward pass computed;
 * grad != 0: the gradient of the loss with respect to that tensor from its
 * backward pass (for a conv or FC with ReLU, with respect to the output
 * after the ReLU, masked by it).  The contents are those of the last
 * psw_stage_step until the next step of the net is issued; a pipelined run
 * may use other step sets.  PSW_ERR_SHAPE for tensor 0 (the caller's batch)
 * or out of range, PSW_ERR_STATE before psw_net_bind. */
int psw_net_tensor(const psw_net *net, int tensor, int grad, float **ptr, int64_t *count);

/* Whether the forward value of tensor `tensor` is stored (host output
 * *stored = 1) or not (0): the output of a BN + ReLU without residual that
 * only one conv reads (the batch-norm and ReLU of Sec. 6's CNNs, before the
 * second conv of a residual block, or between two convs of VGG) is never
 * written while psw_net_set_bn_on_load is on; that conv forms
 * max(y * scale + shift, 0) itself, in one fused multiply-add, from the BN's
 * input y and the step's saved scale and shift (psw_net_bn_saved), in its
 * forward pass and in its weight gradient.  The gradient of every tensor is
 * stored.  Host only, valid from psw_net_create on; PSW_ERR_SHAPE for tensor
 * 0 or out of range. */
int psw_net_tensor_stored(const psw_net *net, int tensor, int *stored);

/* Device pointers of BN operation `op`'s saved statistics of the last
 * psw_stage_step (read-back like psw_net_tensor): mean [c], 1/sqrt(var+eps)
 * [c] and scale_shift [2c] (gamma * invstd, then beta - mean * scale: the
 * affine map of the forward pass, both as float).  PSW_ERR_SHAPE unless op
 * is a BN, PSW_ERR_STATE before psw_net_bind. */
int psw_net_bn_saved(const psw_net *net, int op, float **mean, float **invstd, float **scale_shift);

/* on != 0 (the default): BNs whose output only one conv reads are applied
 * by that conv while loading (psw_net_tensor_stored); on == 0: every BN
 * output is stored by its own apply kernel.  Both give the same results bit
 * for bit.  Takes effect from the next psw_stage_step / psw_pipeline_run /
 * psw_pipeline_capture call; PSW_ERR_NULL for a NULL net. */
int psw_net_set_bn_on_load(psw_net *net, int on);

/* Offset (in floats, inside the packed parameters of the op's stage) and
 * count of operation `op`'s parameters (host outputs). */
int psw_net_param_offset(const psw_net *net, int op, int *stage, int64_t *offset, int64_t *count);

/* Comparison scheme (Sec. 6.7, Sec. 7): with on != 0, every later step's
 * backward pass takes its data gradients (conv and FC transposes, BN's
 * gamma) with the version its forward pass read, r_s = max(0, t - d_s), as
 * weight stashing does, instead of the current version t (the paper's
 * scheme, the default).  Weight gradients and the update are unchanged.
 * The ring already holds version r_s (d_s < ring_depth[s]), so this needs no
 * memory; a multi-device pipeline that stashes keeps d_s extra copies of
 * stage s's weights.  Takes effect from the next psw_stage_step /
 * psw_pipeline_run / psw_pipeline_capture call; PSW_ERR_NULL for a NULL
 * net. */
int psw_net_set_weight_stashing(psw_net *net, int on);

/* Key of the net's dropout masks (default 0); takes effect from the next
 * step.  PSW_ERR_NULL for a NULL net. */
int psw_net_set_dropout_seed(psw_net *net, uint64_t seed);

/* Dry run of psw_stage_step (host only, no device work): the kernel-level
 * plan of step t.  Each record is (op, what, stage, version) where `what`
 * is a PSW_PLAN_* code, `version` the weight version it reads (-1 if
 * none).  A BN whose backward pass has no kernel of its own (it is folded
 * into the backward-data kernels of the convs around it: the next conv's
 * forms its sums, the previous conv's applies it while staging its input)
 * is recorded as PSW_PLAN_BN_BWD_FOLDED instead of PSW_PLAN_BN_BWD.
 * Writes up to cap records; *n_out receives the total count.  Validates
 * exactly as psw_stage_step does (step order excepted). */
typedef struct {
    int32_t op, what, stage;
    int64_t version;
} psw_launch;

enum {
    PSW_PLAN_CONV_FWD = 1, PSW_PLAN_BN_FWD, PSW_PLAN_POOL_FWD, PSW_PLAN_FC_FWD, PSW_PLAN_LOSS,
    PSW_PLAN_RELU_MASK, PSW_PLAN_CONV_BWD_WEIGHT, PSW_PLAN_CONV_BWD_DATA, PSW_PLAN_BN_BWD,
    PSW_PLAN_POOL_BWD, PSW_PLAN_FC_BWD, PSW_PLAN_SGD, PSW_PLAN_DROPOUT_FWD, PSW_PLAN_DROPOUT_BWD,
    PSW_PLAN_BN_BWD_FOLDED
};

int psw_net_plan(const psw_net *net, int64_t t, const int32_t *staleness, psw_launch *out, int cap,
                 int *n_out);

/* Per-kernel timing of psw_stage_step and psw_pipeline_run (for
 * measurement; off by default).  With profiling on, every kernel the
 * library launches there is launched with a start / stop event pair that the
 * runtime stamps from the kernel's own dispatch (hipExtLaunchKernelGGL), and
 * tagged with the kind of launcher that issued it, the kernel's name
 * (template arguments as the compiler spells them, so the name matches a
 * kernel trace) and its algorithmic work.
 * psw_net_profile(net, enable) switches profiling and clears the records;
 * the records are kept until the next psw_net_profile call.
 * psw_net_profile_only does the same but records only the launches of the
 * kernel with exactly the given name (NULL or "" = every kernel), so that
 * one kernel can be timed inside a throughput run at the cost of two events
 * per launch of it.  Events are created on first use and kept until
 * psw_net_destroy.
 * psw_net_profile_read waits for the recorded events and writes the summed
 * milliseconds and kernel launch counts per PSW_PROF_* kind into the host
 * arrays ms[n_kinds] and launches[n_kinds].
 * psw_net_profile_kernels writes one psw_kernel_stat per distinct kernel
 * name (at most cap of them, in decreasing total time) and the number of
 * distinct names to *n_out.  flops and bytes are the summed algorithmic work
 * of the launches: floating-point operations of what the kernel computes
 * (a convolution pass counts 2*N*P*Q*K*C*R*S) and the minimal HBM bytes
 * (each operand read once, each result written once). */
enum {
    PSW_PROF_CONV_FWD = 0, PSW_PROF_CONV_BWD_DATA = 1, PSW_PROF_CONV_BWD_WEIGHT = 2, PSW_PROF_BN_FWD = 3,
    PSW_PROF_BN_BWD = 4, PSW_PROF_POOL = 5, PSW_PROF_FC = 6, PSW_PROF_LOSS = 7, PSW_PROF_SGD = 8,
    PSW_PROF_OTHER = 9, PSW_PROF_KINDS = 10
};
typedef struct psw_kernel_stat {
    char name[192];
    int32_t kind;     /* PSW_PROF_* kind of its first launch */
    int64_t launches;
    double ms;        /* summed event time per launch */
    double flops;     /* summed algorithmic floating-point operations */
    double bytes;     /* summed algorithmic HBM bytes */
} psw_kernel_stat;
int psw_net_profile(psw_net *net, int enable);
int psw_net_profile_only(psw_net *net, int enable, const char *kernel);
int psw_net_profile_read(psw_net *net, int n_kinds, double *ms, int64_t *launches);
int psw_net_profile_kernels(psw_net *net, int cap, psw_kernel_stat *out, int *n_out);
/* psw_net_profile_replay: with reps > 1, every launch recorded from then on
 * is timed in isolation instead: the library waits until the device is idle
 * (hipDeviceSynchronize), then issues the kernel reps times back to back on
 * its stream with the same arguments between a start and a stop event, and
 * records the mean time per launch (ms of psw_kernel_stat and the kinds of
 * psw_net_profile_read are per launch, launches count the recorded launch
 * once).  This is the kernel's own duration plus the dispatch gap between
 * consecutive launches on one stream, without the event pair's cost.  The
 * replays repeat the launch's work on the same buffers (a kernel that
 * accumulates or updates applies it reps times), so the numerical results of
 * a replayed run are not those of the schedule: for timing only.  reps == 1
 * (the default) restores one event pair per launch.  reps in [1, 1000]. */
int psw_net_profile_replay(psw_net *net, int reps);
/* psw_net_profile_timeline: one psw_kernel_span per recorded launch, in
 * issue order (at most cap; *n_out = the record count): start and end in
 * microseconds after the first record's start, and the stream it ran on
 * (0 the caller's, 1 the library's weight-gradient / update stream, 2 the
 * library's forward stream of psw_pipeline_run). */
typedef struct psw_kernel_span {
    char name[96];
    int32_t kind;
    int32_t stream;
    double start_us, end_us;
} psw_kernel_span;
int psw_net_profile_timeline(psw_net *net, int cap, psw_kernel_span *out, int *n_out);

#ifdef __cplusplus
}
#endif
#endif /* PSW_H */
