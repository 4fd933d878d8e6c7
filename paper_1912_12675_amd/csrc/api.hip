// C ABI of libpsw (declared in include/psw.h): argument validation, error
// reporting, and the stale-weight stage scheduler with its per-stage
// weight-version ring.
//
// Schedule (Sec. 3 of the paper, one weight copy per partition, no stashing,
// read as: mini-batch t's forward stage i sees the updates of mini-batches
// < t - d_i, its backward stage sees every update of mini-batches < t):
//   forward of stage s at step t   : version r_s = max(0, t - d_s)
//   backward of stage s at step t  : weight gradients from the activations
//                                    saved by that forward, data gradients
//                                    with version t
//   update of stage s at step t    : version t+1 = SGD(version t)
// The ring of stage s keeps D_s = ring_depth[s] consecutive versions, version
// v in slot v mod D_s.  After step t-1 the resident versions are t-D_s+1..t,
// so any d_s <= D_s-1 is readable; the update of step t writes slot
// (t+1) mod D_s, which holds version t+1-D_s <= t-d_s: only the version the
// forward pass of this same step may read, and that pass has already run on
// the stream.  D_s = 1 updates in place.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/psw.h"
#include "internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_check(hipError_t e, const char* what)
{
    if (e == hipSuccess) return PSW_OK;
    return fail(PSW_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

inline hipStream_t S(void* s) { return (hipStream_t)s; }

bool bad_dims(std::initializer_list<int> v)
{
    for (int x : v)
        if (x <= 0) return true;
    return false;
}

int check_conv(int n, int c, int h, int w, int k, int r, int s, int stride, int pad, int prec, psw::ConvShape* cs)
{
    if (bad_dims({n, c, h, w, k, r, s, stride}) || pad < 0)
        return fail(PSW_ERR_SHAPE, "conv: sizes must be positive (pad >= 0)");
    if (prec != PSW_FP32 && prec != PSW_BF16) return fail(PSW_ERR_UNSUPPORTED, "conv: unknown precision %d", prec);
    const int p = psw::conv_out_dim(h, r, stride, pad), q = psw::conv_out_dim(w, s, stride, pad);
    if (h + 2 * pad < r || w + 2 * pad < s || p <= 0 || q <= 0)
        return fail(PSW_ERR_SHAPE, "conv: kernel larger than padded input");
    if ((int64_t)n * c * h * w > INT32_MAX || (int64_t)n * k * p * q > INT32_MAX ||
        (int64_t)k * c * r * s > INT32_MAX)
        return fail(PSW_ERR_SHAPE, "conv: tensor too large for 32-bit GEMM indexing");
    *cs = psw::ConvShape{n, c, h, w, k, r, s, stride, pad, p, q};
    return PSW_OK;
}

// Scratch of psw_conv_bwd_weight_noalloc: one array per GPU, part of the
// library's device code, so that the entry point allocates nothing.  Host
// code must not pass `scratch` itself to a kernel (in host code the name is
// a stand-in, not a device address): its device address is resolved once per
// device with hipGetSymbolAddress, with that device current, and kept here.
constexpr size_t kScratchBytes = PSW_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) static char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device, nullptr until resolved

int scratch_of_current_device(void** out, const char* what)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_check(e, what);
    if (dev < 0 || dev >= kMaxDevices) return fail(PSW_ERR_UNSUPPORTED, "%s: device %d out of range", what, dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_check(e, what);
        if (!p) return fail(PSW_ERR_HIP, "%s: hipGetSymbolAddress returned no address", what);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return PSW_OK;
}

}  // namespace

extern "C" {

const char* psw_last_error(void) { return g_err.c_str(); }
const char* psw_version(void) { return "psw 0.1 gfx950"; }

int psw_conv_fwd(int n, int c, int h, int w, int k, int r, int s, int stride, int pad, const float* x,
                 const float* wt, const float* bias, int relu, float* y, int prec, void* stream)
{
    psw::ConvShape cs;
    int rc = check_conv(n, c, h, w, k, r, s, stride, pad, prec, &cs);
    if (rc) return rc;
    if (!x || !wt || !y) return fail(PSW_ERR_NULL, "conv_fwd: x, w and y are required");
    return hip_check(psw::conv_fwd(cs, x, wt, bias, relu, y, prec == PSW_BF16, S(stream)), "conv_fwd");
}

int psw_conv_bwd_data(int n, int c, int h, int w, int k, int r, int s, int stride, int pad, const float* wt,
                      const float* dy, float* dx, int accumulate, int prec, void* stream)
{
    psw::ConvShape cs;
    int rc = check_conv(n, c, h, w, k, r, s, stride, pad, prec, &cs);
    if (rc) return rc;
    if (!wt || !dy || !dx) return fail(PSW_ERR_NULL, "conv_bwd_data: w, dy and dx are required");
    return hip_check(psw::conv_bwd_data(cs, wt, dy, dx, accumulate, prec == PSW_BF16, S(stream)), "conv_bwd_data");
}

size_t psw_conv_bwd_weight_ws_bytes(int n, int c, int h, int w, int k, int r, int s, int stride, int pad, int prec)
{
    psw::ConvShape cs;
    if (check_conv(n, c, h, w, k, r, s, stride, pad, prec, &cs)) return 0;
    return psw::conv_bwd_weight_ws_bytes(cs, prec == PSW_BF16);
}

int psw_conv_bwd_weight(int n, int c, int h, int w, int k, int r, int s, int stride, int pad, const float* x,
                        const float* dy, float* dw, float* dbias, int prec, void* ws, size_t ws_bytes, void* stream)
{
    psw::ConvShape cs;
    int rc = check_conv(n, c, h, w, k, r, s, stride, pad, prec, &cs);
    if (rc) return rc;
    if (!x || !dy || !dw || !ws) return fail(PSW_ERR_NULL, "conv_bwd_weight: x, dy, dw and ws are required");
    const size_t need = psw::conv_bwd_weight_ws_bytes(cs, prec == PSW_BF16);
    if (ws_bytes < need) return fail(PSW_ERR_WORKSPACE, "conv_bwd_weight: workspace %zu < %zu bytes", ws_bytes, need);
    return hip_check(psw::conv_bwd_weight(cs, x, dy, dw, dbias, prec == PSW_BF16, ws, ws_bytes, S(stream)),
                     "conv_bwd_weight");
}

int psw_conv_bwd_weight_noalloc(int n, int c, int h, int w, int k, int r, int s, int stride, int pad,
                                const float* x, const float* dy, float* dw, float* dbias, int prec, void* stream)
{
    psw::ConvShape cs;
    int rc = check_conv(n, c, h, w, k, r, s, stride, pad, prec, &cs);
    if (rc) return rc;
    if (!x || !dy || !dw) return fail(PSW_ERR_NULL, "conv_bwd_weight_noalloc: x, dy and dw are required");
    const size_t need = psw::conv_bwd_weight_ws_bytes(cs, prec == PSW_BF16);
    if (need > kScratchBytes)
        return fail(PSW_ERR_WORKSPACE, "conv_bwd_weight_noalloc: shape needs %zu bytes of scratch, the limit is %zu",
                    need, kScratchBytes);
    void* ws = nullptr;
    rc = scratch_of_current_device(&ws, "conv_bwd_weight_noalloc: scratch");
    if (rc) return rc;
    return hip_check(psw::conv_bwd_weight(cs, x, dy, dw, dbias, prec == PSW_BF16, ws, kScratchBytes, S(stream)),
                     "conv_bwd_weight_noalloc");
}

size_t psw_bn_ws_bytes(int n, int c, int h, int w)
{
    if (bad_dims({n, c, h, w})) return 0;
    return psw::bn_ws_bytes(n, c, h, w);
}

static int check_residual(int c, int h, int w, const float* res, int rc, int rh, int rw)
{
    if (!res) return PSW_OK;
    if (rc == c && rh == h && rw == w) return PSW_OK;
    if (rc <= 0 || rc > c || (c - rc) % 2 != 0 || rh <= 0 || rw <= 0 || rh % h != 0 || rw % w != 0 ||
        rh / h != rw / w)
        return fail(PSW_ERR_SHAPE, "bn: residual [%d,%d,%d] does not fit output [%d,%d,%d]", rc, rh, rw, c, h, w);
    return PSW_OK;
}

int psw_bn_relu_fwd(int n, int c, int h, int w, const float* y, const float* gamma, const float* beta, const float* res,
                    int rc, int rh, int rw, int relu, float eps, float momentum, float* z, float* save_mean,
                    float* save_invstd, float* run_mean, float* run_var, void* ws, size_t ws_bytes, void* stream)
{
    if (bad_dims({n, c, h, w})) return fail(PSW_ERR_SHAPE, "bn_fwd: sizes must be positive");
    if (!y || !gamma || !beta || !z || !save_mean || !save_invstd || !ws)
        return fail(PSW_ERR_NULL, "bn_fwd: required pointer is NULL");
    if ((run_mean == nullptr) != (run_var == nullptr))
        return fail(PSW_ERR_NULL, "bn_fwd: run_mean and run_var must both be set or both NULL");
    int e = check_residual(c, h, w, res, rc, rh, rw);
    if (e) return e;
    const size_t need = psw::bn_ws_bytes(n, c, h, w);
    if (ws_bytes < need) return fail(PSW_ERR_WORKSPACE, "bn_fwd: workspace %zu < %zu bytes", ws_bytes, need);
    return hip_check(psw::bn_fwd(n, c, h, w, y, gamma, beta, res, rc, rh, rw, relu, eps, momentum, z, save_mean,
                                 save_invstd, run_mean, run_var, ws, ws_bytes, S(stream)),
                     "bn_fwd");
}

int psw_bn_relu_bwd(int n, int c, int h, int w, const float* dz, const float* z, const float* y, const float* gamma,
                    const float* save_mean, const float* save_invstd, int relu, float* dy, float* dgamma,
                    float* dbeta, float* dres, int rc, int rh, int rw, int res_accumulate, void* ws, size_t ws_bytes,
                    void* stream)
{
    if (bad_dims({n, c, h, w})) return fail(PSW_ERR_SHAPE, "bn_bwd: sizes must be positive");
    if (!dz || !z || !y || !gamma || !save_mean || !save_invstd || !dy || !dgamma || !dbeta || !ws)
        return fail(PSW_ERR_NULL, "bn_bwd: required pointer is NULL");
    int e = check_residual(c, h, w, dres, rc, rh, rw);
    if (e) return e;
    const size_t need = psw::bn_ws_bytes(n, c, h, w);
    if (ws_bytes < need) return fail(PSW_ERR_WORKSPACE, "bn_bwd: workspace %zu < %zu bytes", ws_bytes, need);
    return hip_check(psw::bn_bwd(n, c, h, w, dz, z, y, gamma, save_mean, save_invstd, relu, dy, dgamma, dbeta, dres,
                                 rc, rh, rw, res_accumulate, ws, ws_bytes, S(stream)),
                     "bn_bwd");
}

int psw_pool_fwd(int kind, int n, int c, int h, int w, int k, int stride, const float* x, float* y, int32_t* argmax,
                 void* stream)
{
    if (bad_dims({n, c, h, w})) return fail(PSW_ERR_SHAPE, "pool_fwd: sizes must be positive");
    if (!x || !y) return fail(PSW_ERR_NULL, "pool_fwd: x and y are required");
    if (kind == PSW_POOL_GAVG) return hip_check(psw::gavgpool_fwd(n, c, h, w, x, y, S(stream)), "pool_fwd");
    if (kind != PSW_POOL_MAX) return fail(PSW_ERR_UNSUPPORTED, "pool_fwd: unknown kind %d", kind);
    if (!argmax) return fail(PSW_ERR_NULL, "pool_fwd: max pooling needs argmax");
    if (k <= 0 || stride <= 0 || k > h || k > w) return fail(PSW_ERR_SHAPE, "pool_fwd: bad window");
    if (k != stride) return fail(PSW_ERR_UNSUPPORTED, "pool_fwd: only non-overlapping windows (k == stride)");
    return hip_check(psw::maxpool_fwd(n, c, h, w, k, stride, x, y, argmax, S(stream)), "pool_fwd");
}

int psw_pool_bwd(int kind, int n, int c, int h, int w, int k, int stride, const float* dy, const int32_t* argmax,
                 float* dx, int accumulate, void* stream)
{
    if (bad_dims({n, c, h, w})) return fail(PSW_ERR_SHAPE, "pool_bwd: sizes must be positive");
    if (!dy || !dx) return fail(PSW_ERR_NULL, "pool_bwd: dy and dx are required");
    if (kind == PSW_POOL_GAVG)
        return hip_check(psw::gavgpool_bwd(n, c, h, w, dy, dx, accumulate, S(stream)), "pool_bwd");
    if (kind != PSW_POOL_MAX) return fail(PSW_ERR_UNSUPPORTED, "pool_bwd: unknown kind %d", kind);
    if (!argmax) return fail(PSW_ERR_NULL, "pool_bwd: max pooling needs argmax");
    if (k <= 0 || stride <= 0 || k > h || k > w) return fail(PSW_ERR_SHAPE, "pool_bwd: bad window");
    if (k != stride) return fail(PSW_ERR_UNSUPPORTED, "pool_bwd: only non-overlapping windows (k == stride)");
    return hip_check(psw::maxpool_bwd(n, c, h, w, k, stride, dy, argmax, dx, accumulate, S(stream)), "pool_bwd");
}

int psw_fc_fwd(int n, int in, int out, const float* x, const float* wt, const float* b, int relu, float* y, int prec,
               void* stream)
{
    if (bad_dims({n, in, out})) return fail(PSW_ERR_SHAPE, "fc_fwd: sizes must be positive");
    if (!x || !wt || !y) return fail(PSW_ERR_NULL, "fc_fwd: x, w and y are required");
    if (prec != PSW_FP32 && prec != PSW_BF16) return fail(PSW_ERR_UNSUPPORTED, "fc_fwd: unknown precision");
    return hip_check(psw::fc_fwd(n, in, out, x, wt, b, relu, y, prec == PSW_BF16, S(stream)), "fc_fwd");
}

size_t psw_fc_bwd_ws_bytes(int n, int in, int out)
{
    if (bad_dims({n, in, out})) return 0;
    return psw::fc_bwd_ws_bytes(n, in, out);
}

int psw_fc_bwd(int n, int in, int out, const float* x, const float* wt, const float* dy, float* dx, int dx_accumulate,
               float* dw, float* db, int prec, void* ws, size_t ws_bytes, void* stream)
{
    if (bad_dims({n, in, out})) return fail(PSW_ERR_SHAPE, "fc_bwd: sizes must be positive");
    if (!x || !wt || !dy || !dw || !ws) return fail(PSW_ERR_NULL, "fc_bwd: x, w, dy, dw and ws are required");
    if (prec != PSW_FP32 && prec != PSW_BF16) return fail(PSW_ERR_UNSUPPORTED, "fc_bwd: unknown precision");
    const size_t need = psw::fc_bwd_ws_bytes(n, in, out);
    if (ws_bytes < need) return fail(PSW_ERR_WORKSPACE, "fc_bwd: workspace %zu < %zu bytes", ws_bytes, need);
    return hip_check(psw::fc_bwd(n, in, out, x, wt, dy, dx, dx_accumulate, dw, db, prec == PSW_BF16, ws, ws_bytes,
                                 S(stream)),
                     "fc_bwd");
}

int psw_relu_mask(int64_t count, const float* z, float* g, void* stream)
{
    if (count < 0) return fail(PSW_ERR_SHAPE, "relu_mask: negative count");
    if (count == 0) return PSW_OK;
    if (!z || !g) return fail(PSW_ERR_NULL, "relu_mask: z and g are required");
    return hip_check(psw::relu_mask(count, z, g, S(stream)), "relu_mask");
}

int psw_softmax_xent(int n, int classes, const float* logits, const int32_t* labels, float* loss, float* dlogits,
                     void* stream)
{
    if (bad_dims({n, classes})) return fail(PSW_ERR_SHAPE, "softmax_xent: sizes must be positive");
    if (!logits || !labels || !loss || !dlogits) return fail(PSW_ERR_NULL, "softmax_xent: required pointer is NULL");
    return hip_check(psw::softmax_xent(n, classes, logits, labels, loss, dlogits, S(stream)), "softmax_xent");
}

int psw_dropout(int64_t count, const float* in, float* out, int accumulate, int p24, uint64_t seed, int32_t op,
                int64_t t, void* stream)
{
    if (count < 0 || t < 0) return fail(PSW_ERR_SHAPE, "dropout: count and t must be >= 0");
    if ((count + 3) / 4 > (int64_t)UINT32_MAX + 1) return fail(PSW_ERR_SHAPE, "dropout: count / 4 exceeds 32 bits");
    if (p24 <= 0 || p24 >= (1 << 24)) return fail(PSW_ERR_SHAPE, "dropout: p24 must be in (0, 2^24)");
    if (count > 0 && (!in || !out)) return fail(PSW_ERR_NULL, "dropout: in and out are required");
    return hip_check(psw::dropout_apply(count, in, out, accumulate, p24, seed, (uint32_t)op, t, S(stream)),
                     "dropout");
}

int psw_sgd_momentum_step(int64_t count, const float* w_in, float* w_out, float* v, const float* g, float lr,
                          float mom, float wd, int nesterov, void* stream)
{
    if (count < 0) return fail(PSW_ERR_SHAPE, "sgd: negative count");
    if (count == 0) return PSW_OK;
    if (!w_in || !w_out || !v || !g) return fail(PSW_ERR_NULL, "sgd: required pointer is NULL");
    if (w_out != w_in && w_out < w_in + count && w_in < w_out + count)
        return fail(PSW_ERR_SHAPE, "sgd: w_out partially overlaps w_in");
    return hip_check(psw::sgd_momentum(count, w_in, w_out, v, g, lr, mom, wd, nesterov, S(stream)), "sgd");
}

}  // extern "C"

// ============================================================================
// Network plan and stage scheduler
// ============================================================================
struct Tensor {
    int n, c, h, w;
    int64_t numel() const { return (int64_t)n * c * h * w; }
};

struct psw_net {
    std::vector<psw_layer> ops;
    int batch = 0, prec = 0, S = 0;
    std::vector<Tensor> t;              // n_ops + 1
    std::vector<int> stage_begin, stage_end, ring_depth, stage_of;
    std::vector<int64_t> stage_np;      // params per stage
    std::vector<int64_t> ring_off;      // float offset of each stage's ring
    std::vector<int64_t> flat_off;      // float offset of each stage in momentum/grad
    std::vector<int64_t> poff, pcount;  // per op, inside its stage
    std::vector<int64_t> bn_off;        // per op (BN): offset into running stats, else -1
    int64_t bn_channels = 0;
    // arena layout (bytes)
    std::vector<size_t> act_off, grad_off;  // per tensor (index 0 unused)
    std::vector<size_t> save_off;           // per op: BN mean/invstd/scale,shift or max-pool argmax
    std::vector<char> fuse_stats;           // per conv op: its BN (op+1) statistics come from the conv epilogue
    std::vector<char> fused_now;            // per conv op: the fused kernel ran in the current step
    std::vector<char> fuse_bwd;             // per conv op: its input's BN (op-1) backward sums come from its dgrad
    std::vector<char> fused_bwd_now;        // per conv op: the fused dgrad ran in the current step
    // per BN op without residual: its backward is folded into the convs
    // around it (the next conv's dgrad writes its per-tile sums to the op's
    // own region at fold_off from fold_base in the shared set, and the
    // previous conv's dgrad merges them and forms dy while staging)
    std::vector<char> fold_bn, folded_now;
    std::vector<size_t> fold_off;
    size_t fold_base = 0, fold_bytes = 0;
    // a BN whose output only a global average pool reads: per BN op, that
    // pool op (else -1); the two backward passes run as one kernel
    std::vector<int> gavg_of;
    std::vector<char> gavg_fused;           // per pool op: its backward runs in its BN's kernel
    // per BN op whose 8x8 output only a global average pool reads: that pool
    // op (else -1); the BN apply writes the pooled means too, and the pool
    // op launches nothing when it did (pool_done_now, per step)
    std::vector<int> gavg_fwd_of;
    std::vector<char> pool_done_now;
    // per BN op with both pool fusions: its apply kernel also stores, per
    // (image, channel), the ReLU-pass count and the sum of xhat there (at
    // pstat_off in the step set), and its backward is one elementwise pass
    // from them (bn_bwd_gavg_from_stats)
    std::vector<char> gavg_pstat;
    std::vector<size_t> pstat_off;
    // per BN op: a BN + ReLU without residual whose output only one conv
    // reads; that conv applies it while staging its input (forward and weight
    // gradient) from the BN's input and saved scale and shift, so the output
    // is never stored and a statistics-only launch replaces the apply
    // (bn_on_load_on: psw_net_set_bn_on_load)
    std::vector<char> bn_on_load;
    int bn_on_load_on = 1;

    std::vector<char> grad_accum;           // per op input slot: 0 overwrite, 1 accumulate (in0, in1)
    size_t step_bytes = 0;                  // one step set (activations, saves, gradients, forward ws)
    size_t pgrad_off = 0;                   // parameter gradients in the step set (pipelined runs)
    size_t wsf_off = 0;                     // forward workspace, in the step set
    size_t ws_off = 0, ws_bytes = 0, arena_bytes = 0;  // backward workspace, in the shared set
    size_t wsw_off = 0, wsw_bytes = 0;      // workspace of the backward-weight kernels (shared set)
    // conv weight gradients left as split partial sums for the stage update
    // (psw::sgd_stage), one region per conv in the shared set; the regions of
    // one stage are disjoint, stages reuse them (the weight stream runs the
    // stages one after another)
    std::vector<int32_t> wpart_splits;      // per op: splits, 0 = gradient reduced by conv_bwd_weight
    std::vector<size_t> wpart_off;          // per op: offset of its region from wpart_base
    size_t wpart_base = 0;
    struct SegProto {
        int64_t off, count;
        int op;  // conv op whose partial sums give the gradient, -1: read the gradient array
    };
    std::vector<std::vector<SegProto>> sgd_segs;  // per stage
    // per stage: it has conv layers, whose weight gradients run on the weight
    // stream; a stage without them is updated on the data-gradient stream
    std::vector<char> stage_has_conv;
    // backward-weight kernels run on a second stream of the library, forked
    // from the caller's stream when a conv's output gradient is final and
    // joined before the update (created at bind, default priority)
    hipStream_t side = nullptr;
    std::vector<hipEvent_t> stage_ev;       // per stage: the chain is done with the stage
    hipEvent_t join_ev = nullptr;
    // pipelined runs (psw_pipeline_run): forward stream, further step sets,
    // per-stage update events indexed by version mod upd_q, per step set
    // "weight stream done with the step" events
    hipStream_t fwd = nullptr;
    static constexpr int kMaxSets = 3;
    char* sets[kMaxSets] = {nullptr, nullptr, nullptr};  // step sets: [0] in the arena, more bound for pipelining
    int nsets = 1;
    int upd_q = 0;
    std::vector<hipEvent_t> upd_ev;
    hipEvent_t wdone_ev[kMaxSets] = {nullptr, nullptr, nullptr};
    hipEvent_t fdone_ev = nullptr, start_ev = nullptr;
    // bound memory
    float *ring = nullptr, *momentum = nullptr, *grad = nullptr, *run_mean = nullptr, *run_var = nullptr;
    char* arena = nullptr;
    bool bound = false;
    int64_t next_t = 0;
    // 1: the backward pass takes its data gradients with the forward's
    // version r_s (weight stashing, the comparison scheme), 0: with version t
    int stash = 0;
    uint64_t dropout_seed = 0;  // key of the dropout masks
    // optional per-kernel timing with HIP events (psw_net_profile): while
    // psw_stage_step runs with profiling on, rec is this thread's kernel
    // recorder and every library kernel launch adds one KRec
    struct KRec {
        int kind;
        std::string name;
        psw::Work work;
        hipEvent_t a, b;
        int stream;  // 0 the caller's, 1 the weight stream, 2 the forward stream
        int reps;    // launches between a and b
    };
    struct Recorder final : psw::KernelRecorder {
        psw_net* net = nullptr;
        int kind = PSW_PROF_OTHER;  // the launcher being issued
        std::string only;           // non-empty: time launches of this kernel only
        int replay = 1;             // > 1: isolated back-to-back replays (psw_net_profile_replay)
        bool begin(const std::string& name, hipEvent_t* start, hipEvent_t* stop, int* reps) override
        {
            if (!only.empty() && name != only) return false;
            *start = net->next_event();
            *stop = *start ? net->next_event() : nullptr;
            if (!*start || !*stop) return false;
            if (replay > 1) {
                // the kernel runs alone: everything issued before it is done
                if (hipDeviceSynchronize() != hipSuccess) return false;
                *reps = replay;
            }
            return true;
        }
        void end(std::string&& name, const psw::Work& w, hipEvent_t start, hipEvent_t stop, int reps,
                 hipStream_t st) override
        {
            const int sid = st == net->side ? 1 : (st == net->fwd && st ? 2 : 0);
            net->krecs.push_back(KRec{kind, std::move(name), w, start, stop, sid, reps});
        }
    };
    bool profiling = false;
    Recorder rec;
    std::vector<hipEvent_t> ev_pool;
    size_t ev_used = 0;
    std::vector<KRec> krecs;
    psw_net() { rec.net = this; }
    psw_net(const psw_net&) = delete;
    psw_net& operator=(const psw_net&) = delete;
    ~psw_net()
    {
        for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
        if (side) (void)hipStreamSynchronize(side);
        if (fwd) (void)hipStreamSynchronize(fwd);
        for (hipEvent_t e : stage_ev)
            if (e) (void)hipEventDestroy(e);
        for (hipEvent_t e : upd_ev)
            if (e) (void)hipEventDestroy(e);
        for (hipEvent_t e : wdone_ev)
            if (e) (void)hipEventDestroy(e);
        for (hipEvent_t e : {join_ev, fdone_ev, start_ev})
            if (e) (void)hipEventDestroy(e);
        if (side) (void)hipStreamDestroy(side);
        if (fwd) (void)hipStreamDestroy(fwd);
    }
    hipEvent_t next_event()
    {
        if (ev_used == ev_pool.size()) {
            hipEvent_t e;
            if (hipEventCreate(&e) != hipSuccess) return nullptr;
            ev_pool.push_back(e);
        }
        return ev_pool[ev_used++];
    }
};

namespace psw {
KernelRecorder*& kernel_recorder()
{
    static thread_local KernelRecorder* r = nullptr;
    return r;
}
}  // namespace psw

namespace {

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

int build_net(psw_net* net, const psw_layer* layers, int n_layers, int batch, int c0, int h0, int w0,
              const int32_t* stage_end, int n_stages, const int32_t* ring_depth, int prec)
{
    if (!layers || !stage_end || !ring_depth) return fail(PSW_ERR_NULL, "net_create: required pointer is NULL");
    if (n_layers <= 0 || n_stages <= 0 || n_stages > n_layers || bad_dims({batch, c0, h0, w0}))
        return fail(PSW_ERR_SHAPE, "net_create: bad sizes");
    if (prec != PSW_FP32 && prec != PSW_BF16) return fail(PSW_ERR_UNSUPPORTED, "net_create: unknown precision");
    net->ops.assign(layers, layers + n_layers);
    net->batch = batch;
    net->prec = prec;
    net->S = n_stages;
    net->t.assign(n_layers + 1, Tensor{0, 0, 0, 0});
    net->t[0] = Tensor{batch, c0, h0, w0};
    net->stage_of.assign(n_layers, 0);
    int prev = 0;
    for (int s = 0; s < n_stages; ++s) {
        if (stage_end[s] <= prev || stage_end[s] > n_layers)
            return fail(PSW_ERR_SHAPE, "net_create: stage_end[%d] = %d is not increasing within (0, %d]", s,
                        stage_end[s], n_layers);
        if (ring_depth[s] < 1) return fail(PSW_ERR_SHAPE, "net_create: ring_depth[%d] < 1", s);
        net->stage_begin.push_back(prev);
        net->stage_end.push_back(stage_end[s]);
        net->ring_depth.push_back(ring_depth[s]);
        for (int i = prev; i < stage_end[s]; ++i) net->stage_of[i] = s;
        prev = stage_end[s];
    }
    if (prev != n_layers) return fail(PSW_ERR_SHAPE, "net_create: last stage_end must equal n_layers");
    net->stage_np.assign(n_stages, 0);
    net->poff.assign(n_layers, 0);
    net->pcount.assign(n_layers, 0);
    net->bn_off.assign(n_layers, -1);
    std::vector<int> consumers(n_layers + 1, 0);
    for (int i = 0; i < n_layers; ++i) {
        const psw_layer& o = net->ops[i];
        if (o.in0 < 0 || o.in0 > i) return fail(PSW_ERR_SHAPE, "op %d: in0 %d is not an earlier tensor", i, o.in0);
        if (o.in1 > i || (o.in1 >= 0 && o.kind != PSW_OP_BN))
            return fail(PSW_ERR_SHAPE, "op %d: in1 only allowed on BN and must be earlier", i);
        const Tensor a = net->t[o.in0];
        Tensor out = a;
        int64_t np = 0;
        consumers[o.in0]++;
        if (o.in1 >= 0) consumers[o.in1]++;
        switch (o.kind) {
        case PSW_OP_CONV: {
            if (a.c != o.cin || o.cout <= 0 || o.k <= 0 || o.stride <= 0 || o.pad < 0)
                return fail(PSW_ERR_SHAPE, "op %d: conv channels/geometry do not match its input", i);
            psw::ConvShape cs;
            if (check_conv(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, prec, &cs)) return PSW_ERR_SHAPE;
            out = Tensor{a.n, o.cout, cs.p, cs.q};
            np = (int64_t)o.cout * o.cin * o.k * o.k + ((o.flags & PSW_F_BIAS) ? o.cout : 0);
            break;
        }
        case PSW_OP_BN:
            if (a.c != o.cin || o.cout != o.cin) return fail(PSW_ERR_SHAPE, "op %d: bn channels", i);
            if (o.in1 >= 0) {
                const Tensor r = net->t[o.in1];
                if (r.n != a.n || check_residual(a.c, a.h, a.w, (const float*)1, r.c, r.h, r.w))
                    return fail(PSW_ERR_SHAPE, "op %d: residual shape does not fit", i);
            }
            np = 2 * (int64_t)o.cin;
            net->bn_off[i] = net->bn_channels;
            net->bn_channels += o.cin;
            break;
        case PSW_OP_MAXPOOL:
            if (o.k <= 0 || o.stride != o.k || o.k > a.h || o.k > a.w)
                return fail(PSW_ERR_UNSUPPORTED, "op %d: max-pool needs k == stride <= input", i);
            out.h = (a.h - o.k) / o.stride + 1;
            out.w = (a.w - o.k) / o.stride + 1;
            break;
        case PSW_OP_GAVG:
            out.h = out.w = 1;
            break;
        case PSW_OP_DROPOUT:
            if (a.c != o.cin || o.cout != o.cin) return fail(PSW_ERR_SHAPE, "op %d: dropout channels", i);
            if (o.k <= 0 || o.k >= (1 << 24)) return fail(PSW_ERR_SHAPE, "op %d: dropout threshold outside (0, 2^24)", i);
            if (((int64_t)a.numel() + 3) / 4 > (int64_t)UINT32_MAX + 1)
                return fail(PSW_ERR_SHAPE, "op %d: dropout tensor too large", i);
            break;
        case PSW_OP_FC:
            if ((int64_t)a.c * a.h * a.w != o.cin || o.cout <= 0)
                return fail(PSW_ERR_SHAPE, "op %d: fc input features %lld != cin %d", i, (long long)a.c * a.h * a.w,
                            o.cin);
            out = Tensor{a.n, o.cout, 1, 1};
            np = (int64_t)o.cout * o.cin + ((o.flags & PSW_F_BIAS) ? o.cout : 0);
            break;
        default:
            return fail(PSW_ERR_UNSUPPORTED, "op %d: unknown kind %d", i, o.kind);
        }
        const int s = net->stage_of[i];
        net->poff[i] = net->stage_np[s];
        net->pcount[i] = np;
        net->stage_np[s] += np;
        net->t[i + 1] = out;
    }
    for (int i = 1; i < n_layers; ++i)
        if (consumers[i] == 0) return fail(PSW_ERR_SHAPE, "tensor %d is never used", i);
    const Tensor lg = net->t[n_layers];
    if (lg.h != 1 || lg.w != 1) return fail(PSW_ERR_SHAPE, "the last operation must produce [batch, classes] logits");
    // gradient write modes in reverse order: the first writer overwrites
    std::vector<char> written(n_layers + 1, 0);
    net->grad_accum.assign(2 * n_layers, 0);
    for (int i = n_layers - 1; i >= 0; --i) {
        const psw_layer& o = net->ops[i];
        if (o.kind == PSW_OP_BN && o.in1 >= 0 && o.in1 > 0) {
            net->grad_accum[2 * i + 1] = written[o.in1];
            written[o.in1] = 1;
        }
        if (o.in0 > 0) {
            net->grad_accum[2 * i] = written[o.in0];
            if (o.kind == PSW_OP_BN && written[o.in0])
                return fail(PSW_ERR_UNSUPPORTED, "op %d: a BN input must have no other consumer", i);
            written[o.in0] = 1;
        }
    }
    for (int i = 0; i < n_layers; ++i)
        if (net->ops[i].kind == PSW_OP_BN && net->ops[i].in0 == 0)
            return fail(PSW_ERR_UNSUPPORTED, "op %d: BN directly on the input batch", i);
    // parameter and ring offsets
    int64_t fo = 0, ro = 0;
    for (int s = 0; s < n_stages; ++s) {
        net->flat_off.push_back(fo);
        net->ring_off.push_back(ro);
        fo += net->stage_np[s];
        ro += net->stage_np[s] * net->ring_depth[s];
    }
    // arena = [step set][shared set].  The step set holds everything one
    // step writes and a later stream of the same step reads: activations,
    // saved BN statistics / max-pool argmax, every tensor's gradient, the
    // parameter gradients of a pipelined run, and the forward workspace; a
    // pipelined run alternates between two step sets (psw_net_bind_pipeline)
    // so that step t+1 never writes what step t's weight stream still reads.
    // The shared set holds the backward and backward-weight workspaces, each
    // used by one stream only.  Offsets are relative to their set.
    size_t off = 0;
    net->act_off.assign(n_layers + 1, 0);
    net->grad_off.assign(n_layers + 1, 0);
    net->save_off.assign(n_layers, 0);
    for (int i = 1; i <= n_layers; ++i) {
        net->act_off[i] = off;
        off = align256(off + (size_t)net->t[i].numel() * sizeof(float));
    }
    size_t wsw = 0;
    size_t ws = 0;
    net->fuse_stats.assign(n_layers, 0);
    net->fused_now.assign(n_layers, 0);
    net->fuse_bwd.assign(n_layers, 0);
    net->fused_bwd_now.assign(n_layers, 0);
    for (int i = 0; i < n_layers; ++i) {
        const psw_layer& o = net->ops[i];
        const Tensor a = net->t[o.in0];
        if (o.kind == PSW_OP_BN) {
            net->save_off[i] = off;
            off = align256(off + 4 * (size_t)o.cin * sizeof(float));  // mean, invstd, (scale, shift)
            ws = std::max(ws, psw::bn_ws_bytes(a.n, a.c, a.h, a.w));
        } else if (o.kind == PSW_OP_MAXPOOL) {
            net->save_off[i] = off;
            off = align256(off + (size_t)net->t[i + 1].numel() * sizeof(int32_t));
        } else if (o.kind == PSW_OP_CONV) {
            psw::ConvShape cs;
            check_conv(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, prec, &cs);
            wsw = std::max(wsw, psw::conv_bwd_weight_ws_bytes(cs, prec == PSW_BF16));
            // BN right after this conv, on its output only: statistics in the conv epilogue
            const bool next_bn = i + 1 < n_layers && net->ops[i + 1].kind == PSW_OP_BN && net->ops[i + 1].in0 == i + 1;
            const bool plain = !(o.flags & (PSW_F_BIAS | PSW_F_RELU));
            const size_t pf = psw::conv_fwd_bnstats_part_floats(cs);
            net->fuse_stats[i] = next_bn && plain && pf > 0;
            if (net->fuse_stats[i]) ws = std::max(ws, pf * sizeof(float));
            // input produced by the BN right before this conv: the conv is that
            // tensor's lowest-index consumer, so its dgrad is the last writer of
            // the BN output's gradient and can also form the BN backward sums
            const bool prev_bn = i > 0 && net->ops[i - 1].kind == PSW_OP_BN && o.in0 == i && net->ops[i - 1].in0 > 0;
            const int tb = psw::conv_bwd_data_bnsums_tiles(cs);
            net->fuse_bwd[i] = prev_bn && tb > 0;
            if (net->fuse_bwd[i]) ws = std::max(ws, (size_t)tb * cs.c * 2 * sizeof(float));
        } else if (o.kind == PSW_OP_FC) {
            ws = std::max(ws, psw::fc_bwd_ws_bytes(a.n, o.cin, o.cout));
        }
    }
    // BN backward folded into the neighbouring convs' backward-data kernels:
    // a BN (without residual, or with an identity residual whose gradient it
    // writes first) after a stride-1 direct-kernel conv of its own stage,
    // before a conv whose dgrad forms its sums, whose input gradient it
    // writes once (fp32)
    net->fold_bn.assign(n_layers, 0);
    net->folded_now.assign(n_layers, 0);
    net->fold_off.assign(n_layers, 0);
    size_t fold = 0;
    for (int i = 1; i + 1 < n_layers; ++i) {
        const psw_layer& o = net->ops[i];
        const psw_layer& pc = net->ops[i - 1];
        const psw_layer& nc = net->ops[i + 1];
        if (o.kind != PSW_OP_BN || o.in0 != i) continue;
        if (o.in1 == 0) continue;  // the residual is the net input: no gradient to write
        if (o.in1 > 0) {           // identity residual whose gradient this BN writes first
            const Tensor r = net->t[o.in1], yb = net->t[i];
            if (r.c != yb.c || r.h != yb.h || r.w != yb.w || net->grad_accum[2 * i + 1]) continue;
        }
        if (pc.kind != PSW_OP_CONV || pc.in0 <= 0 || (pc.flags & PSW_F_RELU)) continue;
        // the residual's gradient (written by the fold) must not be the
        // folded conv's own input gradient (x -> conv -> BN(+x)): inside one
        // launch some workgroups would write it while others still read it
        if (o.in1 > 0 && o.in1 == pc.in0) continue;
        if (!net->fuse_bwd[i + 1] || net->grad_accum[2 * i]) continue;
        if (net->stage_of[i - 1] != net->stage_of[i]) continue;
        const Tensor a = net->t[pc.in0];
        psw::ConvShape cs;
        check_conv(a.n, a.c, a.h, a.w, pc.cout, pc.k, pc.k, pc.stride, pc.pad, prec, &cs);
        if (!psw::conv_bwd_data_fold_ok(cs)) continue;
        const Tensor z = net->t[i + 1];
        psw::ConvShape ncs;
        check_conv(z.n, z.c, z.h, z.w, nc.cout, nc.k, nc.k, nc.stride, nc.pad, prec, &ncs);
        net->fold_bn[i] = 1;
        net->fold_off[i] = fold;  // per-tile sums [c][T][2]
        fold = align256(fold + (size_t)psw::conv_bwd_data_bnsums_tiles(ncs) * o.cin * 2 * sizeof(float));
    }
    net->fold_bytes = fold;
    // BN -> global average pool, nothing else reading the BN output: the
    // pool's gradient is uniform per (image, channel), and one kernel per
    // channel does the pool backward and the BN backward (bn_bwd_gavg)
    net->gavg_of.assign(n_layers, -1);
    net->gavg_fused.assign(n_layers, 0);
    net->gavg_fwd_of.assign(n_layers, -1);
    net->pool_done_now.assign(n_layers, 0);
    for (int j = 0; j < n_layers; ++j) {
        const psw_layer& pg = net->ops[j];
        if (pg.kind != PSW_OP_GAVG || pg.in0 < 2 || consumers[pg.in0] != 1) continue;
        const Tensor zt = net->t[pg.in0];
        if (net->ops[pg.in0 - 1].kind == PSW_OP_BN && zt.h * zt.w == 64) net->gavg_fwd_of[pg.in0 - 1] = j;
    }
    for (int j = 0; j < n_layers; ++j) {
        const psw_layer& pg = net->ops[j];
        if (pg.kind != PSW_OP_GAVG || pg.in0 < 2) continue;
        const int b = pg.in0 - 1;  // the op producing the pool's input
        const psw_layer& o = net->ops[b];
        if (o.kind != PSW_OP_BN || consumers[pg.in0] != 1 || net->grad_accum[2 * j] || net->fold_bn[b]) continue;
        if (o.in1 == 0 || (o.in1 > 0 && net->grad_accum[2 * b + 1])) continue;  // it writes the residual's gradient first
        if (o.in1 > 0) {  // identity residual only
            const Tensor r = net->t[o.in1], yb = net->t[o.in0];
            if (r.c != yb.c || r.h != yb.h || r.w != yb.w) continue;
        }
        const Tensor zt = net->t[pg.in0];
        if ((zt.h * zt.w) % 4) continue;
        net->gavg_of[b] = j;
        net->gavg_fused[j] = 1;
    }
    net->gavg_pstat.assign(n_layers, 0);
    net->pstat_off.assign(n_layers, 0);
    for (int b = 1; b < n_layers; ++b) {
        if (net->gavg_of[b] < 0 || net->gavg_fwd_of[b] < 0 || !net->fuse_stats[b - 1] || net->ops[b].in0 != b) continue;
        net->gavg_pstat[b] = 1;
        net->pstat_off[b] = off;
        off = align256(off + 2 * (size_t)net->t[b + 1].n * net->ops[b].cin * sizeof(float));
    }
    // split partial sums of the conv weight gradients, reduced by the stage update
    net->wpart_splits.assign(n_layers, 0);
    net->wpart_off.assign(n_layers, 0);
    net->sgd_segs.assign(n_stages, {});
    net->stage_has_conv.assign(n_stages, 0);
    for (int i = 0; i < n_layers; ++i)
        if (net->ops[i].kind == PSW_OP_CONV) net->stage_has_conv[net->stage_of[i]] = 1;
    size_t wpart = 0;
    for (int s = 0; s < n_stages; ++s) {
        size_t cur = 0;
        auto& segs = net->sgd_segs[s];
        for (int i = net->stage_begin[s]; i < net->stage_end[s]; ++i) {
            const psw_layer& o = net->ops[i];
            if (net->pcount[i] <= 0) continue;
            int splits = 0;
            if (o.kind == PSW_OP_CONV && !(o.flags & PSW_F_BIAS)) {
                const Tensor a = net->t[o.in0];
                psw::ConvShape cs;
                check_conv(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, prec, &cs);
                splits = psw::conv_bwd_weight_part_splits(cs, prec == PSW_BF16);
            }
            if (splits > 0) {
                net->wpart_splits[i] = splits;
                net->wpart_off[i] = cur;
                cur = align256(cur + (size_t)splits * net->pcount[i] * sizeof(float));
                segs.push_back({net->poff[i], net->pcount[i], i});
            } else if (!segs.empty() && segs.back().op < 0 && segs.back().off + segs.back().count == net->poff[i]) {
                segs.back().count += net->pcount[i];
            } else {
                segs.push_back({net->poff[i], net->pcount[i], -1});
            }
        }
        wpart = std::max(wpart, cur);
    }
    // BN + ReLU applied by its one consumer conv while loading: the BN's
    // statistics come from the conv before it, the consumer's forward and
    // weight gradient (split partials) run on the direct kernels, which take
    // the BN's input and scale / shift, and the BN's backward never reads its
    // output (its sums come from the consumer's dgrad, the ReLU mask from y
    // and the scale / shift)
    net->bn_on_load.assign(n_layers, 0);
    for (int j = 1; j + 1 < n_layers; ++j) {
        const psw_layer& o = net->ops[j];
        const psw_layer& c = net->ops[j + 1];
        if (o.kind != PSW_OP_BN || o.in0 != j || o.in1 >= 0 || !(o.flags & PSW_F_RELU)) continue;
        if (!net->fuse_stats[j - 1] || consumers[j + 1] != 1) continue;
        if (c.kind != PSW_OP_CONV || c.in0 != j + 1 || (c.flags & (PSW_F_BIAS | PSW_F_RELU))) continue;
        if (!net->fuse_bwd[j + 1] || net->wpart_splits[j + 1] <= 0 || net->t[j].w % 4) continue;
        const Tensor a = net->t[j + 1];
        psw::ConvShape cs;
        check_conv(a.n, a.c, a.h, a.w, c.cout, c.k, c.k, c.stride, c.pad, prec, &cs);
        if (!psw::conv_fwd_in_bn_ok(cs)) continue;
        net->bn_on_load[j] = 1;
    }
    for (int i = 1; i <= n_layers; ++i) {  // gradients of every tensor
        net->grad_off[i] = off;
        off = align256(off + (size_t)net->t[i].numel() * sizeof(float));
    }
    int64_t np_all = 0;
    for (int s = 0; s < n_stages; ++s) np_all += net->stage_np[s];
    net->pgrad_off = off;  // parameter gradients, stage-major (pipelined runs)
    off = align256(off + (size_t)np_all * sizeof(float));
    net->ws_bytes = align256(ws);
    net->wsf_off = off;
    off += net->ws_bytes;
    net->step_bytes = off;
    off = 0;  // shared set
    net->ws_off = off;
    off += net->ws_bytes;
    net->wsw_off = off;
    net->wsw_bytes = align256(wsw);
    off += net->wsw_bytes;
    net->wpart_base = off;
    off += wpart;
    net->fold_base = off;
    off += net->fold_bytes;
    net->arena_bytes = net->step_bytes + off;
    g_err.clear();
    return PSW_OK;
}

int check_staleness(const psw_net* net, int64_t t, const int32_t* staleness)
{
    if (!staleness) return fail(PSW_ERR_NULL, "staleness array is required");
    if (t < 0) return fail(PSW_ERR_STEP_ORDER, "t must be >= 0");
    for (int s = 0; s < net->S; ++s)
        if (staleness[s] < 0 || staleness[s] >= net->ring_depth[s])
            return fail(PSW_ERR_STALENESS, "stage %d: staleness %d outside [0, ring_depth-1 = %d]", s, staleness[s],
                        net->ring_depth[s] - 1);
    return PSW_OK;
}

inline int64_t fwd_version(int64_t t, int d) { return t - d > 0 ? t - d : 0; }

float* slot_ptr(const psw_net* net, int s, int64_t version)
{
    const int64_t slot = version % net->ring_depth[s];
    return net->ring + net->ring_off[s] + slot * net->stage_np[s];
}

}  // namespace

extern "C" {

int psw_net_create(const psw_layer* layers, int n_layers, int batch, int c0, int h0, int w0, const int32_t* stage_end,
                   int n_stages, const int32_t* ring_depth, int prec, psw_net** out)
{
    if (!out) return fail(PSW_ERR_NULL, "net_create: out is NULL");
    *out = nullptr;
    psw_net* net = new psw_net();
    int rc = build_net(net, layers, n_layers, batch, c0, h0, w0, stage_end, n_stages, ring_depth, prec);
    if (rc) {
        delete net;
        return rc;
    }
    *out = net;
    return PSW_OK;
}

void psw_net_destroy(psw_net* net) { delete net; }

int psw_net_sizes(const psw_net* net, int64_t* stage_params, int64_t* ring_floats, int64_t* n_params,
                  int64_t* bn_channels, int64_t* arena_bytes)
{
    if (!net) return fail(PSW_ERR_NULL, "net_sizes: net is NULL");
    int64_t rf = 0, np = 0;
    for (int s = 0; s < net->S; ++s) {
        if (stage_params) stage_params[s] = net->stage_np[s];
        rf += net->stage_np[s] * net->ring_depth[s];
        np += net->stage_np[s];
    }
    if (ring_floats) *ring_floats = rf;
    if (n_params) *n_params = np;
    if (bn_channels) *bn_channels = net->bn_channels;
    if (arena_bytes) *arena_bytes = (int64_t)net->arena_bytes;
    return PSW_OK;
}

int psw_net_bind(psw_net* net, float* ring, float* momentum, float* grad, float* run_mean, float* run_var, void* arena,
                 size_t arena_bytes)
{
    if (!net || !ring || !momentum || !grad || !arena) return fail(PSW_ERR_NULL, "net_bind: required pointer is NULL");
    if ((run_mean == nullptr) != (run_var == nullptr))
        return fail(PSW_ERR_NULL, "net_bind: run_mean and run_var must both be set or both NULL");
    if (arena_bytes < net->arena_bytes)
        return fail(PSW_ERR_WORKSPACE, "net_bind: arena %zu < %zu bytes", arena_bytes, net->arena_bytes);
    if (((uintptr_t)arena) % 256 != 0) return fail(PSW_ERR_SHAPE, "net_bind: arena must be 256-byte aligned");
    net->ring = ring;
    net->momentum = momentum;
    net->grad = grad;
    net->run_mean = run_mean;
    net->run_var = run_var;
    net->arena = (char*)arena;
    if (!net->side) {
        hipError_t e = hipStreamCreateWithFlags(&net->side, hipStreamNonBlocking);
        if (e != hipSuccess) {
            net->side = nullptr;
            return hip_check(e, "net_bind: side stream");
        }
        net->stage_ev.assign(net->S, nullptr);
        for (auto& ev : net->stage_ev) {
            e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
            if (e != hipSuccess) return hip_check(e, "net_bind: events");
        }
        e = hipEventCreateWithFlags(&net->join_ev, hipEventDisableTiming);
        if (e != hipSuccess) return hip_check(e, "net_bind: events");
    }
    net->bound = true;
    return PSW_OK;
}

int psw_net_set_step(psw_net* net, int64_t t)
{
    if (!net) return fail(PSW_ERR_NULL, "net_set_step: net is NULL");
    if (t < 0) return fail(PSW_ERR_STEP_ORDER, "net_set_step: t < 0");
    net->next_t = t;
    return PSW_OK;
}

int psw_net_slot(const psw_net* net, int stage, int64_t version, float** params)
{
    if (!net || !params) return fail(PSW_ERR_NULL, "net_slot: required pointer is NULL");
    if (stage < 0 || stage >= net->S) return fail(PSW_ERR_SHAPE, "net_slot: stage %d out of range", stage);
    if (!net->bound) return fail(PSW_ERR_STATE, "net_slot: net is not bound");
    const int64_t newest = net->next_t;
    if (version < 0 || version > newest || version <= newest - net->ring_depth[stage])
        return fail(PSW_ERR_STALENESS, "net_slot: version %lld of stage %d is not resident (newest %lld, depth %d)",
                    (long long)version, stage, (long long)newest, net->ring_depth[stage]);
    *params = slot_ptr(net, stage, version);
    return PSW_OK;
}

int psw_net_tensor(const psw_net* net, int tensor, int grad, float** ptr, int64_t* count)
{
    if (!net || !ptr) return fail(PSW_ERR_NULL, "net_tensor: required pointer is NULL");
    if (!net->bound) return fail(PSW_ERR_STATE, "net_tensor: net is not bound");
    const int L = (int)net->ops.size();
    if (tensor < 1 || tensor > L) return fail(PSW_ERR_SHAPE, "net_tensor: tensor %d out of range 1..%d", tensor, L);
    *ptr = (float*)(net->arena + (grad ? net->grad_off[tensor] : net->act_off[tensor]));
    if (count) *count = net->t[tensor].numel();
    return PSW_OK;
}

int psw_net_tensor_stored(const psw_net* net, int tensor, int* stored)
{
    if (!net || !stored) return fail(PSW_ERR_NULL, "net_tensor_stored: required pointer is NULL");
    const int L = (int)net->ops.size();
    if (tensor < 1 || tensor > L)
        return fail(PSW_ERR_SHAPE, "net_tensor_stored: tensor %d out of range 1..%d", tensor, L);
    *stored = (net->bn_on_load_on && net->bn_on_load[tensor - 1]) ? 0 : 1;
    return PSW_OK;
}

int psw_net_bn_saved(const psw_net* net, int op, float** mean, float** invstd, float** scale_shift)
{
    if (!net || !mean || !invstd || !scale_shift) return fail(PSW_ERR_NULL, "net_bn_saved: required pointer is NULL");
    if (!net->bound) return fail(PSW_ERR_STATE, "net_bn_saved: net is not bound");
    if (op < 0 || op >= (int)net->ops.size() || net->ops[op].kind != PSW_OP_BN)
        return fail(PSW_ERR_SHAPE, "net_bn_saved: op %d is not a BN", op);
    float* save = (float*)(net->arena + net->save_off[op]);
    const int c = net->ops[op].cin;
    *mean = save;
    *invstd = save + c;
    *scale_shift = save + 2 * c;
    return PSW_OK;
}

int psw_net_set_bn_on_load(psw_net* net, int on)
{
    if (!net) return fail(PSW_ERR_NULL, "net_set_bn_on_load: net is NULL");
    net->bn_on_load_on = on ? 1 : 0;
    g_err.clear();
    return PSW_OK;
}

int psw_net_param_offset(const psw_net* net, int op, int* stage, int64_t* offset, int64_t* count)
{
    if (!net) return fail(PSW_ERR_NULL, "net_param_offset: net is NULL");
    if (op < 0 || op >= (int)net->ops.size()) return fail(PSW_ERR_SHAPE, "net_param_offset: op out of range");
    if (stage) *stage = net->stage_of[op];
    if (offset) *offset = net->poff[op];
    if (count) *count = net->pcount[op];
    return PSW_OK;
}

int psw_net_set_weight_stashing(psw_net* net, int on)
{
    if (!net) return fail(PSW_ERR_NULL, "net_set_weight_stashing: net is NULL");
    net->stash = on ? 1 : 0;
    g_err.clear();
    return PSW_OK;
}

int psw_net_set_dropout_seed(psw_net* net, uint64_t seed)
{
    if (!net) return fail(PSW_ERR_NULL, "net_set_dropout_seed: net is NULL");
    net->dropout_seed = seed;
    g_err.clear();
    return PSW_OK;
}

int psw_net_plan(const psw_net* net, int64_t t, const int32_t* staleness, psw_launch* out, int cap, int* n_out)
{
    if (!net || !n_out) return fail(PSW_ERR_NULL, "net_plan: required pointer is NULL");
    int rc = check_staleness(net, t, staleness);
    if (rc) return rc;
    int n = 0;
    auto rec = [&](int op, int what, int s, int64_t v) {
        if (out && n < cap) out[n] = psw_launch{op, what, s, v};
        ++n;
    };
    const int L = (int)net->ops.size();
    for (int i = 0; i < L; ++i) {
        const psw_layer& o = net->ops[i];
        const int s = net->stage_of[i];
        const int64_t r = fwd_version(t, staleness[s]);
        switch (o.kind) {
        case PSW_OP_CONV: rec(i, PSW_PLAN_CONV_FWD, s, r); break;
        case PSW_OP_BN: rec(i, PSW_PLAN_BN_FWD, s, r); break;
        case PSW_OP_MAXPOOL:
        case PSW_OP_GAVG: rec(i, PSW_PLAN_POOL_FWD, s, -1); break;
        case PSW_OP_FC: rec(i, PSW_PLAN_FC_FWD, s, r); break;
        case PSW_OP_DROPOUT: rec(i, PSW_PLAN_DROPOUT_FWD, s, -1); break;
        }
    }
    rec(L - 1, PSW_PLAN_LOSS, net->stage_of[L - 1], -1);
    for (int i = L - 1; i >= 0; --i) {
        const psw_layer& o = net->ops[i];
        const int s = net->stage_of[i];
        const int64_t vb = net->stash ? fwd_version(t, staleness[s]) : t;  // backward's version
        switch (o.kind) {
        case PSW_OP_CONV:
            if (o.flags & PSW_F_RELU) rec(i, PSW_PLAN_RELU_MASK, s, -1);
            if (o.in0 > 0) rec(i, PSW_PLAN_CONV_BWD_DATA, s, vb);
            break;
        case PSW_OP_BN: rec(i, net->fold_bn[i] ? PSW_PLAN_BN_BWD_FOLDED : PSW_PLAN_BN_BWD, s, vb); break;
        case PSW_OP_MAXPOOL:
        case PSW_OP_GAVG:
            if (o.in0 > 0) rec(i, PSW_PLAN_POOL_BWD, s, -1);
            break;
        case PSW_OP_FC:
            if (o.flags & PSW_F_RELU) rec(i, PSW_PLAN_RELU_MASK, s, -1);
            rec(i, PSW_PLAN_FC_BWD, s, vb);
            break;
        case PSW_OP_DROPOUT:
            if (o.in0 > 0) rec(i, PSW_PLAN_DROPOUT_BWD, s, -1);
            break;
        }
        // when the data-gradient chain is done with a stage: the stage's
        // weight gradients, then its update (version t -> t+1)
        if (i == net->stage_begin[s]) {
            for (int j = net->stage_end[s] - 1; j >= net->stage_begin[s]; --j)
                if (net->ops[j].kind == PSW_OP_CONV) rec(j, PSW_PLAN_CONV_BWD_WEIGHT, s, -1);
            rec(-1, PSW_PLAN_SGD, s, t);
        }
    }
    *n_out = n;
    return PSW_OK;
}

}  // extern "C"

namespace {

// One step's inputs and where its step set lives.
struct StepIO {
    int64_t t;
    std::vector<int64_t> rv;  // forward weight version per stage
    char* P;                  // step set (activations, saves, logits' gradient, forward workspace)
    const float* x;
    const int32_t* labels;
    float* loss_out;
    const float* lr;          // per stage
    float mom, wd;
    int nesterov;
    float* gbase;             // packed parameter gradients (stage-major)
};

struct Issue {
    psw_net* net;
    const StepIO& io;
    hipError_t e = hipSuccess;
    const char* what = "";
    char* A() const { return io.P; }
    float* act(int id) const { return id == 0 ? (float*)io.x : (float*)(io.P + net->act_off[id]); }
    float* grd(int id) const { return (float*)(io.P + net->grad_off[id]); }
    float* save(int i) const { return (float*)(io.P + net->save_off[i]); }
    float* pstat(int i) const { return (float*)(io.P + net->pstat_off[i]); }
    // BN op j is applied by its consumer while loading (its output not stored)
    bool on_load(int j) const { return net->bn_on_load_on && net->bn_on_load[j]; }
    void* wsf() const { return io.P + net->wsf_off; }
    void* wsb() const { return net->arena + net->step_bytes + net->ws_off; }
    void* wsw() const { return net->arena + net->step_bytes + net->wsw_off; }
    float* wpart(int i) const { return (float*)(net->arena + net->step_bytes + net->wpart_base + net->wpart_off[i]); }
    float* fold_part(int i) const { return (float*)(net->arena + net->step_bytes + net->fold_base + net->fold_off[i]); }
    const float* wfwd(int i) const
    {
        const int s = net->stage_of[i];
        return slot_ptr(net, s, io.rv[s]) + net->poff[i];
    }
    const float* wcur(int i) const { return slot_ptr(net, net->stage_of[i], io.t) + net->poff[i]; }
    // weights of the backward pass's data gradients
    const float* wbwd(int i) const { return net->stash ? wfwd(i) : wcur(i); }
    float* gptr(int i) const { return io.gbase + net->flat_off[net->stage_of[i]] + net->poff[i]; }
};

#define PSW_TRY(expr, w)          \
    do {                          \
        is.e = (expr);            \
        if (is.e != hipSuccess) { \
            is.what = (w);        \
            return is.e;          \
        }                         \
    } while (0)

// Forward pass and loss of one step on stream sf.  before_stage(s) runs
// before the first operation of stage s is issued (the pipelined run makes
// sf wait there for the update that produced the stage's version).
template <typename BeforeStage>
hipError_t issue_forward(Issue& is, hipStream_t sf, BeforeStage before_stage)
{
    psw_net* net = is.net;
    const int L = (int)net->ops.size();
    const int bf16 = net->prec == PSW_BF16;
    int& kind = net->rec.kind;
    void* ws = is.wsf();
    const size_t wsb = net->ws_bytes;
    hipError_t e = hipSuccess;
    bool head = false;
    for (int i = 0; i < L; ++i) {
        if (i == 0 || net->stage_of[i] != net->stage_of[i - 1]) PSW_TRY(before_stage(net->stage_of[i]), "stage wait");
        const psw_layer& o = net->ops[i];
        const Tensor a = net->t[o.in0];
        const float* W = is.wfwd(i);
        switch (o.kind) {
        case PSW_OP_CONV: {
            psw::ConvShape cs;
            check_conv(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, net->prec, &cs);
            const float* b = (o.flags & PSW_F_BIAS) ? W + (int64_t)o.cout * o.cin * o.k * o.k : nullptr;
            kind = PSW_PROF_CONV_FWD;
            net->fused_now[i] = 0;
            // input from a BN applied on load: stage the BN's input through its
            // scale / shift and ReLU (no fallback: the BN output is not stored)
            const int bj = o.in0 - 1;
            const bool ibn = bj >= 1 && is.on_load(bj);
            const float* xin = ibn ? is.act(net->ops[bj].in0) : is.act(o.in0);
            const float* inbn = ibn ? is.save(bj) + 2 * net->ops[bj].cin : nullptr;
            if (net->fuse_stats[i]) {  // the next op's BN statistics come out of this conv
                psw::BnStatsFuse bn{(float*)ws};
                e = psw::conv_fwd_bnstats(cs, xin, W, is.act(i + 1), bn, wsb / sizeof(float), bf16, sf, inbn);
                if (e == hipSuccess)
                    net->fused_now[i] = 1;
                else if (e != hipErrorNotSupported)  // not supported: nothing launched, unfused path below
                    PSW_TRY(e, "conv_fwd_bnstats");
            }
            if (!net->fused_now[i])
                PSW_TRY(psw::conv_fwd(cs, xin, W, b, (o.flags & PSW_F_RELU) != 0, is.act(i + 1), bf16, sf, inbn),
                        "conv_fwd");
            break;
        }
        case PSW_OP_BN: {
            const Tensor r = o.in1 >= 0 ? net->t[o.in1] : Tensor{0, 0, 0, 0};
            float* save = is.save(i);
            if (net->gavg_fwd_of[i] >= 0) net->pool_done_now[net->gavg_fwd_of[i]] = 0;
            float* rm = net->run_mean ? net->run_mean + net->bn_off[i] : nullptr;
            float* rvv = net->run_var ? net->run_var + net->bn_off[i] : nullptr;
            kind = PSW_PROF_BN_FWD;
            if (i > 0 && net->fused_now[i - 1]) {  // per-tile statistics written by the conv into ws
                const psw_layer& cv = net->ops[i - 1];
                const Tensor ci = net->t[cv.in0];
                psw::ConvShape ccs;
                check_conv(ci.n, ci.c, ci.h, ci.w, cv.cout, cv.k, cv.k, cv.stride, cv.pad, net->prec, &ccs);
                const int T = psw::conv_fwd_bnstats_tiles(ccs);
                const int P = a.n * a.h * a.w / T;
                if (is.on_load(i)) {  // the consumer conv applies it: statistics only
                    PSW_TRY(psw::bn_stats_from_partials(o.cin, (const float*)ws, T, P, W, W + o.cin, 1e-5f, 0.1f, save,
                                                        save + o.cin, save + 2 * o.cin, rm, rvv, sf),
                            "bn_stats");
                    break;
                }
                const int pj = net->gavg_fwd_of[i];  // the global pool reading this output alone, if any
                e = psw::bn_apply_from_partials(a.n, a.c, a.h, a.w, is.act(o.in0), (const float*)ws, T, P, W,
                                                W + o.cin, o.in1 >= 0 ? is.act(o.in1) : nullptr, r.c, r.h, r.w,
                                                (o.flags & PSW_F_RELU) != 0, 1e-5f, 0.1f, is.act(i + 1), save,
                                                save + o.cin, save + 2 * o.cin, rm, rvv, sf,
                                                pj >= 0 ? is.act(pj + 1) : nullptr,
                                                (pj >= 0 && net->gavg_pstat[i]) ? is.pstat(i) : nullptr);
                if (e == hipSuccess) {
                    if (pj >= 0) net->pool_done_now[pj] = 1;
                    break;
                }
                if (e != hipErrorNotSupported) PSW_TRY(e, "bn_apply");
                // not supported: nothing launched, the statistics are recomputed below
            }
            if (is.on_load(i) || net->gavg_pstat[i]) {  // excluded when the net was created
                is.what = "BN with fused statistics: the conv before it did not produce them";
                return hipErrorNotSupported;
            }
            PSW_TRY(psw::bn_fwd(a.n, a.c, a.h, a.w, is.act(o.in0), W, W + o.cin, o.in1 >= 0 ? is.act(o.in1) : nullptr,
                                r.c, r.h, r.w, (o.flags & PSW_F_RELU) != 0, 1e-5f, 0.1f, is.act(i + 1), save,
                                save + o.cin, rm, rvv, ws, wsb, sf, save + 2 * o.cin),
                    "bn_fwd");
            break;
        }
        case PSW_OP_MAXPOOL:
            kind = PSW_PROF_POOL;
            PSW_TRY(psw::maxpool_fwd(a.n, a.c, a.h, a.w, o.k, o.stride, is.act(o.in0), is.act(i + 1),
                                     (int32_t*)is.save(i), sf),
                    "maxpool_fwd");
            break;
        case PSW_OP_GAVG:
            kind = PSW_PROF_POOL;
            if (net->pool_done_now[i]) break;  // written by its BN's apply kernel
            PSW_TRY(psw::gavgpool_fwd(a.n, a.c, a.h, a.w, is.act(o.in0), is.act(i + 1), sf), "gavgpool_fwd");
            break;
        case PSW_OP_DROPOUT:
            kind = PSW_PROF_OTHER;
            PSW_TRY(psw::dropout_apply(a.numel(), is.act(o.in0), is.act(i + 1), 0, o.k, net->dropout_seed, (uint32_t)i,
                                       is.io.t, sf),
                    "dropout");
            break;
        case PSW_OP_FC: {
            const float* b = (o.flags & PSW_F_BIAS) ? W + (int64_t)o.cout * o.cin : nullptr;
            kind = PSW_PROF_FC;
            if (i == L - 1 && !(o.flags & PSW_F_RELU)) {  // the classifier: with the loss in one launch if small
                e = psw::fc_softmax_xent(a.n, o.cin, o.cout, is.act(o.in0), W, b, is.act(i + 1), bf16,
                                         is.io.labels, is.io.loss_out, is.grd(L), sf);
                if (e == hipSuccess) {
                    head = true;
                    break;
                }
                if (e != hipErrorNotSupported) PSW_TRY(e, "fc_softmax_xent");
            }
            PSW_TRY(psw::fc_fwd(a.n, o.cin, o.cout, is.act(o.in0), W, b, (o.flags & PSW_F_RELU) != 0, is.act(i + 1),
                                bf16, sf),
                    "fc_fwd");
            break;
        }
        }
    }
    if (head) return hipSuccess;  // the loss came with the classifier
    const Tensor lg = net->t[L];
    kind = PSW_PROF_LOSS;
    PSW_TRY(psw::softmax_xent(lg.n, lg.c, is.act(L), is.io.labels, is.io.loss_out, is.grd(L), sf), "softmax_xent");
    return hipSuccess;
}

// Backward pass and updates of one step: the data-gradient chain on sb;
// before_stage(s) runs before the chain's first operation of stage s.  When
// the chain has finished stage s, sw waits for it, computes the stage's conv
// weight gradients (they share only the step's activations with the chain)
// and writes version t+1 of stage s (all of the stage's parameter gradients
// are then complete, and nothing later in the step reads the stage's version
// t); a stage without convs is updated on sb.  after_update(s, stream) then
// runs with the stream that issued the update.
template <typename BeforeStage, typename AfterUpdate>
hipError_t issue_backward(Issue& is, hipStream_t sb, hipStream_t sw, BeforeStage before_stage,
                          AfterUpdate after_update)
{
    psw_net* net = is.net;
    const StepIO& io = is.io;
    const int L = (int)net->ops.size();
    const int bf16 = net->prec == PSW_BF16;
    int& kind = net->rec.kind;
    void* ws = is.wsb();
    const size_t wsb = net->ws_bytes;
    void* wsw = is.wsw();
    const size_t wswb = net->wsw_bytes;
    hipError_t e = hipSuccess;
    for (int i = L - 1; i >= 0; --i) {
        const psw_layer& o = net->ops[i];
        const Tensor a = net->t[o.in0];
        const Tensor y = net->t[i + 1];
        if (i == net->stage_end[net->stage_of[i]] - 1)
            PSW_TRY(before_stage(net->stage_of[i]), "backward order");
        float* g = is.grd(i + 1);
        float* din = o.in0 > 0 ? is.grd(o.in0) : nullptr;
        const int acc0 = net->grad_accum[2 * i];
        switch (o.kind) {
        case PSW_OP_CONV: {
            psw::ConvShape cs;
            check_conv(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, net->prec, &cs);
            kind = PSW_PROF_OTHER;
            if (o.flags & PSW_F_RELU) PSW_TRY(psw::relu_mask(y.numel(), is.act(i + 1), g, sb), "relu_mask");
            kind = PSW_PROF_CONV_BWD_DATA;
            net->fused_bwd_now[i] = 0;
            // BN op i+1 folded: this dgrad forms its input g (the BN's input
            // gradient, also written out) from that BN's output gradient
            const bool fold_in = i + 1 < L && net->folded_now[i + 1];
            psw::BnFold fold;
            if (fold_in) {
                const psw_layer& fb = net->ops[i + 1];
                const psw_layer& nc = net->ops[i + 2];
                const Tensor z = net->t[i + 2];
                psw::ConvShape ncs;
                check_conv(z.n, z.c, z.h, z.w, nc.cout, nc.k, nc.k, nc.stride, nc.pad, net->prec, &ncs);
                const float* fsave = is.save(i + 1);
                float* dgb = is.gptr(i + 1);
                fold.g = is.grd(i + 2);
                fold.y = is.act(i + 1);
                fold.part = is.fold_part(i + 1);
                fold.T = psw::conv_bwd_data_bnsums_tiles(ncs);
                fold.count = (double)y.n * y.h * y.w;
                fold.gamma = is.wbwd(i + 1);
                fold.mean = fsave;
                fold.invstd = fsave + fb.cin;
                fold.scale = fsave + 2 * fb.cin;
                fold.relu = (fb.flags & PSW_F_RELU) != 0;
                fold.dy = g;
                fold.dgamma = dgb;
                fold.dbeta = dgb + fb.cin;
                if (fb.in1 >= 0) {  // identity residual: mask from z, g' to the residual's gradient
                    fold.z = is.act(i + 2);
                    fold.dres = is.grd(fb.in1);
                }
            }
            if (din && net->fuse_bwd[i]) {  // BN op i-1's backward sums out of this dgrad
                const psw_layer& bo = net->ops[i - 1];
                const float* bsave = is.save(i - 1);
                psw::BnBwdFuse bnb{(float*)ws, is.act(i), is.act(bo.in0), bsave, bsave + bo.cin,
                                   (bo.flags & PSW_F_RELU) != 0};
                if (bo.in1 < 0) {  // no residual: the ReLU mask comes from y and the forward's scale / shift
                    bnb.scale = bsave + 2 * bo.cin;
                    bnb.shift = bsave + 3 * bo.cin;
                }
                if (net->fold_bn[i - 1]) bnb.part = is.fold_part(i - 1);  // merged by the dgrad of op i-2
                e = fold_in ? psw::conv_bwd_data_fold(cs, is.wbwd(i), din, acc0, &bnb, fold, bf16, sb)
                            : psw::conv_bwd_data_bnsums(cs, is.wbwd(i), g, din, acc0, bnb, bf16, sb);
                if (e == hipSuccess)
                    net->fused_bwd_now[i] = 1;
                else if (e != hipErrorNotSupported)  // not supported: nothing launched, unfused path below
                    PSW_TRY(e, "conv_bwd_data_bnsums");
            }
            if (i >= 1) net->folded_now[i - 1] = net->fused_bwd_now[i] && net->fold_bn[i - 1];
            if (din && !net->fused_bwd_now[i]) {
                if (fold_in)  // covered by construction (the fold's conditions when the net was created)
                    PSW_TRY(psw::conv_bwd_data_fold(cs, is.wbwd(i), din, acc0, nullptr, fold, bf16, sb),
                            "conv_bwd_data (folded BN backward)");
                else
                    PSW_TRY(psw::conv_bwd_data(cs, is.wbwd(i), g, din, acc0, bf16, sb), "conv_bwd_data");
            }
            break;
        }
        case PSW_OP_BN: {
            if (net->folded_now[i]) break;  // done by the dgrads of ops i+1 (sums) and i-1 (dy)
            const float* save = is.save(i);
            const Tensor r = o.in1 >= 0 ? net->t[o.in1] : Tensor{0, 0, 0, 0};
            float* dres = o.in1 > 0 ? is.grd(o.in1) : nullptr;
            float* dg = is.gptr(i);
            if (!din) {  // rejected when the net is created
                is.what = "BN directly on the input batch";
                return hipErrorInvalidValue;
            }
            kind = PSW_PROF_BN_BWD;
            bool done = false;
            if (net->gavg_of[i] >= 0 && net->gavg_pstat[i]) {  // from the forward's plane statistics
                PSW_TRY(psw::bn_bwd_gavg_from_stats(a.n, a.c, a.h, a.w, is.grd(net->gavg_of[i] + 1), is.pstat(i),
                                                    is.act(i + 1), is.act(o.in0), is.wbwd(i), save, save + o.cin,
                                                    (o.flags & PSW_F_RELU) != 0, g, din, dg, dg + o.cin, dres, sb),
                        "bn_bwd_gavg_from_stats");
                done = true;
            } else if (net->gavg_of[i] >= 0) {  // with the global average pool's backward: dh = the pool output's gradient
                PSW_TRY(psw::bn_bwd_gavg(a.n, a.c, a.h, a.w, is.grd(net->gavg_of[i] + 1), is.act(i + 1),
                                         is.act(o.in0), is.wbwd(i), save, save + o.cin,
                                         (o.flags & PSW_F_RELU) != 0, g, din, dg, dg + o.cin, dres, sb),
                        "bn_bwd_gavg");
                done = true;
            }
            if (!done && i + 1 < L && net->fused_bwd_now[i + 1]) {  // sums written by the next conv's dgrad into ws
                const psw_layer& cv = net->ops[i + 1];
                psw::ConvShape ccs;
                check_conv(y.n, y.c, y.h, y.w, cv.cout, cv.k, cv.k, cv.stride, cv.pad, net->prec, &ccs);
                const int T = psw::conv_bwd_data_bnsums_tiles(ccs);
                // without a residual the ReLU mask comes from y and the forward's scale / shift
                const float* scale = o.in1 < 0 ? save + 2 * o.cin : nullptr;
                e = psw::bn_bwd_from_partials(a.n, a.c, a.h, a.w, g, is.act(i + 1), is.act(o.in0), is.wbwd(i), save,
                                              save + o.cin, scale, (const float*)ws, T, (o.flags & PSW_F_RELU) != 0,
                                              din, dg, dg + o.cin, dres, r.c, r.h, r.w, net->grad_accum[2 * i + 1], sb);
                if (e == hipSuccess)
                    done = true;
                else if (e != hipErrorNotSupported)  // not supported: nothing launched, sums recomputed below
                    PSW_TRY(e, "bn_bwd_from_partials");
            }
            if (!done && is.on_load(i)) {  // excluded when the net was created: bn_bwd reads the BN output
                is.what = "BN applied on load: backward sums not fused into its consumer's dgrad";
                return hipErrorNotSupported;
            }
            if (!done)
                PSW_TRY(psw::bn_bwd(a.n, a.c, a.h, a.w, g, is.act(i + 1), is.act(o.in0), is.wbwd(i), save,
                                    save + o.cin, (o.flags & PSW_F_RELU) != 0, din, dg, dg + o.cin, dres, r.c, r.h,
                                    r.w, net->grad_accum[2 * i + 1], ws, wsb, sb),
                        "bn_bwd");
            break;
        }
        case PSW_OP_MAXPOOL:
            kind = PSW_PROF_POOL;
            if (din)
                PSW_TRY(psw::maxpool_bwd(a.n, a.c, a.h, a.w, o.k, o.stride, g, (const int32_t*)is.save(i), din, acc0,
                                         sb),
                        "maxpool_bwd");
            break;
        case PSW_OP_GAVG:
            kind = PSW_PROF_POOL;
            if (net->gavg_fused[i]) break;  // in its BN's backward kernel (bn_bwd_gavg)
            if (din) PSW_TRY(psw::gavgpool_bwd(a.n, a.c, a.h, a.w, g, din, acc0, sb), "gavgpool_bwd");
            break;
        case PSW_OP_DROPOUT:  // the mask of this step's forward pass, recomputed
            kind = PSW_PROF_OTHER;
            if (din)
                PSW_TRY(psw::dropout_apply(y.numel(), g, din, acc0, o.k, net->dropout_seed, (uint32_t)i, io.t, sb),
                        "dropout");
            break;
        case PSW_OP_FC: {
            kind = PSW_PROF_OTHER;
            if (o.flags & PSW_F_RELU) PSW_TRY(psw::relu_mask(y.numel(), is.act(i + 1), g, sb), "relu_mask");
            float* dw = is.gptr(i);
            float* db = (o.flags & PSW_F_BIAS) ? dw + (int64_t)o.cout * o.cin : nullptr;
            kind = PSW_PROF_FC;
            PSW_TRY(psw::fc_bwd(a.n, o.cin, o.cout, is.act(o.in0), is.wbwd(i), g, din, acc0, dw, db, bf16, ws, wsb,
                                sb),
                    "fc_bwd");
            break;
        }
        }
        const int s = net->stage_of[i];
        if (i == net->stage_begin[s]) {
            // the chain is done with stage s: its weight gradients (from the
            // step's activations and the now final output gradients) and its
            // update run on sw, beside the chain's next stage; a stage
            // without convs is updated on the chain's stream itself
            const hipStream_t su = net->stage_has_conv[s] ? sw : sb;
            if (su != sb) {
                PSW_TRY(hipEventRecord(net->stage_ev[s], sb), "stage join");
                PSW_TRY(hipStreamWaitEvent(sw, net->stage_ev[s], 0), "stage join");
            }
            // consecutive convs of one shape whose partial sums the update
            // reduces share a launch (each keeps its own operands and sums)
            const float* gx[psw::kWgradGroupMax];
            const float* gdy[psw::kWgradGroupMax];
            const float* gbn[psw::kWgradGroupMax];  // input BN applied on load, else null
            float* gpart[psw::kWgradGroupMax];
            int gn = 0;
            psw::ConvShape gcs{};
            auto flush = [&]() -> hipError_t {
                if (gn == 0) return hipSuccess;
                kind = PSW_PROF_CONV_BWD_WEIGHT;
                const int m = gn;
                gn = 0;
                return psw::conv_bwd_weight_partials_group(gcs, gx, gdy, gpart, m, bf16, sw, gbn);
            };
            for (int j = net->stage_end[s] - 1; j >= net->stage_begin[s]; --j) {
                const psw_layer& c = net->ops[j];
                if (c.kind != PSW_OP_CONV) continue;
                const Tensor ca = net->t[c.in0];
                psw::ConvShape ccs;
                check_conv(ca.n, ca.c, ca.h, ca.w, c.cout, c.k, c.k, c.stride, c.pad, net->prec, &ccs);
                float* dw = is.gptr(j);
                float* db = (c.flags & PSW_F_BIAS) ? dw + (int64_t)c.cout * c.cin * c.k * c.k : nullptr;
                if (net->wpart_splits[j] > 0) {  // reduced by the stage update below
                    if (gn > 0 && (gn == psw::kWgradGroupMax || memcmp(&gcs, &ccs, sizeof ccs) != 0))
                        PSW_TRY(flush(), "conv_bwd_weight");
                    gcs = ccs;
                    const int bj = c.in0 - 1;  // input from a BN applied on load: its input and scale / shift
                    const bool ibn = bj >= 1 && is.on_load(bj);
                    gx[gn] = ibn ? is.act(net->ops[bj].in0) : is.act(c.in0);
                    gbn[gn] = ibn ? is.save(bj) + 2 * net->ops[bj].cin : nullptr;
                    gdy[gn] = is.grd(j + 1);
                    gpart[gn] = is.wpart(j);
                    ++gn;
                } else {
                    PSW_TRY(flush(), "conv_bwd_weight");
                    kind = PSW_PROF_CONV_BWD_WEIGHT;
                    PSW_TRY(psw::conv_bwd_weight(ccs, is.act(c.in0), is.grd(j + 1), dw, db, bf16, wsw, wswb, sw),
                            "conv_bwd_weight");
                }
            }
            PSW_TRY(flush(), "conv_bwd_weight");
            kind = PSW_PROF_SGD;
            psw::SgdSeg segs[64];
            const auto& proto = net->sgd_segs[s];
            for (size_t q0 = 0; q0 < proto.size(); q0 += 64) {
                const int m = (int)std::min<size_t>(64, proto.size() - q0);
                for (int q = 0; q < m; ++q) {
                    const auto& pr = proto[q0 + q];
                    segs[q] = {pr.off, pr.count, pr.op >= 0 ? is.wpart(pr.op) : nullptr,
                               pr.op >= 0 ? net->wpart_splits[pr.op] : 0};
                }
                PSW_TRY(psw::sgd_stage(segs, m, slot_ptr(net, s, io.t), slot_ptr(net, s, io.t + 1),
                                       net->momentum + net->flat_off[s], io.gbase + net->flat_off[s], io.lr[s], io.mom,
                                       io.wd, io.nesterov, su),
                        "sgd");
            }
            PSW_TRY(after_update(s, su), "update event");
        }
    }
    return hipSuccess;
}

#undef PSW_TRY

struct RecorderScope {
    explicit RecorderScope(psw::KernelRecorder* r) { psw::kernel_recorder() = r; }
    ~RecorderScope() { psw::kernel_recorder() = nullptr; }
};

}  // namespace

extern "C" {

int psw_stage_step(psw_net* net, int64_t t, const int32_t* staleness, const float* lr, float mom, float wd,
                   int nesterov, const float* x, const int32_t* labels, float* loss_out, int32_t* versions_out,
                   void* stream)
{
    if (!net) return fail(PSW_ERR_NULL, "stage_step: net is NULL");
    if (!net->bound) return fail(PSW_ERR_STATE, "stage_step: net is not bound");
    if (!lr || !x || !labels || !loss_out) return fail(PSW_ERR_NULL, "stage_step: required pointer is NULL");
    int rc = check_staleness(net, t, staleness);
    if (rc) return rc;
    if (t != net->next_t)
        return fail(PSW_ERR_STEP_ORDER, "stage_step: expected t = %lld, got %lld", (long long)net->next_t, (long long)t);
    hipStream_t st = S(stream);
    StepIO io{t, std::vector<int64_t>(net->S), net->arena, x, labels, loss_out, lr, mom, wd, nesterov, net->grad};
    for (int s = 0; s < net->S; ++s) io.rv[s] = fwd_version(t, staleness[s]);
    Issue is{net, io};
    net->rec.kind = PSW_PROF_OTHER;
    RecorderScope rec_scope(net->profiling ? &net->rec : nullptr);
    // forward and the data-gradient chain on the caller's stream; weight
    // gradients and updates on the side stream, joined back at the end (also
    // when a launcher fails part way)
    hipError_t e = issue_forward(is, st, [](int) { return hipSuccess; });
    if (e == hipSuccess)
        e = issue_backward(is, st, net->side, [](int) { return hipSuccess; },
                           [](int, hipStream_t) { return hipSuccess; });
    hipError_t ej = hipEventRecord(net->join_ev, net->side);
    if (ej == hipSuccess) ej = hipStreamWaitEvent(st, net->join_ev, 0);
    if (e != hipSuccess) return hip_check(e, is.what);
    if (ej != hipSuccess) return hip_check(ej, "join");
    if (versions_out)
        for (int s = 0; s < net->S; ++s) versions_out[s] = (int32_t)io.rv[s];
    net->next_t = t + 1;
    return PSW_OK;
}

int psw_net_pipeline_bytes(const psw_net* net, int64_t* bytes)
{
    if (!net || !bytes) return fail(PSW_ERR_NULL, "net_pipeline_bytes: required pointer is NULL");
    *bytes = (int64_t)net->step_bytes;
    return PSW_OK;
}

int psw_net_bind_pipeline(psw_net* net, void* step_set, size_t bytes)
{
    if (!net || !step_set) return fail(PSW_ERR_NULL, "net_bind_pipeline: required pointer is NULL");
    if (!net->bound) return fail(PSW_ERR_STATE, "net_bind_pipeline: bind the net first");
    if (bytes < net->step_bytes)
        return fail(PSW_ERR_WORKSPACE, "net_bind_pipeline: %zu < %zu bytes", bytes, net->step_bytes);
    const int extra = (int)std::min<size_t>(bytes / net->step_bytes, psw_net::kMaxSets - 1);
    if (((uintptr_t)step_set) % 256 != 0) return fail(PSW_ERR_SHAPE, "net_bind_pipeline: must be 256-byte aligned");
    if (!net->fwd) {
        hipError_t e = hipStreamCreateWithFlags(&net->fwd, hipStreamNonBlocking);
        if (e != hipSuccess) {
            net->fwd = nullptr;
            return hip_check(e, "net_bind_pipeline: forward stream");
        }
        int D = 1;
        for (int d : net->ring_depth) D = std::max(D, d);
        net->upd_q = D + 1;
        net->upd_ev.assign((size_t)net->S * net->upd_q, nullptr);
        std::vector<hipEvent_t*> evs;
        for (auto& ev : net->upd_ev) evs.push_back(&ev);
        for (auto& ev : net->wdone_ev) evs.push_back(&ev);
        evs.push_back(&net->fdone_ev);
        evs.push_back(&net->start_ev);
        for (hipEvent_t* ev : evs) {
            e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
            if (e != hipSuccess) return hip_check(e, "net_bind_pipeline: events");
        }
    }
    net->sets[0] = net->arena;
    for (int k = 0; k < extra; ++k) net->sets[1 + k] = (char*)step_set + (size_t)k * net->step_bytes;
    net->nsets = 1 + extra;
    return PSW_OK;
}

}  // extern "C"

namespace {

// Issues steps t0 .. t0+n_steps-1 as a pipeline joined into sb (validated
// by the caller).  Returns a PSW status; *issued = steps fully issued.
int issue_pipeline(psw_net* net, int64_t t0, int n_steps, const int32_t* staleness, const float* lr, float mom,
                   float wd, int nesterov, const float* x, const int32_t* labels, int n_batches, float* losses,
                   int32_t* versions_out, hipStream_t sb, int64_t* issued)
{
    hipStream_t sf = net->fwd, sw = net->side;
    const Tensor in = net->t[0];
    const size_t xs = (size_t)in.numel();
    const int S_ = net->S, Q = net->upd_q;
    *issued = 0;
    // everything the caller enqueued before (inputs, earlier versions) comes first
    hipError_t e = hipEventRecord(net->start_ev, sb);
    if (e == hipSuccess) e = hipStreamWaitEvent(sf, net->start_ev, 0);
    if (e == hipSuccess) e = hipStreamWaitEvent(sw, net->start_ev, 0);
    if (e != hipSuccess) return hip_check(e, "pipeline: start");
    const char* what = "";
    for (int i = 0; i < n_steps && e == hipSuccess; ++i) {
        const int64_t t = t0 + i;
        const int NS = net->nsets;
        const int p = (int)(t % NS);
        hipEvent_t wdone = net->wdone_ev[p];
        char* P = net->sets[p];
        StepIO io{t, std::vector<int64_t>(S_), P, x + (size_t)(i % n_batches) * xs,
                  labels + (size_t)(i % n_batches) * in.n, losses + i, lr + (size_t)i * S_, mom, wd, nesterov,
                  (float*)(P + net->pgrad_off)};
        for (int s = 0; s < S_; ++s) io.rv[s] = fwd_version(t, staleness[(size_t)i * S_ + s]);
        Issue is{net, io};
        // forward of t: its step set is free once step t-NS is done with it
        // (the weight stream's last update of a step follows the chain's end)
        if (i >= NS) {
            e = hipStreamWaitEvent(sf, wdone, 0);
            if (e != hipSuccess) {
                what = "pipeline: step set";
                break;
            }
        }
        // stage s reads version r = rv[s]; wait for the update that wrote it
        // when it was written inside this run
        // (the weight stream runs in order, so the wait for step t-NS above
        // already covers every update of steps <= t-NS)
        e = issue_forward(is, sf, [&](int s) -> hipError_t {
            const int64_t r = io.rv[s];
            if (r - 1 < t0 || (i >= NS && r - 1 <= t - NS && net->stage_has_conv[s])) return hipSuccess;
            return hipStreamWaitEvent(sf, net->upd_ev[(size_t)s * Q + (size_t)(r % Q)], 0);
        });
        if (e != hipSuccess) {
            what = is.what;
            break;
        }
        // backward of t after its forward
        e = hipEventRecord(net->fdone_ev, sf);
        if (e == hipSuccess) e = hipStreamWaitEvent(sb, net->fdone_ev, 0);
        if (e != hipSuccess) {
            what = "pipeline: backward order";
            break;
        }
        // stage s of backward t reads version t (written by the update of step
        // t-1 on the weight stream) unless it stashes; the forward's waits
        // already cover d_s = 0 and stashing (both read the version r_s)
        e = issue_backward(
            is, sb, sw,
            [&](int s) -> hipError_t {
                if (net->stash || t - 1 < t0 || io.rv[s] == t || !net->stage_has_conv[s]) return hipSuccess;
                return hipStreamWaitEvent(sb, net->upd_ev[(size_t)s * Q + (size_t)(t % Q)], 0);
            },
            [&](int s, hipStream_t su) -> hipError_t {
                return hipEventRecord(net->upd_ev[(size_t)s * Q + (size_t)((t + 1) % Q)], su);
            });
        if (e != hipSuccess) {
            what = is.what;
            break;
        }
        // the chain's end reaches the weight stream through stage 0's weight
        // gradients; a stage 0 without convs (no work on sw) is joined here
        if (!net->stage_has_conv[0]) {
            e = hipEventRecord(net->stage_ev[0], sb);
            if (e == hipSuccess) e = hipStreamWaitEvent(sw, net->stage_ev[0], 0);
        }
        if (e == hipSuccess) e = hipEventRecord(wdone, sw);
        if (e != hipSuccess) {
            what = "pipeline: step done";
            break;
        }
        if (versions_out)
            for (int s = 0; s < S_; ++s) versions_out[(size_t)i * S_ + s] = (int32_t)io.rv[s];
        ++*issued;
    }
    // join: sb waits for the forward and weight streams
    hipError_t ej = hipEventRecord(net->join_ev, sw);
    if (ej == hipSuccess) ej = hipStreamWaitEvent(sb, net->join_ev, 0);
    if (ej == hipSuccess) ej = hipEventRecord(net->fdone_ev, sf);
    if (ej == hipSuccess) ej = hipStreamWaitEvent(sb, net->fdone_ev, 0);
    if (e != hipSuccess) return hip_check(e, what);
    if (ej != hipSuccess) return hip_check(ej, "pipeline: join");
    return PSW_OK;
}

int check_pipeline_args(const psw_net* net, int64_t t0, int n_steps, const int32_t* staleness, const float* lr,
                        const float* x, const int32_t* labels, int n_batches, const float* losses, const char* who)
{
    if (!net) return fail(PSW_ERR_NULL, "%s: net is NULL", who);
    if (!net->bound || net->nsets < 2) return fail(PSW_ERR_STATE, "%s: bind the net and its pipeline sets first", who);
    if (!staleness || !lr || !x || !labels || !losses) return fail(PSW_ERR_NULL, "%s: required pointer is NULL", who);
    if (n_steps < 0 || n_batches < 1) return fail(PSW_ERR_SHAPE, "%s: n_steps >= 0 and n_batches >= 1", who);
    for (int i = 0; i < n_steps; ++i) {
        int rc = check_staleness(net, t0 + i, staleness + (size_t)i * net->S);
        if (rc) return rc;
    }
    return PSW_OK;
}

int64_t gcd64(int64_t a, int64_t b) { return b ? gcd64(b, a % b) : a; }

// period of the per-step buffers: ring slots (t mod D_s) and step sets (t mod nsets)
int64_t replay_period(const psw_net* net)
{
    int64_t p = net->nsets;
    for (int d : net->ring_depth) p = p / gcd64(p, d) * d;
    return p;
}

}  // namespace

struct psw_graph {
    psw_net* net = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    int64_t t0 = 0, period = 1;
    int n_steps = 0;
    ~psw_graph()
    {
        if (exec) (void)hipGraphExecDestroy(exec);
        if (graph) (void)hipGraphDestroy(graph);
    }
};

extern "C" {

int psw_pipeline_run(psw_net* net, int64_t t0, int n_steps, const int32_t* staleness, const float* lr, float mom,
                     float wd, int nesterov, const float* x, const int32_t* labels, int n_batches, float* losses,
                     int32_t* versions_out, void* stream)
{
    int rc = check_pipeline_args(net, t0, n_steps, staleness, lr, x, labels, n_batches, losses, "pipeline_run");
    if (rc) return rc;
    if (t0 != net->next_t)
        return fail(PSW_ERR_STEP_ORDER, "pipeline_run: expected t0 = %lld, got %lld", (long long)net->next_t,
                    (long long)t0);
    if (n_steps == 0) return PSW_OK;
    net->rec.kind = PSW_PROF_OTHER;
    RecorderScope rec_scope(net->profiling ? &net->rec : nullptr);
    int64_t issued = 0;
    rc = issue_pipeline(net, t0, n_steps, staleness, lr, mom, wd, nesterov, x, labels, n_batches, losses,
                        versions_out, S(stream), &issued);
    net->next_t = t0 + issued;
    return rc;
}

int psw_pipeline_capture(psw_net* net, int n_steps, const int32_t* staleness, const float* lr, float mom, float wd,
                         int nesterov, const float* x, const int32_t* labels, int n_batches, float* losses,
                         psw_graph** out)
{
    if (!out) return fail(PSW_ERR_NULL, "pipeline_capture: out is NULL");
    *out = nullptr;
    const int64_t t0 = net ? net->next_t : 0;
    int rc = check_pipeline_args(net, t0, n_steps, staleness, lr, x, labels, n_batches, losses, "pipeline_capture");
    if (rc) return rc;
    for (const psw_layer& o : net->ops)  // a replay would repeat the captured steps' masks
        if (o.kind == PSW_OP_DROPOUT)
            return fail(PSW_ERR_UNSUPPORTED, "pipeline_capture: dropout masks depend on the step; run nets with "
                        "dropout with psw_pipeline_run");
    const int64_t period = replay_period(net);
    if (n_steps <= 0 || n_steps % period != 0)
        return fail(PSW_ERR_SHAPE, "pipeline_capture: n_steps must be a positive multiple of %lld", (long long)period);
    for (int i = 0; i < n_steps; ++i)
        for (int s = 0; s < net->S; ++s)
            if (t0 + i - staleness[(size_t)i * net->S + s] < 0)
                return fail(PSW_ERR_STALENESS, "pipeline_capture: step %lld clamps its version at 0 (pipeline fill); "
                            "run the fill with psw_pipeline_run first", (long long)(t0 + i));
    psw_graph* g = new psw_graph;
    g->net = net;
    g->t0 = t0;
    g->period = period;
    g->n_steps = n_steps;
    hipStream_t cap = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&cap, hipStreamNonBlocking);
    if (e != hipSuccess) {
        delete g;
        return hip_check(e, "pipeline_capture: stream");
    }
    RecorderScope rec_scope(nullptr);  // no per-kernel events inside a graph
    e = hipStreamBeginCapture(cap, hipStreamCaptureModeThreadLocal);
    int64_t issued = 0;
    if (e == hipSuccess)
        rc = issue_pipeline(net, t0, n_steps, staleness, lr, mom, wd, nesterov, x, labels, n_batches, losses, nullptr,
                            cap, &issued);
    hipGraph_t graph = nullptr;
    hipError_t ee = e == hipSuccess ? hipStreamEndCapture(cap, &graph) : e;
    (void)hipStreamDestroy(cap);
    g->graph = graph;
    if (e != hipSuccess || ee != hipSuccess || rc != PSW_OK) {
        delete g;
        if (rc != PSW_OK) return rc;
        return hip_check(e != hipSuccess ? e : ee, "pipeline_capture");
    }
    e = hipGraphInstantiate(&g->exec, graph, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        g->exec = nullptr;
        delete g;
        return hip_check(e, "pipeline_capture: instantiate");
    }
    *out = g;
    return PSW_OK;
}

int psw_graph_launch(psw_graph* g, void* stream)
{
    if (!g || !g->exec) return fail(PSW_ERR_NULL, "graph_launch: graph is NULL");
    psw_net* net = g->net;
    if ((net->next_t - g->t0) % g->period != 0 || net->next_t < g->t0)
        return fail(PSW_ERR_STEP_ORDER, "graph_launch: the net is at step %lld; this graph replays from steps "
                    "%lld + k*%lld", (long long)net->next_t, (long long)g->t0, (long long)g->period);
    hipError_t e = hipGraphLaunch(g->exec, S(stream));
    if (e != hipSuccess) return hip_check(e, "graph_launch");
    net->next_t += g->n_steps;
    return PSW_OK;
}

int psw_graph_destroy(psw_graph* g)
{
    delete g;
    return PSW_OK;
}

int psw_net_profile(psw_net* net, int enable)
{
    return psw_net_profile_only(net, enable, nullptr);
}

int psw_net_profile_replay(psw_net* net, int reps)
{
    if (!net) return fail(PSW_ERR_NULL, "net_profile_replay: net is NULL");
    if (reps < 1 || reps > 1000) return fail(PSW_ERR_SHAPE, "net_profile_replay: reps = %d outside [1, 1000]", reps);
    net->rec.replay = reps;
    return PSW_OK;
}

int psw_net_profile_only(psw_net* net, int enable, const char* kernel)
{
    if (!net) return fail(PSW_ERR_NULL, "net_profile: net is NULL");
    net->profiling = enable != 0;
    net->rec.only = kernel ? kernel : "";
    net->krecs.clear();
    net->ev_used = 0;
    return PSW_OK;
}

namespace {
hipError_t krec_ms(const psw_net::KRec& r, double* ms)
{
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return e;
    float t = 0.f;
    e = hipEventElapsedTime(&t, r.a, r.b);
    *ms = (double)t / r.reps;  // per launch
    return e;
}
}  // namespace

int psw_net_profile_read(psw_net* net, int n_kinds, double* ms, int64_t* launches)
{
    if (!net || !ms || !launches) return fail(PSW_ERR_NULL, "net_profile_read: required pointer is NULL");
    for (int k = 0; k < n_kinds; ++k) {
        ms[k] = 0.0;
        launches[k] = 0;
    }
    for (const auto& r : net->krecs) {
        double t = 0.0;
        hipError_t e = krec_ms(r, &t);
        if (e != hipSuccess) return hip_check(e, "net_profile_read");
        if (r.kind >= 0 && r.kind < n_kinds) {
            ms[r.kind] += t;
            launches[r.kind] += 1;
        }
    }
    return PSW_OK;
}

int psw_net_profile_timeline(psw_net* net, int cap, psw_kernel_span* out, int* n_out)
{
    if (!net || !n_out || (cap > 0 && !out)) return fail(PSW_ERR_NULL, "net_profile_timeline: required pointer is NULL");
    *n_out = (int)net->krecs.size();
    if (net->krecs.empty()) return PSW_OK;
    const psw_net::KRec& first = net->krecs.front();
    hipError_t e = hipEventSynchronize(net->krecs.back().b);
    if (e != hipSuccess) return hip_check(e, "net_profile_timeline");
    for (int i = 0; i < cap && i < (int)net->krecs.size(); ++i) {
        const psw_net::KRec& r = net->krecs[i];
        float t0 = 0.f, t1 = 0.f;
        e = hipEventSynchronize(r.b);
        if (e == hipSuccess) e = hipEventElapsedTime(&t0, first.a, r.a);
        if (e == hipSuccess) e = hipEventElapsedTime(&t1, first.a, r.b);
        if (e != hipSuccess) return hip_check(e, "net_profile_timeline");
        psw_kernel_span sp{};
        snprintf(sp.name, sizeof(sp.name), "%s", r.name.c_str());
        sp.kind = r.kind;
        sp.stream = r.stream;
        sp.start_us = 1e3 * t0;
        sp.end_us = 1e3 * t1;
        out[i] = sp;
    }
    return PSW_OK;
}

int psw_net_profile_kernels(psw_net* net, int cap, psw_kernel_stat* out, int* n_out)
{
    if (!net || !n_out || (cap > 0 && !out)) return fail(PSW_ERR_NULL, "net_profile_kernels: required pointer is NULL");
    std::vector<psw_kernel_stat> st;
    std::vector<std::string> names;
    for (const auto& r : net->krecs) {
        double t = 0.0;
        hipError_t e = krec_ms(r, &t);
        if (e != hipSuccess) return hip_check(e, "net_profile_kernels");
        size_t j = 0;
        while (j < names.size() && names[j] != r.name) ++j;
        if (j == names.size()) {
            names.push_back(r.name);
            psw_kernel_stat k{};
            snprintf(k.name, sizeof(k.name), "%s", r.name.c_str());
            k.kind = r.kind;
            st.push_back(k);
        }
        st[j].launches += 1;
        st[j].ms += t;
        st[j].flops += r.work.flops;
        st[j].bytes += r.work.bytes;
    }
    std::stable_sort(st.begin(), st.end(), [](const psw_kernel_stat& x, const psw_kernel_stat& y) { return x.ms > y.ms; });
    *n_out = (int)st.size();
    for (int i = 0; i < cap && i < (int)st.size(); ++i) out[i] = st[i];
    return PSW_OK;
}

}  // extern "C"
