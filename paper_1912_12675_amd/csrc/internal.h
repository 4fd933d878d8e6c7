// Internal launchers of libpsw (not part of the public C ABI).
// All tensors are NCHW float32 in device memory; conv weights are KCRS.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

namespace psw {

// ---- streaming stores ----------------------------------------------------
// Large outputs that later kernels read back (activations, gradients, split
// partial sums) are stored non-temporally: they stream to memory while the
// kernel runs instead of staying dirty in the XCD's L2, which the end of a
// kernel would otherwise write back before the next one starts.
__device__ __forceinline__ void store_stream(float* p, float v) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ void store_stream2(float* p, float2 v)
{
    typedef float f2v __attribute__((ext_vector_type(2)));
    __builtin_nontemporal_store(f2v{v.x, v.y}, reinterpret_cast<f2v*>(p));
}
__device__ __forceinline__ void store_stream4(float* p, float4 v)
{
    typedef float f4v __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(f4v{v.x, v.y, v.z, v.w}, reinterpret_cast<f4v*>(p));
}

// ---- kernel timing hook -------------------------------------------------
// While a recorder is installed on the calling thread (the scheduler does so
// in its profiling mode), every kernel the library launches is timed with a
// start / stop event pair and reported with its name (template arguments
// spelled as the compiler prints them) and its algorithmic work: the
// floating-point operations and the minimal HBM bytes (each input read once,
// each output written once) of what the kernel computes.  begin() decides
// how: *reps == 1 launches the kernel once with hipExtLaunchKernelGGL and the
// pair stamped from its own dispatch; *reps > 1 replays it: the pair is
// recorded on the stream around reps back-to-back launches of the same
// kernel with the same arguments (the recorder has waited for the device to
// be idle first, so the kernel runs alone).
struct Work {
    double flops;
    double bytes;
};

class KernelRecorder {
public:
    // false: do not time this launch; else *start / *stop are the events and
    // *reps (1 on entry) the number of back-to-back launches between them
    virtual bool begin(const std::string& name, hipEvent_t* start, hipEvent_t* stop, int* reps) = 0;
    virtual void end(std::string&& name, const Work& w, hipEvent_t start, hipEvent_t stop, int reps,
                     hipStream_t st) = 0;

protected:
    ~KernelRecorder() = default;
};

KernelRecorder*& kernel_recorder();  // this thread's recorder, nullptr when off

inline void kname_arg(std::string& s, int v) { s += std::to_string(v); }
inline void kname_arg(std::string& s, bool v) { s += v ? "true" : "false"; }
template <typename... T>
std::string kname(const char* base, T... v)
{
    std::string s = base;
    if constexpr (sizeof...(v) > 0) {
        s += '<';
        bool first = true;
        ((s += first ? "" : ", ", first = false, kname_arg(s, v)), ...);
        s += '>';
    }
    return s;
}

#define PSW_LAUNCH(NAME, WORK, KERNEL, GRID, BLOCK, SHMEM, STREAM, ...)                              \
    do {                                                                                          \
        ::psw::KernelRecorder* psw_rec_ = ::psw::kernel_recorder();                               \
        hipEvent_t psw_e0_ = nullptr, psw_e1_ = nullptr;                                          \
        int psw_reps_ = 1;                                                                        \
        std::string psw_name_;                                                                    \
        if (psw_rec_) {                                                                           \
            psw_name_ = NAME;                                                                     \
            if (!psw_rec_->begin(psw_name_, &psw_e0_, &psw_e1_, &psw_reps_)) psw_rec_ = nullptr;  \
        }                                                                                         \
        if (psw_rec_ && psw_reps_ > 1) {                                                          \
            (void)hipEventRecord(psw_e0_, STREAM);                                                \
            for (int psw_i_ = 0; psw_i_ < psw_reps_; ++psw_i_)                                    \
                hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, __VA_ARGS__);              \
            (void)hipEventRecord(psw_e1_, STREAM);                                                \
        } else if (psw_rec_) {                                                                    \
            hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, psw_e0_, psw_e1_, 0, __VA_ARGS__); \
        } else {                                                                                  \
            hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, __VA_ARGS__);                  \
        }                                                                                         \
        if (psw_rec_) psw_rec_->end(std::move(psw_name_), WORK, psw_e0_, psw_e1_, psw_reps_, STREAM); \
    } while (0)

constexpr double kF = 4.0;  // bytes per float

struct ConvShape {
    int n, c, h, w;        // input
    int k, r, s;           // output channels, kernel
    int stride, pad;
    int p, q;              // output spatial size
};

inline int conv_out_dim(int in, int k, int stride, int pad) { return (in + 2 * pad - k) / stride + 1; }

// algorithmic work of one pass of a convolution (the three passes have the
// same multiply-add count); bytes: x, w and y once each
inline Work conv_work(int n, int c, int h, int w, int k, int r, int s, int p, int q)
{
    return Work{2.0 * n * p * q * (double)k * c * r * s, kF * ((double)n * c * h * w + (double)k * c * r * s + (double)n * k * p * q)};
}
inline Work conv_work(const ConvShape& cs) { return conv_work(cs.n, cs.c, cs.h, cs.w, cs.k, cs.r, cs.s, cs.p, cs.q); }

// Batch-norm statistics fused into a convolution's epilogue: every workgroup
// writes the (mean, M2) of each of its output channels over its P pixels to
// part[channel][tile][2]; bn_apply_from_partials merges them.
struct BnStatsFuse {
    float* part;
};

// Batch-norm backward sums fused into the epilogue of the backward-data
// kernel that produces dz (the gradient of the BN output): with
// g = dz * [z > 0] (relu) or dz and xhat = (y - mean) * invstd, every
// workgroup writes (sum g, sum g*xhat) of each channel over its pixels to
// part[channel][tile][2]; bn_bwd_from_partials merges them.
// For a BN without residual the ReLU mask is recomputed from y instead of
// read from z: z > 0 exactly when fmaf(y, scale, shift) > 0 with the
// forward's own per-channel scale and shift (the forward evaluates that
// same fused multiply-add), so scale != nullptr means z is not read.
struct BnBwdFuse {
    float* part;
    const float* z;       // BN output (its ReLU mask); unused when scale is set
    const float* y;       // BN input
    const float* mean;
    const float* invstd;
    int relu;
    const float* scale = nullptr;  // forward scale / shift (BN without residual)
    const float* shift = nullptr;
};

// Backward of a BN without residual folded into the staging of the
// backward-data conv that reads its result.  Every workgroup first merges the
// BN's per-tile sums part[c][T][2] (written by the next conv's backward-data
// epilogue, see BnBwdFuse) in a fixed order in fp64 into, per channel,
// a = gamma*invstd, b = mean g', d = mean g'*xhat (workgroup 0 also writes
// dbeta = sum g' and dgamma = sum g'*xhat); then the conv's input
// dy = a*(g' - b - xhat*d) is formed per element while staging, from the BN
// output gradient g (g' = g masked by the ReLU, the mask recomputed as
// fmaf(y, scale, shift) > 0) and the BN input y, xhat = (y - mean)*invstd.
// The rows a workgroup owns are also written to dy, which the weight
// gradient reads.  For a BN with an identity residual (dres set) the ReLU
// mask is z > 0 with z the BN output, and g' is written to dres (the
// residual's gradient, overwritten).  The channel count must be a power of
// two.
struct BnFold {
    const float* g = nullptr;
    const float* y = nullptr;
    const float* part = nullptr;
    int T = 0;                     // tiles (partials per channel)
    double count = 0.0;            // elements per channel, n*h*w
    const float* gamma = nullptr;
    const float* mean = nullptr;
    const float* invstd = nullptr;
    const float* scale = nullptr;  // shift at scale + c; read when relu is set
    int relu = 0;
    float* dy = nullptr;
    float* dgamma = nullptr;
    float* dbeta = nullptr;
    const float* z = nullptr;      // BN output (residual BN only)
    float* dres = nullptr;         // residual's gradient (residual BN only)
};
constexpr int kFoldMaxChannels = 128;
// largest input of a forward conv that applies its input's BN while loading
constexpr int kInBnMaxChannels = 128;

// ---- convolution (implicit GEMM on MFMA) ----
// Forward conv + fused BN statistics (direct kernel only); returns
// hipErrorNotSupported when the shape has no direct configuration.
// in_bn (may be null): see conv_fwd.
hipError_t conv_fwd_bnstats(const ConvShape& cs, const float* x, const float* w, float* y, const BnStatsFuse& bn,
                            size_t part_capacity_floats, int bf16, hipStream_t st, const float* in_bn = nullptr);
size_t conv_fwd_bnstats_part_floats(const ConvShape& cs);
int conv_fwd_bnstats_tiles(const ConvShape& cs);  // tiles T (partials per channel), 0 if not fused
// BN forward (+residual, +ReLU) whose statistics come as per-tile (mean, M2)
// partials over P pixels each: every block merges its channel's T partials
// in a fixed order (double precision), block 0 of a channel stores the saved
// statistics and running statistics, and every block normalises its part.
// pool: when set (an 8x8 output that only a global average pool reads), the
// per-(image, channel) means of the output are written there as well;
// hipErrorNotSupported (nothing launched) unless h * w == 64.  pstat (with
// pool only): per (image, channel) the number of elements where the ReLU
// passed and the sum of xhat = (y - mean) * invstd over them, [n][c][2].
hipError_t bn_apply_from_partials(int n, int c, int h, int w, const float* y, const float* part, int T, int P,
                                  const float* gamma, const float* beta, const float* res, int rc, int rh, int rw,
                                  int relu, float eps, float momentum, float* z, float* save_mean, float* save_invstd,
                                  float* save_scale, float* run_mean, float* run_var, hipStream_t st,
                                  float* pool = nullptr, float* pstat = nullptr);
// The statistics of bn_apply_from_partials alone (saved mean, invstd, scale
// and shift, running statistics; the same values bit for bit), for a BN
// whose output is never stored because its one consumer applies it while
// loading (DirArgs::in_bn, the weight gradient's in_bn).  save_scale is
// required.
hipError_t bn_stats_from_partials(int c, const float* part, int T, int P, const float* gamma, const float* beta,
                                  float eps, float momentum, float* save_mean, float* save_invstd, float* save_scale,
                                  float* run_mean, float* run_var, hipStream_t st);
// Direct 3x3 / pad 1 kernel (forward, or backward-data of a stride-1 layer
// when transpose is set); hipErrorNotSupported when no tile config fits.
// bf16: both operands rounded to bfloat16 (nearest even), fp32 accumulation.
hipError_t conv3x3_direct(int n, int C, int H, int W, int K, int stride, const float* x, const float* w, float* y,
                          int accumulate, bool transpose, hipStream_t st, const BnStatsFuse* bn = nullptr,
                          const BnBwdFuse* bnb = nullptr, const BnFold* fold = nullptr, bool bf16 = false,
                          const float* in_bn = nullptr);
// whether conv3x3_direct takes the shape (same arguments)
bool conv3x3_direct_covers(int n, int C, int H, int W, int K, int stride, bool transpose);
// number of pixel tiles (workgroups along x) of the direct forward kernel, 0 if none
int conv3x3_direct_tiles(int n, int C, int H, int W, int K, int stride);
// Backward-data of a 3x3 / pad 1 / stride 2 conv (layer channels CL in, KL
// out, input H x W); hipErrorNotSupported when no tile config fits.
hipError_t conv3x3_dgrad_s2(int n, int CL, int H, int W, int KL, const float* w, const float* dy, float* dx,
                            int accumulate, hipStream_t st, const BnBwdFuse* bnb = nullptr, bool bf16 = false);
int dgrad_bnsums_tiles(int n, int CL, int H, int W, int KL, int stride);
// Backward data with the preceding BN's backward sums fused (direct kernel
// or stride-2 kernel only); tiles = partials per channel, 0 if not fused.
int conv_bwd_data_bnsums_tiles(const ConvShape& cs);
hipError_t conv_bwd_data_bnsums(const ConvShape& cs, const float* w, const float* dy, float* dx, int accumulate,
                                const BnBwdFuse& bnb, int bf16, hipStream_t st);
// Backward data whose input is formed from the preceding BN's folded
// backward (stride-1 direct kernel only; conv_bwd_data_fold_ok says
// whether the shape is covered); bnb, if set, as for conv_bwd_data_bnsums.
bool conv_bwd_data_fold_ok(const ConvShape& cs);
hipError_t conv_bwd_data_fold(const ConvShape& cs, const float* w, float* dx, int accumulate, const BnBwdFuse* bnb,
                              const BnFold& fold, int bf16, hipStream_t st);
// BN backward (+ residual) from per-tile (sum g, sum g*xhat) partials:
// merges them in a fixed order, writes dgamma, dbeta (block 0 of a channel)
// and dy, and dres for an identity or option-A (2x subsampled, zero-padded
// channels) residual.  scale (scale[c], shift[c] after it) replaces z for
// the ReLU mask of a BN without residual.  hipErrorNotSupported (nothing
// launched) for other residual shapes or misaligned operands.
hipError_t bn_bwd_from_partials(int n, int c, int h, int w, const float* dz, const float* z, const float* y,
                                const float* gamma, const float* mean, const float* invstd, const float* scale,
                                const float* part, int T, int relu, float* dy, float* dgamma, float* dbeta,
                                float* dres, int rc, int rh, int rw, int res_accumulate, hipStream_t st);
// Backward-weight partial sums of a 3x3 / pad 1 conv (dW-shaped, one per
// workgroup); conv3x3_wgrad_splits is 0 when no configuration covers it.
int conv3x3_wgrad_splits(int n, int C, int H, int W, int K, int stride);
hipError_t conv3x3_wgrad(int n, int C, int H, int W, int K, int stride, const float* x, const float* dy, float* part,
                         hipStream_t st, bool bf16 = false);
// The same for `count` (<= kWgradGroupMax) convolutions of one shape in one
// launch: member i reads x[i], dy[i] and writes its partial sums to part[i].
constexpr int kWgradGroupMax = 8;
// in_bn (may be null, else one pointer per member, each may be null): see
// the in_bn of WgArgs.
hipError_t conv3x3_wgrad_group(int n, int C, int H, int W, int K, int stride, const float* const* x,
                               const float* const* dy, float* const* part, int count, hipStream_t st,
                               bool bf16 = false, const float* const* in_bn = nullptr);
// in_bn (may be null): x is the raw input of a BN + ReLU whose output is not
// stored, in_bn its per-channel scale [c] and shift [c] (DirArgs::in_bn);
// only the direct kernel takes it (conv_fwd_in_bn_ok), otherwise
// hipErrorNotSupported with nothing launched.
hipError_t conv_fwd(const ConvShape& cs, const float* x, const float* w, const float* bias, int relu,
                    float* y, int bf16, hipStream_t st, const float* in_bn = nullptr);
// whether conv_fwd / conv_fwd_bnstats take an in_bn for this shape (no bias,
// no ReLU)
bool conv_fwd_in_bn_ok(const ConvShape& cs);
hipError_t conv_bwd_data(const ConvShape& cs, const float* w, const float* dy, float* dx, int accumulate,
                         int bf16, hipStream_t st);
size_t conv_bwd_weight_ws_bytes(const ConvShape& cs, int bf16);
hipError_t conv_bwd_weight(const ConvShape& cs, const float* x, const float* dy, float* dw, float* db,
                           int bf16, void* ws, size_t ws_bytes, hipStream_t st);
// Weight gradient left as split partial sums part[z][k*c*r*s], z < splits,
// for a consumer that reduces them (sgd_stage): splits = 0 when the shape has
// no split form, and then conv_bwd_weight_partials returns
// hipErrorNotSupported without launching.
int conv_bwd_weight_part_splits(const ConvShape& cs, int bf16);
hipError_t conv_bwd_weight_partials(const ConvShape& cs, const float* x, const float* dy, float* part, int bf16,
                                    hipStream_t st);
// The same for `count` convolutions of shape cs in one launch; in_bn (may be
// null): per member, null or the scale / shift of a BN + ReLU applied to x
// on load (conv3x3_wgrad_group).
hipError_t conv_bwd_weight_partials_group(const ConvShape& cs, const float* const* x, const float* const* dy,
                                          float* const* part, int count, int bf16, hipStream_t st,
                                          const float* const* in_bn = nullptr);

// ---- batch norm (+ residual) (+ ReLU) ----
size_t bn_ws_bytes(int n, int c, int h, int w);
hipError_t bn_fwd(int n, int c, int h, int w, const float* y, const float* gamma, const float* beta,
                  const float* res, int rc, int rh, int rw, int relu, float eps, float momentum, float* z,
                  float* save_mean, float* save_invstd, float* run_mean, float* run_var, void* ws,
                  size_t ws_bytes, hipStream_t st, float* save_scale = nullptr);
hipError_t bn_bwd(int n, int c, int h, int w, const float* dz, const float* z, const float* y,
                  const float* gamma, const float* save_mean, const float* save_invstd, int relu, float* dy,
                  float* dgamma, float* dbeta, float* dres, int rc, int rh, int rw, int res_accumulate,
                  void* ws, size_t ws_bytes, hipStream_t st);

// Backward of a BN whose output is read only by a global average pool, with
// that pool's backward: dh [n][c] is the pooled output's gradient; writes the
// BN output's gradient dz (dh / (h w) at every pixel), dy, dgamma, dbeta and,
// for an identity residual, its gradient (overwritten: the BN must be its
// first writer).  One workgroup per channel; hipErrorNotSupported (nothing
// launched) unless h w % 4 == 0 and the tensors are 16-byte aligned.
hipError_t bn_bwd_gavg(int n, int c, int h, int w, const float* dh, const float* z, const float* y,
                       const float* gamma, const float* mean, const float* invstd, int relu, float* dz, float* dy,
                       float* dgamma, float* dbeta, float* dres, hipStream_t st);
// bn_bwd_gavg from the plane statistics the forward stored (pstat of
// bn_apply_from_partials: per (image, channel) the ReLU-pass count and the
// sum of xhat there): one elementwise pass over many workgroups per channel.
hipError_t bn_bwd_gavg_from_stats(int n, int c, int h, int w, const float* dh, const float* pstat, const float* z,
                                  const float* y, const float* gamma, const float* mean, const float* invstd, int relu,
                                  float* dz, float* dy, float* dgamma, float* dbeta, float* dres, hipStream_t st);

// ---- pooling ----
hipError_t maxpool_fwd(int n, int c, int h, int w, int k, int stride, const float* x, float* y,
                       int32_t* argmax, hipStream_t st);
hipError_t maxpool_bwd(int n, int c, int h, int w, int k, int stride, const float* dy,
                       const int32_t* argmax, float* dx, int accumulate, hipStream_t st);
hipError_t gavgpool_fwd(int n, int c, int h, int w, const float* x, float* y, hipStream_t st);
hipError_t gavgpool_bwd(int n, int c, int h, int w, const float* dy, float* dx, int accumulate,
                        hipStream_t st);

// ---- fully connected (GEMM on MFMA) ----
// Small FC as the last layer: logits, mean softmax cross-entropy and its
// gradient in one launch; hipErrorNotSupported (nothing launched) when the
// layer is not small.
hipError_t fc_softmax_xent(int n, int in, int out, const float* x, const float* w, const float* b, float* logits,
                           int bf16, const int32_t* labels, float* loss, float* dlogits, hipStream_t st);
hipError_t fc_fwd(int n, int in, int out, const float* x, const float* w, const float* b, int relu, float* y,
                  int bf16, hipStream_t st);
size_t fc_bwd_ws_bytes(int n, int in, int out);
hipError_t fc_bwd(int n, int in, int out, const float* x, const float* w, const float* dy, float* dx,
                  int dx_accumulate, float* dw, float* db, int bf16, void* ws, size_t ws_bytes,
                  hipStream_t st);

// ---- misc ----
hipError_t relu_mask(int64_t count, const float* z, float* g, hipStream_t st);
hipError_t softmax_xent(int n, int classes, const float* logits, const int32_t* labels, float* loss,
                        float* dlogits, hipStream_t st);
hipError_t sgd_momentum(int64_t count, const float* w_in, float* w_out, float* v, const float* g, float lr,
                        float mom, float wd, int nesterov, hipStream_t st);
// One SGD-momentum update over a stage's packed parameters, described as
// segments [off, off + count) (offsets relative to w_in / w_out / v / g).  A
// segment with part != nullptr takes its gradient as the sum of `splits`
// partial sums part[z][i] (z ascending within each of 16 residue classes
// z mod 16, then the 16 class sums in order, as the split reduction of
// conv_bwd_weight adds them) and also writes that sum to g; other segments
// read g.
struct SgdSeg {
    int64_t off, count;
    const float* part;
    int32_t splits;
};
hipError_t sgd_stage(const SgdSeg* segs, int nseg, const float* w_in, float* w_out, float* v, float* g, float lr,
                     float mom, float wd, int nesterov, hipStream_t st);
hipError_t channel_sum(int n, int c, int hw, const float* x, float* out, void* ws, size_t ws_bytes,
                       hipStream_t st);
// Dropout with counter-based masks (Philox4x32-10): out (+)= keep * in * scale
// over n floats, the mask of operation `op` at step t under `seed`, drop
// probability p24 / 2^24 (0 < p24 < 2^24); the same call with the gradients
// is the backward pass.
hipError_t dropout_apply(int64_t n, const float* in, float* out, int accumulate, int p24, uint64_t seed, uint32_t op,
                         int64_t t, hipStream_t st);
size_t channel_sum_ws_bytes(int n, int c, int hw);

}  // namespace psw
