// Batch norm (+residual, +ReLU), pooling, fully-connected GEMMs, softmax
// cross-entropy and the SGD-momentum update for gfx950.
//
// Reductions (BN statistics, BN backward sums, bias gradients, the loss) are
// deterministic: every partial sum has a fixed owner and partials are
// combined in a fixed order; BN sums are accumulated in double so the
// E[y^2]-E[y]^2 form loses nothing at these sizes.
#include <algorithm>

#include "internal.h"

namespace psw {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef unsigned short v8us __attribute__((ext_vector_type(8)));

constexpr int kBlock = 256;

__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, 64);
    return v;
}

__device__ __forceinline__ float wave_sum_f(float v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, 64);
    return v;
}

// Sum over the block in a fixed order; result valid in thread 0.
__device__ __forceinline__ double block_sum(double v, double* sh)
{
    v = wave_sum(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) sh[wave] = v;
    __syncthreads();
    double t = 0.0;
    if (threadIdx.x == 0)
        for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += sh[i];
    __syncthreads();
    return t;
}

// Two sums over the block at once, fixed order; results valid in thread 0.
__device__ __forceinline__ void block_sum2(double& a, double& b, double* sh)
{
    a = wave_sum(a);
    b = wave_sum(b);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = (int)(blockDim.x >> 6);
    if (lane == 0) {
        sh[wave] = a;
        sh[nw + wave] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double ta = 0.0, tb = 0.0;
        for (int i = 0; i < nw; ++i) {
            ta += sh[i];
            tb += sh[nw + i];
        }
        a = ta;
        b = tb;
    }
    __syncthreads();
}

int channel_splits(int n, int c)
{
    int sp = (1024 + c - 1) / c;
    if (sp > n) sp = n;
    if (sp < 1) sp = 1;
    return sp;
}

// ---------------------------------------------------------------- BN -------
// mode 0: sum y, sum y^2              (forward statistics)
// mode 1: sum g, sum g*xhat with g = dz*[z>0 if relu]   (backward sums)
// mode 2: sum x                       (bias gradient; second slot unused)
__global__ __launch_bounds__(kBlock) void chan_partials(int mode, int n, int c, int hw, int split, const float* x,
                                                         const float* z, const float* y, const float* mean,
                                                         const float* invstd, int relu, double* part)
{
    __shared__ double sh[kBlock / 64];
    const int ch = blockIdx.x, sp = blockIdx.y;
    const int i0 = (int)((int64_t)n * sp / split), i1 = (int)((int64_t)n * (sp + 1) / split);
    const int64_t total = (int64_t)(i1 - i0) * hw;
    double s1 = 0.0, s2 = 0.0;
    const double mu = mode == 1 ? (double)mean[ch] : 0.0;
    const double is = mode == 1 ? (double)invstd[ch] : 0.0;
    for (int64_t idx = threadIdx.x; idx < total; idx += kBlock) {
        const int img = i0 + (int)(idx / hw);
        const int off = (int)(idx - (int64_t)(img - i0) * hw);
        const size_t g = ((size_t)img * c + ch) * hw + off;
        const double v = x[g];
        if (mode == 0) {
            s1 += v;
            s2 += v * v;
        } else if (mode == 1) {
            const double gg = (relu && !(z[g] > 0.f)) ? 0.0 : v;
            s1 += gg;
            s2 += gg * ((double)y[g] - mu) * is;
        } else {
            s1 += v;
        }
    }
    s1 = block_sum(s1, sh);
    s2 = block_sum(s2, sh);
    if (threadIdx.x == 0) {
        part[((size_t)ch * split + sp) * 2 + 0] = s1;
        part[((size_t)ch * split + sp) * 2 + 1] = s2;
    }
}

__global__ void bn_fwd_finalize(int c, int split, double count, const double* part, const float* gamma,
                                const float* beta, float eps, float momentum, float* save_mean, float* save_invstd,
                                float* run_mean, float* run_var, float* coef, float* save_scale)
{
    const int ch = blockIdx.x * blockDim.x + threadIdx.x;
    if (ch >= c) return;
    double s1 = 0.0, s2 = 0.0;
    for (int sp = 0; sp < split; ++sp) {
        s1 += part[((size_t)ch * split + sp) * 2 + 0];
        s2 += part[((size_t)ch * split + sp) * 2 + 1];
    }
    const double mean = s1 / count;
    double var = s2 / count - mean * mean;
    if (var < 0.0) var = 0.0;
    const double invstd = 1.0 / sqrt(var + (double)eps);
    save_mean[ch] = (float)mean;
    save_invstd[ch] = (float)invstd;
    if (run_mean) run_mean[ch] = (float)((1.0 - momentum) * run_mean[ch] + momentum * mean);
    if (run_var)
        run_var[ch] = (float)((1.0 - momentum) * run_var[ch] +
                              momentum * (count > 1.0 ? var * count / (count - 1.0) : var));
    const double scale = (double)gamma[ch] * invstd;
    coef[2 * ch + 0] = (float)scale;
    coef[2 * ch + 1] = (float)((double)beta[ch] - mean * scale);
    if (save_scale) {
        save_scale[ch] = coef[2 * ch + 0];
        save_scale[c + ch] = coef[2 * ch + 1];
    }
}

__global__ void bn_fwd_apply(int64_t total, int c, int hw, const float* y, const float* coef, const float* res,
                             int rc, int rh, int rw, int h, int w, int relu, float* z)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int64_t nc = i / hw;
    const int ch = (int)(nc % c);
    float v = __fmaf_rn(y[i], coef[2 * ch], coef[2 * ch + 1]);
    if (res) {
        if (rc == c && rh == h && rw == w) {
            v += res[i];
        } else {
            const int lo = (c - rc) / 2, cc = ch - lo;
            if (cc >= 0 && cc < rc) {
                const int img = (int)(nc / c), off = (int)(i - nc * hw);
                const int hh = off / w, ww = off - hh * w;
                v += res[(((size_t)img * rc + cc) * rh + hh * (rh / h)) * rw + ww * (rw / w)];
            }
        }
    }
    if (relu) v = fmaxf(v, 0.f);
    z[i] = v;
}

__global__ void bn_bwd_finalize(int c, int split, double count, const double* part, const float* gamma,
                                const float* invstd, float* dgamma, float* dbeta, float* coef)
{
    const int ch = blockIdx.x * blockDim.x + threadIdx.x;
    if (ch >= c) return;
    double s1 = 0.0, s2 = 0.0;
    for (int sp = 0; sp < split; ++sp) {
        s1 += part[((size_t)ch * split + sp) * 2 + 0];
        s2 += part[((size_t)ch * split + sp) * 2 + 1];
    }
    dbeta[ch] = (float)s1;
    dgamma[ch] = (float)s2;
    coef[3 * ch + 0] = (float)((double)gamma[ch] * (double)invstd[ch]);
    coef[3 * ch + 1] = (float)(s1 / count);
    coef[3 * ch + 2] = (float)(s2 / count);
}

__global__ void bn_bwd_apply(int64_t total, int c, int hw, const float* dz, const float* z, const float* y,
                             const float* mean, const float* invstd, const float* coef, int relu, float* dy,
                             float* dres_identity, int res_accumulate)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int ch = (int)((i / hw) % c);
    const float g = (relu && !(z[i] > 0.f)) ? 0.f : dz[i];
    const float xh = (y[i] - mean[ch]) * invstd[ch];
    dy[i] = coef[3 * ch] * (g - coef[3 * ch + 1] - xh * coef[3 * ch + 2]);
    if (dres_identity) dres_identity[i] = res_accumulate ? dres_identity[i] + g : g;
}

// option-A shortcut backward: dres[n][cr][hr][wr] gets g[n][cr+lo][hr/sh][wr/sw]
// at subsampled positions and zero elsewhere
__global__ void shortcut_a_bwd(int64_t total, int c, int h, int w, int rc, int rh, int rw, const float* dz,
                               const float* z, int relu, float* dres, int accumulate)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int rhw = rh * rw;
    const int64_t ncr = i / rhw;
    const int off = (int)(i - ncr * rhw);
    const int cr = (int)(ncr % rc), img = (int)(ncr / rc);
    const int hr = off / rw, wr = off - hr * rw;
    const int sh = rh / h, sw = rw / w;
    float g = 0.f;
    if (hr % sh == 0 && wr % sw == 0) {
        const int ch = cr + (c - rc) / 2;
        const size_t j = (((size_t)img * c + ch) * h + hr / sh) * w + wr / sw;
        g = (relu && !(z[j] > 0.f)) ? 0.f : dz[j];
    }
    dres[i] = accumulate ? dres[i] + g : g;
}

__global__ void chan_sum_finalize(int c, int split, const double* part, float* out)
{
    const int ch = blockIdx.x * blockDim.x + threadIdx.x;
    if (ch >= c) return;
    double s = 0.0;
    for (int sp = 0; sp < split; ++sp) s += part[((size_t)ch * split + sp) * 2];
    out[ch] = (float)s;
}

// -------------------------------------------------------------- pooling ----
__global__ void maxpool_fwd_k(int64_t total, int h, int w, int p, int q, int k, int stride, const float* x,
                              float* y, int32_t* argmax)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int64_t nc = i / ((int64_t)p * q);
    const int pq = (int)(i - nc * p * q);
    const int pp = pq / q, qq = pq - pp * q;
    const float* xp = x + nc * h * w;
    float best = 0.f;
    int bi = -1;
    for (int r = 0; r < k; ++r)
        for (int s = 0; s < k; ++s) {
            const int ih = pp * stride + r, iw = qq * stride + s;
            const float v = xp[ih * w + iw];
            if (bi < 0 || v > best) {
                best = v;
                bi = ih * w + iw;
            }
        }
    y[i] = best;
    argmax[i] = bi;
}

// non-overlapping windows (k == stride): each input element belongs to at
// most one window, so the backward pass is a gather with no conflicts
__global__ void maxpool_bwd_k(int64_t total, int h, int w, int p, int q, int k, const float* dy,
                              const int32_t* argmax, float* dx, int accumulate)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int64_t nc = i / ((int64_t)h * w);
    const int hw = (int)(i - nc * h * w);
    const int ih = hw / w, iw = hw - ih * w;
    const int pp = ih / k, qq = iw / k;
    float g = 0.f;
    if (pp < p && qq < q) {
        const int64_t o = nc * p * q + pp * q + qq;
        if (argmax[o] == hw) g = dy[o];
    }
    dx[i] = accumulate ? dx[i] + g : g;
}

__global__ void gavg_fwd_k(int64_t planes, int hw, const float* x, float* y)
{
    const int64_t plane = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (plane >= planes) return;
    float s = 0.f;
    for (int i = lane; i < hw; i += 64) s += x[plane * hw + i];
    s = wave_sum_f(s);
    if (lane == 0) y[plane] = s / (float)hw;
}

__global__ void gavg_bwd_k(int64_t total, int hw, const float* dy, float* dx, int accumulate)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const float g = dy[i / hw] / (float)hw;
    dx[i] = accumulate ? dx[i] + g : g;
}

// Backward of a BN whose output feeds only a global average pool (the last
// BN of a CIFAR ResNet): the pool's gradient dh[n][c] / hw is the BN output's
// gradient at every pixel of (n, c), so one workgroup per channel forms the
// channel's sums  sum g', sum g' xhat  (g' = that gradient where the ReLU
// passed, z > 0; double, each thread's elements in order, then the block in
// a fixed order), and a second pass over the channel (now in L2) writes
// dy = gamma invstd (g' - sum g' / M - xhat sum g' xhat / M), the pool's
// gradient dz (so every tensor's gradient stays readable) and the identity
// residual's gradient g' (its first writer).  One launch replaces
// the pool backward, the sums, their finalisation and the apply.
__global__ __launch_bounds__(kBlock) void bn_bwd_gavg_k(int n, int c, int hw, const float* dh, const float* z,
                                                         const float* y, const float* gamma, const float* mean,
                                                         const float* invstd, int relu, float* dz, float* dy,
                                                         float* dgamma, float* dbeta, float* dres)
{
    __shared__ double sh[2 * kBlock / 64];
    __shared__ float coef[3];
    const int ch = blockIdx.x;
    const int hw4 = hw >> 2, units = n * hw4;
    const float mu = mean[ch], is = invstd[ch];
    const double mud = (double)mu, isd = (double)is;
    double s1 = 0.0, s2 = 0.0;
#pragma unroll 4
    for (int u = threadIdx.x; u < units; u += kBlock) {
        const int img = u / hw4, off = (u - img * hw4) * 4;
        const size_t i = ((size_t)img * c + ch) * hw + off;
        const float g = dh[(size_t)img * c + ch] / (float)hw;
        const float4 yv = *reinterpret_cast<const float4*>(y + i);
        const float4 zv = *reinterpret_cast<const float4*>(z + i);
        const float yy[4] = {yv.x, yv.y, yv.z, yv.w}, zz[4] = {zv.x, zv.y, zv.z, zv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const double gg = (relu && !(zz[e] > 0.f)) ? 0.0 : (double)g;
            s1 += gg;
            s2 += gg * ((double)yy[e] - mud) * isd;
        }
    }
    block_sum2(s1, s2, sh);
    if (threadIdx.x == 0) {
        const double cnt = (double)n * hw;
        coef[0] = (float)((double)gamma[ch] * isd);
        coef[1] = (float)(s1 / cnt);
        coef[2] = (float)(s2 / cnt);
        dbeta[ch] = (float)s1;
        dgamma[ch] = (float)s2;
    }
    __syncthreads();
    const float a = coef[0], b = coef[1], d = coef[2];
#pragma unroll 4
    for (int u = threadIdx.x; u < units; u += kBlock) {
        const int img = u / hw4, off = (u - img * hw4) * 4;
        const size_t i = ((size_t)img * c + ch) * hw + off;
        const float g = dh[(size_t)img * c + ch] / (float)hw;
        const float4 yv = *reinterpret_cast<const float4*>(y + i);
        const float4 zv = *reinterpret_cast<const float4*>(z + i);
        const float yy[4] = {yv.x, yv.y, yv.z, yv.w}, zz[4] = {zv.x, zv.y, zv.z, zv.w};
        float o[4], gm[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            gm[e] = (relu && !(zz[e] > 0.f)) ? 0.f : g;
            const float xh = (yy[e] - mu) * is;
            o[e] = a * (gm[e] - b - xh * d);
        }
        store_stream4(dz + i, make_float4(g, g, g, g));
        store_stream4(dy + i, make_float4(o[0], o[1], o[2], o[3]));
        if (dres) store_stream4(dres + i, make_float4(gm[0], gm[1], gm[2], gm[3]));
    }
}

// The same backward from the plane statistics the forward's apply kernel
// stored (per image and channel: the number of pixels where the ReLU passed
// and the sum of xhat there): with the pool's gradient g = dh / hw uniform
// over a plane, sum g' = sum_n g_n cnt_n and sum g' xhat = sum_n g_n sx_n,
// so the channel's sums come from 2n numbers and one elementwise pass
// remains, spread over many workgroups per channel (grid (c, blocks per
// channel), U float4 per thread).
template <int U>
__global__ __launch_bounds__(kBlock) void bn_bwd_gavg_stats_k(int n, int c, int hw, const float* dh,
                                                               const float* pstat, const float* z, const float* y,
                                                               const float* gamma, const float* mean,
                                                               const float* invstd, int relu, float* dz, float* dy,
                                                               float* dgamma, float* dbeta, float* dres)
{
    __shared__ double sh[2 * kBlock / 64];
    __shared__ float coef[3];
    const int ch = blockIdx.x;
    const int hw4 = hw >> 2, units = n * hw4;
    const int u0 = blockIdx.y * (U * kBlock), u1 = min(u0 + U * kBlock, units);
    // the elements first (their latency passes under the sums)
    size_t idx[U];
    float4 yv[U], zv[U];
    float gq[U];
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const int u = u0 + (int)threadIdx.x + q * kBlock;
        idx[q] = 0;
        yv[q] = zv[q] = make_float4(0.f, 0.f, 0.f, 0.f);
        gq[q] = 0.f;
        if (u < u1) {
            const int img = u / hw4, off = (u - img * hw4) * 4;
            idx[q] = ((size_t)img * c + ch) * hw + off;
            yv[q] = *reinterpret_cast<const float4*>(y + idx[q]);
            zv[q] = *reinterpret_cast<const float4*>(z + idx[q]);
            gq[q] = dh[(size_t)img * c + ch] / (float)hw;
        }
    }
    double s1 = 0.0, s2 = 0.0;
    for (int img = threadIdx.x; img < n; img += kBlock) {
        const double g = (double)(dh[(size_t)img * c + ch] / (float)hw);
        s1 += g * (double)pstat[((size_t)img * c + ch) * 2 + 0];
        s2 += g * (double)pstat[((size_t)img * c + ch) * 2 + 1];
    }
    block_sum2(s1, s2, sh);
    const float mu = mean[ch], is = invstd[ch];
    if (threadIdx.x == 0) {
        const double cnt = (double)n * hw;
        coef[0] = (float)((double)gamma[ch] * (double)is);
        coef[1] = (float)(s1 / cnt);
        coef[2] = (float)(s2 / cnt);
        if (blockIdx.y == 0) {
            dbeta[ch] = (float)s1;
            dgamma[ch] = (float)s2;
        }
    }
    __syncthreads();
    const float a = coef[0], b = coef[1], d = coef[2];
#pragma unroll
    for (int q = 0; q < U; ++q) {
        if (u0 + (int)threadIdx.x + q * kBlock >= u1) continue;
        const float g = gq[q];
        const float yy[4] = {yv[q].x, yv[q].y, yv[q].z, yv[q].w}, zz[4] = {zv[q].x, zv[q].y, zv[q].z, zv[q].w};
        float o[4], gm[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            gm[e] = (relu && !(zz[e] > 0.f)) ? 0.f : g;
            const float xh = (yy[e] - mu) * is;
            o[e] = a * (gm[e] - b - xh * d);
        }
        store_stream4(dz + idx[q], make_float4(g, g, g, g));
        store_stream4(dy + idx[q], make_float4(o[0], o[1], o[2], o[3]));
        if (dres) store_stream4(dres + idx[q], make_float4(gm[0], gm[1], gm[2], gm[3]));
    }
}

// -------------------------------------------------------------- misc -------
__global__ void relu_mask_k(int64_t count, const float* z, float* g)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count && !(z[i] > 0.f)) g[i] = 0.f;
}

__global__ __launch_bounds__(kBlock) void softmax_xent_k(int n, int classes, const float* logits,
                                                          const int32_t* labels, float* loss, float* dlogits)
{
    __shared__ double sh[kBlock / 64];
    double part = 0.0;
    for (int row = threadIdx.x; row < n; row += kBlock) {
        const float* z = logits + (size_t)row * classes;
        float mx = z[0];
        for (int j = 1; j < classes; ++j) mx = fmaxf(mx, z[j]);
        float se = 0.f;
        for (int j = 0; j < classes; ++j) se += expf(z[j] - mx);
        const float lse = mx + logf(se);
        const int lab = labels[row];
        part += (double)(lse - z[lab]);
        for (int j = 0; j < classes; ++j)
            dlogits[(size_t)row * classes + j] = (expf(z[j] - lse) - (j == lab ? 1.f : 0.f)) / (float)n;
    }
    const double t = block_sum(part, sh);
    if (threadIdx.x == 0) loss[0] = (float)(t / n);
}

__device__ __forceinline__ void sgd_one(int64_t i, float gv, const float* w_in, float* w_out, float* v, float lr,
                                        float mom, float wd, int nesterov)
{
    const float w = w_in[i];
    const float d = gv + wd * w;
    const float vv = mom * v[i] + d;
    v[i] = vv;
    w_out[i] = w - lr * (nesterov ? d + mom * vv : vv);
}

__global__ void sgd_k(int64_t count, const float* w_in, float* w_out, float* v, const float* g, float lr, float mom,
                      float wd, int nesterov)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= count) return;
    sgd_one(i, g[i], w_in, w_out, v, lr, mom, wd, nesterov);
}

// Stage update with the split reduction of its conv weight gradients folded
// in.  A workgroup owns one segment's range: kSgdOut consecutive parameters
// (one 128-byte line) of a split segment, its kSgdGroups lane groups summing
// residue classes of the splits, or kSgdBlock parameters of a plain segment.
constexpr int kSgdBlock = 512, kSgdOut = 32, kSgdGroups = kSgdBlock / kSgdOut, kSgdMaxSegs = 48;
static_assert(kSgdGroups == 16, "split order: 16 residue classes");
struct SgdSegDev {
    int64_t off, count;
    const float* part;
    int32_t splits, first_block;
};
struct SgdSegs {
    SgdSegDev s[kSgdMaxSegs];
    int32_t n;
};

__global__ __launch_bounds__(kSgdBlock) void sgd_stage_k(SgdSegs segs, const float* w_in, float* w_out, float* v,
                                                         float* g, float lr, float mom, float wd, int nesterov)
{
    __shared__ float sh[kSgdGroups][kSgdOut + 1];
    // the block's segment: static indices only (kernel-argument loads)
    int64_t off = segs.s[0].off, count = segs.s[0].count;
    const float* part = segs.s[0].part;
    int splits = segs.s[0].splits, first = 0;
#pragma unroll
    for (int k = 1; k < kSgdMaxSegs; ++k)
        if (k < segs.n && (int)blockIdx.x >= segs.s[k].first_block) {
            off = segs.s[k].off;
            count = segs.s[k].count;
            part = segs.s[k].part;
            splits = segs.s[k].splits;
            first = segs.s[k].first_block;
        }
    const int b = blockIdx.x - first, tid = threadIdx.x;
    if (!part) {
        const int64_t i = (int64_t)b * kSgdBlock + tid;
        if (i < count) sgd_one(off + i, g[off + i], w_in, w_out, v, lr, mom, wd, nesterov);
        return;
    }
    const int o = tid % kSgdOut, zl = tid / kSgdOut;
    const int64_t i = (int64_t)b * kSgdOut + o;
    float acc = 0.f;
    if (i < count) {
        int z = zl;
        for (; z + 7 * kSgdGroups < splits; z += 8 * kSgdGroups) {
            float pv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) pv[u] = part[(int64_t)(z + u * kSgdGroups) * count + i];
#pragma unroll
            for (int u = 0; u < 8; ++u) acc += pv[u];
        }
        for (; z < splits; z += kSgdGroups) acc += part[(int64_t)z * count + i];
    }
    sh[zl][o] = acc;
    __syncthreads();
    if (zl == 0 && i < count) {
        float t = 0.f;
        for (int q = 0; q < kSgdGroups; ++q) t += sh[q][o];
        g[off + i] = t;
        sgd_one(off + i, t, w_in, w_out, v, lr, mom, wd, nesterov);
    }
}

// ------------------------------------------------------ FC GEMM (MFMA) -----
// C[m][n] = sum_k A(m,k) B(k,n); A(m,k) = A[m*sam + k*sak], B(k,n) = B[k*sbk + n*sbn]
struct GemmArgs {
    const float* A;
    const float* B;
    float* C;
    const float* bias;  // per column n (direct mode only)
    int M, N, K;
    int64_t sam, sak, sbk, sbn;
    int kchunk;
    int relu, accumulate;
    int partial;  // 1: write raw sums to C + z*M*N
};

__device__ __forceinline__ float round_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) != 0x7f800000u) u += 0x7fffu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xffff0000u);
}

template <int BM, int BN, int WM, int WN, bool BF16, bool AK, bool BKC>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a)
{
    constexpr int BK = BF16 ? 32 : 16;
    constexpr int KSTEP = BF16 ? 32 : 4;
    constexpr int TM = BM / WM / 16, TN = BN / WN / 16;
    __shared__ float As[BK][BM + 4];
    __shared__ float Bs[BK][BN + 4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int kbeg = blockIdx.z * a.kchunk;
    const int kend = min(a.K, kbeg + a.kchunk);
    v4f acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
#pragma unroll
        for (int e = 0; e < (BM * BK + 255) / 256; ++e) {
            const int idx = e * 256 + tid;
            if (idx < BM * BK) {
                int kk, mm;
                if (AK) { kk = idx % BK; mm = idx / BK; } else { mm = idx % BM; kk = idx / BM; }
                const int m = m0 + mm, k = k0 + kk;
                const float v = (m < a.M && k < kend) ? a.A[(int64_t)m * a.sam + (int64_t)k * a.sak] : 0.f;
                As[kk][mm] = BF16 ? round_bf16(v) : v;
            }
        }
#pragma unroll
        for (int e = 0; e < (BN * BK + 255) / 256; ++e) {
            const int idx = e * 256 + tid;
            if (idx < BN * BK) {
                int kk, nn;
                if (BKC) { kk = idx % BK; nn = idx / BK; } else { nn = idx % BN; kk = idx / BN; }
                const int n = n0 + nn, k = k0 + kk;
                const float v = (n < a.N && k < kend) ? a.B[(int64_t)k * a.sbk + (int64_t)n * a.sbn] : 0.f;
                Bs[kk][nn] = BF16 ? round_bf16(v) : v;
            }
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < BK; ks += KSTEP) {
            if constexpr (!BF16) {
                float af[TM], bfr[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) af[i] = As[ks + (lane >> 4)][wm * (BM / WM) + i * 16 + (lane & 15)];
#pragma unroll
                for (int j = 0; j < TN; ++j) bfr[j] = Bs[ks + (lane >> 4)][wn * (BN / WN) + j * 16 + (lane & 15)];
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bfr[j], acc[i][j], 0, 0, 0);
            } else {
                v8bf af[TM], bfr[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    v8us u;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        u[e] = (unsigned short)(__float_as_uint(
                                   As[ks + 8 * (lane >> 4) + e][wm * (BM / WM) + i * 16 + (lane & 15)]) >> 16);
                    af[i] = __builtin_bit_cast(v8bf, u);
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    v8us u;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        u[e] = (unsigned short)(__float_as_uint(
                                   Bs[ks + 8 * (lane >> 4) + e][wn * (BN / WN) + j * 16 + (lane & 15)]) >> 16);
                    bfr[j] = __builtin_bit_cast(v8bf, u);
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + wn * (BN / WN) + j * 16 + (lane & 15);
            if (n >= a.N) continue;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = m0 + wm * (BM / WM) + i * 16 + 4 * (lane >> 4) + v;
                if (m >= a.M) continue;
                float val = acc[i][j][v];
                if (a.partial) {
                    a.C[((int64_t)blockIdx.z * a.M + m) * a.N + n] = val;
                } else {
                    if (a.bias) val += a.bias[n];
                    if (a.relu) val = fmaxf(val, 0.f);
                    float* dst = a.C + (int64_t)m * a.N + n;
                    *dst = a.accumulate ? *dst + val : val;
                }
            }
        }
}

__global__ void gemm_reduce(const float* part, int splits, int M, int N, const float* bias, int relu, int accumulate,
                            float* C)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t count = (int64_t)M * N;
    if (i >= count) return;
    float v = 0.f;
    for (int z = 0; z < splits; ++z) v += part[(int64_t)z * count + i];
    if (bias) v += bias[i % N];
    if (relu) v = fmaxf(v, 0.f);
    C[i] = accumulate ? C[i] + v : v;
}

template <bool AK, bool BKC>
hipError_t gemm(GemmArgs a, int bf16, void* ws, size_t ws_bytes, hipStream_t st)
{
    constexpr int BM = 64, BN = 64;
    const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    const int BK = bf16 ? 32 : 16;
    int splits = 1;
    if (tiles < 512 && ws) {
        splits = (1024 + tiles - 1) / tiles;
        const int maxs = (a.K + 4 * BK - 1) / (4 * BK);  // at least four BK slices per split
        if (splits > maxs) splits = maxs;
        while (splits > 1 && (size_t)splits * a.M * a.N * sizeof(float) > ws_bytes) --splits;
        if (splits < 1) splits = 1;
    }
    const int per = (a.K + splits - 1) / splits;
    a.kchunk = ((per + BK - 1) / BK) * BK;
    splits = (a.K + a.kchunk - 1) / a.kchunk;
    if (splits < 1) splits = 1;
    float* out = a.C;
    const float* bias = a.bias;
    const int relu = a.relu, accum = a.accumulate;
    if (splits > 1) {
        a.partial = 1;
        a.C = (float*)ws;
    }
    dim3 grid((a.N + BN - 1) / BN, (a.M + BM - 1) / BM, splits);
    const Work gw{2.0 * a.M * a.N * (double)a.K, kF * ((double)a.M * a.K + (double)a.K * a.N + (double)a.M * a.N)};
    if (bf16)
        PSW_LAUNCH(kname("gemm_kernel", BM, BN, 2, 2, true, AK, BKC), gw, (gemm_kernel<BM, BN, 2, 2, true, AK, BKC>),
                   grid, dim3(256), 0, st, a);
    else
        PSW_LAUNCH(kname("gemm_kernel", BM, BN, 2, 2, false, AK, BKC), gw, (gemm_kernel<BM, BN, 2, 2, false, AK, BKC>),
                   grid, dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || splits == 1) return e;
    const int64_t count = (int64_t)a.M * a.N;
    PSW_LAUNCH(kname("gemm_reduce"), (Work{(double)splits * count, kF * (splits + 1.0 + accum) * count}), gemm_reduce,
               dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, (const float*)ws, splits,
                       a.M, a.N, bias, relu, accum, out);
    return hipGetLastError();
}

inline unsigned blocks_for(int64_t n, int b = kBlock) { return (unsigned)((n + b - 1) / b); }

// ------------------------------------------ small fully-connected layers --
// The classifier of the CIFAR nets (e.g. 128 x 64 -> 10) is far too small for
// the tiled GEMM: one launch per direction does it on the vector units, every
// sum in a fixed order (k, o or i ascending).  bf16 mode rounds both operands
// of every product, as the GEMM does.
constexpr int kHeadBlock = 1024;
constexpr int kSmallFcLogits = 4096;  // n*out (logits held in LDS)
constexpr int kFcMaxN = 256, kFcMaxOut = 64, kFcKC = 32, kFcKW = 16;

bool small_fc(int n, int in, int out)
{
    return n <= kFcMaxN && out <= kFcMaxOut && (int64_t)n * out <= kSmallFcLogits && in <= 4096;
}

// y[i][o] = sum_k x[i][k] w[o][k] (+ b[o]) (relu), k ascending, from LDS
// chunks of kFcKC columns; with labels: also the mean softmax cross-entropy
// and its gradient (as softmax_xent_k).  One workgroup.
__global__ __launch_bounds__(kHeadBlock) void fc_small_fwd_k(int n, int in, int out, const float* x, const float* w,
                                                             const float* b, int relu, int bf16, float* y,
                                                             const int32_t* labels, float* loss, float* dlogits)
{
    constexpr int KP = kFcKC + 1;
    __shared__ float xs[kFcMaxN * KP];
    __shared__ float ws[kFcMaxOut * KP];
    __shared__ float z[kSmallFcLogits];
    __shared__ double sh[kHeadBlock / 64];
    constexpr int Q = kSmallFcLogits / kHeadBlock;
    float acc[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) acc[q] = 0.f;
    // The next chunk's loads are issued before the current chunk's products.
    constexpr int RX = kFcMaxN * kFcKC / kHeadBlock, RW = kFcMaxOut * kFcKC / kHeadBlock;
    float vx[RX], vw[RW];
    auto load_chunk = [&](int k0) {
#pragma unroll
        for (int r = 0; r < RX; ++r) {
            const int idx = threadIdx.x + r * kHeadBlock, i = idx / kFcKC, k = k0 + idx % kFcKC;
            vx[r] = (i < n && k < in) ? x[(size_t)i * in + k] : 0.f;
        }
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const int idx = threadIdx.x + r * kHeadBlock, o = idx / kFcKC, k = k0 + idx % kFcKC;
            vw[r] = (o < out && k < in) ? w[(size_t)o * in + k] : 0.f;
        }
    };
    load_chunk(0);
    for (int k0 = 0; k0 < in; k0 += kFcKC) {
        __syncthreads();
#pragma unroll
        for (int r = 0; r < RX; ++r) {
            const int idx = threadIdx.x + r * kHeadBlock;
            xs[(idx / kFcKC) * KP + idx % kFcKC] = bf16 ? round_bf16(vx[r]) : vx[r];
        }
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const int idx = threadIdx.x + r * kHeadBlock;
            ws[(idx / kFcKC) * KP + idx % kFcKC] = bf16 ? round_bf16(vw[r]) : vw[r];
        }
        __syncthreads();
        if (k0 + kFcKC < in) load_chunk(k0 + kFcKC);
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int e = threadIdx.x + q * kHeadBlock;
            if (e < n * out) {
                const int i = e / out, o = e - (e / out) * out;
                const float* xr = xs + i * KP;
                const float* wr = ws + o * KP;
#pragma unroll 8
                for (int kk = 0; kk < kFcKC; ++kk) acc[q] = fmaf(xr[kk], wr[kk], acc[q]);
            }
        }
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int e = threadIdx.x + q * kHeadBlock;
        if (e < n * out) {
            float v = acc[q];
            if (b) v += b[e - (e / out) * out];
            if (relu) v = fmaxf(v, 0.f);
            y[e] = v;
            z[e] = v;
        }
    }
    if (!labels) return;
    __syncthreads();
    double part = 0.0;
    for (int row = threadIdx.x; row < n; row += kHeadBlock) {
        const float* zr = z + row * out;
        float mx = zr[0];
        for (int j = 1; j < out; ++j) mx = fmaxf(mx, zr[j]);
        float se = 0.f;
        for (int j = 0; j < out; ++j) se += expf(zr[j] - mx);
        const float lse = mx + logf(se);
        const int lab = labels[row];
        part += (double)(lse - zr[lab]);
        for (int j = 0; j < out; ++j)
            dlogits[(size_t)row * out + j] = (expf(zr[j] - lse) - (j == lab ? 1.f : 0.f)) / (float)n;
    }
    const double t = block_sum(part, sh);
    if (threadIdx.x == 0) loss[0] = (float)(t / n);
}

// Blocks [0, nbx): dx[i][k] (+)= sum_o dy[i][o] w[o][k], o ascending, one
// output per thread.  Blocks [nbx, nbx + nbw): dw[o][k] = sum_i dy[i][o]
// x[i][k], i ascending, for kFcKW columns k from LDS copies of dy and of those
// columns of x; the first of them also db[o] = sum_i dy[i][o].  Global loads
// are issued in batches before their values are used.
__global__ __launch_bounds__(kBlock) void fc_small_bwd_k(int n, int in, int out, const float* x, const float* w,
                                                         const float* dy, float* dx, int dx_accumulate, float* dw,
                                                         float* db, int bf16, int nbx)
{
    __shared__ float dys[kSmallFcLogits];
    __shared__ float xs[kFcMaxN * (kFcKW + 1)];
    const int bid = blockIdx.x, tid = threadIdx.x;
    if (bid < nbx) {
        const int64_t e = (int64_t)bid * kBlock + tid;
        if (e >= (int64_t)n * in) return;
        const int i = (int)(e / in), k = (int)(e - (e / in) * in);
        const float old = dx_accumulate ? dx[e] : 0.f;
        float acc = 0.f;
        constexpr int U = 8;
        for (int o0 = 0; o0 < out; o0 += U) {
            float g[U], wv[U];
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int o = o0 + j;
                g[j] = o < out ? dy[(size_t)i * out + o] : 0.f;
                wv[j] = o < out ? w[(size_t)o * in + k] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < U; ++j)
                if (o0 + j < out) acc = fmaf(bf16 ? round_bf16(g[j]) : g[j], bf16 ? round_bf16(wv[j]) : wv[j], acc);
        }
        dx[e] = dx_accumulate ? old + acc : acc;
        return;
    }
    const int k0 = (bid - nbx) * kFcKW;
    constexpr int RD = kSmallFcLogits / kBlock, RX = kFcMaxN * kFcKW / kBlock;
    float vd[RD], vx[RX];
#pragma unroll
    for (int r = 0; r < RD; ++r) {
        const int idx = tid + r * kBlock;
        vd[r] = idx < n * out ? dy[idx] : 0.f;
    }
#pragma unroll
    for (int r = 0; r < RX; ++r) {
        const int idx = tid + r * kBlock, i = idx / kFcKW, k = k0 + idx % kFcKW;
        vx[r] = (i < n && k < in) ? x[(size_t)i * in + k] : 0.f;
    }
#pragma unroll
    for (int r = 0; r < RD; ++r) dys[tid + r * kBlock] = vd[r];
#pragma unroll
    for (int r = 0; r < RX; ++r) {
        const int idx = tid + r * kBlock;
        xs[(idx / kFcKW) * (kFcKW + 1) + idx % kFcKW] = bf16 ? round_bf16(vx[r]) : vx[r];
    }
    __syncthreads();
    if (db && bid == nbx && tid < out) {
        float acc = 0.f;
        for (int i = 0; i < n; ++i) acc += dys[i * out + tid];
        db[tid] = acc;
    }
    for (int t = tid; t < out * kFcKW; t += kBlock) {
        const int o = t / kFcKW, kk = t % kFcKW, k = k0 + kk;
        if (k >= in) continue;
        float acc = 0.f;
        for (int i = 0; i < n; ++i) {
            const float g = dys[i * out + o];
            acc = fmaf(bf16 ? round_bf16(g) : g, xs[i * (kFcKW + 1) + kk], acc);
        }
        dw[(size_t)o * in + k] = acc;
    }
}



}  // namespace

// ------------------------------------------------------------ launchers -----
size_t channel_sum_ws_bytes(int n, int c, int hw)
{
    (void)hw;
    return (size_t)c * channel_splits(n, c) * 2 * sizeof(double);
}

hipError_t channel_sum(int n, int c, int hw, const float* x, float* out, void* ws, size_t ws_bytes, hipStream_t st)
{
    const int sp = channel_splits(n, c);
    if (ws_bytes < channel_sum_ws_bytes(n, c, hw)) return hipErrorInvalidValue;
    const double elems = (double)n * c * hw;
    PSW_LAUNCH(kname("chan_partials"), (Work{elems, kF * elems}), chan_partials, dim3(c, sp), dim3(kBlock), 0, st, 2,
               n, c, hw, sp, x, (const float*)nullptr, (const float*)nullptr, (const float*)nullptr,
               (const float*)nullptr, 0, (double*)ws);
    PSW_LAUNCH(kname("chan_sum_finalize"), (Work{(double)c * sp, 16.0 * c * sp + kF * c}), chan_sum_finalize,
               dim3(blocks_for(c)), dim3(kBlock), 0, st, c, sp, (const double*)ws, out);
    return hipGetLastError();
}

size_t bn_ws_bytes(int n, int c, int h, int w)
{
    (void)h; (void)w;
    return (size_t)c * channel_splits(n, c) * 2 * sizeof(double) + (size_t)c * 3 * sizeof(float) + 256;
}

hipError_t bn_fwd(int n, int c, int h, int w, const float* y, const float* gamma, const float* beta, const float* res,
                  int rc, int rh, int rw, int relu, float eps, float momentum, float* z, float* save_mean,
                  float* save_invstd, float* run_mean, float* run_var, void* ws, size_t ws_bytes, hipStream_t st,
                  float* save_scale)
{
    if (ws_bytes < bn_ws_bytes(n, c, h, w)) return hipErrorInvalidValue;
    const int sp = channel_splits(n, c);
    const int hw = h * w;
    double* part = (double*)ws;
    float* coef = (float*)((char*)ws + (size_t)c * sp * 2 * sizeof(double));
    const int64_t total = (int64_t)n * c * hw;
    PSW_LAUNCH(kname("chan_partials"), (Work{3.0 * total, kF * total}), chan_partials, dim3(c, sp), dim3(kBlock), 0, st,
               0, n, c, hw, sp, y, (const float*)nullptr, (const float*)nullptr, (const float*)nullptr,
               (const float*)nullptr, 0, part);
    PSW_LAUNCH(kname("bn_fwd_finalize"), (Work{2.0 * c * sp, 16.0 * c * sp + 6 * kF * c}), bn_fwd_finalize,
               dim3(blocks_for(c)), dim3(kBlock), 0, st, c, sp, (double)n * hw, (const double*)part, gamma, beta, eps,
               momentum, save_mean, save_invstd, run_mean, run_var, coef, save_scale);
    const double rbytes = res ? kF * (double)n * std::min(c, rc) * hw : 0.0;
    PSW_LAUNCH(kname("bn_fwd_apply"), (Work{3.0 * total, kF * 2.0 * total + rbytes}), bn_fwd_apply,
               dim3(blocks_for(total)), dim3(kBlock), 0, st, total, c, hw, y, (const float*)coef, res, rc, rh, rw, h, w,
               relu, z);
    return hipGetLastError();
}

hipError_t bn_bwd(int n, int c, int h, int w, const float* dz, const float* z, const float* y, const float* gamma,
                  const float* save_mean, const float* save_invstd, int relu, float* dy, float* dgamma,
                  float* dbeta, float* dres, int rc, int rh, int rw, int res_accumulate, void* ws, size_t ws_bytes,
                  hipStream_t st)
{
    if (ws_bytes < bn_ws_bytes(n, c, h, w)) return hipErrorInvalidValue;
    const int sp = channel_splits(n, c);
    const int hw = h * w;
    double* part = (double*)ws;
    float* coef = (float*)((char*)ws + (size_t)c * sp * 2 * sizeof(double));
    const int64_t total = (int64_t)n * c * hw;
    PSW_LAUNCH(kname("chan_partials"), (Work{5.0 * total, 3 * kF * total}), chan_partials, dim3(c, sp), dim3(kBlock), 0,
               st, 1, n, c, hw, sp, dz, z, y, save_mean, save_invstd, relu, part);
    PSW_LAUNCH(kname("bn_bwd_finalize"), (Work{2.0 * c * sp, 16.0 * c * sp + 7 * kF * c}), bn_bwd_finalize,
               dim3(blocks_for(c)), dim3(kBlock), 0, st, c, sp, (double)n * hw, (const double*)part, gamma, save_invstd,
               dgamma, dbeta, coef);
    const bool identity = dres && rc == c && rh == h && rw == w;
    PSW_LAUNCH(kname("bn_bwd_apply"),
               (Work{6.0 * total, kF * (4.0 + (identity ? 1.0 + res_accumulate : 0.0)) * total}), bn_bwd_apply,
               dim3(blocks_for(total)), dim3(kBlock), 0, st, total, c, hw, dz, z, y, save_mean, save_invstd,
               (const float*)coef, relu, dy, identity ? dres : (float*)nullptr, res_accumulate);
    if (dres && !identity) {
        const int64_t rtotal = (int64_t)n * rc * rh * rw;
        PSW_LAUNCH(kname("shortcut_a_bwd"), (Work{0.0, kF * ((1.0 + res_accumulate) * rtotal + 2.0 * n * rc * hw)}),
                   shortcut_a_bwd, dim3(blocks_for(rtotal)), dim3(kBlock), 0, st, rtotal, c, h, w, rc, rh, rw, dz, z,
                   relu, dres, res_accumulate);
    }
    return hipGetLastError();
}

namespace {
// Both kernels run on grid (c, blocks per channel): every block first merges
// its channel's T per-tile partials in a fixed order (so all blocks of a
// channel see bit-identical coefficients), then transforms its share of the
// channel's n*hw elements.  Element loops walk float4 units of one channel
// (unit u: image u / hw4, offset 4*(u % hw4)) with 32-bit index arithmetic.
// A block of either kernel covers U float4 units per thread of one channel;
// U is chosen per launch (apply_units_per_thread) so that small layers get
// more, shorter blocks.

// forward: tile partials (mean_t, M2_t over P pixels each), merged in one
// pass in double:
//   mean = (1/T) sum mean_t,  M2 = sum (M2_t + P mean_t^2) - T P mean^2
// (exact products of fp32 values; the double sums lose nothing that the
// fp32 tile statistics did not already round).  The element loads are
// issued before the merge so that the two memory latencies overlap, and
// every load precedes every store.  Block y == 0 also stores the channel's
// scale and shift, which the backward recomputes the ReLU mask from.
// Per-tile statistics of one channel held in registers by the BN kernels:
// thread t takes tiles t, t + kBlock, ... (the order of the sums), up to
// kMergeTilesPerThread of them; larger tables are read in the merge loop.
constexpr int kMergeTilesPerThread = 4;
__device__ __forceinline__ void load_tile_stats(const float* pp, int T, float2 (&pv)[kMergeTilesPerThread])
{
#pragma unroll
    for (int k = 0; k < kMergeTilesPerThread; ++k) {
        const int t = (int)threadIdx.x + k * kBlock;
        pv[k] = (t < T && T <= kMergeTilesPerThread * kBlock) ? *reinterpret_cast<const float2*>(pp + 2 * t)
                                                              : make_float2(0.f, 0.f);
    }
}

// the merge of one channel's T tile statistics (thread t: tiles t,
// t + kBlock, ... in order, from pv or, for larger tables, from pp; then the
// block in a fixed order), and thread 0's coefficients: coef = (scale,
// shift, mean, invstd) as stored; block y == 0 also stores the saved and
// running statistics
__device__ __forceinline__ void bn_merge_finish(const float* pp, int T, int P,
                                                const float2 (&pv)[kMergeTilesPerThread], double* sh, float* coef,
                                                int c, int ch, const float* gamma, const float* beta, float eps,
                                                float momentum, float* save_mean, float* save_invstd,
                                                float* save_scale, float* run_mean, float* run_var)
{
    double s1 = 0.0, s2 = 0.0;
    if (T <= kMergeTilesPerThread * kBlock) {
#pragma unroll
        for (int k = 0; k < kMergeTilesPerThread; ++k)
            if ((int)threadIdx.x + k * kBlock < T) {
                const double m = (double)pv[k].x;
                s1 += m;
                s2 += (double)pv[k].y + (double)P * m * m;
            }
    } else {
        for (int t = threadIdx.x; t < T; t += kBlock) {
            const double m = (double)pp[2 * t];
            s1 += m;
            s2 += (double)pp[2 * t + 1] + (double)P * m * m;
        }
    }
    block_sum2(s1, s2, sh);
    if (threadIdx.x == 0) {
        const double cnt = (double)T * P;
        const double mean = s1 / T;
        double var = (s2 - cnt * mean * mean) / cnt;
        if (var < 0.0) var = 0.0;
        const double invstd = 1.0 / sqrt(var + (double)eps);
        const double scale = (double)gamma[ch] * invstd;
        coef[0] = (float)scale;
        coef[1] = (float)((double)beta[ch] - mean * scale);
        coef[2] = (float)mean;
        coef[3] = (float)invstd;
        if (blockIdx.y == 0) {
            save_mean[ch] = (float)mean;
            save_invstd[ch] = (float)invstd;
            if (save_scale) {
                save_scale[ch] = coef[0];
                save_scale[c + ch] = coef[1];
            }
            if (run_mean) {
                run_mean[ch] = (float)((1.0 - momentum) * run_mean[ch] + momentum * mean);
                run_var[ch] = (float)((1.0 - momentum) * run_var[ch] + momentum * (cnt > 1.0 ? var * cnt / (cnt - 1.0) : var));
            }
        }
    }
}

// The statistics alone (one block per channel), for a BN whose output is
// never stored: its only consumer, a convolution, stages
// max(fma(y, scale, shift), 0) itself from y and the saved scale and shift
// (the values this kernel's coefficients give, bit for bit, as the apply
// kernel would).
__global__ __launch_bounds__(kBlock) void bn_stats_partials_k(int c, const float* part, int T, int P,
                                                               const float* gamma, const float* beta, float eps,
                                                               float momentum, float* save_mean, float* save_invstd,
                                                               float* save_scale, float* run_mean, float* run_var)
{
    __shared__ double sh[2 * kBlock / 64];
    __shared__ float coef[4];
    const int ch = blockIdx.x;
    const float* pp = part + (size_t)ch * T * 2;
    float2 pv[kMergeTilesPerThread];
    load_tile_stats(pp, T, pv);
    bn_merge_finish(pp, T, P, pv, sh, coef, c, ch, gamma, beta, eps, momentum, save_mean, save_invstd, save_scale,
                    run_mean, run_var);
}

template <int U>
__global__ __launch_bounds__(kBlock) void bn_apply_partials_k(int n, int c, int hw, const float* y, const float* part,
                                                               int T, int P, const float* gamma, const float* beta,
                                                               const float* res, int rc, int rh, int rw, int h, int w,
                                                               int relu, float eps, float momentum, float* z,
                                                               float* save_mean, float* save_invstd, float* save_scale,
                                                               float* run_mean, float* run_var, float* pool,
                                                               float* pstat)
{
    __shared__ double sh[2 * kBlock / 64];
    __shared__ float coef[4];
    const int ch = blockIdx.x;
    const int hw4 = hw >> 2;
    const int units = n * hw4;
    const int u0 = blockIdx.y * (U * kBlock);
    const int u1 = min(u0 + U * kBlock, units);
    const bool identity = res && rc == c && rh == h && rw == w;
    const int lo = (c - rc) / 2, cc = ch - lo;
    const bool shortcut_a = res && !identity && cc >= 0 && cc < rc;
    // the per-tile statistics are loaded first, so that their merge below
    // runs while the tensor loads are in flight (loads complete in order)
    const float* pp = part + (size_t)ch * T * 2;
    float2 pv[kMergeTilesPerThread];
    load_tile_stats(pp, T, pv);
    size_t idx[U];
    float4 yv[U], rv[U];
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const int u = u0 + threadIdx.x + q * kBlock;
        yv[q] = rv[q] = make_float4(0.f, 0.f, 0.f, 0.f);
        idx[q] = 0;
        if (u < u1) {
            const int img = u / hw4, off = (u - img * hw4) * 4;
            idx[q] = ((size_t)img * c + ch) * hw + off;
            yv[q] = *reinterpret_cast<const float4*>(y + idx[q]);
            if (identity) {
                rv[q] = *reinterpret_cast<const float4*>(res + idx[q]);
            } else if (shortcut_a) {  // option-A shortcut: subsampled, channel-padded residual
                const int hh = off / w, ww = off - hh * w;  // w % 4 == 0: the four elements share a row
                const int sw = rw / w;
                const float* rp = res + (((size_t)img * rc + cc) * rh + hh * (rh / h)) * rw + ww * sw;
                rv[q] = make_float4(rp[0], rp[sw], rp[2 * sw], rp[3 * sw]);
            }
        }
    }
    bn_merge_finish(pp, T, P, pv, sh, coef, c, ch, gamma, beta, eps, momentum, save_mean, save_invstd, save_scale,
                    run_mean, run_var);
    __syncthreads();
    const float sc = coef[0], sf = coef[1];
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const bool live = u0 + (int)threadIdx.x + q * kBlock < u1;
        float v[4] = {__fmaf_rn(yv[q].x, sc, sf), __fmaf_rn(yv[q].y, sc, sf), __fmaf_rn(yv[q].z, sc, sf),
                      __fmaf_rn(yv[q].w, sc, sf)};
        if (res) {
            v[0] += rv[q].x; v[1] += rv[q].y; v[2] += rv[q].z; v[3] += rv[q].w;
        }
        if (relu) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = fmaxf(v[e], 0.f);
        }
        if (live) store_stream4(z + idx[q], make_float4(v[0], v[1], v[2], v[3]));
        if (pool) {  // a global average pool reads this BN's output alone: the 16 units of
                     // an 8x8 plane are 16 consecutive lanes (rows of 16 live or dead together)
            float ps = (v[0] + v[1]) + (v[2] + v[3]);
#pragma unroll
            for (int off = 8; off > 0; off >>= 1) ps += __shfl_xor(ps, off, 16);
            // and, for the backward, the plane's ReLU count and sum of xhat
            // where the ReLU passes: the pool's gradient is uniform over the
            // plane, so the BN backward's sums follow from these two numbers
            float pc = 0.f, px = 0.f;
            if (pstat) {
                const float mu = coef[2], is = coef[3];
                const float yy[4] = {yv[q].x, yv[q].y, yv[q].z, yv[q].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const bool pass = !relu || v[e] > 0.f;
                    pc += pass ? 1.f : 0.f;
                    px += pass ? (yy[e] - mu) * is : 0.f;
                }
#pragma unroll
                for (int off = 8; off > 0; off >>= 1) {
                    pc += __shfl_xor(pc, off, 16);
                    px += __shfl_xor(px, off, 16);
                }
            }
            if (live && (threadIdx.x & 15) == 0) {
                const int u = u0 + (int)threadIdx.x + q * kBlock;
                pool[(size_t)(u / hw4) * c + ch] = ps / (float)hw;
                if (pstat) {
                    pstat[((size_t)(u / hw4) * c + ch) * 2 + 0] = pc;
                    pstat[((size_t)(u / hw4) * c + ch) * 2 + 1] = px;
                }
            }
        }
    }
}

// backward: tile partials (sum g, sum g*xhat) with g = dz*[z > 0] (relu);
//   dbeta = sum g, dgamma = sum g*xhat,
//   dy = gamma*invstd*(g - dbeta/M - xhat*dgamma/M),
// and the residual's gradient: dres (+)= g (identity), or for the option-A
// shortcut (residual of 2x the resolution, channels padded by lo on each
// side) g at the even positions of channel ch - lo and zero elsewhere.
// With scale set (a BN without residual) the mask is fmaf(y, scale, shift)
// > 0, the forward's own pre-activation, and z is not read.
template <int U>
__global__ __launch_bounds__(kBlock) void bn_bwd_partials_k(int n, int c, int hw, int w, const float* dz,
                                                             const float* z, const float* y, const float* gamma,
                                                             const float* mean, const float* invstd,
                                                             const float* scale, const float* part, int T, int relu,
                                                             float* dy, float* dgamma, float* dbeta, float* dres,
                                                             int rc, int res_mode, int res_accumulate)
{
    __shared__ double sh[2 * kBlock / 64];
    __shared__ float coef[3];
    const int ch = blockIdx.x;
    const int hw4 = hw >> 2;
    const int units = n * hw4;
    const int u0 = blockIdx.y * (U * kBlock);
    const int u1 = min(u0 + U * kBlock, units);
    const bool ymask = relu && scale, zmask = relu && !scale;
    const float sc = ymask ? scale[ch] : 0.f, sf = ymask ? scale[c + ch] : 0.f;
    const int cc = ch - (c - rc) / 2;  // residual channel (option A)
    const bool identity = res_mode == 1, shortcut_a = res_mode == 2 && cc >= 0 && cc < rc;
    const float* pp = part + (size_t)ch * T * 2;  // loaded first, as in bn_apply_partials_k
    float2 pv[kMergeTilesPerThread];
    load_tile_stats(pp, T, pv);
    size_t idx[U];
    float4 gv[U], zv[U], yv[U], ov[U];
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const int u = u0 + threadIdx.x + q * kBlock;
        gv[q] = yv[q] = ov[q] = make_float4(0.f, 0.f, 0.f, 0.f);
        zv[q] = make_float4(1.f, 1.f, 1.f, 1.f);
        idx[q] = 0;
        if (u < u1) {
            const int img = u / hw4, off = (u - img * hw4) * 4;
            idx[q] = ((size_t)img * c + ch) * hw + off;
            gv[q] = *reinterpret_cast<const float4*>(dz + idx[q]);
            yv[q] = *reinterpret_cast<const float4*>(y + idx[q]);
            if (zmask) zv[q] = *reinterpret_cast<const float4*>(z + idx[q]);
            if (identity && res_accumulate) ov[q] = *reinterpret_cast<const float4*>(dres + idx[q]);
        }
    }
    double s1 = 0.0, s2 = 0.0;
    if (T <= kMergeTilesPerThread * kBlock) {
#pragma unroll
        for (int k = 0; k < kMergeTilesPerThread; ++k)
            if ((int)threadIdx.x + k * kBlock < T) {
                s1 += (double)pv[k].x;
                s2 += (double)pv[k].y;
            }
    } else {
        for (int t = threadIdx.x; t < T; t += kBlock) {
            s1 += (double)pp[2 * t];
            s2 += (double)pp[2 * t + 1];
        }
    }
    block_sum2(s1, s2, sh);
    const float mu = mean[ch], is = invstd[ch];
    if (threadIdx.x == 0) {
        const double cnt = (double)n * hw;
        coef[0] = (float)((double)gamma[ch] * (double)is);
        coef[1] = (float)(s1 / cnt);
        coef[2] = (float)(s2 / cnt);
        if (blockIdx.y == 0) {
            dbeta[ch] = (float)s1;
            dgamma[ch] = (float)s2;
        }
    }
    __syncthreads();
    const float a = coef[0], b = coef[1], d = coef[2];
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const int u = u0 + (int)threadIdx.x + q * kBlock;
        if (u >= u1) continue;
        float g[4] = {gv[q].x, gv[q].y, gv[q].z, gv[q].w};
        const float zz[4] = {zv[q].x, zv[q].y, zv[q].z, zv[q].w};
        const float yy[4] = {yv[q].x, yv[q].y, yv[q].z, yv[q].w};
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bool pass = ymask ? __fmaf_rn(yy[e], sc, sf) > 0.f : zz[e] > 0.f;
            if (relu && !pass) g[e] = 0.f;
            const float xh = (yy[e] - mu) * is;
            o[e] = a * (g[e] - b - xh * d);
        }
        store_stream4(dy + idx[q], make_float4(o[0], o[1], o[2], o[3]));
        if (identity) {
            store_stream4(dres + idx[q], make_float4(g[0] + ov[q].x, g[1] + ov[q].y, g[2] + ov[q].z, g[3] + ov[q].w));
        } else if (shortcut_a) {  // residual rows 2hh (g at even columns) and 2hh+1 (zero)
            const int img = u / hw4, off = (u - img * hw4) * 4;
            const int hh = off / w, ww = off - hh * w;
            float4* r0 = reinterpret_cast<float4*>(dres + (((size_t)img * rc + cc) * (2 * (hw / w)) + 2 * hh) * (2 * w) + 2 * ww);
            float4* r1 = r0 + (2 * w) / 4;
            float4 e0 = make_float4(g[0], 0.f, g[1], 0.f), e1 = make_float4(g[2], 0.f, g[3], 0.f);
            if (res_accumulate) {
                const float4 o0 = r0[0], o1 = r0[1];
                e0.x += o0.x; e0.y += o0.y; e0.z += o0.z; e0.w += o0.w;
                e1.x += o1.x; e1.y += o1.y; e1.z += o1.z; e1.w += o1.w;
            }
            r0[0] = e0;
            r0[1] = e1;
            if (!res_accumulate) {
                r1[0] = make_float4(0.f, 0.f, 0.f, 0.f);
                r1[1] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// units per thread: the largest of 4, 2, 1 that still gives >= 1024 blocks
// (four per CU), else 1
int apply_units_per_thread(int64_t units_total)
{
    for (int u = 4; u > 1; u /= 2)
        if (units_total / ((int64_t)u * kBlock) >= 1024) return u;
    return 1;
}
}  // namespace

hipError_t bn_apply_from_partials(int n, int c, int h, int w, const float* y, const float* part, int T, int P,
                                  const float* gamma, const float* beta, const float* res, int rc, int rh, int rw,
                                  int relu, float eps, float momentum, float* z, float* save_mean, float* save_invstd,
                                  float* save_scale, float* run_mean, float* run_var, hipStream_t st, float* pool,
                                  float* pstat)
{
    if (pool && h * w != 64) return hipErrorNotSupported;
    if (pstat && (!pool || (uintptr_t)pstat % 8)) return hipErrorNotSupported;
    const bool identity = res && rc == c && rh == h && rw == w;
    if (w % 4 || !aligned16(y) || !aligned16(z) || (identity && !aligned16(res)) || (uintptr_t)part % 8)
        return hipErrorNotSupported;
    const int64_t units = (int64_t)n * h * w / 4;
    if (units > INT32_MAX) return hipErrorNotSupported;
    const int U = apply_units_per_thread(units * c);
    const unsigned per_ch = (unsigned)((units + U * kBlock - 1) / (U * kBlock));
    const double total = (double)n * c * h * w;
    const double rbytes = res ? kF * (double)n * std::min(c, rc) * h * w : 0.0;
    Work wk{3.0 * total, 2 * kF * total + rbytes + 2 * kF * T * c};
    if (pool) wk.bytes += kF * (double)n * c * (pstat ? 3.0 : 1.0);  // the pooled means (and plane statistics) written
#define PSW_BN_APPLY(UU)                                                                                          \
    PSW_LAUNCH(kname("bn_apply_partials_k", UU), wk, bn_apply_partials_k<UU>, dim3(c, per_ch), dim3(kBlock), 0, st, n, c, \
               h * w, y, part, T, P, gamma, beta, res, rc, rh, rw, h, w, relu, eps, momentum, z, save_mean,          \
               save_invstd, save_scale, run_mean, run_var, pool, pstat)
    if (U == 4)
        PSW_BN_APPLY(4);
    else if (U == 2)
        PSW_BN_APPLY(2);
    else
        PSW_BN_APPLY(1);
#undef PSW_BN_APPLY
    return hipGetLastError();
}

hipError_t bn_stats_from_partials(int c, const float* part, int T, int P, const float* gamma, const float* beta,
                                  float eps, float momentum, float* save_mean, float* save_invstd, float* save_scale,
                                  float* run_mean, float* run_var, hipStream_t st)
{
    if (!save_scale || (uintptr_t)part % 8) return hipErrorNotSupported;
    const Work wk{8.0 * c * T, 2 * kF * (double)T * c + 4 * kF * c};  // the partials read, four floats per channel written
    PSW_LAUNCH(kname("bn_stats_partials_k"), wk, bn_stats_partials_k, dim3(c), dim3(kBlock), 0, st, c, part, T, P,
               gamma, beta, eps, momentum, save_mean, save_invstd, save_scale, run_mean, run_var);
    return hipGetLastError();
}

hipError_t bn_bwd_from_partials(int n, int c, int h, int w, const float* dz, const float* z, const float* y,
                                const float* gamma, const float* mean, const float* invstd, const float* scale,
                                const float* part, int T, int relu, float* dy, float* dgamma, float* dbeta,
                                float* dres, int rc, int rh, int rw, int res_accumulate, hipStream_t st)
{
    int res_mode = 0;
    if (dres) {
        if (rc == c && rh == h && rw == w) res_mode = 1;
        else if (rh == 2 * h && rw == 2 * w && rc <= c && (c - rc) % 2 == 0) res_mode = 2;
        else return hipErrorNotSupported;
    }
    if (relu && !scale && !z) return hipErrorInvalidValue;
    if (w % 4 || !aligned16(dz) || !aligned16(y) || !aligned16(dy) || (z && !aligned16(z)) || (uintptr_t)part % 8 ||
        (dres && !aligned16(dres)))
        return hipErrorNotSupported;
    const int64_t units = (int64_t)n * h * w / 4;
    if (units > INT32_MAX) return hipErrorNotSupported;
    const int U = apply_units_per_thread(units * c);
    const unsigned per_ch = (unsigned)((units + U * kBlock - 1) / (U * kBlock));
    const double total = (double)n * c * h * w;
    double bytes = kF * ((relu && !scale ? 4.0 : 3.0) * total) + 2 * kF * T * c;  // dz, y, (z), dy
    if (res_mode == 1) bytes += kF * (1.0 + res_accumulate) * total;
    if (res_mode == 2) bytes += kF * (double)n * rc * rh * rw + (res_accumulate ? kF * (double)n * rc * h * w * 2 : 0.0);
#define PSW_BN_BWD(UU)                                                                                            \
    PSW_LAUNCH(kname("bn_bwd_partials_k", UU), (Work{6.0 * total, bytes}), bn_bwd_partials_k<UU>, dim3(c, per_ch),     \
               dim3(kBlock), 0, st, n, c, h * w, w, dz, z, y, gamma, mean, invstd, scale, part, T, relu, dy, dgamma,   \
               dbeta, dres, rc, res_mode, res_accumulate)
    if (U == 4)
        PSW_BN_BWD(4);
    else if (U == 2)
        PSW_BN_BWD(2);
    else
        PSW_BN_BWD(1);
#undef PSW_BN_BWD
    return hipGetLastError();
}

hipError_t bn_bwd_gavg(int n, int c, int h, int w, const float* dh, const float* z, const float* y,
                       const float* gamma, const float* mean, const float* invstd, int relu, float* dz, float* dy,
                       float* dgamma, float* dbeta, float* dres, hipStream_t st)
{
    const int hw = h * w;
    if (hw % 4 || !aligned16(z) || !aligned16(y) || !aligned16(dz) || !aligned16(dy) || (dres && !aligned16(dres)))
        return hipErrorNotSupported;
    if ((int64_t)n * hw > INT32_MAX) return hipErrorNotSupported;
    const double total = (double)n * c * hw;
    // y and z read (their second pass hits L2), dz, dy (and the residual's gradient) written
    const Work wk{8.0 * total, kF * ((4.0 + (dres ? 1.0 : 0.0)) * total + (double)n * c)};
    PSW_LAUNCH(kname("bn_bwd_gavg_k"), wk, bn_bwd_gavg_k, dim3(c), dim3(kBlock), 0, st, n, c, hw, dh, z, y, gamma, mean,
               invstd, relu, dz, dy, dgamma, dbeta, dres);
    return hipGetLastError();
}

hipError_t bn_bwd_gavg_from_stats(int n, int c, int h, int w, const float* dh, const float* pstat, const float* z,
                                  const float* y, const float* gamma, const float* mean, const float* invstd, int relu,
                                  float* dz, float* dy, float* dgamma, float* dbeta, float* dres, hipStream_t st)
{
    const int hw = h * w;
    if (hw % 4 || !aligned16(z) || !aligned16(y) || !aligned16(dz) || !aligned16(dy) || (dres && !aligned16(dres)) ||
        (uintptr_t)pstat % 8)
        return hipErrorNotSupported;
    const int64_t units = (int64_t)n * hw / 4;
    if (units > INT32_MAX) return hipErrorNotSupported;
    const int U = apply_units_per_thread(units * c);
    const unsigned per_ch = (unsigned)((units + U * kBlock - 1) / (U * kBlock));
    const double total = (double)n * c * hw;
    // y and z read, dz, dy (and the residual's gradient) written, the plane statistics and dh read
    const Work wk{6.0 * total, kF * ((4.0 + (dres ? 1.0 : 0.0)) * total + 3.0 * n * c)};
#define PSW_BN_GS(UU)                                                                                             \
    PSW_LAUNCH(kname("bn_bwd_gavg_stats_k", UU), wk, bn_bwd_gavg_stats_k<UU>, dim3(c, per_ch), dim3(kBlock), 0, st, n, \
               c, hw, dh, pstat, z, y, gamma, mean, invstd, relu, dz, dy, dgamma, dbeta, dres)
    if (U == 4)
        PSW_BN_GS(4);
    else if (U == 2)
        PSW_BN_GS(2);
    else
        PSW_BN_GS(1);
#undef PSW_BN_GS
    return hipGetLastError();
}

hipError_t maxpool_fwd(int n, int c, int h, int w, int k, int stride, const float* x, float* y, int32_t* argmax,
                       hipStream_t st)
{
    const int p = (h - k) / stride + 1, q = (w - k) / stride + 1;
    const int64_t total = (int64_t)n * c * p * q;
    PSW_LAUNCH(kname("maxpool_fwd_k"), (Work{(double)total * k * k, kF * ((double)n * c * h * w + 2.0 * total)}),
               maxpool_fwd_k, dim3(blocks_for(total)), dim3(kBlock), 0, st, total, h, w, p, q, k, stride, x, y, argmax);
    return hipGetLastError();
}

hipError_t maxpool_bwd(int n, int c, int h, int w, int k, int stride, const float* dy, const int32_t* argmax,
                       float* dx, int accumulate, hipStream_t st)
{
    const int p = (h - k) / stride + 1, q = (w - k) / stride + 1;
    const int64_t total = (int64_t)n * c * h * w;
    PSW_LAUNCH(kname("maxpool_bwd_k"), (Work{0.0, kF * (2.0 * n * c * p * q + (1.0 + accumulate) * total)}),
               maxpool_bwd_k, dim3(blocks_for(total)), dim3(kBlock), 0, st, total, h, w, p, q, k, dy, argmax, dx,
               accumulate);
    return hipGetLastError();
}

hipError_t gavgpool_fwd(int n, int c, int h, int w, const float* x, float* y, hipStream_t st)
{
    const int64_t planes = (int64_t)n * c;
    PSW_LAUNCH(kname("gavg_fwd_k"), (Work{(double)planes * h * w, kF * planes * (h * w + 1.0)}), gavg_fwd_k,
               dim3(blocks_for(planes, 4)), dim3(kBlock), 0, st, planes, h * w, x, y);
    return hipGetLastError();
}

hipError_t gavgpool_bwd(int n, int c, int h, int w, const float* dy, float* dx, int accumulate, hipStream_t st)
{
    const int64_t total = (int64_t)n * c * h * w;
    PSW_LAUNCH(kname("gavg_bwd_k"), (Work{(double)total, kF * ((double)n * c + (1.0 + accumulate) * total)}),
               gavg_bwd_k, dim3(blocks_for(total)), dim3(kBlock), 0, st, total, h * w, dy, dx, accumulate);
    return hipGetLastError();
}

hipError_t relu_mask(int64_t count, const float* z, float* g, hipStream_t st)
{
    PSW_LAUNCH(kname("relu_mask_k"), (Work{(double)count, 3 * kF * count}), relu_mask_k, dim3(blocks_for(count)),
               dim3(kBlock), 0, st, count, z, g);
    return hipGetLastError();
}

hipError_t softmax_xent(int n, int classes, const float* logits, const int32_t* labels, float* loss, float* dlogits,
                        hipStream_t st)
{
    PSW_LAUNCH(kname("softmax_xent_k"), (Work{5.0 * n * classes, kF * (2.0 * n * classes + n + 1.0)}), softmax_xent_k,
               dim3(1), dim3(kBlock), 0, st, n, classes, logits, labels, loss, dlogits);
    return hipGetLastError();
}

hipError_t sgd_momentum(int64_t count, const float* w_in, float* w_out, float* v, const float* g, float lr, float mom,
                        float wd, int nesterov, hipStream_t st)
{
    if (count <= 0) return hipSuccess;
    PSW_LAUNCH(kname("sgd_k"), (Work{5.0 * count, 5 * kF * count}), sgd_k, dim3(blocks_for(count)), dim3(kBlock), 0, st,
               count, w_in, w_out, v, g, lr, mom, wd, nesterov);
    return hipGetLastError();
}

hipError_t sgd_stage(const SgdSeg* segs, int nseg, const float* w_in, float* w_out, float* v, float* g, float lr,
                     float mom, float wd, int nesterov, hipStream_t st)
{
    for (int a0 = 0; a0 < nseg; a0 += kSgdMaxSegs) {
        SgdSegs ss{};
        int64_t nb = 0;
        double fl = 0.0, bytes = 0.0;
        ss.n = 0;
        for (int k = a0; k < nseg && k < a0 + kSgdMaxSegs; ++k) {
            const SgdSeg& q = segs[k];
            if (q.count <= 0) continue;
            SgdSegDev& d = ss.s[ss.n++];
            d.off = q.off;
            d.count = q.count;
            d.part = q.splits > 0 ? q.part : nullptr;
            d.splits = q.splits > 0 ? q.splits : 0;
            d.first_block = (int32_t)nb;
            nb += d.part ? (q.count + kSgdOut - 1) / kSgdOut : (q.count + kSgdBlock - 1) / kSgdBlock;
            fl += 5.0 * q.count + (d.part ? (double)d.splits * q.count : 0.0);
            bytes += kF * (5.0 * q.count + (d.part ? (double)d.splits * q.count : 0.0));
        }
        if (!ss.n) continue;
        if (nb > INT32_MAX) return hipErrorInvalidValue;
        PSW_LAUNCH(kname("sgd_stage_k"), (Work{fl, bytes}), sgd_stage_k, dim3((unsigned)nb), dim3(kSgdBlock), 0, st, ss,
                   w_in, w_out, v, g, lr, mom, wd, nesterov);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// ------------------------------------------------------------- dropout -----
// Masks from Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds
// on a 4-word counter; each round takes the two 32x32 -> 64-bit products of
// counter words 0 and 2 with the round multipliers, and the new counter is
// (hi(word 2 product) ^ word 1 ^ key 0, lo(word 2 product), hi(word 0
// product) ^ word 3 ^ key 1, lo(word 0 product)); the key grows by the two
// Weyl increments between rounds.  Thread q draws the words of elements
// 4q .. 4q+3 from counter (q, op, t mod 2^32, t / 2^32) under key
// (seed mod 2^32, seed / 2^32); element j is kept iff the top 24 bits of its
// word are >= p24, and kept values are scaled by 2^24 / (2^24 - p24).
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        if (round) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint32_t hi0 = __umulhi(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
        const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
        c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    }
    return c;
}

struct DropKey {
    uint32_t k0, k1, op, t_lo, t_hi;
    int p24;
    float scale;
};

// out[j] (+)= keep(j) ? in[j] * scale : 0, four elements per thread
__global__ void dropout_k(int64_t n, const float* in, float* out, int accumulate, DropKey dk)
{
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t j0 = q * 4;
    if (j0 >= n) return;
    const uint4 r = philox4x32_10(make_uint4((uint32_t)q, dk.op, dk.t_lo, dk.t_hi), dk.k0, dk.k1);
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
    float v[4], o[4] = {0.f, 0.f, 0.f, 0.f};
    const bool full = j0 + 4 <= n && (uintptr_t)(in + j0) % 16 == 0 && (uintptr_t)(out + j0) % 16 == 0;
    if (full) {
        const float4 a = *reinterpret_cast<const float4*>(in + j0);
        v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w;
        if (accumulate) {
            const float4 b = *reinterpret_cast<const float4*>(out + j0);
            o[0] = b.x, o[1] = b.y, o[2] = b.z, o[3] = b.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[e] = j0 + e < n ? in[j0 + e] : 0.f;
            if (accumulate && j0 + e < n) o[e] = out[j0 + e];
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float d = (int)(w[e] >> 8) >= dk.p24 ? v[e] * dk.scale : 0.f;
        o[e] = accumulate ? o[e] + d : d;
    }
    if (full) {
        *reinterpret_cast<float4*>(out + j0) = make_float4(o[0], o[1], o[2], o[3]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (j0 + e < n) out[j0 + e] = o[e];
    }
}

hipError_t dropout_apply(int64_t n, const float* in, float* out, int accumulate, int p24, uint64_t seed, uint32_t op,
                         int64_t t, hipStream_t st)
{
    if (n < 0 || p24 <= 0 || p24 >= (1 << 24) || t < 0) return hipErrorInvalidValue;
    if ((n + 3) / 4 > (int64_t)UINT32_MAX + 1) return hipErrorInvalidValue;  // counter word 0 is j / 4
    if (n == 0) return hipSuccess;
    DropKey dk{(uint32_t)seed, (uint32_t)(seed >> 32), op, (uint32_t)t, (uint32_t)((uint64_t)t >> 32), p24,
               (float)(16777216.0 / (16777216.0 - p24))};
    const int64_t quads = (n + 3) / 4;
    PSW_LAUNCH(kname("dropout_k"), (Work{(double)n, kF * (2.0 + accumulate) * n}),
               dropout_k, dim3(blocks_for(quads)), dim3(kBlock), 0, st, n, in, out, accumulate, dk);
    return hipGetLastError();
}

hipError_t fc_fwd(int n, int in, int out, const float* x, const float* w, const float* b, int relu, float* y, int bf16,
                  hipStream_t st)
{
    if (small_fc(n, in, out)) {
        const double fl = 2.0 * n * out * (double)in;
        PSW_LAUNCH(kname("fc_small_fwd_k"), (Work{fl, kF * ((double)n * in + (double)out * in + (double)n * out)}),
                   fc_small_fwd_k, dim3(1), dim3(kHeadBlock), 0, st, n, in, out, x, w, b, relu, bf16, y,
                   (const int32_t*)nullptr, (float*)nullptr, (float*)nullptr);
        return hipGetLastError();
    }
    GemmArgs a{};
    a.A = x; a.B = w; a.C = y; a.bias = b; a.relu = relu;
    a.M = n; a.N = out; a.K = in;
    a.sam = in; a.sak = 1;    // x[n][i]
    a.sbk = 1; a.sbn = in;    // w[o][i]
    return gemm<true, true>(a, bf16, nullptr, 0, st);
}

hipError_t fc_softmax_xent(int n, int in, int out, const float* x, const float* w, const float* b, float* logits,
                           int bf16, const int32_t* labels, float* loss, float* dlogits, hipStream_t st)
{
    if (!small_fc(n, in, out)) return hipErrorNotSupported;
    const double fl = 2.0 * n * out * (double)in + 5.0 * n * out;
    PSW_LAUNCH(kname("fc_small_fwd_k"),
               (Work{fl, kF * ((double)n * in + (double)out * in + 3.0 * n * out + n + 1.0)}), fc_small_fwd_k, dim3(1),
               dim3(kHeadBlock), 0, st, n, in, out, x, w, b, 0, bf16, logits, labels, loss, dlogits);
    return hipGetLastError();
}

size_t fc_bwd_ws_bytes(int n, int in, int out)
{
    // [db partials: out x 2 doubles, padded][split-K partials of the dx GEMM]
    const int tiles = ((n + 63) / 64) * ((in + 63) / 64);
    int splits = tiles < 512 ? (1024 + tiles - 1) / tiles : 1;
    const int maxs = (out + 63) / 64;
    if (splits > maxs) splits = maxs;
    if (splits < 1) splits = 1;
    const size_t head = (((size_t)out * 2 * sizeof(double)) + 255) / 256 * 256;
    return head + (size_t)splits * n * in * sizeof(float);
}

hipError_t fc_bwd(int n, int in, int out, const float* x, const float* w, const float* dy, float* dx, int dx_accumulate,
                  float* dw, float* db, int bf16, void* ws, size_t ws_bytes, hipStream_t st)
{
    if (ws_bytes < fc_bwd_ws_bytes(n, in, out)) return hipErrorInvalidValue;
    if (small_fc(n, in, out)) {
        const int nbx = dx ? (int)blocks_for((int64_t)n * in) : 0, nbw = (in + kFcKW - 1) / kFcKW;
        const double fl = 2.0 * (dx ? 2.0 : 1.0) * n * out * (double)in + (double)n * out;
        const double bytes = kF * ((double)n * out + (double)out * in + (double)n * in * (dx ? 2.0 + dx_accumulate : 1.0) +
                                   (double)out * in + out);
        PSW_LAUNCH(kname("fc_small_bwd_k"), (Work{fl, bytes}), fc_small_bwd_k, dim3(nbx + nbw), dim3(kBlock), 0,
                   st, n, in, out, x, w, dy, dx, dx_accumulate, dw, db, bf16, nbx);
        return hipGetLastError();
    }
    const size_t head = (((size_t)out * 2 * sizeof(double)) + 255) / 256 * 256;
    hipError_t e = hipSuccess;
    if (dx) {
        GemmArgs a{};
        a.A = dy; a.B = w; a.C = dx; a.accumulate = dx_accumulate;
        a.M = n; a.N = in; a.K = out;
        a.sam = out; a.sak = 1;   // dy[n][o]
        a.sbk = in; a.sbn = 1;    // w[o][i]
        e = gemm<true, false>(a, bf16, (char*)ws + head, ws_bytes - head, st);
        if (e != hipSuccess) return e;
    }
    {
        GemmArgs a{};
        a.A = dy; a.B = x; a.C = dw;
        a.M = out; a.N = in; a.K = n;
        a.sam = 1; a.sak = out;   // dy[n][o] read as A(m=o, k=n)
        a.sbk = in; a.sbn = 1;    // x[n][i]
        e = gemm<false, false>(a, bf16, nullptr, 0, st);
        if (e != hipSuccess) return e;
    }
    if (db) {
        // db[o] = sum_n dy[n][o]: the column sums of dy viewed as [n][out][1]
        // (not a product, so never rounded to bf16)
        PSW_LAUNCH(kname("chan_partials"), (Work{(double)n * out, kF * n * out}), chan_partials, dim3(out, 1),
                   dim3(kBlock), 0, st, 2, n, out, 1, 1, dy, (const float*)nullptr, (const float*)nullptr,
                   (const float*)nullptr, (const float*)nullptr, 0, (double*)ws);
        PSW_LAUNCH(kname("chan_sum_finalize"), (Work{(double)out, 16.0 * out + kF * out}), chan_sum_finalize,
                   dim3(blocks_for(out)), dim3(kBlock), 0, st, out, 1, (const double*)ws, db);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace psw
