// Backward-weight of a 3x3 / pad 1 convolution (stride 1 or 2) on CDNA4
// matrix cores, NCHW fp32:
//   dW[k][c][r][s] = sum_{n,p,q} dy[n][k][p][q] * x[n][c][p*S+r-1][q*S+s-1]
// (Sec. 2 of the paper: the weight gradient of layer l from x^(l-1) and
// delta^(l)).
//
// A workgroup reduces over TPW consecutive (image, TH-row band) tiles and
// writes one
// dW-shaped partial sum; the partials are added in a fixed order by the
// reduction kernel of conv.hip, so the result is bit-reproducible.
// In the workgroup, wave (kb, cb, wpx) owns the 16x16 output blocks
// (output channels kb*16.., input channels cb*16..) of all 9 taps (9 MFMA
// accumulators) and the pixel quads wpx, wpx+WPX, ...; waves that differ only
// in wpx are summed through LDS in wpx order at the end.
//
// MFMA v_mfma_f32_16x16x4_f32 with k = 4 consecutive output pixels of one
// row: A[m=k_out][k=pixel] from dy, B[k=pixel][n=c_in] from x shifted by the
// tap.  Both tiles sit in LDS pixel-major (channels innermost) with a pixel
// stride chosen so that the four lane groups (four pixels) of an operand
// read land in disjoint banks.
#include "internal.h"

namespace psw {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

struct WgArgs {
    const float* x;   // [n][C][H][W]
    const float* dy;  // [n][K][HO][WO]
    float* part;      // [gridDim.x][K][C][9]
    int n, C, H, W, K, HO;
};

// smallest v >= lo with (v * mult) % 32 == 16
constexpr int bank_stride(int lo, int mult)
{
    int v = lo;
    while ((v * mult) % 32 != 16) ++v;
    return v;
}

template <int STRIDE, int WO, int TH, int KBW, int CBW, int WPX, int TPW>
__global__ __launch_bounds__(64 * KBW * CBW * WPX) void conv3x3_wgrad(WgArgs a)
{
    constexpr int NT = 64 * KBW * CBW * WPX;
    constexpr int WIN = WO * STRIDE;
    constexpr int WS = WIN + (STRIDE == 1 ? 2 : 1);   // staged input columns: -1 .. WIN (-1 .. WIN-1 for stride 2)
    constexpr int HRR = (TH - 1) * STRIDE + 3;        // staged input rows
    constexpr int KC = 16 * KBW, CCH = 16 * CBW;
    constexpr int KSTR = bank_stride(KC, 1);          // dy pixel stride
    constexpr int CSTR = bank_stride(CCH, STRIDE);    // x pixel stride
    constexpr int NPIX = TH * WO;
    constexpr int QUADS = NPIX / 4;
    static_assert(WO % 4 == 0, "pixel quads stay inside one row");
    constexpr int DS_FLOATS = NPIX * KSTR;
    constexpr int XS_FLOATS = HRR * WS * CSTR;
    constexpr int RED_FLOATS = (WPX > 1) ? (WPX - 1) * KBW * CBW * 9 * 4 * 64 : 0;
    constexpr int LDS_FLOATS = (DS_FLOATS + XS_FLOATS) > RED_FLOATS ? (DS_FLOATS + XS_FLOATS) : RED_FLOATS;
    __shared__ float lds[LDS_FLOATS];
    float* Ds = lds;
    float* Xs = lds + DS_FLOATS;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int kb = wave % KBW, cb = (wave / KBW) % CBW, wpx = wave / (KBW * CBW);
    const int g = lane >> 4, j = lane & 15;
    const int tiles = a.HO / TH;  // row bands per image

    v4f acc[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};

    // zero padding columns of the x tile (never written by the staging loop)
    for (int i = tid; i < HRR * CCH; i += NT) {
        const int rr = i / CCH, c = i - (i / CCH) * CCH;
        Xs[(rr * WS + 0) * CSTR + c] = 0.f;
        if (STRIDE == 1) Xs[(rr * WS + WS - 1) * CSTR + c] = 0.f;
    }

    for (int it = 0; it < TPW; ++it) {
        const int tl = blockIdx.x * TPW + it;
        const int img = tl / tiles;
        const int oh0 = (tl - img * tiles) * TH;
        __syncthreads();  // previous tile's LDS reads are done
        for (int i = tid; i < KC * NPIX; i += NT) {
            const int k = i / NPIX, pix = i - (i / NPIX) * NPIX;
            Ds[pix * KSTR + k] = a.dy[(((size_t)img * a.K + k) * a.HO + oh0) * WO + pix];
        }
        const int ih0 = oh0 * STRIDE - 1;
        for (int i = tid; i < CCH * HRR * WIN; i += NT) {
            const int c = i / (HRR * WIN);
            const int rem = i - c * (HRR * WIN);
            const int rr = rem / WIN, iw = rem - (rem / WIN) * WIN;
            const int ih = ih0 + rr;
            float v = 0.f;
            if (ih >= 0 && ih < a.H) v = a.x[(((size_t)img * a.C + c) * a.H + ih) * WIN + iw];
            Xs[(rr * WS + iw + 1) * CSTR + c] = v;
        }
        __syncthreads();
        const float* dsl = Ds + g * KSTR + kb * 16 + j;
        const float* xsl = Xs + g * STRIDE * CSTR + cb * 16 + j;
        for (int qd = wpx; qd < QUADS; qd += WPX) {
            const int pix0 = qd * 4;
            const int row = pix0 / WO, col0 = pix0 - (pix0 / WO) * WO;
            const float av = dsl[pix0 * KSTR];
            const float* xb = xsl + ((row * STRIDE) * WS + col0 * STRIDE) * CSTR;
#pragma unroll
            for (int r = 0; r < 3; ++r)
#pragma unroll
                for (int s = 0; s < 3; ++s) {
                    const float bv = xb[(r * WS + s) * CSTR];
                    acc[r * 3 + s] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[r * 3 + s], 0, 0, 0);
                }
        }
    }

    if constexpr (WPX > 1) {
        __syncthreads();  // LDS tiles are no longer read: reuse for the reduction
        if (wpx > 0) {
            float* dst = lds + ((((wpx - 1) * KBW + kb) * CBW + cb) * 9) * 4 * 64;
#pragma unroll
            for (int t = 0; t < 9; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) dst[(t * 4 + i) * 64 + lane] = acc[t][i];
        }
        __syncthreads();
        if (wpx != 0) return;
        for (int w = 1; w < WPX; ++w) {
            const float* src = lds + ((((w - 1) * KBW + kb) * CBW + cb) * 9) * 4 * 64;
#pragma unroll
            for (int t = 0; t < 9; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[t][i] += src[(t * 4 + i) * 64 + lane];
        }
    }
    // D lane l, register i: output channel kb*16 + 4g + i, input channel cb*16 + j
    float* out = a.part + (size_t)blockIdx.x * a.K * a.C * 9;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int k = kb * 16 + 4 * g + i, c = cb * 16 + j;
        float* o = out + ((size_t)k * a.C + c) * 9;
#pragma unroll
        for (int t = 0; t < 9; ++t) o[t] = acc[t][i];
    }
}

// Which configuration covers a shape; 0 = none.
int wgrad_config(int n, int C, int H, int W, int K, int stride)
{
    if (stride == 1 && H == 32 && W == 32 && C == 16 && K == 16) return 1;
    if (stride == 1 && H == 16 && W == 16 && C == 32 && K == 32) return 2;
    if (stride == 1 && H == 8 && W == 8 && C == 64 && K == 64 && n % 2 == 0) return 3;
    if (stride == 2 && H == 32 && W == 32 && C == 16 && K == 32) return 4;
    if (stride == 2 && H == 16 && W == 16 && C == 32 && K == 64 && n % 2 == 0) return 5;
    return 0;
}

}  // namespace

// Number of partial sums (workgroups) for a shape; 0 when not covered.
int conv3x3_wgrad_splits(int n, int C, int H, int W, int K, int stride)
{
    switch (wgrad_config(n, C, H, W, K, stride)) {
    case 1: return n * 2;       // one 16-row band (of 32) per workgroup
    case 2: return n;           // one image per workgroup
    case 3: return n / 2;       // two images per workgroup
    case 4: return n * 2;       // one 8-row band (of 16 output rows) per workgroup
    case 5: return n / 2;       // two images per workgroup
    default: return 0;
    }
}

hipError_t conv3x3_wgrad(int n, int C, int H, int W, int K, int stride, const float* x, const float* dy, float* part,
                         hipStream_t st)
{
    const int cfg = wgrad_config(n, C, H, W, K, stride);
    if (!cfg) return hipErrorNotSupported;
    WgArgs a{x, dy, part, n, C, H, W, K, H / stride};
    const int splits = conv3x3_wgrad_splits(n, C, H, W, K, stride);
    const int nt = cfg == 1 ? 256 : cfg == 2 ? 512 : cfg == 3 ? 1024 : cfg == 4 ? 256 : 512;
    switch (cfg) {
    case 1:
        hipLaunchKernelGGL((conv3x3_wgrad<1, 32, 16, 1, 1, 4, 1>), dim3(splits), dim3(nt), 0, st, a);
        break;
    case 2:
        hipLaunchKernelGGL((conv3x3_wgrad<1, 16, 16, 2, 2, 2, 1>), dim3(splits), dim3(nt), 0, st, a);
        break;
    case 3:
        hipLaunchKernelGGL((conv3x3_wgrad<1, 8, 8, 4, 4, 1, 2>), dim3(splits), dim3(nt), 0, st, a);
        break;
    case 4:
        hipLaunchKernelGGL((conv3x3_wgrad<2, 16, 8, 2, 1, 2, 1>), dim3(splits), dim3(nt), 0, st, a);
        break;
    case 5:
        hipLaunchKernelGGL((conv3x3_wgrad<2, 8, 8, 4, 2, 1, 2>), dim3(splits), dim3(nt), 0, st, a);
        break;
    }
    return hipGetLastError();
}

}  // namespace psw
