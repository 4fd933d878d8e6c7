// Direct 3x3 convolution (pad 1, stride 1 or 2) on CDNA4 matrix cores, NCHW
// fp32: the forward pass of the CIFAR ResNet / VGG conv layers and the
// backward-data pass of their stride-1 layers (a stride-1 3x3 conv whose
// weights are transposed over (k,c) and flipped over (r,s)).
//
// A workgroup owns one image, TH output rows (all WO columns) and 16*WK
// output channels.  Input channels are processed in chunks of CC: the
// chunk's halo tile  [CC][(TH-1)*STRIDE+3][WIN+halo]  is staged in LDS with
// float4 loads (zero rows/columns supply the padding), and the chunk's
// weights are staged in LDS already in MFMA-fragment order so that every
// wave reads its A operand with one conflict-free ds_read per k-step.
//
// MFMA v_mfma_f32_16x16x4_f32, D[m][n] += A[m][k] B[k][n] with
//   m = output channel (16 per wave), n = output pixel (16 per block),
//   k = (4 input channels) x one tap (r,s): lane group g = lane/16 supplies
//   channel c0+4*c4+g, lane%16 the channel (A) or pixel (B).
// D lane l, register i holds channel 4*(l/16)+i of pixel l%16, so the 16
// lanes of a group store 16 consecutive pixels of one NCHW plane.
#include "internal.h"

namespace psw {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

struct DirArgs {
    const float* x;  // input  [n][C][H][W]
    const float* w;  // layer weights as stored, KCRS
    float* y;        // output [n][K][HO][WO]
    int C, H, K, HO;
    int accumulate;
};

constexpr int round4(int v) { return (v + 3) / 4 * 4; }

template <int WO, int STRIDE, int TH, int CC, int WK, int WP, int NBW, bool TRANS>
__global__ __launch_bounds__(64 * WK * WP) void conv3x3_direct(DirArgs a)
{
    constexpr int NT = 64 * WK * WP;
    constexpr int WIN = WO * STRIDE;                       // input width
    constexpr int HR = (TH - 1) * STRIDE + 3;              // staged input rows
    constexpr int RSTR = round4(WIN + (STRIDE == 1 ? 5 : 4));  // LDS row stride (cols 3 .. WIN+4)
    constexpr int PS0 = HR * RSTR;
    constexpr int PS = PS0 + ((16 - PS0 % 32) + 32) % 32;  // plane stride = 16 mod 32: lane groups hit disjoint banks
    constexpr int KSTEPS = CC / 4 * 9;
    constexpr int TK = 16 * WK;
    static_assert(TH * WO == 16 * NBW * WP, "pixel tiling");
    static_assert(CC % 4 == 0 && WIN % 4 == 0, "tiling");
    __shared__ __attribute__((aligned(16))) float Xs[CC * PS];
    __shared__ float Wf[WK * KSTEPS * 64];

    const int tiles = a.HO / TH;
    const int img = blockIdx.x / tiles;
    const int oh0 = (blockIdx.x - img * tiles) * TH;
    const int ih0 = oh0 * STRIDE - 1;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wk = wave % WK, wp = wave / WK;
    const int mblk = blockIdx.y * TK;
    const int g = lane >> 4, j = lane & 15;

    int boff[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int pix = (wp * NBW + nb) * 16 + j;
        const int row = pix / WO, col = pix - (pix / WO) * WO;
        boff[nb] = g * PS + row * STRIDE * RSTR + col * STRIDE + 3;
    }
    v4f acc[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) acc[nb] = v4f{0.f, 0.f, 0.f, 0.f};

    // halo columns: never overwritten by the staging loop below
    for (int i = tid; i < CC * HR; i += NT) {
        const int c = i / HR, rr = i - (i / HR) * HR;
        Xs[c * PS + rr * RSTR + 3] = 0.f;
        if (STRIDE == 1) Xs[c * PS + rr * RSTR + WIN + 4] = 0.f;
    }

    for (int c0 = 0; c0 < a.C; c0 += CC) {
        __syncthreads();  // the previous chunk's LDS reads are complete
        // input halo tile, float4 per thread (rows outside the image are zero)
        constexpr int Q4 = WIN / 4;
        for (int i = tid; i < CC * HR * Q4; i += NT) {
            const int c = i / (HR * Q4);
            const int rem = i - c * (HR * Q4);
            const int rr = rem / Q4, q4 = rem - (rem / Q4) * Q4;
            const int ih = ih0 + rr;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (ih >= 0 && ih < a.H)
                v = *reinterpret_cast<const float4*>(a.x + (((size_t)img * a.C + c0 + c) * a.H + ih) * WIN + q4 * 4);
            *reinterpret_cast<float4*>(&Xs[c * PS + rr * RSTR + 4 + q4 * 4]) = v;
        }
        // weights of (TK output channels) x (CC input channels), fragment order
        for (int i = tid; i < TK * CC * 9; i += NT) {
            int m, c, rs;
            float v;
            if (!TRANS) {  // w[m][c][rs]: each output channel's CC*9 run is contiguous
                m = i / (CC * 9);
                const int rem = i - m * (CC * 9);
                c = rem / 9;
                rs = rem - c * 9;
                v = a.w[((size_t)(mblk + m) * a.C + c0 + c) * 9 + rs];
            } else {       // w_layer[c][m][8-rs]: each input channel's TK*9 run is contiguous
                c = i / (TK * 9);
                const int rem = i - c * (TK * 9);
                m = rem / 9;
                const int rsl = rem - m * 9;
                rs = 8 - rsl;
                v = a.w[((size_t)(c0 + c) * a.K + mblk + m) * 9 + rsl];
            }
            const int kb = m >> 4, ml = m & 15, c4 = c >> 2, gg = c & 3;
            Wf[((kb * (CC / 4) + c4) * 9 + rs) * 64 + gg * 16 + ml] = v;
        }
        __syncthreads();
        const float* wf = Wf + wk * KSTEPS * 64 + lane;
#pragma unroll
        for (int c4 = 0; c4 < CC / 4; ++c4)
#pragma unroll
            for (int r = 0; r < 3; ++r)
#pragma unroll
                for (int s = 0; s < 3; ++s) {
                    const float av = wf[((c4 * 9) + r * 3 + s) * 64];
#pragma unroll
                    for (int nb = 0; nb < NBW; ++nb) {
                        const float bv = Xs[boff[nb] + c4 * 4 * PS + r * RSTR + s];
                        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[nb], 0, 0, 0);
                    }
                }
    }

#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int pix = (wp * NBW + nb) * 16 + j;
        const int row = pix / WO, col = pix - (pix / WO) * WO;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = mblk + wk * 16 + 4 * g + i;
            float* dst = a.y + (((size_t)img * a.K + m) * a.HO + oh0 + row) * WO + col;
            *dst = a.accumulate ? *dst + acc[nb][i] : acc[nb][i];
        }
    }
}

template <int WO, int STRIDE, int TH, int CC, int WK, int WP, int NBW>
hipError_t launch_direct(const DirArgs& a, int n, bool trans, hipStream_t st)
{
    dim3 grid(n * (a.HO / TH), a.K / (16 * WK));
    dim3 block(64 * WK * WP);
    if (trans)
        hipLaunchKernelGGL((conv3x3_direct<WO, STRIDE, TH, CC, WK, WP, NBW, true>), grid, block, 0, st, a);
    else
        hipLaunchKernelGGL((conv3x3_direct<WO, STRIDE, TH, CC, WK, WP, NBW, false>), grid, block, 0, st, a);
    return hipGetLastError();
}

}  // namespace

// Returns hipErrorNotSupported (nothing launched) when no tile configuration
// covers the shape; the caller then uses the general implicit GEMM.
hipError_t conv3x3_direct(int n, int C, int H, int W, int K, int stride, const float* x, const float* w, float* y,
                          int accumulate, bool transpose, hipStream_t st)
{
    if (stride != 1 && stride != 2) return hipErrorNotSupported;
    if (H % stride || W % stride || C % 16) return hipErrorNotSupported;
    const int HO = H / stride, WO = W / stride;
    DirArgs a{x, w, y, C, H, K, HO, accumulate};
    if (stride == 1) {
        if (WO == 32 && HO % 4 == 0 && K % 16 == 0) return launch_direct<32, 1, 4, 16, 1, 4, 2>(a, n, transpose, st);
        if (WO == 16 && HO % 4 == 0 && K % 32 == 0) return launch_direct<16, 1, 4, 16, 2, 2, 2>(a, n, transpose, st);
        if (WO == 8 && HO % 2 == 0 && K % 64 == 0) return launch_direct<8, 1, 2, 16, 4, 1, 1>(a, n, transpose, st);
    } else if (!transpose) {
        if (WO == 16 && HO % 4 == 0 && K % 32 == 0) return launch_direct<16, 2, 4, 16, 2, 2, 2>(a, n, false, st);
        if (WO == 8 && HO % 2 == 0 && K % 64 == 0) return launch_direct<8, 2, 2, 16, 4, 1, 1>(a, n, false, st);
    }
    return hipErrorNotSupported;
}

}  // namespace psw
