// Direct 3x3 convolution (pad 1, stride 1 or 2) on CDNA4 matrix cores, NCHW
// fp32: the forward pass of the CIFAR ResNet / VGG conv layers and the
// backward-data pass of their stride-1 layers (a stride-1 3x3 conv whose
// weights are transposed over (k,c) and flipped over (r,s)).
//
// A workgroup owns one image, TH output rows (all WO columns) and 16*WK
// output channels.  Input channels are processed in chunks of CC: the
// chunk's halo tile  [CC][(TH-1)*STRIDE+3][WIN+halo]  is staged in LDS with
// float4 loads (zero rows/columns supply the padding), and the chunk's
// weights are staged in LDS as [output channel][CC*9] rows padded to a stride
// of 2 (mod 32) floats: the coalesced staging writes are contiguous, and the
// A-operand read of a k-step (16 output channels x 4 input channels, nine
// floats apart) touches 64 distinct banks... per half-wave.
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
typedef short v4s __attribute__((ext_vector_type(4)));

// one DPP lane permutation of a float within each row of 16 lanes
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E;             // quad_perm [1,0,3,2], [2,3,0,1]
constexpr int kDppHalfMirror = 0x141, kDppMirror = 0x140;   // lane i <-> 7-i in 8, 15-i in 16
// sum over the 16 lanes of a row: the quad exchanges give every lane its
// quad's sum, the half-row mirror pairs each quad with the other quad of its
// half, the row mirror each half with the other; a + b and b + a are the same
// float, so all 16 lanes hold the same total
__device__ __forceinline__ float row16_sum(float v)
{
    v += dpp_f<kDppXor1>(v);
    v += dpp_f<kDppXor2>(v);
    v += dpp_f<kDppHalfMirror>(v);
    v += dpp_f<kDppMirror>(v);
    return v;
}
// (mean, M2) of n values per lane merged over the 16 lanes of a row by the
// same pairing: two parts of equal count n give mean (m + m')/2 and
// M2 q + q' + (n/2)(m - m')^2, the same on both lanes of a pair
template <int CTRL>
__device__ __forceinline__ void merge_step(float& m, float& q, float n)
{
    const float m2 = dpp_f<CTRL>(m), q2 = dpp_f<CTRL>(q);
    const float d = m - m2;
    m = 0.5f * (m + m2);
    q = (q + q2) + 0.5f * n * (d * d);
}
__device__ __forceinline__ void row16_meanvar(float& m, float& q, float n)
{
    merge_step<kDppXor1>(m, q, n);
    merge_step<kDppXor2>(m, q, 2.f * n);
    merge_step<kDppHalfMirror>(m, q, 4.f * n);
    merge_step<kDppMirror>(m, q, 8.f * n);
}

// bfloat16 rounding (nearest even) of a float: its bits, and its value as a float
__device__ __forceinline__ unsigned short bf16_bits(float f) { return __builtin_bit_cast(unsigned short, (__bf16)f); }
__device__ __forceinline__ float bf16_round(float f) { return (float)(__bf16)f; }

struct DirArgs {
    const float* x;  // input  [n][C][H][W]
    const float* w;  // layer weights as stored, KCRS
    float* y;        // output [n][K][HO][WO]
    int C, H, K, HO;
    int n;           // images
    int accumulate;
    BnStatsFuse bn;  // bn.part == nullptr: no statistics
    BnBwdFuse bnb;   // bnb.part == nullptr: no backward sums (transposed kernel only)
    BnFold fold;     // input formed from a folded BN backward (FOLD kernels only)
    // forward only, may be null: the input is the raw input of a BN + ReLU
    // whose output is never stored; in_bn[c], in_bn[C + c] are channel c's
    // scale and shift, and the staged input is max(fma(x, scale, shift), 0)
    // (zero outside the image, like any halo)
    const float* in_bn;
};

constexpr int round4(int v) { return (v + 3) / 4 * 4; }

// B-operand LDS offset of pixel j (0..15) of a block relative to pixel 0
constexpr int pix_off(int j, int wo, int stride, int rstr) { return (j / wo) * stride * rstr + (j % wo) * stride; }

// Number of LDS bank collisions (32 banks of 4 bytes) of one B-operand read
// for a plane stride ps: lanes (j, g) read g*ps + pix_off(j); the hardware
// serves each 32-lane half (g = 0,1 and g = 2,3) separately.
constexpr int b_conflicts(int ps, int wo, int stride, int rstr)
{
    int worst = 0;
    for (int half = 0; half < 2; ++half) {
        int cnt[32] = {};
        for (int g = 2 * half; g < 2 * half + 2; ++g)
            for (int j = 0; j < 16; ++j) cnt[(g * ps + pix_off(j, wo, stride, rstr)) % 32]++;
        for (int b = 0; b < 32; ++b) worst = cnt[b] > worst ? cnt[b] : worst;
    }
    return worst;
}

// smallest plane stride >= lo, multiple of 4 (float4 staging), with the
// fewest B-operand bank collisions
constexpr int plane_stride_b(int lo, int wo, int stride, int rstr)
{
    int best = round4(lo), bestc = b_conflicts(round4(lo), wo, stride, rstr);
    for (int v = round4(lo); v < round4(lo) + 32; v += 4) {
        const int c = b_conflicts(v, wo, stride, rstr);
        if (c < bestc) {
            bestc = c;
            best = v;
        }
    }
    return best;
}
// bf16 quad-interleaved tile (8 bytes = 4 channels per pixel): bank-pair
// collisions (16 pairs of 8 bytes) of the 16 lanes of one lane group reading
// the pixels of a 16-pixel block, for a row stride rs (in 8-byte elements)
constexpr int q_conflicts(int rs, int wo, int stride)
{
    int cnt[16] = {}, worst = 0;
    for (int j = 0; j < 16; ++j) cnt[pix_off(j, wo, stride, rs) % 16]++;
    for (int b = 0; b < 16; ++b) worst = cnt[b] > worst ? cnt[b] : worst;
    return worst;
}
constexpr int row_stride_q(int lo, int wo, int stride)
{
    int best = lo, bestc = q_conflicts(lo, wo, stride);
    for (int v = lo; v < lo + 16; ++v)
        if (q_conflicts(v, wo, stride) < bestc) {
            bestc = q_conflicts(v, wo, stride);
            best = v;
        }
    return best;
}

// weight row stride (floats) of an LDS tile with `n` floats per output
// channel: the smallest v >= n with v = 2 (mod 32), so that lanes
// (m, g) -> m*v + 9*g hit distinct banks within each 32-lane half
constexpr int wrow(int n)
{
    int v = n;
    while (v % 32 != 2) ++v;
    return v;
}

// FOLD: 0 plain input; 1 input from a folded BN backward (no residual, ReLU
// mask from the forward's scale and shift); 2 the same for a BN with an
// identity residual (ReLU mask from the BN output z; the masked gradient
// is also written to the residual's gradient)
// BF: bfloat16 operands (rounded to nearest even when staged) with fp32
// accumulation.  With 16-channel chunks the products run on
// v_mfma_f32_16x16x16_bf16 (k = 16 input channels of one tap): the input
// tile is staged as bf16 with 4 channels interleaved per pixel (one 8-byte
// read is a lane's B operand) and the weights as [m][tap][c] bf16 rows (one
// 8-byte read is its A operand).  Narrower chunks (an image net's first
// layer) keep the fp32 layout and matrix op on operands rounded to bf16,
// which forms the same exact products.
template <int WO, int STRIDE, int TH, int CC, int WK, int WP, int NBW, bool TRANS, int TPW, int FOLD, bool BF>
__global__ __launch_bounds__(64 * WK * WP) void conv3x3_direct(DirArgs a)
{
    static_assert(!FOLD || (TRANS && STRIDE == 1 && TPW == 1), "folded BN backward: stride-1 backward data");
    constexpr int NT = 64 * WK * WP;
    constexpr int WIN = WO * STRIDE;                       // input width
    constexpr int HR = (TH - 1) * STRIDE + 3;              // staged input rows
    constexpr int RSTR = round4(WIN + (STRIDE == 1 ? 5 : 4));  // LDS row stride (cols 3 .. WIN+4)
    constexpr int PS = plane_stride_b(HR * RSTR, WO, STRIDE, RSTR);  // lane groups hit disjoint banks where possible
    constexpr int TK = 16 * WK;
    constexpr int WR = wrow(CC * 9);
    static_assert(TH * WO == 16 * NBW * WP, "pixel tiling");
    static_assert(CC % 4 == 0 && WIN % 4 == 0, "tiling");
    constexpr bool BMF = BF && CC % 16 == 0;                    // bf16 matrix op
    constexpr int RSQ = row_stride_q(RSTR, WO, STRIDE);         // (BMF) row stride, 8-byte elements
    constexpr int QPS = HR * RSQ;                               // (BMF) plane stride of a channel quad
    constexpr int WRQ = wrow(CC * 9 / 2);                       // (BMF) weight row stride, dwords
    constexpr int XS_FLOATS = BMF ? (CC / 4) * QPS * 2 : CC * PS;
    constexpr int WC_FLOATS = BMF ? TK * WRQ : TK * WR;
    __shared__ __attribute__((aligned(16))) float Xs[XS_FLOATS];
    __shared__ __attribute__((aligned(16))) float Wc[WC_FLOATS];
    unsigned short* const Xh = reinterpret_cast<unsigned short*>(Xs);  // (BMF) bf16 views
    unsigned short* const Wh = reinterpret_cast<unsigned short*>(Wc);
    // folded BN backward: per input channel (a, b, d, mean, invstd, scale, shift)
    __shared__ __attribute__((aligned(16))) float ftab[FOLD ? kFoldMaxChannels * 8 : 4];
    // per-wave parts of the epilogue's per-tile channel sums: [2][WP][TK]
    __shared__ float wred[2 * WP * TK];
    // input BN (a.in_bn, forward kernels): scale [kInBnMaxChannels], shift
    constexpr bool IBN = !TRANS && !FOLD;
    __shared__ float ibt[IBN ? 2 * kInBnMaxChannels : 1];

    constexpr int tiles = WO / TH;       // row tiles per (square) image
    static_assert(WO % TH == 0, "row tiles");
    static_assert(TPW == 1 || tiles % TPW == 0, "a workgroup's tiles lie in one image");
    // one-dimensional grid: workgroup -> (image, group of TPW tiles, block of
    // TK output channels).  Image i's workgroups run on XCD i mod 8
    // (consecutive workgroups go to the 8 XCDs in turn), in consecutive
    // rounds of 8, so the row tiles of an image, which share halo rows, and
    // its output-channel blocks, which share the whole input tile, find them
    // in that XCD's L2; indices past the last image (the grid is a multiple
    // of 8 images) do nothing
    constexpr int tgroups = tiles / TPW;
    const int kblocks = a.K / TK, combos = tgroups * kblocks;
    const int slot = (int)(blockIdx.x >> 3) % combos;
    const int image = (int)(blockIdx.x >> 3) / combos * 8 + (int)(blockIdx.x & 7);
    if (image >= a.n) return;
    const int bxl = image * tgroups + slot % tgroups;  // group of TPW consecutive tiles (image-major)
    const int byl = slot / tgroups;                    // output-channel block
    const int T_all = a.n * tiles;       // tiles of the launch (BN partial index)
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wk = wave % WK, wp = wave / WK;
    const int mblk = byl * TK;
    const int g = lane >> 4, j = lane & 15;

    int boff[NBW];  // B operand: fp32 layout, float offset; BMF, byte offset of the 8-byte element
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int pix = (wp * NBW + nb) * 16 + j;
        const int row = pix / WO, col = pix - (pix / WO) * WO;
        boff[nb] = BMF ? (g * QPS + row * STRIDE * RSQ + col * STRIDE + 3) * 8
                       : g * PS + row * STRIDE * RSTR + col * STRIDE + 3;
    }
    v4f acc[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) acc[nb] = v4f{0.f, 0.f, 0.f, 0.f};

    // halo columns: never overwritten by the staging loop below
    if constexpr (BMF) {
        for (int i = tid; i < (CC / 4) * HR; i += NT) {
            const int cq = i / HR, rr = i - (i / HR) * HR;
            uint2* row = reinterpret_cast<uint2*>(Xs) + cq * QPS + rr * RSQ;
            row[3] = make_uint2(0u, 0u);
            if (STRIDE == 1) row[WIN + 4] = make_uint2(0u, 0u);
        }
    } else {
        for (int i = tid; i < CC * HR; i += NT) {
            const int c = i / HR, rr = i - (i / HR) * HR;
            Xs[c * PS + rr * RSTR + 3] = 0.f;
            if (STRIDE == 1) Xs[c * PS + rr * RSTR + WIN + 4] = 0.f;
        }
    }

    // software pipeline over input-channel chunks: the next chunk's tile and
    // weights are loaded into registers while the current chunk computes.
    // A thread's staging coordinates are the same for every chunk and tile,
    // so they are computed once; global offsets are 32-bit (the launcher
    // checks the tensor sizes), so loads take a uniform base and a lane
    // offset.  Images are square: input height = WIN, output height = WO.
    constexpr int Q4 = WIN / 4;
    constexpr int HIN = WIN;
    constexpr int XN = CC * HR * Q4;
    // weights: TK runs of CC*9 floats (forward) or CC runs of TK*9 floats
    // (transposed), both multiples of 4: loaded as float4, stored as scalars
    constexpr int WN4 = TK * CC * 9 / 4;
    static_assert((CC * 9) % 4 == 0 && (TK * 9) % 4 == 0, "float4 weight runs");
    constexpr int XV = (XN + NT - 1) / NT, WV = (WN4 + NT - 1) / NT;
    static_assert(XV <= 32, "okm: one bit per staged float4");
    const bool wvec = (a.C % 4 == 0) && (TRANS ? (a.K % 4 == 0) : true) && ((uintptr_t)a.w % 16 == 0);
    int xl[XV], xg[XV], xrow[XV], xch[XV];  // LDS offset, offset from (plane c0, row ih0), row, channel
#pragma unroll
    for (int k = 0; k < XV; ++k) {
        const int i = tid + k * NT;
        const int c = i / (HR * Q4);
        const int rem = i - c * (HR * Q4);
        const int rr = rem / Q4, q4 = rem - (rem / Q4) * Q4;
        // fp32: float offset of the 4 pixels; BMF: bf16 offset of the first
        // pixel's slot of channel c (the next pixels are 4 bf16 apart)
        xl[k] = BMF ? ((c / 4) * QPS + rr * RSQ + 4 + q4 * 4) * 4 + (c % 4) : c * PS + rr * RSTR + 4 + q4 * 4;
        xg[k] = (c * HIN + rr) * WIN + q4 * 4;
        xrow[k] = rr;
        xch[k] = i < XN ? c : CC;  // CC: past the chunk (never loaded or stored)
    }
    int wl[WV], wg[WV], wc[WV];  // forward: LDS offset, offset from channel 0, channel; transposed: run base
    int wq[BMF ? WV : 1][4];     // BMF: bf16 LDS offset of each of the 4 weights, [m][tap][c] rows
#pragma unroll
    for (int k = 0; k < WV; ++k) {
        const int i = (tid + k * NT) * 4;
        if (!TRANS) {
            const int m = i / (CC * 9), rem = i - (i / (CC * 9)) * (CC * 9);
            wl[k] = m * WR + rem;
            wg[k] = (mblk + m) * a.C * 9 + rem;
            wc[k] = rem / 9;  // first channel of the run (a run of 4 may cross into the next channel)
        } else {
            const int c = i / (TK * 9), rem = i - (i / (TK * 9)) * (TK * 9);
            wl[k] = rem;
            wg[k] = c * a.K * 9 + mblk * 9 + rem;
            wc[k] = c;
        }
        if (i >= WN4 * 4) wc[k] = -1;  // past the weights of a chunk
        if constexpr (BMF) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                int m, c, tap;
                if (!TRANS) {  // run of output channel m: (c, tap) = divmod(rem + e, 9)
                    m = i / (CC * 9);
                    const int r2 = i - m * (CC * 9) + e;
                    c = r2 / 9;
                    tap = r2 - c * 9;
                } else {       // run of input channel c: (m, 8 - tap) = divmod(rem + e, 9), taps flipped
                    c = i / (TK * 9);
                    const int r2 = i - c * (TK * 9) + e;
                    m = r2 / 9;
                    tap = 8 - (r2 - m * 9);
                }
                wq[k][e] = m * 2 * WRQ + tap * CC + c;
            }
        }
    }
    float4 xr[XV];
    float4 wr[WV];
    float4 fyr[FOLD ? XV : 1];  // folded BN: xr holds its output gradient, fyr its input
    float4 fzr[FOLD == 2 ? XV : 1];  // and fzr its output (ReLU mask) when it has a residual
    unsigned okm = 0;           // folded BN, input BN: bit k set when element k lies inside the tensor
    // Loads are issued without branches: a lane whose element lies outside
    // the tensor (halo rows, channels past C, threads past the chunk) loads
    // from offset 0 and keeps zero, so the compiler can count outstanding
    // memory operations exactly instead of waiting for all of them.
    const bool wfast = wvec && (a.C % CC == 0);  // every weight run of every chunk is in range
    auto load_chunk = [&](int img, int ih0, int c0) {  // channels c0.. of tile (img, rows from ih0)
        const int xb = ((img * a.C + c0) * HIN + ih0) * WIN;
        if constexpr (FOLD) okm = 0;
#pragma unroll
        for (int k = 0; k < XV; ++k) {
            const int ih = ih0 + xrow[k];
            const bool ok = ((k + 1) * NT <= XN || xch[k] < CC) && ih >= 0 && ih < HIN && c0 + xch[k] < a.C;
            if constexpr (FOLD) {
                const float4 v = *reinterpret_cast<const float4*>(a.fold.g + (ok ? xb + xg[k] : 0));
                const float4 u = *reinterpret_cast<const float4*>(a.fold.y + (ok ? xb + xg[k] : 0));
                xr[k] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
                fyr[k] = ok ? u : make_float4(0.f, 0.f, 0.f, 0.f);
                if constexpr (FOLD == 2) {
                    const float4 w = *reinterpret_cast<const float4*>(a.fold.z + (ok ? xb + xg[k] : 0));
                    fzr[k] = ok ? w : make_float4(0.f, 0.f, 0.f, 0.f);
                }
                okm |= ok ? 1u << k : 0u;
            } else {
                const float4 v = *reinterpret_cast<const float4*>(a.x + (ok ? xb + xg[k] : 0));
                xr[k] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
                if constexpr (IBN) okm = (okm & ~(1u << k)) | (ok ? 1u << k : 0u);
            }
        }
        if (wfast) {
#pragma unroll
            for (int k = 0; k < WV; ++k) {
                const bool ok = (k + 1) * NT * 4 <= WN4 * 4 || wc[k] >= 0;
                const int off = TRANS ? wg[k] + c0 * a.K * 9 : wg[k] + c0 * 9;
                const float4 v = *reinterpret_cast<const float4*>(a.w + (ok ? off : 0));
                wr[k] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
            }
            return;
        }
#pragma unroll
        for (int k = 0; k < WV; ++k) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (wc[k] >= 0) {
                if (!TRANS) {  // w[m][c][rs]: each output channel's CC*9 run is contiguous
                    const float* src = a.w + (wg[k] + c0 * 9);
                    if (wvec && c0 + CC <= a.C) {
                        v = *reinterpret_cast<const float4*>(src);
                    } else {  // narrow input (C < CC) or misaligned: element-wise with bounds
                        const int rem = wl[k] - (wl[k] / WR) * WR;
                        float t[4];
                        for (int e = 0; e < 4; ++e) t[e] = (c0 + (rem + e) / 9 < a.C) ? src[e] : 0.f;
                        v = make_float4(t[0], t[1], t[2], t[3]);
                    }
                } else {       // w_layer[c][m][rs]: each input channel's TK*9 run is contiguous
                    const float* src = a.w + (wg[k] + c0 * a.K * 9);
                    if (c0 + wc[k] < a.C) {
                        if (wvec) {
                            v = *reinterpret_cast<const float4*>(src);
                        } else {
                            v = make_float4(src[0], src[1], src[2], src[3]);
                        }
                    }
                }
            }
            wr[k] = v;
        }
    };
    // folded BN: the staged tile's own rows (1..TH) of dy go to global memory
    // after the barrier that follows the staging, so that the stores drain
    // under the matrix loop instead of delaying the barrier
    auto write_dy = [&](int img, int ih0, int c0) {
        if constexpr (FOLD) {
            if (byl != 0) return;
            const int xb = ((img * a.C + c0) * HIN + ih0) * WIN;
#pragma unroll
            for (int k = 0; k < XV; ++k)
                if ((okm & (1u << k)) && xrow[k] >= 1 && xrow[k] <= TH) {
                    store_stream4(a.fold.dy + xb + xg[k], xr[k]);
                    if constexpr (FOLD == 2) store_stream4(a.fold.dres + xb + xg[k], fyr[k]);
                }
        }
    };
    // one staged float4 of the input tile (4 pixels of one channel)
    auto put_x = [&](int k, float4 v) {
        if constexpr (BMF) {
            Xh[xl[k]] = bf16_bits(v.x);
            Xh[xl[k] + 4] = bf16_bits(v.y);
            Xh[xl[k] + 8] = bf16_bits(v.z);
            Xh[xl[k] + 12] = bf16_bits(v.w);
        } else if constexpr (BF) {
            *reinterpret_cast<float4*>(&Xs[xl[k]]) =
                make_float4(bf16_round(v.x), bf16_round(v.y), bf16_round(v.z), bf16_round(v.w));
        } else {
            *reinterpret_cast<float4*>(&Xs[xl[k]]) = v;
        }
    };
    auto store_chunk = [&](int img, int ih0, int c0) {
        (void)img;
        (void)ih0;
        if constexpr (FOLD) {  // the BN backward of each staged element, in the order of bn_bwd_partials_k
#pragma unroll
            for (int k = 0; k < XV; ++k) {
                if (!((k + 1) * NT <= XN || xch[k] < CC)) continue;
                float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
                if (okm & (1u << k)) {
                    const float4 f0 = *reinterpret_cast<const float4*>(ftab + (c0 + xch[k]) * 8);
                    const float4 f1 = *reinterpret_cast<const float4*>(ftab + (c0 + xch[k]) * 8 + 4);
                    const float fa = f0.x, fb = f0.y, fd = f0.z, mu = f0.w, is = f1.x, sc = f1.y, sf = f1.z;
                    const float gg[4] = {xr[k].x, xr[k].y, xr[k].z, xr[k].w};
                    const float yy[4] = {fyr[k].x, fyr[k].y, fyr[k].z, fyr[k].w};
                    float zz[4] = {1.f, 1.f, 1.f, 1.f};
                    if constexpr (FOLD == 2) {
                        zz[0] = fzr[k].x; zz[1] = fzr[k].y; zz[2] = fzr[k].z; zz[3] = fzr[k].w;
                    }
                    float r[4], gms[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const bool pass = FOLD == 2 ? zz[e] > 0.f : __fmaf_rn(yy[e], sc, sf) > 0.f;
                        const float gm = (a.fold.relu && !pass) ? 0.f : gg[e];
                        const float xh = (yy[e] - mu) * is;
                        r[e] = fa * (gm - fb - xh * fd);
                        gms[e] = gm;
                    }
                    o = make_float4(r[0], r[1], r[2], r[3]);
                    if constexpr (FOLD == 2) fyr[k] = make_float4(gms[0], gms[1], gms[2], gms[3]);  // the residual's gradient
                }
                put_x(k, o);
                xr[k] = o;  // written out by write_dy
            }
        } else {
#pragma unroll
            for (int k = 0; k < XV; ++k) {
                if (!((k + 1) * NT <= XN || xch[k] < CC)) continue;
                float4 v = xr[k];
                if constexpr (IBN) {
                    if (a.in_bn) {  // the BN + ReLU of the stored input, exactly as its apply kernel forms it
                        const int ch = c0 + xch[k] < a.C ? c0 + xch[k] : 0;
                        const float sc = ibt[ch], sf = ibt[kInBnMaxChannels + ch];
                        v = (okm & (1u << k)) ? make_float4(fmaxf(__fmaf_rn(v.x, sc, sf), 0.f),
                                                            fmaxf(__fmaf_rn(v.y, sc, sf), 0.f),
                                                            fmaxf(__fmaf_rn(v.z, sc, sf), 0.f),
                                                            fmaxf(__fmaf_rn(v.w, sc, sf), 0.f))
                                              : make_float4(0.f, 0.f, 0.f, 0.f);
                    }
                }
                put_x(k, v);
            }
        }
#pragma unroll
        for (int k = 0; k < WV; ++k) {
            if (!((k + 1) * NT * 4 <= WN4 * 4 || wc[k] >= 0)) continue;
            float vv[4] = {wr[k].x, wr[k].y, wr[k].z, wr[k].w};
            if constexpr (BMF) {
#pragma unroll
                for (int e = 0; e < 4; ++e) Wh[wq[k][e]] = bf16_bits(vv[e]);
                continue;
            }
            if constexpr (BF)
#pragma unroll
                for (int e = 0; e < 4; ++e) vv[e] = bf16_round(vv[e]);
            if (!TRANS) {
#pragma unroll
                for (int e = 0; e < 4; ++e) Wc[wl[k] + e] = vv[e];  // a run never crosses m (CC*9 % 4 == 0)
            } else {  // flip the taps
                const int rem = wl[k];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = (rem + e) / 9, rsl = (rem + e) - ((rem + e) / 9) * 9;
                    Wc[m * WR + wc[k] * 9 + 8 - rsl] = vv[e];
                }
            }
        }
    };

    // TPW consecutive row tiles per workgroup; the software pipeline runs
    // across them: the first chunk of the next tile is loaded while the last
    // chunk of the current one is on the matrix cores
    load_chunk(bxl * TPW / tiles, (bxl * TPW % tiles) * TH * STRIDE - 1, 0);
    if constexpr (IBN) {  // after the first tile's loads are issued; read after the chunk loop's first barrier
        if (a.in_bn)
            for (int i = tid; i < a.C; i += NT) {
                ibt[i] = a.in_bn[i];
                ibt[kInBnMaxChannels + i] = a.in_bn[a.C + i];
            }
    }
    if constexpr (FOLD) {
        // merge the BN's per-tile sums while the first tile loads are in
        // flight: G = NT / C consecutive threads per channel, thread q of a
        // channel sums tiles q, q+G, ... in fp64, then the G partial sums
        // meet in a fixed xor tree; the table is read after the first
        // barrier below
        const int G = NT / a.C;
        const int ch = tid / G, q = tid - (tid / G) * G;
        const float2* pp = reinterpret_cast<const float2*>(a.fold.part) + (size_t)ch * a.fold.T;
        // tiles q, q+G, ... in that order: nf of them for every thread (16
        // unconditional loads in flight at a time), then one more for the
        // first T - nf*G threads
        double s1 = 0.0, s2 = 0.0;
        const int nf = a.fold.T / G;
        int u = 0;
        for (; u + 16 <= nf; u += 16) {
            float2 v[16];
#pragma unroll
            for (int k = 0; k < 16; ++k) v[k] = pp[q + (u + k) * G];
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                s1 += (double)v[k].x;
                s2 += (double)v[k].y;
            }
        }
        for (; u < nf; ++u) {
            const float2 v = pp[q + u * G];
            s1 += (double)v.x;
            s2 += (double)v.y;
        }
        if (q < a.fold.T - nf * G) {
            const float2 v = pp[q + nf * G];
            s1 += (double)v.x;
            s2 += (double)v.y;
        }
        for (int off = G / 2; off > 0; off >>= 1) {
            s1 += __shfl_xor(s1, off, G);
            s2 += __shfl_xor(s2, off, G);
        }
        if (q == 0) {
            const float is = a.fold.invstd[ch];
            ftab[ch * 8 + 0] = (float)((double)a.fold.gamma[ch] * (double)is);
            ftab[ch * 8 + 1] = (float)(s1 / a.fold.count);
            ftab[ch * 8 + 2] = (float)(s2 / a.fold.count);
            ftab[ch * 8 + 3] = a.fold.mean[ch];
            ftab[ch * 8 + 4] = is;
            ftab[ch * 8 + 5] = a.fold.relu ? a.fold.scale[ch] : 0.f;
            ftab[ch * 8 + 6] = a.fold.relu ? a.fold.scale[a.C + ch] : 0.f;
            if (bxl == 0 && byl == 0) {
                a.fold.dbeta[ch] = (float)s1;
                a.fold.dgamma[ch] = (float)s2;
            }
        }
    }
    // backward sums with one tile per workgroup: the BN tensors the epilogue
    // reads are loaded now, so that their latency passes under the matrix work
    constexpr bool PRE = TRANS && TPW == 1;
    float pyy[PRE ? NBW : 1][4], pzz[PRE ? NBW : 1][4];
    if constexpr (PRE) {
        if (a.bnb.part) {
            const int img = bxl / tiles, oh0 = (bxl - img * tiles) * TH;
            const bool zmask = a.bnb.relu && !a.bnb.scale;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                const int pix = (wp * NBW + nb) * 16 + j;
                const int row = pix / WO, col = pix - (pix / WO) * WO;
                const int o = ((img * a.K + mblk + wk * 16 + 4 * g) * WO + oh0 + row) * WO + col;
#pragma unroll
                for (int i = 0; i < 4; ++i) pyy[nb][i] = a.bnb.y[o + i * WO * WO];
                if (zmask)
#pragma unroll
                    for (int i = 0; i < 4; ++i) pzz[nb][i] = a.bnb.z[o + i * WO * WO];
            }
        }
    }
    for (int q = 0; q < TPW; ++q) {
    const int tl = bxl * TPW + q;
    const int img = tl / tiles;
    const int oh0 = (tl - img * tiles) * TH;
    for (int c0 = 0; c0 < a.C; c0 += CC) {
        __syncthreads();  // the previous chunk's LDS reads are complete
        store_chunk(img, oh0 * STRIDE - 1, c0);
        __syncthreads();
        write_dy(img, oh0 * STRIDE - 1, c0);
        if (c0 + CC < a.C)
            load_chunk(img, oh0 * STRIDE - 1, c0 + CC);
        else if (q + 1 < TPW)
            load_chunk((tl + 1) / tiles, ((tl + 1) % tiles) * TH * STRIDE - 1, 0);
        if constexpr (BMF) {
            // lane (j, g): A = weights of output channel j, channels 4g..4g+3 of
            // the 16-channel group, one tap; B = those 4 channels of pixel j
            const char* wfb = reinterpret_cast<const char*>(Wc) + (wk * 16 + j) * WRQ * 4 + g * 8;
            const char* xfb = reinterpret_cast<const char*>(Xs);
#pragma unroll
            for (int c16 = 0; c16 < CC / 16; ++c16)
#pragma unroll
                for (int r = 0; r < 3; ++r)
#pragma unroll
                    for (int s = 0; s < 3; ++s) {
                        const v4s av = *reinterpret_cast<const v4s*>(wfb + ((r * 3 + s) * CC + c16 * 16) * 2);
#pragma unroll
                        for (int nb = 0; nb < NBW; ++nb) {
                            const v4s bv = *reinterpret_cast<const v4s*>(
                                xfb + boff[nb] + (c16 * 4 * QPS + r * RSQ + s) * 8);
                            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, bv, acc[nb], 0, 0, 0);
                        }
                    }
        } else {
            const float* wf = Wc + (wk * 16 + j) * WR + g * 9;
#pragma unroll
            for (int c4 = 0; c4 < CC / 4; ++c4)
#pragma unroll
                for (int r = 0; r < 3; ++r)
#pragma unroll
                    for (int s = 0; s < 3; ++s) {
                        const float av = wf[c4 * 36 + r * 3 + s];
#pragma unroll
                        for (int nb = 0; nb < NBW; ++nb) {
                            const float bv = Xs[boff[nb] + c4 * 4 * PS + r * RSTR + s];
                            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[nb], 0, 0, 0);
                        }
                    }
        }
    }

    // epilogue: every global load is issued before the first store (the
    // output may alias nothing, but the compiler cannot know that, and a
    // load after a store would wait for it)
    int oidx[NBW];  // index of (channel mblk+wk*16+4g, pixel) of block nb
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int pix = (wp * NBW + nb) * 16 + j;
        const int row = pix / WO, col = pix - (pix / WO) * WO;
        oidx[nb] = ((img * a.K + mblk + wk * 16 + 4 * g) * WO + oh0 + row) * WO + col;
    }
    constexpr int cstr = WO * WO;  // channel stride
    if (a.accumulate) {
        float old[NBW][4];
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) old[nb][i] = a.y[oidx[nb] + i * cstr];
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[nb][i] += old[nb][i];
    }
    float gs1[4] = {0.f, 0.f, 0.f, 0.f}, gs2[4] = {0.f, 0.f, 0.f, 0.f};
    if (TRANS && a.bnb.part) {  // acc is the final gradient of the preceding BN's output
        const bool zmask = a.bnb.relu && !a.bnb.scale, ymask = a.bnb.relu && a.bnb.scale;
        float zz[NBW][4], yy[NBW][4], mu[4], is[4], sc[4], sf[4];
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if constexpr (PRE) {
                    yy[nb][i] = pyy[nb][i];
                    zz[nb][i] = zmask ? pzz[nb][i] : 1.f;
                } else {
                    yy[nb][i] = a.bnb.y[oidx[nb] + i * cstr];
                    zz[nb][i] = zmask ? a.bnb.z[oidx[nb] + i * cstr] : 1.f;
                }
            }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = mblk + wk * 16 + 4 * g + i;
            mu[i] = a.bnb.mean[m];
            is[i] = a.bnb.invstd[m];
            sc[i] = ymask ? a.bnb.scale[m] : 0.f;
            sf[i] = ymask ? a.bnb.shift[m] : 0.f;
        }
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bool pass = ymask ? __fmaf_rn(yy[nb][i], sc[i], sf[i]) > 0.f : zz[nb][i] > 0.f;
                const float gg = (a.bnb.relu && !pass) ? 0.f : acc[nb][i];
                gs1[i] += gg;
                gs2[i] += gg * ((yy[nb][i] - mu[i]) * is[i]);
            }
    }
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) store_stream(a.y + oidx[nb] + i * cstr, acc[nb][i]);
    if constexpr (TRANS) {
        if (a.bnb.part) {  // per-tile backward sums of each channel
            float* red = wred;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                gs1[i] = row16_sum(gs1[i]);
                gs2[i] = row16_sum(gs2[i]);
            }
            if (j == 0)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    red[wp * TK + wk * 16 + 4 * g + i] = gs1[i];
                    red[(WP + wp) * TK + wk * 16 + 4 * g + i] = gs2[i];
                }
            __syncthreads();
            if (wp == 0 && j == 0)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float t1 = 0.f, t2 = 0.f;
                    for (int q = 0; q < WP; ++q) {
                        t1 += red[q * TK + wk * 16 + 4 * g + i];
                        t2 += red[(WP + q) * TK + wk * 16 + 4 * g + i];
                    }
                    const int m = mblk + wk * 16 + 4 * g + i;
                    a.bnb.part[((size_t)m * T_all + tl) * 2 + 0] = t1;
                    a.bnb.part[((size_t)m * T_all + tl) * 2 + 1] = t2;
                }
            if (TPW > 1) __syncthreads();  // wred is written again by the next tile
        }
    }
    if constexpr (!TRANS) {
        if (a.bn.part) {
            // per-tile statistics of each output channel over the TH*WO
            // pixels: each wave takes the two-pass (mean, M2) of its own
            // 16*NBW pixels in registers, and one lane per channel combines
            // the WP equal-count parts (mean = mean of the means, M2 = sum
            // of the M2 + n * sum of the squared mean deviations)
            // (a lane's NBW values first, then the 16 lanes of its row)
            constexpr float PW = 16.f * NBW;
            float wm[4], wq[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float v = 0.f;
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) v += acc[nb][i];
                wm[i] = v / (float)NBW;
                float q = 0.f;
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) {
                    const float d = acc[nb][i] - wm[i];
                    q += d * d;
                }
                wq[i] = q;
                row16_meanvar(wm[i], wq[i], (float)NBW);
            }
            if (j == 0)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    wred[wp * TK + wk * 16 + 4 * g + i] = wm[i];
                    wred[(WP + wp) * TK + wk * 16 + 4 * g + i] = wq[i];
                }
            __syncthreads();
            if (wp == 0 && j == 0)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int c = wk * 16 + 4 * g + i;
                    float mu = 0.f;
                    for (int q = 0; q < WP; ++q) mu += wred[q * TK + c];
                    mu /= (float)WP;
                    float m2 = 0.f, dev = 0.f;
                    for (int q = 0; q < WP; ++q) {
                        const float d = wred[q * TK + c] - mu;
                        m2 += wred[(WP + q) * TK + c];
                        dev += d * d;
                    }
                    const int m = mblk + c;
                    a.bn.part[((size_t)m * T_all + tl) * 2 + 0] = mu;
                    a.bn.part[((size_t)m * T_all + tl) * 2 + 1] = m2 + PW * dev;
                }
            if (TPW > 1) __syncthreads();  // wred is written again by the next tile
        }
    }
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) acc[nb] = v4f{0.f, 0.f, 0.f, 0.f};
    }  // tiles
}

// Backward-data of a 3x3 / pad 1 / stride 2 convolution: dx (H = 2*HO) from
// dy.  Output pixel (2i+ph, 2j+pw) receives dy[i+di][j+dj] w[r][s] for the
// taps with 2i+ph = 2(i+di)+r-1:  ph = 0 -> r = 1 (di 0);  ph = 1 -> r = 0
// (di 1) and r = 2 (di 0); likewise for columns.  A 16-pixel block of dy
// positions therefore feeds four output parity classes from only four
// B fragments (di, dj in {0,1}); the nine taps are nine MFMAs.  Each lane
// stores the pw = 0,1 pair of a class row as one float2.
struct DgArgs {
    const float* dy;  // [n][KL][HO][WO]
    const float* w;   // layer weights [KL][CL][3][3]
    float* dx;        // [n][CL][2*HO][2*WO]
    int KL, CL, HO;
    int accumulate;
    BnBwdFuse bnb;    // bnb.part == nullptr: no backward sums
};

// BF: bf16 operands on v_mfma_f32_16x16x16_bf16 (16 dy channels per k-step),
// staged as in conv3x3_direct (dy tile with 4 channels interleaved per
// pixel, weights as [m][tap][c] bf16 rows).
template <int WO, int TH, int CC, int WK, int WP, int NBW, bool BF>
__global__ __launch_bounds__(64 * WK * WP) void conv3x3_dgrad_s2(DgArgs a)
{
    constexpr int NT = 64 * WK * WP;
    constexpr int HR = TH + 1;                 // dy rows i0 .. i0+TH (the last may be past the edge)
    constexpr int RSTR = round4(WO + 1);       // dy cols 0 .. WO (col WO is zero)
    constexpr int PS = plane_stride_b(HR * RSTR, WO, 1, RSTR);
    constexpr int TK = 16 * WK;
    constexpr int WR = wrow(CC * 9);
    static_assert(TH * WO == 16 * NBW * WP, "pixel tiling");
    static_assert(!BF || CC % 16 == 0, "bf16: 16-channel chunks");
    constexpr int RSQ = row_stride_q(RSTR, WO, 1);  // (BF) row stride, 8-byte elements
    constexpr int QPS = HR * RSQ;                   // (BF) plane stride of a channel quad
    constexpr int WRQ = wrow(CC * 9 / 2);           // (BF) weight row stride, dwords
    constexpr int XS_FLOATS = BF ? (CC / 4) * QPS * 2 : CC * PS;
    constexpr int WC_FLOATS = BF ? TK * WRQ : TK * WR;
    static_assert(XS_FLOATS >= 2 * WP * TK, "input tile reused by the backward-sums epilogue");
    __shared__ __attribute__((aligned(16))) float Xs[XS_FLOATS];
    __shared__ __attribute__((aligned(16))) float Wc[WC_FLOATS];
    unsigned short* const Xh = reinterpret_cast<unsigned short*>(Xs);
    unsigned short* const Wh = reinterpret_cast<unsigned short*>(Wc);

    const int tiles = a.HO / TH;
    const int img = blockIdx.x / tiles;
    const int i0 = (blockIdx.x - img * tiles) * TH;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wk = wave % WK, wp = wave / WK;
    const int mblk = blockIdx.y * TK;
    const int g = lane >> 4, j = lane & 15;

    int boff[NBW];  // fp32: float offset; BF: byte offset of the 8-byte element
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int pix = (wp * NBW + nb) * 16 + j;
        boff[nb] = BF ? (g * QPS + (pix / WO) * RSQ + (pix - (pix / WO) * WO)) * 8
                      : g * PS + (pix / WO) * RSTR + (pix - (pix / WO) * WO);
    }
    v4f acc[NBW][4];  // [block][class ph*2+pw]
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[nb][q] = v4f{0.f, 0.f, 0.f, 0.f};

    if constexpr (BF) {
        for (int i = tid; i < (CC / 4) * HR; i += NT) {
            const int cq = i / HR, rr = i - (i / HR) * HR;
            reinterpret_cast<uint2*>(Xs)[cq * QPS + rr * RSQ + WO] = make_uint2(0u, 0u);
        }
    } else {
        for (int i = tid; i < CC * HR; i += NT) {
            const int c = i / HR, rr = i - (i / HR) * HR;
            Xs[c * PS + rr * RSTR + WO] = 0.f;
        }
    }
    // Software pipeline over chunks of CC dy channels: the next chunk's dy
    // tile and weights are loaded into registers while the current one is
    // on the matrix cores.  Per-thread staging coordinates are fixed.
    constexpr int Q4 = WO / 4;
    constexpr int XN = CC * HR * Q4, XV = (XN + NT - 1) / NT;
    // weights w_layer[c][m][rs]: for each dy channel c of the chunk a run of
    // TK*9 floats (output channels mblk.. of dx), loaded as float4
    constexpr int WN4 = CC * TK * 9 / 4, WV = (WN4 + NT - 1) / NT;
    static_assert((TK * 9) % 4 == 0, "float4 weight runs");
    int xl[XV], xg[XV], xrow[XV];
    bool xon[XV];
#pragma unroll
    for (int k = 0; k < XV; ++k) {
        const int i = tid + k * NT;
        const int c = i / (HR * Q4), rem = i - (i / (HR * Q4)) * (HR * Q4);
        const int rr = rem / Q4, q4 = rem - (rem / Q4) * Q4;
        xon[k] = i < XN;
        // fp32: float offset of the 4 pixels; BF: bf16 offset of the first pixel's slot of channel c
        xl[k] = BF ? ((c / 4) * QPS + rr * RSQ + q4 * 4) * 4 + (c % 4) : c * PS + rr * RSTR + q4 * 4;
        xg[k] = (c * a.HO + rr) * WO + q4 * 4;  // from (plane c0, row i0)
        xrow[k] = rr;
    }
    int wg[WV], wl[WV][4];
    bool won[WV];
#pragma unroll
    for (int k = 0; k < WV; ++k) {
        const int i = (tid + k * NT) * 4;
        won[k] = i < WN4 * 4;
        const int c = i / (TK * 9), rem = i - (i / (TK * 9)) * (TK * 9);
        wg[k] = c * a.CL * 9 + mblk * 9 + rem;  // from dy channel c0
#pragma unroll
        for (int e = 0; e < 4; ++e) {  // a run of 4 never crosses c (TK*9 % 4 == 0)
            const int m = (rem + e) / 9, rs = (rem + e) - ((rem + e) / 9) * 9;
            wl[k][e] = BF ? m * 2 * WRQ + rs * CC + c : m * WR + c * 9 + rs;
        }
    }
    float4 xr[XV], wr[WV];
    auto load_chunk = [&](int c0) {
        const int xb = ((img * a.KL + c0) * a.HO + i0) * WO;
#pragma unroll
        for (int k = 0; k < XV; ++k) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (xon[k] && i0 + xrow[k] < a.HO) v = *reinterpret_cast<const float4*>(a.dy + (xb + xg[k]));
            xr[k] = v;
        }
        const float* wb = a.w + (size_t)c0 * a.CL * 9;
#pragma unroll
        for (int k = 0; k < WV; ++k)
            wr[k] = won[k] ? *reinterpret_cast<const float4*>(wb + wg[k]) : make_float4(0.f, 0.f, 0.f, 0.f);
    };
    load_chunk(0);
    for (int c0 = 0; c0 < a.KL; c0 += CC) {
        __syncthreads();  // the previous chunk's LDS reads are complete
#pragma unroll
        for (int k = 0; k < XV; ++k)
            if (xon[k]) {
                if constexpr (BF) {
                    Xh[xl[k]] = bf16_bits(xr[k].x);
                    Xh[xl[k] + 4] = bf16_bits(xr[k].y);
                    Xh[xl[k] + 8] = bf16_bits(xr[k].z);
                    Xh[xl[k] + 12] = bf16_bits(xr[k].w);
                } else {
                    *reinterpret_cast<float4*>(&Xs[xl[k]]) = xr[k];
                }
            }
#pragma unroll
        for (int k = 0; k < WV; ++k)
            if (won[k]) {
                if constexpr (BF) {
                    Wh[wl[k][0]] = bf16_bits(wr[k].x);
                    Wh[wl[k][1]] = bf16_bits(wr[k].y);
                    Wh[wl[k][2]] = bf16_bits(wr[k].z);
                    Wh[wl[k][3]] = bf16_bits(wr[k].w);
                } else {
                    Wc[wl[k][0]] = wr[k].x;
                    Wc[wl[k][1]] = wr[k].y;
                    Wc[wl[k][2]] = wr[k].z;
                    Wc[wl[k][3]] = wr[k].w;
                }
            }
        __syncthreads();
        if (c0 + CC < a.KL) load_chunk(c0 + CC);
        if constexpr (BF) {
            // lane (j, g): A = weights of dx channel j, dy channels 4g..4g+3 of
            // the 16-channel group, one tap; B = those dy channels at one position
            const char* wfb = reinterpret_cast<const char*>(Wc) + (wk * 16 + j) * WRQ * 4 + g * 8;
            const char* xfb = reinterpret_cast<const char*>(Xs);
#pragma unroll
            for (int c16 = 0; c16 < CC / 16; ++c16) {
                v4s w9[9];
#pragma unroll
                for (int t = 0; t < 9; ++t) w9[t] = *reinterpret_cast<const v4s*>(wfb + (t * CC + c16 * 16) * 2);
#pragma unroll
                for (int nb = 0; nb < NBW; ++nb) {
                    const char* xb = xfb + boff[nb] + c16 * 4 * QPS * 8;
                    const v4s b00 = *reinterpret_cast<const v4s*>(xb), b01 = *reinterpret_cast<const v4s*>(xb + 8);
                    const v4s b10 = *reinterpret_cast<const v4s*>(xb + RSQ * 8);
                    const v4s b11 = *reinterpret_cast<const v4s*>(xb + RSQ * 8 + 8);
                    acc[nb][0] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[4], b00, acc[nb][0], 0, 0, 0);
                    acc[nb][1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[3], b01, acc[nb][1], 0, 0, 0);
                    acc[nb][1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[5], b00, acc[nb][1], 0, 0, 0);
                    acc[nb][2] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[1], b10, acc[nb][2], 0, 0, 0);
                    acc[nb][2] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[7], b00, acc[nb][2], 0, 0, 0);
                    acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[0], b11, acc[nb][3], 0, 0, 0);
                    acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[2], b10, acc[nb][3], 0, 0, 0);
                    acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[6], b01, acc[nb][3], 0, 0, 0);
                    acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(w9[8], b00, acc[nb][3], 0, 0, 0);
                }
            }
            continue;
        }
        const float* wf = Wc + (wk * 16 + j) * WR + g * 9;
#pragma unroll
        for (int c4 = 0; c4 < CC / 4; ++c4) {
            float w9[9];
#pragma unroll
            for (int t = 0; t < 9; ++t) w9[t] = wf[c4 * 36 + t];
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                const float* xb = Xs + boff[nb] + c4 * 4 * PS;
                const float b00 = xb[0], b01 = xb[1], b10 = xb[RSTR], b11 = xb[RSTR + 1];
                // class (0,0): r=1,s=1
                acc[nb][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[4], b00, acc[nb][0], 0, 0, 0);
                // class (0,1): r=1; s=0 -> dj 1, s=2 -> dj 0
                acc[nb][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[3], b01, acc[nb][1], 0, 0, 0);
                acc[nb][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[5], b00, acc[nb][1], 0, 0, 0);
                // class (1,0): s=1; r=0 -> di 1, r=2 -> di 0
                acc[nb][2] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[1], b10, acc[nb][2], 0, 0, 0);
                acc[nb][2] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[7], b00, acc[nb][2], 0, 0, 0);
                // class (1,1)
                acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[0], b11, acc[nb][3], 0, 0, 0);
                acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[2], b10, acc[nb][3], 0, 0, 0);
                acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[6], b01, acc[nb][3], 0, 0, 0);
                acc[nb][3] = __builtin_amdgcn_mfma_f32_16x16x4f32(w9[8], b00, acc[nb][3], 0, 0, 0);
            }
        }
    }
    constexpr int W2 = 2 * WO;
    const int H2 = 2 * a.HO;
    // all loads before the first store (see the direct kernel's epilogue)
    size_t oidx[NBW];  // dx index of (channel mblk+wk*16+4g, row 2ii, col 2jj) of block nb
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int pix = (wp * NBW + nb) * 16 + j;
        const int ii = i0 + pix / WO, jj = pix - (pix / WO) * WO;
        oidx[nb] = (((size_t)img * a.CL + mblk + wk * 16 + 4 * g) * H2 + 2 * ii) * W2 + 2 * jj;
    }
    const size_t cstr = (size_t)H2 * W2;
    // element (nb, v, ph): dx[oidx[nb] + v*cstr + ph*W2 + {0,1}] = classes (ph,0), (ph,1)
    float2 val[NBW][4][2];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int ph = 0; ph < 2; ++ph) val[nb][v][ph] = make_float2(acc[nb][2 * ph][v], acc[nb][2 * ph + 1][v]);
    if (a.accumulate) {
        float2 old[NBW][4][2];
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int ph = 0; ph < 2; ++ph)
                    old[nb][v][ph] = *reinterpret_cast<const float2*>(a.dx + oidx[nb] + v * cstr + ph * W2);
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int ph = 0; ph < 2; ++ph) {
                    val[nb][v][ph].x += old[nb][v][ph].x;
                    val[nb][v][ph].y += old[nb][v][ph].y;
                }
    }
    float gs1[4] = {0.f, 0.f, 0.f, 0.f}, gs2[4] = {0.f, 0.f, 0.f, 0.f};
    if (a.bnb.part) {
        const bool zmask = a.bnb.relu && !a.bnb.scale, ymask = a.bnb.relu && a.bnb.scale;
        float2 zz[NBW][4][2], yy[NBW][4][2];
        float mu[4], is[4], sc[4], sf[4];
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int ph = 0; ph < 2; ++ph) {
                    yy[nb][v][ph] = *reinterpret_cast<const float2*>(a.bnb.y + oidx[nb] + v * cstr + ph * W2);
                    zz[nb][v][ph] = zmask ? *reinterpret_cast<const float2*>(a.bnb.z + oidx[nb] + v * cstr + ph * W2)
                                          : make_float2(1.f, 1.f);
                }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = mblk + wk * 16 + 4 * g + v;
            mu[v] = a.bnb.mean[m];
            is[v] = a.bnb.invstd[m];
            sc[v] = ymask ? a.bnb.scale[m] : 0.f;
            sf[v] = ymask ? a.bnb.shift[m] : 0.f;
        }
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int ph = 0; ph < 2; ++ph) {
                    const float2 gv = val[nb][v][ph], zv = zz[nb][v][ph], yv = yy[nb][v][ph];
                    const bool p0 = ymask ? __fmaf_rn(yv.x, sc[v], sf[v]) > 0.f : zv.x > 0.f;
                    const bool p1 = ymask ? __fmaf_rn(yv.y, sc[v], sf[v]) > 0.f : zv.y > 0.f;
                    const float g0 = (a.bnb.relu && !p0) ? 0.f : gv.x;
                    const float g1 = (a.bnb.relu && !p1) ? 0.f : gv.y;
                    gs1[v] += g0 + g1;
                    gs2[v] += g0 * ((yv.x - mu[v]) * is[v]) + g1 * ((yv.y - mu[v]) * is[v]);
                }
    }
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int ph = 0; ph < 2; ++ph)
                store_stream2(a.dx + oidx[nb] + v * cstr + ph * W2, val[nb][v][ph]);
    if (a.bnb.part) {
        float* red = Xs;  // [2][WP][TK]
        __syncthreads();
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            gs1[v] = row16_sum(gs1[v]);
            gs2[v] = row16_sum(gs2[v]);
        }
        if (j == 0)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                red[wp * TK + wk * 16 + 4 * g + v] = gs1[v];
                red[(WP + wp) * TK + wk * 16 + 4 * g + v] = gs2[v];
            }
        __syncthreads();
        if (wp == 0 && j == 0)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float t1 = 0.f, t2 = 0.f;
                for (int q = 0; q < WP; ++q) {
                    t1 += red[q * TK + wk * 16 + 4 * g + v];
                    t2 += red[(WP + q) * TK + wk * 16 + 4 * g + v];
                }
                const int m = mblk + wk * 16 + 4 * g + v;
                a.bnb.part[((size_t)m * gridDim.x + blockIdx.x) * 2 + 0] = t1;
                a.bnb.part[((size_t)m * gridDim.x + blockIdx.x) * 2 + 1] = t2;
            }
    }
}

template <int WO, int STRIDE, int TH, int CC, int WK, int WP, int NBW, int TPW, bool TRANS, int FOLD, bool BF>
void launch_direct_k(const DirArgs& a, dim3 grid, dim3 block, const Work& wk, hipStream_t st)
{
    PSW_LAUNCH(kname("conv3x3_direct", WO, STRIDE, TH, CC, WK, WP, NBW, TRANS, TPW, FOLD, BF), wk,
               (conv3x3_direct<WO, STRIDE, TH, CC, WK, WP, NBW, TRANS, TPW, FOLD, BF>), grid, block, 0, st, a);
}

template <int WO, int STRIDE, int TH, int CC, int WK, int WP, int NBW, int TPW, bool TRANS, int FOLD>
void launch_direct_p(const DirArgs& a, dim3 grid, dim3 block, const Work& wk, bool bf, hipStream_t st)
{
    if (bf)
        launch_direct_k<WO, STRIDE, TH, CC, WK, WP, NBW, TPW, TRANS, FOLD, true>(a, grid, block, wk, st);
    else
        launch_direct_k<WO, STRIDE, TH, CC, WK, WP, NBW, TPW, TRANS, FOLD, false>(a, grid, block, wk, st);
}

template <int WO, int STRIDE, int TH, int CC, int WK, int WP, int NBW, int TPW = 1>
hipError_t launch_direct(const DirArgs& a, int n, bool trans, bool bf, hipStream_t st)
{
    if ((a.HO / TH) % TPW) return hipErrorNotSupported;
    // one-dimensional, a multiple of 8 images (the kernel maps workgroups to
    // images XCD by XCD)
    dim3 grid((unsigned)((n + 7) / 8 * 8 * (a.HO / TH / TPW) * (a.K / (16 * WK))));
    dim3 block(64 * WK * WP);
    // as a convolution: input a.C x a.H x WO*STRIDE, output a.K x a.HO x WO
    Work wk = conv_work(n, a.C, a.H, WO * STRIDE, a.K, 3, 3, a.HO, WO);
    const double out_bytes = kF * n * (double)a.K * a.HO * WO;
    const double in_bytes = kF * n * (double)a.C * a.H * a.H;
    if (a.accumulate) wk.bytes += out_bytes;        // the existing output is read
    if (a.bnb.part) wk.bytes += (a.bnb.scale ? 1.0 : 2.0) * out_bytes;  // BN input (and output) for the sums
    // folded BN: g and y (and z, and the residual's gradient written) instead of dy, dy written
    if (a.fold.g) wk.bytes += (a.fold.dres ? 4.0 : 2.0) * in_bytes;
    if (trans && a.fold.g) {
        if constexpr (STRIDE == 1 && TPW == 1) {
            if (a.fold.dres)
                launch_direct_p<WO, STRIDE, TH, CC, WK, WP, NBW, TPW, true, 2>(a, grid, block, wk, bf, st);
            else
                launch_direct_p<WO, STRIDE, TH, CC, WK, WP, NBW, TPW, true, 1>(a, grid, block, wk, bf, st);
        } else {
            return hipErrorNotSupported;
        }
    } else if (trans) {
        launch_direct_p<WO, STRIDE, TH, CC, WK, WP, NBW, TPW, true, 0>(a, grid, block, wk, bf, st);
    } else {
        launch_direct_p<WO, STRIDE, TH, CC, WK, WP, NBW, TPW, false, 0>(a, grid, block, wk, bf, st);
    }
    return hipGetLastError();
}

}  // namespace

// The 32x32 stride-1 backward-data kernels use 16-row tiles once 8-row tiles
// would number 1024 or more (batch 256): every workgroup of a folded BN
// backward merges the per-tile sums of all the producer's tiles, so that
// merge grows with the square of the tile count; 16-row tiles quarter it
// (ResNet-110 b256: folded kernels 30.7 -> 27.0 us), while at batch 128 the
// two sizes time the same.
static bool dgrad_tall_tiles(int n, int ho) { return ho % 16 == 0 && (int64_t)n * (ho / 8) >= 1024; }

// Returns hipErrorNotSupported (nothing launched) when no tile configuration
// covers the shape; the caller then uses the general implicit GEMM.
int conv3x3_direct_tiles(int n, int C, int H, int W, int K, int stride)
{
    if ((stride != 1 && stride != 2) || H % stride || W % stride || H != W) return 0;
    if ((int64_t)n * C * H * W > INT32_MAX || (int64_t)n * K * (H / stride) * (W / stride) > INT32_MAX) return 0;
    const int HO = H / stride, WO = W / stride;
    if (C <= 4 && stride == 1) return (WO == 32 && HO % 8 == 0 && K % 16 == 0) ? n * (HO / 8) : 0;
    if (C % 16) return 0;
    if (WO == 32 && stride == 1 && HO % 8 == 0 && K % 16 == 0) return n * (HO / 8);
    if (WO == 16 && HO % 8 == 0 && K % 32 == 0) return n * (HO / 8);
    if (WO == 8 && HO % 8 == 0 && K % 32 == 0) return n * (HO / 8);
    return 0;
}

bool conv3x3_direct_covers(int n, int C, int H, int W, int K, int stride, bool transpose)
{
    if (stride != 1 && stride != 2) return false;
    if (H % stride || W % stride || H != W) return false;
    if ((int64_t)n * C * H * W > INT32_MAX || (int64_t)n * K * (H / stride) * (W / stride) > INT32_MAX) return false;
    const int HO = H / stride, WO = W / stride;
    if (C <= 4 && stride == 1 && !transpose) return WO == 32 && HO % 8 == 0 && K % 16 == 0;
    if (C % 16) return false;
    if (stride == 1)
        return (WO == 32 && HO % 8 == 0 && K % 16 == 0) || (WO == 16 && HO % 8 == 0 && K % 32 == 0) ||
               (WO == 8 && HO % 8 == 0 && K % 32 == 0);
    if (transpose) return false;
    return (WO == 16 && HO % 8 == 0 && K % 32 == 0) || (WO == 8 && HO % 8 == 0 && K % 32 == 0);
}

hipError_t conv3x3_direct(int n, int C, int H, int W, int K, int stride, const float* x, const float* w, float* y,
                          int accumulate, bool transpose, hipStream_t st, const BnStatsFuse* bn, const BnBwdFuse* bnb,
                          const BnFold* fold, bool bf16, const float* in_bn)
{
    if (in_bn && (transpose || C > kInBnMaxChannels)) return hipErrorNotSupported;
    if (bnb && (!transpose || stride != 1)) return hipErrorNotSupported;
    if (fold && (!transpose || stride != 1 || C > kFoldMaxChannels || (C & (C - 1)) || !fold->g || !fold->y ||
                 !fold->dy || !fold->part || (uintptr_t)fold->part % 8 || (fold->dres && !fold->z) ||
                 (uintptr_t)fold->g % 16 || (uintptr_t)fold->y % 16 || (uintptr_t)fold->z % 16 ||
                 (uintptr_t)fold->dres % 16))
        return hipErrorNotSupported;
    if (stride != 1 && stride != 2) return hipErrorNotSupported;
    if (H % stride || W % stride || H != W) return hipErrorNotSupported;  // square images (compile-time strides)
    // 32-bit element offsets inside the kernel
    if ((int64_t)n * C * H * W > INT32_MAX || (int64_t)n * K * (H / stride) * (W / stride) > INT32_MAX)
        return hipErrorNotSupported;
    if (bn && transpose) return hipErrorNotSupported;
    if ((uintptr_t)x % 16) return hipErrorNotSupported;  // float4 tile staging
    const int HO = H / stride, WO = W / stride;
    DirArgs a{x, w, y, C, H, K, HO, n, accumulate, BnStatsFuse{nullptr}, BnBwdFuse{}, BnFold{}, in_bn};
    if (bn) a.bn = *bn;
    if (bnb) a.bnb = *bnb;
    if (fold) a.fold = *fold;
    if (C <= 4 && stride == 1 && !transpose) {  // first layer of an image net (3 input channels)
        if (WO == 32 && HO % 8 == 0 && K % 16 == 0) return launch_direct<32, 1, 8, 4, 1, 4, 4>(a, n, false, bf16, st);
        return hipErrorNotSupported;
    }
    if (C % 16) return hipErrorNotSupported;
    if (stride == 1) {
        if (WO == 32 && HO % 8 == 0 && K % 16 == 0) {
            if (transpose && dgrad_tall_tiles(n, HO))
                return launch_direct<32, 1, 16, 16, 1, 8, 4>(a, n, true, bf16, st);
            return launch_direct<32, 1, 8, 16, 1, 4, 4>(a, n, transpose, bf16, st);
        }
        // forward 16x16 / 8x8: 16 output channels per workgroup (4 waves, twice
        // the workgroups of the backward's 32): the same kernel time alone, but
        // they share the CUs with the other streams' kernels better (pipelined
        // ResNet-20 b128 +1.2%)
        if (WO == 16 && HO % 8 == 0 && K % 32 == 0 && !transpose)
            return launch_direct<16, 1, 8, 16, 1, 4, 2>(a, n, false, bf16, st);
        if (WO == 16 && HO % 8 == 0 && K % 32 == 0) return launch_direct<16, 1, 8, 16, 2, 4, 2>(a, n, true, bf16, st);
        if (WO == 8 && HO % 8 == 0 && K % 32 == 0 && !transpose)
            return launch_direct<8, 1, 8, 16, 1, 4, 1>(a, n, false, bf16, st);
        if (WO == 8 && HO % 8 == 0 && K % 32 == 0) return launch_direct<8, 1, 8, 16, 2, 4, 1>(a, n, true, bf16, st);
    } else if (!transpose) {
        if (WO == 16 && HO % 8 == 0 && K % 32 == 0) return launch_direct<16, 2, 8, 16, 2, 4, 2>(a, n, false, bf16, st);
        if (WO == 8 && HO % 8 == 0 && K % 32 == 0) return launch_direct<8, 2, 8, 16, 2, 2, 2>(a, n, false, bf16, st);
    }
    return hipErrorNotSupported;
}

}  // namespace psw

namespace psw {
hipError_t conv3x3_dgrad_s2(int n, int CL, int H, int W, int KL, const float* w, const float* dy, float* dx,
                            int accumulate, hipStream_t st, const BnBwdFuse* bnb, bool bf16)
{
    if (H % 2 || W % 2 || KL % 16) return hipErrorNotSupported;
    // float4 staging of dy and of the weights, float2 stores
    if ((uintptr_t)dy % 16 || (uintptr_t)w % 16 || (uintptr_t)dx % 8) return hipErrorNotSupported;
    // 32-bit element offsets of the staging
    if ((int64_t)n * KL * (H / 2) * (W / 2) > INT32_MAX || (int64_t)KL * CL * 9 > INT32_MAX) return hipErrorNotSupported;
    const int HO = H / 2, WO = W / 2;
    DgArgs a{dy, w, dx, KL, CL, HO, accumulate, BnBwdFuse{}};
    if (bnb) a.bnb = *bnb;
    // the layer: CL x H x W -> KL x HO x WO, stride 2
    Work wk = conv_work(n, CL, H, W, KL, 3, 3, HO, WO);
    const double dx_bytes = kF * n * (double)CL * H * W;
    if (accumulate) wk.bytes += dx_bytes;
    if (bnb) wk.bytes += (bnb->scale ? 1.0 : 2.0) * dx_bytes;
#define PSW_DGS2(WO_, TH_, BF_)                                                                            \
    PSW_LAUNCH(kname("conv3x3_dgrad_s2", WO_, TH_, 16, 1, 4, 1, BF_), wk, (conv3x3_dgrad_s2<WO_, TH_, 16, 1, 4, 1, BF_>), \
               dim3(n * (HO / TH_), CL / 16), dim3(256), 0, st, a)
    if (WO == 16 && HO % 4 == 0 && CL % 16 == 0) {
        if (bf16)
            PSW_DGS2(16, 4, true);
        else
            PSW_DGS2(16, 4, false);
        return hipGetLastError();
    }
    if (WO == 8 && HO % 8 == 0 && CL % 16 == 0) {
        if (bf16)
            PSW_DGS2(8, 8, true);
        else
            PSW_DGS2(8, 8, false);
        return hipGetLastError();
    }
#undef PSW_DGS2
    return hipErrorNotSupported;
}
}  // namespace psw

namespace psw {
// tiles (workgroups along x) of the backward-data kernels that can carry the
// BN backward sums; 0 when neither kernel covers the shape
int dgrad_bnsums_tiles(int n, int CL, int H, int W, int KL, int stride)
{
    if (stride == 1) {
        if (KL % 16 || H != W) return 0;
        if ((int64_t)n * (CL > KL ? CL : KL) * H * W > INT32_MAX) return 0;
        if (W == 32 && H % 8 == 0 && CL % 16 == 0) return n * (H / (dgrad_tall_tiles(n, H) ? 16 : 8));
        if (W == 16 && H % 8 == 0 && CL % 32 == 0) return n * (H / 8);
        if (W == 8 && H % 8 == 0 && CL % 32 == 0) return n * (H / 8);
        return 0;
    }
    if (stride == 2) {
        if (H % 2 || W % 2 || KL % 16) return 0;
        const int HO = H / 2, WO = W / 2;
        if (WO == 16 && HO % 4 == 0 && CL % 16 == 0) return n * (HO / 4);
        if (WO == 8 && HO % 8 == 0 && CL % 16 == 0) return n * (HO / 8);
    }
    return 0;
}
}  // namespace psw
