// Backward-weight of a 3x3 / pad 1 convolution (stride 1 or 2) on CDNA4
// matrix cores, NCHW fp32:
//   dW[k][c][r][s] = sum_{n,p,q} dy[n][k][p][q] * x[n][c][p*S+r-1][q*S+s-1]
// (Sec. 2 of the paper: the weight gradient of layer l from x^(l-1) and
// delta^(l)).
//
// A workgroup reduces over IPW * TPW consecutive (image, TH-row band) tiles
// and writes one dW-shaped partial sum; the partials are added in a fixed
// order by the stage update (or the reduction kernel of conv.hip), so the
// result is bit-reproducible.  Its waves form IPW groups, each with its own
// LDS tiles walking TPW of the tiles; the groups' sums meet in LDS in group
// order at the end, so a workgroup covers IPW times the pixels of one group
// and writes IPW times fewer partial sums than one group per workgroup would.
// One launch may cover several convolutions of the same shape (the
// same-shape layers of a pipeline stage), and each has its own operands and
// partial sums.  The grid is one-dimensional: a workgroup's unit (member,
// partial-sum index) and its combination of CBW-block input channels and
// KBW-block output channels follow from its index so that the combinations
// of one unit, which read the same input or output-gradient tile, run on
// one XCD (consecutive workgroups go to the 8 XCDs in turn) at nearly the
// same time, and the tiles come from that XCD's L2 after the first read.  In
// the workgroup, wave (kb, cb, wpx) owns the 16x16 output blocks (output channels
// kb*16.., input channels of block cb) of all 9 taps (9 MFMA accumulators)
// and the pixel quads wpx, wpx+WPX, ...; waves that differ only in wpx are
// summed through LDS in wpx order at the end.
//
// The bands are walked in chunks of RC output rows, software-pipelined: the
// next chunk's dy rows and input rows (with their halo) are loaded into
// registers while the matrix cores work on the current chunk in LDS.
//
// MFMA v_mfma_f32_16x16x4_f32 with k = 4 consecutive output pixels of one
// row: A[m=k_out][k=pixel] from dy, B[k=pixel][n=c_in] from x shifted by the
// tap.  Both tiles sit in LDS plane-major (one plane per channel, as in NCHW)
// with a plane stride of 2 (mod 32) floats: an operand read by lanes
// (channel j, pixel g) hits bank 2j + g (stride 1), all distinct within a
// 32-lane half.  Input rows are stored with the data columns 16-byte aligned
// (input column -1 at offset 3), so staging writes are 8-byte stores.
#include "internal.h"

namespace psw {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));

// 4 floats rounded to bfloat16 (nearest even), packed as a matrix operand
__device__ __forceinline__ v4s bf16x4(float a, float b, float c, float d)
{
    return v4s{__builtin_bit_cast(short, (__bf16)a), __builtin_bit_cast(short, (__bf16)b),
               __builtin_bit_cast(short, (__bf16)c), __builtin_bit_cast(short, (__bf16)d)};
}

struct WgArgs {
    const float* x[kWgradGroupMax];   // member i: [n][C][H][W]
    const float* dy[kWgradGroupMax];  // [n][K][HO][WO]
    float* part[kWgradGroupMax];      // [splits][K][C][9]
    // may be null: member i's x is the raw input of a BN + ReLU whose output
    // is not stored; in_bn[i][c], in_bn[i][C + c] are channel c's scale and
    // shift, and the input used is max(fma(x, scale, shift), 0)
    const float* in_bn[kWgradGroupMax];
    int n, C, H, W, K, HO;
    int splits;                       // workgroups (partial sums) per member
    int units;                        // splits * members
    int cgroups, combos;              // input-channel groups; combos = cgroups * output-channel groups
};

// smallest v >= lo with v % 32 == 2
constexpr int plane_stride(int lo)
{
    int v = lo;
    while (v % 32 != 2) ++v;
    return v;
}

constexpr int round4(int v) { return (v + 3) / 4 * 4; }

// BF: bf16 operands with fp32 accumulation on v_mfma_f32_16x16x16_bf16, k =
// 16 consecutive output pixels (4 pixel quads; lane group g supplies quad g):
// the fp32 tiles are staged as before and each lane rounds its 4 dy values
// and its 4 shifted input values to bf16 when it reads them.
// IBN: some member may have an input BN (WgArgs::in_bn); without it the
// staging has no such path.
template <int STRIDE, int WO, int TH, int KBW, int CBW, int WPX, int TPW, int RC, bool BF, int IPW, bool IBN>
__global__ __launch_bounds__(64 * KBW * CBW * WPX * IPW) void conv3x3_wgrad(WgArgs a)
{
    constexpr int NT = 64 * KBW * CBW * WPX;  // threads of one group
    constexpr int WIN = WO * STRIDE;
    constexpr int XRS = round4(WIN + (STRIDE == 1 ? 5 : 4));  // input row: cols -1 .. WIN(-1) at offsets 3 ..
    constexpr int HRC = (RC - 1) * STRIDE + 3;                // staged input rows per chunk
    constexpr int KC = 16 * KBW, CCH = 16 * CBW;
    constexpr int NPC = RC * WO;                              // output pixels per chunk
    constexpr int QC = NPC / 4;                               // pixel quads per chunk
    constexpr int DPS = plane_stride(NPC);                    // dy plane stride
    constexpr int XPS = plane_stride(HRC * XRS);              // x plane stride
    constexpr int NCH = TPW * (TH / RC);                      // chunks per workgroup
    static_assert(WO % 4 == 0 && TH % RC == 0 && QC % WPX == 0, "tiling");
    static_assert(!BF || QC % (4 * WPX) == 0, "bf16: 16-pixel blocks");
    constexpr int DS_FLOATS = KC * DPS;
    constexpr int XS_FLOATS = CCH * XPS;
    constexpr int ACC_FLOATS = 9 * 4 * 64;  // one wave's accumulators
    // final sums: within each group over wpx, then over the groups
    constexpr int RED1 = (WPX > 1) ? IPW * (WPX - 1) * KBW * CBW * ACC_FLOATS : 0;
    constexpr int RED2 = (IPW > 1) ? (IPW - 1) * KBW * CBW * ACC_FLOATS : 0;
    constexpr int TILE_FLOATS = IPW * (DS_FLOATS + XS_FLOATS);
    constexpr int LDS_FLOATS = TILE_FLOATS > RED1 ? (TILE_FLOATS > RED2 ? TILE_FLOATS : RED2) : (RED1 > RED2 ? RED1 : RED2);
    static_assert(LDS_FLOATS * 4 <= 65536, "LDS");
    __shared__ __attribute__((aligned(16))) float lds[LDS_FLOATS];
    __shared__ float bnt[IBN ? 2 * CCH : 1];  // the member's input BN over this workgroup's channels: scale, shift

    const int wave_all = threadIdx.x >> 6;
    const int ip = wave_all / (KBW * CBW * WPX);  // group
    const int tid = threadIdx.x - ip * NT, lane = tid & 63, wave = tid >> 6;
    const int kb = wave % KBW, cb = (wave / KBW) % CBW, wpx = wave / (KBW * CBW);
    float* Ds = lds + ip * (DS_FLOATS + XS_FLOATS);
    float* Xs = Ds + DS_FLOATS;
    const int g = lane >> 4, j = lane & 15;
    // workgroup index -> (unit, channel combination): units u = 8g + x for
    // g >= 0 run on XCD x, each unit's combinations in consecutive rounds of
    // 8 workgroups; indices past the last unit (the grid is a multiple of 8
    // units) do nothing
    const int wgi = blockIdx.x;
    const int slot = (wgi >> 3) % a.combos;
    const int unit = ((wgi >> 3) / a.combos) * 8 + (wgi & 7);
    if (unit >= a.units) return;
    const int mem = unit / a.splits;                // member of the group
    const int bx = unit - mem * a.splits;           // partial-sum index within it
    const int cgi = slot % a.cgroups, kgi = slot / a.cgroups;
    const float* gx = a.x[mem];
    const float* gdy = a.dy[mem];
    const float* ibn = IBN ? a.in_bn[mem] : nullptr;
    const int bands = a.HO / TH;         // row bands per image
    const int cbase = cgi * CCH;  // first input channel of this workgroup
    const int kbase = kgi * KC;   // first output channel of this workgroup

    v4f acc[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};

    // zero halo columns of the x tile (never written by the staging below)
    for (int i = tid; i < HRC * CCH; i += NT) {
        const int c = i / HRC, rr = i - (i / HRC) * HRC;
        Xs[c * XPS + rr * XRS + 3] = 0.f;
        if (STRIDE == 1) Xs[c * XPS + rr * XRS + WIN + 4] = 0.f;
    }

    // chunk ch: tile ch / (TH/RC) of this workgroup, rows (ch % (TH/RC))*RC ..
    constexpr int DN4 = KC * NPC / 4, XN4 = CCH * HRC * WIN / 4;
    constexpr int DV = (DN4 + NT - 1) / NT, XV = (XN4 + NT - 1) / NT;
    float4 dr[DV], xr[XV];
    auto load_chunk = [&](int ch) {
        const int tl = (bx * IPW + ip) * TPW + ch / (TH / RC);
        const int img = tl / bands;
        const int oh0 = (tl - img * bands) * TH + (ch % (TH / RC)) * RC;
        const int ih0 = oh0 * STRIDE - 1;
#pragma unroll
        for (int v = 0; v < DV; ++v) {
            const int i4 = tid + v * NT;
            float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
            if (i4 < DN4) {
                const int i = i4 * 4;
                const int k = i / NPC, pix = i - (i / NPC) * NPC;
                val = *reinterpret_cast<const float4*>(gdy + (((size_t)img * a.K + kbase + k) * a.HO + oh0) * WO + pix);
            }
            dr[v] = val;
        }
        // with an input BN, elements outside the input start as NaN: the
        // staging's max(fma(x, scale, shift), 0) then gives exactly 0 there
        const float fill = ibn ? __builtin_nanf("") : 0.f;
#pragma unroll
        for (int v = 0; v < XV; ++v) {
            const int i4 = tid + v * NT;
            float4 val = make_float4(fill, fill, fill, fill);
            if (i4 < XN4) {
                const int i = i4 * 4;
                const int c = i / (HRC * WIN);
                const int rem = i - c * (HRC * WIN);
                const int rr = rem / WIN, iw = rem - (rem / WIN) * WIN;
                const int ih = ih0 + rr;
                if (ih >= 0 && ih < a.H && cbase + c < a.C)
                    val = *reinterpret_cast<const float4*>(gx + (((size_t)img * a.C + cbase + c) * a.H + ih) * WIN + iw);
            }
            xr[v] = val;
        }
    };
    auto store_chunk = [&]() {
#pragma unroll
        for (int v = 0; v < DV; ++v) {
            const int i4 = tid + v * NT;
            if (i4 < DN4) {
                const int i = i4 * 4;
                const int k = i / NPC, pix = i - (i / NPC) * NPC;
                float2* d = reinterpret_cast<float2*>(Ds + k * DPS + pix);  // DPS and pix even: 8-byte aligned
                d[0] = make_float2(dr[v].x, dr[v].y);
                d[1] = make_float2(dr[v].z, dr[v].w);
            }
        }
#pragma unroll
        for (int v = 0; v < XV; ++v) {
            const int i4 = tid + v * NT;
            if (i4 < XN4) {
                const int i = i4 * 4;
                const int c = i / (HRC * WIN);
                const int rem = i - c * (HRC * WIN);
                const int rr = rem / WIN, iw = rem - (rem / WIN) * WIN;
                float4 val = xr[v];
                if (IBN && ibn) {  // the BN + ReLU of the stored input, exactly as its apply kernel forms it
                    const float sc = bnt[c], sf = bnt[CCH + c];
                    val = make_float4(fmaxf(__fmaf_rn(val.x, sc, sf), 0.f), fmaxf(__fmaf_rn(val.y, sc, sf), 0.f),
                                      fmaxf(__fmaf_rn(val.z, sc, sf), 0.f), fmaxf(__fmaf_rn(val.w, sc, sf), 0.f));
                }
                float2* d = reinterpret_cast<float2*>(Xs + c * XPS + rr * XRS + 4 + iw);  // even offset
                d[0] = make_float2(val.x, val.y);
                d[1] = make_float2(val.z, val.w);
            }
        }
    };

    const float* dsl = Ds + (kb * 16 + j) * DPS + g;
    const float* xsl = Xs + (cb * 16 + j) * XPS + g * STRIDE + 3;
    // the input BN's coefficients (read after the chunk loop's first
    // barrier; loaded before the first chunk: issued after it, their wait
    // held the staging of the 32x32 layers back by 6 us)
    if (IBN && ibn && threadIdx.x < CCH) {
        const int c = cbase + (int)threadIdx.x < a.C ? cbase + (int)threadIdx.x : 0;
        bnt[threadIdx.x] = ibn[c];
        bnt[CCH + threadIdx.x] = ibn[a.C + c];
    }
    load_chunk(0);
    for (int ch = 0; ch < NCH; ++ch) {
        __syncthreads();  // the previous chunk's LDS reads are done
        store_chunk();
        __syncthreads();
        if (ch + 1 < NCH) load_chunk(ch + 1);
        if constexpr (BF) {
            const float* dsb = Ds + (kb * 16 + j) * DPS;
            const float* xsb = Xs + (cb * 16 + j) * XPS + 3;
#pragma unroll
            for (int qb = 0; qb < QC / (4 * WPX); ++qb) {
                const int pix0 = ((qb * WPX + wpx) * 4 + g) * 4;  // this lane group's pixel quad
                const int row = pix0 / WO, col0 = pix0 - (pix0 / WO) * WO;
                const float2 d0 = *reinterpret_cast<const float2*>(dsb + pix0);
                const float2 d1 = *reinterpret_cast<const float2*>(dsb + pix0 + 2);
                const v4s av = bf16x4(d0.x, d0.y, d1.x, d1.y);
                const float* xb = xsb + (row * STRIDE) * XRS + col0 * STRIDE;
#pragma unroll
                for (int r = 0; r < 3; ++r)
#pragma unroll
                    for (int s = 0; s < 3; ++s) {
                        const float* p = xb + r * XRS + s;
                        const v4s bv = bf16x4(p[0], p[STRIDE], p[2 * STRIDE], p[3 * STRIDE]);
                        acc[r * 3 + s] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, bv, acc[r * 3 + s], 0, 0, 0);
                    }
            }
            continue;
        }
#pragma unroll
        for (int qi = 0; qi < QC / WPX; ++qi) {
            const int pix0 = (qi * WPX + wpx) * 4;
            const int row = pix0 / WO, col0 = pix0 - (pix0 / WO) * WO;
            const float av = dsl[pix0];
            const float* xb = xsl + (row * STRIDE) * XRS + col0 * STRIDE;
#pragma unroll
            for (int r = 0; r < 3; ++r)
#pragma unroll
                for (int s = 0; s < 3; ++s) {
                    const float bv = xb[r * XRS + s];
                    acc[r * 3 + s] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[r * 3 + s], 0, 0, 0);
                }
        }
    }

    // sums in a fixed order: within each group over wpx, then over the groups
    if constexpr (WPX > 1) {
        __syncthreads();  // LDS tiles are no longer read: reuse for the reduction
        if (wpx > 0) {
            float* dst = lds + ((((ip * (WPX - 1) + wpx - 1) * KBW + kb) * CBW + cb)) * ACC_FLOATS;
#pragma unroll
            for (int t = 0; t < 9; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) dst[(t * 4 + i) * 64 + lane] = acc[t][i];
        }
        __syncthreads();
        if (wpx == 0)
            for (int w = 1; w < WPX; ++w) {
                const float* src = lds + ((((ip * (WPX - 1) + w - 1) * KBW + kb) * CBW + cb)) * ACC_FLOATS;
#pragma unroll
                for (int t = 0; t < 9; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[t][i] += src[(t * 4 + i) * 64 + lane];
            }
    }
    if constexpr (IPW > 1) {
        __syncthreads();
        if (wpx == 0 && ip > 0) {
            float* dst = lds + (((ip - 1) * KBW + kb) * CBW + cb) * ACC_FLOATS;
#pragma unroll
            for (int t = 0; t < 9; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) dst[(t * 4 + i) * 64 + lane] = acc[t][i];
        }
        __syncthreads();
        if (wpx == 0 && ip == 0)
            for (int q = 1; q < IPW; ++q) {
                const float* src = lds + (((q - 1) * KBW + kb) * CBW + cb) * ACC_FLOATS;
#pragma unroll
                for (int t = 0; t < 9; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[t][i] += src[(t * 4 + i) * 64 + lane];
            }
    }
    if (wpx != 0 || ip != 0) return;
    // D lane l, register i: output channel kb*16 + 4g + i, input channel cb*16 + j
    float* out = a.part[mem] + (size_t)bx * a.K * a.C * 9;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int k = kbase + kb * 16 + 4 * g + i, c = cbase + cb * 16 + j;
        if (c >= a.C) continue;  // zero-filled channels of a narrow input (C < 16)
        float* o = out + ((size_t)k * a.C + c) * 9;
#pragma unroll
        for (int t = 0; t < 9; ++t) o[t] = acc[t][i];  // 36-byte runs per lane: plain stores, merged in L2
    }
}

// Which configuration covers a shape; 0 = none.
int wgrad_config(int n, int C, int H, int W, int K, int stride)
{
    if (stride == 1 && H == 32 && W == 32 && C == 16 && K == 16) return 1;
    if (stride == 1 && H == 16 && W == 16 && C == 32 && K == 32 && n % 4 == 0) return 2;
    if (stride == 1 && H == 8 && W == 8 && C == 64 && K == 64 && n % 8 == 0) return 3;
    if (stride == 2 && H == 32 && W == 32 && C == 16 && K == 32) return 4;
    if (stride == 2 && H == 16 && W == 16 && C == 32 && K == 64 && n % 2 == 0) return 5;
    if (stride == 1 && H == 32 && W == 32 && C < 16 && K == 16) return 6;
    return 0;
}

// At batch 256 and above, the 16x16 and 8x8 layers give each group twice
// the images: half the workgroups and half the split partial sums that the
// stage update reads (ResNet-110 b256: those weight gradients 37.0 / 32.4 ->
// 34.3 / 29.9 us, the updates 214 -> 192 us per step); at batch 128 the
// extra work per workgroup costs more than the halved sums save.
bool wgrad_wide(int n) { return n >= 256 && n % 16 == 0; }

}  // namespace

// Number of partial sums (workgroups) for a shape; 0 when not covered.
int conv3x3_wgrad_splits(int n, int C, int H, int W, int K, int stride)
{
    switch (wgrad_config(n, C, H, W, K, stride)) {  // two groups of waves per workgroup
    case 1: return n;           // one 16-row band (of 32) per group: one image per workgroup
    case 2: return wgrad_wide(n) ? n / 8 : n / 4;   // two (four) images per group, 16 of the 32 output channels
    case 3: return wgrad_wide(n) ? n / 16 : n / 8;  // four (eight) images per group, 32 of the 64 output channels
    case 4: return n;           // one 8-row band (of 16 output rows) per group
    case 5: return n / 2;       // one image per group
    case 6: return 2 * n;       // one 8-row band per group, input channels zero-filled to 16
    default: return 0;
    }
}

hipError_t conv3x3_wgrad_group(int n, int C, int H, int W, int K, int stride, const float* const* x,
                               const float* const* dy, float* const* part, int count, hipStream_t st, bool bf16,
                               const float* const* in_bn)
{
    const int cfg = wgrad_config(n, C, H, W, K, stride);
    if (!cfg || count < 1 || count > kWgradGroupMax) return hipErrorNotSupported;
    WgArgs a{};
    for (int i = 0; i < count; ++i) {
        if ((uintptr_t)x[i] % 16 || (uintptr_t)dy[i] % 16) return hipErrorNotSupported;  // float4 staging
        a.x[i] = x[i];
        a.dy[i] = dy[i];
        a.part[i] = part[i];
        a.in_bn[i] = in_bn ? in_bn[i] : nullptr;
    }
    a.n = n; a.C = C; a.H = H; a.W = W; a.K = K; a.HO = H / stride;
    const int splits = conv3x3_wgrad_splits(n, C, H, W, K, stride);
    a.splits = splits;
    const int cgroups = (C + 15) / 16;  // one 16-channel block per workgroup (grid.y)
    // output-channel groups: configurations 2-5 split K over the grid (the
    // stride-2 layers' small launches then fill the chip: twice the
    // workgroups with the same partial sums)
    const int kgroups = (cfg == 2 || cfg == 4) ? K / 16 : (cfg == 3 || cfg == 5) ? K / 32 : 1;
    a.units = splits * count;
    a.cgroups = cgroups;
    a.combos = cgroups * kgroups;
    const dim3 grid((unsigned)((a.units + 7) / 8 * 8 * a.combos));
    Work wk = conv_work(n, C, H, W, K, 3, 3, H / stride, W / stride);
    wk.flops *= count;
    wk.bytes *= count;
#define PSW_WG1(S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_, BF_, IBN_)                                            \
    PSW_LAUNCH(kname("conv3x3_wgrad", S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_, BF_, 2, IBN_), wk,               \
               (conv3x3_wgrad<S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_, BF_, 2, IBN_>), grid, dim3(512), 0, st, a)
#define PSW_WG(S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_)                                                          \
    do {                                                                                                        \
        if (bf16 && any_bn) PSW_WG1(S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_, true, true);                     \
        else if (bf16) PSW_WG1(S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_, true, false);                         \
        else if (any_bn) PSW_WG1(S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_, false, true);                       \
        else PSW_WG1(S_, WO_, TH_, KBW_, CBW_, WPX_, TPW_, RC_, false, false);                                  \
    } while (0)
    bool any_bn = false;
    for (int i = 0; i < count; ++i) any_bn = any_bn || a.in_bn[i];
    switch (cfg) {
    case 1:  // with an input BN the 4-row chunks' staging would pass 128 VGPRs (one workgroup per CU)
        if (any_bn) PSW_WG(1, 32, 16, 1, 1, 4, 1, 2);
        else PSW_WG(1, 32, 16, 1, 1, 4, 1, 4);
        break;
    case 6: PSW_WG(1, 32, 8, 1, 1, 4, 1, 4); break;  // a narrow input: twice the workgroups
    case 2:
        if (wgrad_wide(n)) PSW_WG(1, 16, 16, 1, 1, 4, 4, 8);
        else PSW_WG(1, 16, 16, 1, 1, 4, 2, 8);
        break;
    case 3:
        if (wgrad_wide(n)) PSW_WG(1, 8, 8, 2, 1, 2, 8, 8);
        else PSW_WG(1, 8, 8, 2, 1, 2, 4, 8);
        break;
    case 4: PSW_WG(2, 16, 8, 1, 1, 4, 1, 4); break;
    case 5: PSW_WG(2, 8, 8, 2, 1, 2, 1, 4); break;
    }
#undef PSW_WG
#undef PSW_WG1
    return hipGetLastError();
}

hipError_t conv3x3_wgrad(int n, int C, int H, int W, int K, int stride, const float* x, const float* dy, float* part,
                         hipStream_t st, bool bf16)
{
    return conv3x3_wgrad_group(n, C, H, W, K, stride, &x, &dy, &part, 1, st, bf16);
}

}  // namespace psw
