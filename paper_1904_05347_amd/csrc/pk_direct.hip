// pk_direct.hip -- tiled direct convolution for a short reduction
// (KH * KW * Cin <= 32, e.g. the first layer of an image network, Cin = 3).
//
// The implicit GEMM spends most of its time on a K loop that is only one or
// two blocks deep here, while the layer is bound by writing its output.  This
// kernel follows the paper's tiled convolution (Section 4.1.1): a work-group
// owns a tile of output pixels, loads the input patch those pixels need --
// the tile plus its halo -- into LDS once, so neighbouring windows reuse it,
// and each wave computes several outputs from it.  The products run on the
// fp32 MFMA as a 32-pixel x 32-channel x K block per wave step:
//   A(p, k) = patch[(r*sh + kh)][(p*sw + kw)][ci]     (LDS, one read per k)
//   B(k, c) = f[kh][kw][ci][c]                        (registers, loaded once)
// with k = (kh*KW + kw)*Cin + ci padded to an even count (B = 0 there).
//
// Tile: 8 output rows x 32 output columns x 64 output channels per
// work-group (grid.z walks further groups of 64 channels); 4 waves, each
// owning 2 rows x 32 columns x 64 channels = 4 MFMA blocks.
#include <hip/hip_runtime.h>

#include "pk_configs.hpp"

namespace pk {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int DT_ROWS = 8;       // output rows per work-group
constexpr int DT_COLS = 32;      // output columns per work-group (one MFMA block of pixels)
constexpr int DT_CH = 64;        // output channels per work-group
constexpr int DT_WAVES = 4;
constexpr int DT_ROWS_PER_WAVE = DT_ROWS / DT_WAVES;
constexpr int DT_KMAX = 32;      // longest reduction this kernel takes
constexpr int DT_LDS_FLOATS = 12 * 1024;  // input patch capacity (48 KiB)

// Floats of the input patch a work-group stages: the launch sizes LDS to it,
// so small patches leave room for more resident work-groups.
int64_t direct_patch_floats(int64_t KH, int64_t KW, int64_t Cin, int64_t sh, int64_t sw)
{
    return ((DT_ROWS - 1) * sh + KH) * ((DT_COLS - 1) * sw + KW) * Cin;
}

__global__ void __launch_bounds__(64 * DT_WAVES) direct_conv_kernel(KernelArgs p)
{
    extern __shared__ float patch[];  // direct_patch_floats() floats
    const float *x = p.A;
    const float *f = p.B;
    float *y = p.C;
    const int H = p.H, W = p.W, Cin = p.Cin, KH = p.KH, KW = p.KW, sh = p.sh, sw = p.sw;
    const int Ho = p.Ho, Wo = p.Wo, Cout = p.N, K = p.K;

    const int tiles_w = (Wo + DT_COLS - 1) / DT_COLS;
    const int ho0 = (blockIdx.x / tiles_w) * DT_ROWS;
    const int wo0 = (blockIdx.x % tiles_w) * DT_COLS;
    const int n = blockIdx.y;
    const int c0 = blockIdx.z * DT_CH;

    // input patch rows ih0 .. ih0 + PH - 1, columns iw0 .. iw0 + PW - 1, all channels
    const int PH = (DT_ROWS - 1) * sh + KH;
    const int PW = (DT_COLS - 1) * sw + KW;
    const int row_len = PW * Cin;
    const int ih0 = ho0 * sh - p.pt;
    const int iw0 = wo0 * sw - p.pl;
    const float *img = x + (int64_t)n * H * W * Cin;
    for (int e = threadIdx.x; e < PH * row_len; e += blockDim.x) {
        const int r = e / row_len;
        const int q = e - r * row_len;
        const int col = q / Cin, ci = q - col * Cin;
        const int ih = ih0 + r, iw = iw0 + col;
        float v = 0.f;
        if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W) v = img[((int64_t)ih * W + iw) * Cin + ci];
        patch[e] = v;
    }

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int l32 = lane & 31, h = lane >> 5;

    // Per k-step s this lane supplies k = 2s + h: its patch offset and filter values.
    int off[DT_KMAX / 2];
    float bv[2][DT_KMAX / 2];
#pragma unroll
    for (int s = 0; s < DT_KMAX / 2; ++s) {
        const int k = 2 * s + h;
        int o = 0;
        float b0 = 0.f, b1 = 0.f;
        if (k < K) {
            const int tap = k / Cin, ci = k - tap * Cin;
            const int kh = tap / KW, kw = tap - kh * KW;
            o = (kh * PW + kw) * Cin + ci;
            const int co0 = c0 + l32, co1 = c0 + 32 + l32;
            if (co0 < Cout) b0 = f[(int64_t)k * Cout + co0];
            if (co1 < Cout) b1 = f[(int64_t)k * Cout + co1];
        }
        off[s] = o;
        bv[0][s] = b0;
        bv[1][s] = b1;
    }
    __syncthreads();

    f32x16 acc[DT_ROWS_PER_WAVE][2];
#pragma unroll
    for (int r = 0; r < DT_ROWS_PER_WAVE; ++r)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[r][j][i] = 0.f;

    const int ksteps = (K + 1) / 2;
    const bool tail_lane = (K & 1) && h == 1;
#pragma unroll
    for (int r = 0; r < DT_ROWS_PER_WAVE; ++r) {
        const int prow = (wave * DT_ROWS_PER_WAVE + r) * sh;     // patch row of tap kh = 0
        const float *base = patch + prow * row_len + l32 * sw * Cin;
#pragma unroll
        for (int s = 0; s < DT_KMAX / 2; ++s) {
            if (s < ksteps) {
                // for odd K the upper half-wave's last k is past the window:
                // its filter value is 0 and its input value must be 0 too
                // (an infinite input would otherwise give 0 * inf = NaN)
                const float a = (s == ksteps - 1 && tail_lane) ? 0.f : base[off[s]];
                acc[r][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv[0][s], acc[r][0], 0, 0, 0);
                acc[r][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv[1][s], acc[r][1], 0, 0, 0);
            }
        }
    }

    // acc[r][j][i]: pixel column 8*(i/4) + 4*h + i%4 of row r, channel c0 + 32*j + l32
#pragma unroll
    for (int r = 0; r < DT_ROWS_PER_WAVE; ++r) {
        const int ho = ho0 + wave * DT_ROWS_PER_WAVE + r;
        if (ho >= Ho) continue;
        float *yrow = y + (((int64_t)n * Ho + ho) * Wo) * Cout;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int wo = wo0 + 8 * (i >> 2) + 4 * h + (i & 3);
            if (wo >= Wo) continue;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int co = c0 + 32 * j + l32;
                if (co < Cout) yrow[(int64_t)wo * Cout + co] = acc[r][j][i];
            }
        }
    }
}

hipError_t launch_direct(const KernelArgs &a, hipStream_t stream)
{
    const unsigned tiles = (unsigned)(((a.Ho + DT_ROWS - 1) / DT_ROWS) * ((a.Wo + DT_COLS - 1) / DT_COLS));
    const dim3 grid(tiles, (unsigned)a.batch, (unsigned)((a.N + DT_CH - 1) / DT_CH));
    const size_t lds = (size_t)direct_patch_floats(a.KH, a.KW, a.Cin, a.sh, a.sw) * sizeof(float);
    hipLaunchKernelGGL(direct_conv_kernel, grid, dim3(64 * DT_WAVES), lds, stream, a);
    return hipGetLastError();
}

}  // namespace

bool direct_conv_fits(int64_t KH, int64_t KW, int64_t Cin, int64_t sh, int64_t sw)
{
    if (KH > DT_KMAX || KW > DT_KMAX || Cin > DT_KMAX || sh > 64 || sw > 64) return false;
    if (KH * KW * Cin > DT_KMAX) return false;
    return direct_patch_floats(KH, KW, Cin, sh, sw) <= DT_LDS_FLOATS;
}

const Config *configs_direct(int *count)
{
    static const Config kTable[] = {
        {"direct_8x32x64_k32", KIND_DIRECT, DT_ROWS * DT_COLS, DT_CH, DT_KMAX, DT_WAVES, 1, 0, 0, 1, 1, 1, 0,
         (int)(DT_LDS_FLOATS * sizeof(float)), &launch_direct},
    };
    *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
    return kTable;
}

}  // namespace pk
