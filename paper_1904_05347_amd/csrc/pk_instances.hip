// pk_instances.hip -- the kernel instances of the tile-parameter space.
//
// Naming: <kind>_<BM>x<BN>x<BK>_w<WAVES_M>x<WAVES_N>_<layout>_v<VA><VB>
//   kind    gemm or conv (implicit GEMM over an NHWC image)
//   layout  gemm: nn / tn / nt / tt (storage of A and B); conv: the filter is
//           always K x Cout ('n')
//   v       elements per global load of A and of B
#include "pk_configs.hpp"
#include "pk_kernel.hpp"

namespace pk {

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB>
static hipError_t launch_gemm(const KernelArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.tiles_m * a.tiles_n), 1u, (unsigned)a.splits);
    const dim3 block(64 * WAVES_M * WAVES_N);
    hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB>),
                       grid, block, 0, stream, a);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB>
static constexpr int lds_bytes()
{
    return (int)sizeof(float) * GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB>::LDS_FLOATS;
}

#define PK_GEMM(name, BM, BN, BK, WM, WN, TA, TB, VA, VB)                                              \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, VA, VB,                                            \
     lds_bytes<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>(),                \
     &launch_gemm<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>}

#define PK_CONV(name, BM, BN, BK, WM, WN, VA, VB)                                                      \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, VA, VB,                                              \
     lds_bytes<BM, BN, BK, WM, WN, A_CONV, false, VA, VB>(),                                          \
     &launch_gemm<BM, BN, BK, WM, WN, A_CONV, false, VA, VB>}

const Config *configs(int *count)
{
    static const Config kTable[] = {
    // 16-byte loads, large tiles: the 1024..4096 sweep
    PK_GEMM(gemm_128x128x16_w2x2_nn_v44, 128, 128, 16, 2, 2, 0, 0, 4, 4),
    PK_GEMM(gemm_128x128x16_w2x2_tn_v44, 128, 128, 16, 2, 2, 1, 0, 4, 4),
    PK_GEMM(gemm_128x128x16_w2x2_nt_v44, 128, 128, 16, 2, 2, 0, 1, 4, 4),
    PK_GEMM(gemm_128x128x16_w2x2_tt_v44, 128, 128, 16, 2, 2, 1, 1, 4, 4),
    // 16-byte loads, small tiles: small or skinny products
    PK_GEMM(gemm_64x64x16_w2x2_nn_v44, 64, 64, 16, 2, 2, 0, 0, 4, 4),
    PK_GEMM(gemm_64x64x16_w2x2_tn_v44, 64, 64, 16, 2, 2, 1, 0, 4, 4),
    PK_GEMM(gemm_64x64x16_w2x2_nt_v44, 64, 64, 16, 2, 2, 0, 1, 4, 4),
    PK_GEMM(gemm_64x64x16_w2x2_tt_v44, 64, 64, 16, 2, 2, 1, 1, 4, 4),
    // scalar loads: any alignment, any leading dimension
    PK_GEMM(gemm_64x64x16_w2x2_nn_v11, 64, 64, 16, 2, 2, 0, 0, 1, 1),
    PK_GEMM(gemm_64x64x16_w2x2_tn_v11, 64, 64, 16, 2, 2, 1, 0, 1, 1),
    PK_GEMM(gemm_64x64x16_w2x2_nt_v11, 64, 64, 16, 2, 2, 0, 1, 1, 1),
    PK_GEMM(gemm_64x64x16_w2x2_tt_v11, 64, 64, 16, 2, 2, 1, 1, 1, 1),
    // implicit-GEMM convolution
    PK_CONV(conv_128x128x16_w2x2_v44, 128, 128, 16, 2, 2, 4, 4),
    PK_CONV(conv_128x64x16_w2x2_v44, 128, 64, 16, 2, 2, 4, 4),
    PK_CONV(conv_64x64x16_w2x2_v44, 64, 64, 16, 2, 2, 4, 4),
    PK_CONV(conv_128x64x16_w2x2_v14, 128, 64, 16, 2, 2, 1, 4),
    PK_CONV(conv_64x64x16_w2x2_v11, 64, 64, 16, 2, 2, 1, 1),
    };
    *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
    return kTable;
}

// ---------------------------------------------------------------- helpers

hipError_t launch_splitk_reduce(const float *ws, float *C, int M, int N, int64_t ldc, int splits,
                                float beta, hipStream_t stream)
{
    const int64_t total = (int64_t)M * N;
    const int64_t blocks = (total + 255) / 256;
    const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3(grid), dim3(256), 0, stream, ws, C, M, N, ldc, splits, beta);
    return hipGetLastError();
}

hipError_t launch_scale(float *C, int M, int N, int64_t ldc, float beta, hipStream_t stream)
{
    const int64_t total = (int64_t)M * N;
    const int64_t blocks = (total + 255) / 256;
    const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
    hipLaunchKernelGGL(scale_kernel, dim3(grid), dim3(256), 0, stream, C, M, N, ldc, beta);
    return hipGetLastError();
}

}  // namespace pk
