// pk_instance_common.hpp -- how one tile configuration becomes a kernel
// instance and a registry entry.  Included by the pk_inst_*.hip files, each of
// which instantiates one group of configurations (compiled in parallel).
#pragma once

#include "pk_configs.hpp"
#include "pk_kernel.hpp"

namespace pk {
// Whether a launch needs the epilogue that reads C: beta != 0 on an unsplit
// product (split partial sums never read C; the reduction applies beta).
// Convolutions always have beta == 0, so their instances never compile it.
template <int AMODE>
static bool reads_c(const KernelArgs &a)
{
    return AMODE != A_CONV && a.beta != 0.f && a.splits <= 1;
}

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC>
static hipError_t launch_gemm(const KernelArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.tiles_m * a.tiles_n), (unsigned)(a.nbatch > 1 ? a.nbatch : 1), (unsigned)a.splits);
    const dim3 block(64 * WAVES_M * WAVES_N);
    if constexpr (AMODE != A_CONV) {
        if (reads_c<AMODE>(a)) {
            hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, true>),
                               grid, block, 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, false>),
                       grid, block, 0, stream, a);
    return hipGetLastError();
}

// Persistent launch: as many work-groups as the CUs hold at once (from the
// occupancy the compiled kernel allows), each walking its share of the tiles.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC>
static hipError_t launch_gemm_persistent(const KernelArgs &a, hipStream_t stream)
{
    const bool beta = reads_c<AMODE>(a);
    auto kernel = gemm_persistent_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, false>;
    if constexpr (AMODE != A_CONV) {
        if (beta) kernel = gemm_persistent_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, true>;
    }
    const int threads = 64 * WAVES_M * WAVES_N;
    static int per_cu[2] = {0, 0};  // resident work-groups per CU (same on every MI355X)
    if (per_cu[beta] == 0) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1) n = 1;
        per_cu[beta] = n;
    }
    const int64_t items = (int64_t)a.tiles_m * a.tiles_n * a.splits;
    int64_t grid = (int64_t)per_cu[beta] * device_cu_count();
    if (grid > items) grid = items;
    if (grid >= a.xcds && a.xcds > 1) grid -= grid % a.xcds;
    hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(threads), 0, stream, a);
    return hipGetLastError();
}

// Stream-K: work-groups one CU holds at once, per epilogue form.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC>
static int resident_streamk(int beta)
{
    static int per_cu[2] = {0, 0};  // the same on every MI355X
    const int b = beta ? 1 : 0;
    if (per_cu[b] == 0) {
        auto kernel = gemm_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, false>;
        if constexpr (AMODE != A_CONV) {
            if (b) kernel = gemm_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, true>;
        }
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, 64 * WAVES_M * WAVES_N, 0) != hipSuccess ||
            n < 1)
            n = 1;
        per_cu[b] = n;
    }
    return per_cu[b];
}

// Stream-K launch: a.sk_groups work-groups (planned by the caller together
// with the workspace), after zeroing the tiles' arrival counters.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC>
static hipError_t launch_gemm_streamk(const KernelArgs &a, hipStream_t stream)
{
    if (a.sk_groups < 1 || !a.sk_part || !a.sk_cnt || a.sk_nkb < 1) return hipErrorInvalidValue;
    const hipError_t z = launch_zero_ints(a.sk_cnt, a.tiles_m * a.tiles_n, stream);
    if (z != hipSuccess) return z;
    const dim3 grid((unsigned)a.sk_groups), block(64 * WAVES_M * WAVES_N);
    if constexpr (AMODE != A_CONV) {
        if (reads_c<AMODE>(a)) {
            hipLaunchKernelGGL((gemm_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, true>),
                               grid, block, 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((gemm_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, false>),
                       grid, block, 0, stream, a);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int AMODE, bool TB, int OCC>
static int resident_dma_streamk(int beta)
{
    static int per_cu[2] = {0, 0};  // the same on every MI355X
    const int b = beta ? 1 : 0;
    if (per_cu[b] == 0) {
        auto kernel = gemm_dma_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, STAGES, AMODE, TB, OCC, false>;
        if constexpr (AMODE != A_CONV) {
            if (b) kernel = gemm_dma_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, STAGES, AMODE, TB, OCC, true>;
        }
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, 64 * WAVES_M * WAVES_N, 0) != hipSuccess ||
            n < 1)
            n = 1;
        per_cu[b] = n;
    }
    return per_cu[b];
}

// Stream-K launch of the direct-to-LDS contraction (as launch_gemm_streamk).
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int AMODE, bool TB, int OCC>
static hipError_t launch_gemm_dma_streamk(const KernelArgs &a, hipStream_t stream)
{
    if (a.sk_groups < 1 || !a.sk_part || !a.sk_cnt || a.sk_nkb < 1) return hipErrorInvalidValue;
    const hipError_t z = launch_zero_ints(a.sk_cnt, a.tiles_m * a.tiles_n, stream);
    if (z != hipSuccess) return z;
    const dim3 grid((unsigned)a.sk_groups), block(64 * WAVES_M * WAVES_N);
    if constexpr (AMODE != A_CONV) {
        if (reads_c<AMODE>(a)) {
            hipLaunchKernelGGL((gemm_dma_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, STAGES, AMODE, TB, OCC, true>),
                               grid, block, 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((gemm_dma_streamk_kernel<BM, BN, BK, WAVES_M, WAVES_N, STAGES, AMODE, TB, OCC, false>), grid,
                       block, 0, stream, a);
    return hipGetLastError();
}

// K split among groups of waves, operands copied straight into LDS.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int KS, int STAGES, int AMODE, bool TB, int OCC>
static hipError_t launch_gemm_dma_ksplit(const KernelArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.tiles_m * a.tiles_n), (unsigned)(a.nbatch > 1 ? a.nbatch : 1), (unsigned)a.splits);
    const dim3 block(64 * WAVES_M * WAVES_N * KS);
    if constexpr (AMODE != A_CONV) {
        if (reads_c<AMODE>(a)) {
            hipLaunchKernelGGL(
                (gemm_dma_ksplit_kernel<BM, BN, BK, WAVES_M, WAVES_N, KS, STAGES, AMODE, TB, OCC, true>), grid,
                block, 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((gemm_dma_ksplit_kernel<BM, BN, BK, WAVES_M, WAVES_N, KS, STAGES, AMODE, TB, OCC, false>),
                       grid, block, 0, stream, a);
    return hipGetLastError();
}

// B-resident streaming launch: as many work-groups as the CUs hold, a
// multiple of (XCD count) x (column blocks N / BN), each walking a contiguous
// range of row tiles of one column block.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int OCC>
static hipError_t launch_gemm_bres(const KernelArgs &a, hipStream_t stream)
{
    if (a.K != BK || a.N % BN != 0 || a.N < BN || a.splits > 1 || a.nbatch > 1) return hipErrorInvalidValue;
    const bool beta = reads_c<A_KCONTIG>(a);
    auto kernel = beta ? gemm_bres_kernel<BM, BN, BK, WAVES_M, WAVES_N, OCC, true>
                       : gemm_bres_kernel<BM, BN, BK, WAVES_M, WAVES_N, OCC, false>;
    const int threads = 64 * WAVES_M * WAVES_N;
    static int per_cu[2] = {0, 0};
    if (per_cu[beta] == 0) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1) n = 1;
        per_cu[beta] = n;
    }
    const int64_t tiles = (a.M + BM - 1) / BM;
    const int64_t ncb = a.N / BN;
    const int64_t x = a.xcds > 1 ? a.xcds : 1;
    // row groups per column block: a multiple of x, at most one per tile (and x)
    int64_t groups = (int64_t)per_cu[beta] * device_cu_count() / ncb;
    groups -= groups % x;
    if (groups > tiles) groups = (tiles + x - 1) / x * x;
    if (groups < x) groups = x;
    hipLaunchKernelGGL(kernel, dim3((unsigned)(groups * ncb)), dim3(threads), 0, stream, a);
    return hipGetLastError();
}

// K split among KS groups of waves inside each work-group; a split across
// work-groups (grid z) divides the K-blocks first, as in launch_gemm.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int KS, int AHEAD, int AMODE, bool B_KCONTIG, int VA,
          int VB, int OCC>
static hipError_t launch_gemm_ksplit(const KernelArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.tiles_m * a.tiles_n), (unsigned)(a.nbatch > 1 ? a.nbatch : 1), (unsigned)a.splits);
    const dim3 block(64 * WAVES_M * WAVES_N * KS);
    if (reads_c<AMODE>(a)) {
        hipLaunchKernelGGL(
            (gemm_ksplit_kernel<BM, BN, BK, WAVES_M, WAVES_N, KS, AHEAD, AMODE, B_KCONTIG, VA, VB, OCC, true>), grid, block,
            0, stream, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((gemm_ksplit_kernel<BM, BN, BK, WAVES_M, WAVES_N, KS, AHEAD, AMODE, B_KCONTIG, VA, VB, OCC, false>),
                       grid, block, 0, stream, a);
    return hipGetLastError();
}

// Direct-to-LDS staging (same grid as launch_gemm; dense operands).  The
// host checks that the rows one tile addresses span less than 2 GiB.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int AMODE, bool TB, int OCC>
static hipError_t launch_gemm_dma(const KernelArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.tiles_m * a.tiles_n), (unsigned)(a.nbatch > 1 ? a.nbatch : 1), (unsigned)a.splits);
    const dim3 block(64 * WAVES_M * WAVES_N);
    if constexpr (AMODE != A_CONV) {
        if (reads_c<AMODE>(a)) {
            hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, BK, WAVES_M, WAVES_N, STAGES, AMODE, TB, OCC, true>), grid,
                               block, 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, BK, WAVES_M, WAVES_N, STAGES, AMODE, TB, OCC, false>), grid, block, 0,
                       stream, a);
    return hipGetLastError();
}

// Loads two K-blocks ahead (same grid as launch_gemm).
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC>
static hipError_t launch_gemm_deep(const KernelArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.tiles_m * a.tiles_n), (unsigned)(a.nbatch > 1 ? a.nbatch : 1), (unsigned)a.splits);
    const dim3 block(64 * WAVES_M * WAVES_N);
    if constexpr (AMODE != A_CONV) {
        if (reads_c<AMODE>(a)) {
            hipLaunchKernelGGL((gemm_deep_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, true>),
                               grid, block, 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((gemm_deep_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, false>), grid,
                       block, 0, stream, a);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC>
static hipError_t launch_gemm_single_stage(const KernelArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.tiles_m * a.tiles_n), (unsigned)(a.nbatch > 1 ? a.nbatch : 1), (unsigned)a.splits);
    const dim3 block(64 * WAVES_M * WAVES_N);
    if constexpr (AMODE != A_CONV) {
        if (reads_c<AMODE>(a)) {
            hipLaunchKernelGGL(
                (gemm_single_stage_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, true>), grid,
                block, 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((gemm_single_stage_kernel<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB, OCC, false>),
                       grid, block, 0, stream, a);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB>
static constexpr int lds_bytes()
{
    return (int)sizeof(float) * GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB>::LDS_FLOATS;
}

#define PK_GEMM(name, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC)                                         \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC, 0,                                    \
     lds_bytes<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>(),                \
     &launch_gemm<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB, OCC>}

#define PK_CONV(name, BM, BN, BK, WM, WN, VA, VB, OCC)                                                 \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, VA, VB, OCC, 0,                                      \
     lds_bytes<BM, BN, BK, WM, WN, A_CONV, false, VA, VB>(),                                          \
     &launch_gemm<BM, BN, BK, WM, WN, A_CONV, false, VA, VB, OCC>}

#define PK_GEMM_P(name, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC)                                       \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC, 1,                                    \
     lds_bytes<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>(),                \
     &launch_gemm_persistent<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB, OCC>}

#define PK_GEMM_1S(name, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC)                                      \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC, 0,                                    \
     lds_bytes<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>() / 2,            \
     &launch_gemm_single_stage<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB, OCC>, 1}

#define PK_GEMM_D(name, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC)                                       \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC, 0,                                    \
     lds_bytes<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>(),                \
     &launch_gemm_deep<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB, OCC>}

#define PK_GEMM_KS(name, BM, BN, BK, WM, WN, KS, AHEAD, TA, TB, VA, VB, OCC)                         \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC, 0,                                    \
     KS * lds_bytes<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>(),           \
     &launch_gemm_ksplit<BM, BN, BK, WM, WN, KS, AHEAD, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB, OCC>, \
     0, 0, nullptr, 0, KS}

#define PK_GEMM_DMA(name, BM, BN, BK, WM, WN, STAGES, TA, TB, OCC)                                    \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, 4, 4, OCC, 0, STAGES * 4 * (BM * BK + BK * BN),     \
     &launch_gemm_dma<BM, BN, BK, WM, WN, STAGES, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), OCC>, 0, 0, nullptr, 0, 1, \
     STAGES}

#define PK_CONV_DMA(name, BM, BN, BK, WM, WN, STAGES, OCC)                                           \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, 4, 4, OCC, 0, STAGES * 4 * (BM * BK + BK * BN),      \
     &launch_gemm_dma<BM, BN, BK, WM, WN, STAGES, A_CONV, false, OCC>, 0, 0, nullptr, 0, 1, STAGES}

#define PK_GEMM_DMA_KS(name, BM, BN, BK, WM, WN, KS, STAGES, TA, TB, OCC)                              \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, 4, 4, OCC, 0, KS * STAGES * 4 * (BM * BK + BK * BN), \
     &launch_gemm_dma_ksplit<BM, BN, BK, WM, WN, KS, STAGES, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), OCC>, \
     0, 0, nullptr, 0, KS, STAGES}

#define PK_CONV_DMA_KS(name, BM, BN, BK, WM, WN, KS, STAGES, OCC)                                    \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, 4, 4, OCC, 0, KS * STAGES * 4 * (BM * BK + BK * BN),     \
     &launch_gemm_dma_ksplit<BM, BN, BK, WM, WN, KS, STAGES, A_CONV, false, OCC>, 0, 0, nullptr, 0, KS, STAGES}

#define PK_GEMM_DMA_SK(name, BM, BN, BK, WM, WN, STAGES, OCC)                                       \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, 0, 0, 4, 4, OCC, 0, STAGES * 4 * (BM * BK + BK * BN),       \
     &launch_gemm_dma_streamk<BM, BN, BK, WM, WN, STAGES, A_KCONTIG, false, OCC>, 0, 1,                \
     &resident_dma_streamk<BM, BN, BK, WM, WN, STAGES, A_KCONTIG, false, OCC>, 0, 1, STAGES}

#define PK_CONV_DMA_SK(name, BM, BN, BK, WM, WN, STAGES, OCC)                                        \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, 4, 4, OCC, 0, STAGES * 4 * (BM * BK + BK * BN),       \
     &launch_gemm_dma_streamk<BM, BN, BK, WM, WN, STAGES, A_CONV, false, OCC>, 0, 1,                   \
     &resident_dma_streamk<BM, BN, BK, WM, WN, STAGES, A_CONV, false, OCC>, 0, 1, STAGES}

#define PK_CONV_D(name, BM, BN, BK, WM, WN, VA, VB, OCC)                                               \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, VA, VB, OCC, 0,                                      \
     lds_bytes<BM, BN, BK, WM, WN, A_CONV, false, VA, VB>(),                                          \
     &launch_gemm_deep<BM, BN, BK, WM, WN, A_CONV, false, VA, VB, OCC>}

#define PK_CONV_P(name, BM, BN, BK, WM, WN, VA, VB, OCC)                                               \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, VA, VB, OCC, 1,                                      \
     lds_bytes<BM, BN, BK, WM, WN, A_CONV, false, VA, VB>(),                                          \
     &launch_gemm_persistent<BM, BN, BK, WM, WN, A_CONV, false, VA, VB, OCC>}


// LDS of the B-resident form: two A stages and B transposed.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N>
static constexpr int bres_lds_bytes()
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, A_KCONTIG, true, 4, 4> G;
    return (int)sizeof(float) * (2 * G::A_STAGE + G::B_STAGE);
}

#define PK_GEMM_BRES(name, BM, BN, BK, WM, WN, OCC)                                                    \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, 0, 0, 4, 4, OCC, 0, bres_lds_bytes<BM, BN, BK, WM, WN>(),   \
     &launch_gemm_bres<BM, BN, BK, WM, WN, OCC>, 0, 0, nullptr, 1}

#define PK_GEMM_SK(name, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC)                                      \
    {#name, KIND_GEMM, BM, BN, BK, WM, WN, TA, TB, VA, VB, OCC, 0,                                    \
     lds_bytes<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB>(),                \
     &launch_gemm_streamk<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB, OCC>, 0, 1, \
     &resident_streamk<BM, BN, BK, WM, WN, (TA ? A_MCONTIG : A_KCONTIG), (TB != 0), VA, VB, OCC>}

#define PK_CONV_SK(name, BM, BN, BK, WM, WN, VA, VB, OCC)                                              \
    {#name, KIND_CONV, BM, BN, BK, WM, WN, 0, 0, VA, VB, OCC, 0,                                      \
     lds_bytes<BM, BN, BK, WM, WN, A_CONV, false, VA, VB>(),                                          \
     &launch_gemm_streamk<BM, BN, BK, WM, WN, A_CONV, false, VA, VB, OCC>, 0, 1,                      \
     &resident_streamk<BM, BN, BK, WM, WN, A_CONV, false, VA, VB, OCC>}

}  // namespace pk
