// pk_configs.hpp -- the compiled tile-parameter space and its registry.
//
// The paper keeps tile sizes as compile-time template parameters and picks a
// configuration per device and problem shape (Sections 3.1 and 5: "h x w"
// registers per thread, "r x c" threads per work-group, optional local memory
// and double buffering).  Here each configuration is one instance of
// pk::gemm_kernel; the registry lists them for the selector and for callers
// that want to force one (tuning, ablations, tests).
#pragma once

#include <hip/hip_runtime.h>

#include "pk_args.hpp"

namespace pk {

enum Kind { KIND_GEMM = 0, KIND_CONV = 1, KIND_DIRECT = 2 };

typedef hipError_t (*LaunchFn)(const KernelArgs &args, hipStream_t stream);

struct Config {
    const char *name;
    int kind;
    int bm, bn, bk;
    int waves_m, waves_n;
    int trans_a, trans_b;  // GEMM: 1 = operand stored transposed; CONV: always 0
    int vec_a, vec_b;
    int occupancy;  // waves per SIMD the registers are allotted for (1 = unconstrained)
    int persistent; // 1 = grid sized to the resident work-groups, each looping over tiles
    int lds_bytes;
    LaunchFn launch;
    int single_stage;  // 1 = one LDS stage (no double buffering; an ablation form)
    int streamk;       // 1 = stream-K: resident work-groups share the (tile, K-block) iterations evenly
    // work-groups of this instance one CU holds at once (occupancy query;
    // beta != 0 selects the epilogue that reads C).  Set for stream-K instances.
    int (*resident)(int beta);
    int bres;  // 1 = op(B) resident in LDS: runs only products with K == bk and N a multiple of bn
    int kgroups = 1;  // groups of waves splitting K inside the work-group (gemm_ksplit_kernel)
    int dma = 0;      // LDS stages filled straight from global memory (gemm_dma_kernel); 0 = register-staged
    // tiled direct convolution (pk_direct_tiled.hip): output rows of a
    // work-group's tile (its columns are bm / tile_rows, its channels bn, its
    // input-channel load width vec_a); 0 for every other kind
    int tile_rows = 0;
};

// LDS a tiled direct convolution instance may ask for at launch (dynamic).
constexpr int kDirectTiledMaxLds = 65536;
// Bytes of LDS tiled direct instance c needs for this window (-1 when the
// sizes are out of range).
size_t direct_tiled_lds_bytes(const Config *c, int64_t KH, int64_t KW, int64_t Cin, int64_t sh, int64_t sw);

// The registry (defined with the kernel instances, host side only).
const Config *configs(int *count);

hipError_t launch_splitk_reduce(const float *ws, float *C, int M, int N, int64_t ldc, int splits,
                                float beta, hipStream_t stream);
// Compute units of the current device (queried once per device).
int device_cu_count();

// Whether a direct convolution configuration takes this window: c, or, when
// c is NULL, the fixed-tile short-reduction kernel that the rules choose
// (reduction of at most 32, input patch fits its LDS buffer).
bool direct_conv_fits(const Config *c, int64_t W, int64_t Wo, int64_t Cout, int64_t KH, int64_t KW, int64_t Cin,
                      int64_t sh, int64_t sw);

hipError_t launch_scale(float *C, int M, int N, int64_t ldc, float beta, hipStream_t stream);
// p[0 .. n) = 0 (a kernel, so that it may be captured in a graph).
hipError_t launch_zero_ints(int *p, int n, hipStream_t stream);

// Winograd F(m x m, 3x3) transforms, m = 2 or 4 (pk_winograd.hip); A = m + 2.
// U: A*A x Cin x Cout, V: A*A x T x Cin, M: A*A x T x Cout, T = N * TH * TW
// tiles of m x m outputs.  vec4: channel count divisible by 4 and every
// pointer 16-byte aligned.
hipError_t launch_wino_filter(int m, const float *f, float *U, int64_t Cin, int64_t Cout, hipStream_t stream);
hipError_t launch_wino_input(int m, const float *x, float *V, int64_t H, int64_t W, int64_t Cin, int64_t pt,
                             int64_t pl, int64_t TH, int64_t TW, int64_t T, bool vec4, hipStream_t stream);
hipError_t launch_wino_output(int m, const float *M, float *y, int64_t Ho, int64_t Wo, int64_t Cout, int64_t TH,
                              int64_t TW, int64_t T, bool vec4, hipStream_t stream);

}  // namespace pk
