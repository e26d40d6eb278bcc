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
};

// The registry (defined with the kernel instances, host side only).
const Config *configs(int *count);

hipError_t launch_splitk_reduce(const float *ws, float *C, int M, int N, int64_t ldc, int splits,
                                float beta, hipStream_t stream);
// Compute units of the current device (queried once per device).
int device_cu_count();

// Whether the tiled direct convolution takes this window (short reduction,
// input patch fits its LDS buffer).
bool direct_conv_fits(int64_t KH, int64_t KW, int64_t Cin, int64_t sh, int64_t sw);

hipError_t launch_scale(float *C, int M, int N, int64_t ldc, float beta, hipStream_t stream);

}  // namespace pk
