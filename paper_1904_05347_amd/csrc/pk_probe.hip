// pk_probe.hip -- measurement probes for the roofline denominators.
//
// mfma_peak_kernel: every wave issues back-to-back v_mfma_f32_32x32x2_f32 on
// eight independent accumulators whose operands never change, so the matrix
// pipe never waits on memory or on a dependency.  Its rate is the fp32 matrix
// throughput the chip sustains under this load (clock, power).
// copy_kernel: a 16-byte-per-lane streaming copy, the HBM bandwidth a plain
// kernel sustains.
#include <hip/hip_runtime.h>

#include "../../include/pk.h"

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256) mfma_peak_kernel(int iters, float seed, float *out)
{
    const float a = seed + threadIdx.x * 1e-7f, b = seed - threadIdx.x * 1e-7f;
    f32x16 acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[i], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[i][r];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// The same issue pattern, but every MFMA reads different operand registers
// holding random fp32 values (loaded from `src`, 16 A and 16 B values per
// lane), so the multipliers see data of the kind a real product feeds them.
__global__ void __launch_bounds__(256) mfma_data_kernel(int iters, const float *src, float *out)
{
    float a[16], b[16];
    const int lane = blockIdx.x * blockDim.x + threadIdx.x;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        a[i] = src[(lane * 32 + i) & 0xFFFFF];
        b[i] = src[(lane * 32 + 16 + i) & 0xFFFFF];
    }
    f32x16 acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int s = 0; s < 16; ++s)
            acc[s & 3] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[s], b[(s * 7) & 15], acc[s & 3], 0, 0, 0);
    }
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) t += acc[i][r];
    out[lane] = t;
}

__global__ void __launch_bounds__(256) copy_kernel(const f32x4 *__restrict__ src, f32x4 *__restrict__ dst, int64_t n4)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) dst[i] = src[i];
}

}  // namespace

extern "C" {

int pk_probe_mfma_peak(int blocks, int iters, float *out, void *stream)
{
    if (blocks < 1) return PK_ERR_INVALID_VALUE;
    if (iters < 1) return PK_ERR_INVALID_VALUE;
    if (!out) return PK_ERR_INVALID_VALUE;
    hipLaunchKernelGGL(mfma_peak_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters, 1.0f, out);
    return hipGetLastError() == hipSuccess ? PK_OK : PK_ERR_LAUNCH;
}

int pk_probe_mfma_data(int blocks, int iters, const float *src, float *out, void *stream)
{
    if (blocks < 1 || iters < 1 || !src || !out) return PK_ERR_INVALID_VALUE;
    hipLaunchKernelGGL(mfma_data_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters, src, out);
    return hipGetLastError() == hipSuccess ? PK_OK : PK_ERR_LAUNCH;
}

int pk_probe_copy(const float *src, float *dst, int64_t n, void *stream)
{
    if (!src || !dst || n < 0 || n % 4 != 0 || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15))
        return PK_ERR_INVALID_VALUE;
    if (n == 0) return PK_OK;
    const int64_t n4 = n / 4;
    int64_t blocks = (n4 + 255) / 256;
    if (blocks > 256 * 64) blocks = 256 * 64;
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                       (const f32x4 *)src, (f32x4 *)dst, n4);
    return hipGetLastError() == hipSuccess ? PK_OK : PK_ERR_LAUNCH;
}

}  // extern "C"
