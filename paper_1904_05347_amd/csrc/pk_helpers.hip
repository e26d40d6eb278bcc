// pk_helpers.hip -- the split-K reduction and the beta-scaling launches.
#include <hip/hip_runtime.h>

#include "pk_configs.hpp"

namespace pk {

// Fixed-order reduction of split-K partials: C = sum_z ws[z] (+ beta * C).
// Element e of the M x N result is summed over z = 0, 1, ... in that order,
// so the result does not depend on scheduling.  Each work-item owns V
// consecutive elements of one row (V = 4 when rows and both buffers allow
// 16-byte accesses) and issues the loads of up to eight partials before the
// first addition, so a split of S costs about S/8 memory round trips
// instead of S.
template <int V>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(const float *ws, float *C, int M, int N,
                                                            int64_t ldc, int splits, float beta)
{
    typedef float VT __attribute__((ext_vector_type(V)));
    constexpr int B = 8;  // partials in flight per work-item
    const int64_t total = (int64_t)M * N;
    const int nv = N / V;
    const int64_t items = (int64_t)M * nv;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t it = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; it < items; it += stride) {
        const int64_t row = it / nv;
        const int col = (int)(it - row * nv) * V;
        const float *p = ws + row * N + col;
        VT s = *reinterpret_cast<const VT *>(p);
        for (int z = 1; z < splits; z += B) {
            VT v[B];
#pragma unroll
            for (int u = 0; u < B; ++u)
                if (z + u < splits) v[u] = *reinterpret_cast<const VT *>(p + (int64_t)(z + u) * total);
#pragma unroll
            for (int u = 0; u < B; ++u)
                if (z + u < splits) s += v[u];
        }
        float *c = C + row * ldc + col;
        if (beta != 0.f) {
#pragma unroll
            for (int j = 0; j < V; ++j) s[j] = fmaf(beta, c[j], s[j]);
        }
        *reinterpret_cast<VT *>(c) = s;
    }
}

// C <- beta * C (alpha == 0 or K == 0).  beta == 0 writes zeros without reading.
__global__ void __launch_bounds__(256) scale_kernel(float *C, int M, int N, int64_t ldc, float beta)
{
    const int64_t total = (int64_t)M * N;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += stride) {
        const int64_t row = e / N, col = e - row * N;
        float *c = C + row * ldc + col;
        *c = beta != 0.f ? beta * *c : 0.f;
    }
}

// Arrival counters of a stream-K launch start at zero.
__global__ void __launch_bounds__(256) zero_ints_kernel(int *p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// ---------------------------------------------------------------- helpers

int device_cu_count()
{
    static int counts[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
    if (counts[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
        counts[dev] = n;
    }
    return counts[dev];
}

hipError_t launch_splitk_reduce(const float *ws, float *C, int M, int N, int64_t ldc, int splits,
                                float beta, hipStream_t stream)
{
    const bool v4 = N % 4 == 0 && ldc % 4 == 0 && reinterpret_cast<uintptr_t>(C) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(ws) % 16 == 0;
    const int64_t items = (int64_t)M * N / (v4 ? 4 : 1);
    const int64_t blocks = (items + 255) / 256;
    const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
    if (v4)
        hipLaunchKernelGGL(splitk_reduce_kernel<4>, dim3(grid), dim3(256), 0, stream, ws, C, M, N, ldc, splits, beta);
    else
        hipLaunchKernelGGL(splitk_reduce_kernel<1>, dim3(grid), dim3(256), 0, stream, ws, C, M, N, ldc, splits, beta);
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

hipError_t launch_zero_ints(int *p, int n, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(zero_ints_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, p, n);
    return hipGetLastError();
}

}  // namespace pk
