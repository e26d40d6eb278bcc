// pk_winograd.hip -- the transforms of the Winograd convolution F(2x2, 3x3)
// (Section 4.1.2: the Lavin-Gray technique the paper adopts), for a 3x3
// window at stride 1.  The product in the middle is the batched contraction of
// pk_kernel.hpp (16 independent Cin-deep products); these kernels are the
// memory-bound steps around it:
//
//   filter:  U[p][ci][co] = (G g G^T)[p],   g = f[.][.][ci][co]        (3x3 -> 4x4)
//   input:   V[p][t][ci]  = (B^T d B)[p],   d = the 4x4 input tile t   (zero outside)
//   product: M[p] = V[p] U[p]               (T x Cin) (Cin x Cout), p = 0..15
//   output:  y(2 x 2 block of tile t, co) = A^T m A,  m[p] = M[p][t][co]
//
// with G = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1],
//      B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1],  A^T = [1 1 1 0; 0 1 -1 -1].
// Tile t = (n, th, tw) covers outputs rows 2th, 2th+1 and columns 2tw, 2tw+1;
// its input tile starts at row 2th - pt, column 2tw - pl.  p = 4*a + b for
// row a, column b of the 4x4 transformed tile.
//
// Layout (all row-major, in the caller's workspace): U is 16 matrices
// Cin x Cout, V is 16 matrices T x Cin, M is 16 matrices T x Cout, so the
// product is a batch of plain NN GEMMs.  Every transform thread handles one
// (tile, channel) pair -- VEC consecutive channels when the channel count
// allows 16-byte access -- so loads and stores are coalesced along the NHWC
// channel dimension.
#include <hip/hip_runtime.h>

#include "pk_configs.hpp"

namespace pk {

namespace {

template <int VEC>
struct VecT;
template <>
struct VecT<1> {
    typedef float type;
};
template <>
struct VecT<4> {
    typedef float4 type;
};

constexpr int WT_THREADS = 256;

// 1-D transforms of four values along one axis (elementwise on vectors).
template <typename T>
__device__ __forceinline__ void input_1d(const T &d0, const T &d1, const T &d2, const T &d3, T &e0, T &e1, T &e2,
                                         T &e3)
{
    e0 = d0 - d2;  // rows of B^T
    e1 = d1 + d2;
    e2 = d2 - d1;
    e3 = d1 - d3;
}

template <typename T>
__device__ __forceinline__ void output_1d(const T &m0, const T &m1, const T &m2, const T &m3, T &r0, T &r1)
{
    r0 = m0 + m1 + m2;  // rows of A^T
    r1 = m1 - m2 - m3;
}

__device__ __forceinline__ void filter_1d(float g0, float g1, float g2, float &u0, float &u1, float &u2, float &u3)
{
    u0 = g0;  // rows of G
    u1 = 0.5f * (g0 + g1 + g2);
    u2 = 0.5f * (g0 - g1 + g2);
    u3 = g2;
}

__global__ void __launch_bounds__(WT_THREADS) wino_filter_kernel(const float *__restrict__ f, float *__restrict__ U,
                                                                 int64_t pairs)
{
    const int64_t e = (int64_t)blockIdx.x * WT_THREADS + threadIdx.x;  // ci * Cout + co
    if (e >= pairs) return;
    float g[3][3];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int c = 0; c < 3; ++c) g[r][c] = f[(int64_t)(r * 3 + c) * pairs + e];
    float t[4][3];  // G g
#pragma unroll
    for (int c = 0; c < 3; ++c) filter_1d(g[0][c], g[1][c], g[2][c], t[0][c], t[1][c], t[2][c], t[3][c]);
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        float u[4];  // (G g) G^T, row a
        filter_1d(t[a][0], t[a][1], t[a][2], u[0], u[1], u[2], u[3]);
#pragma unroll
        for (int b = 0; b < 4; ++b) U[(int64_t)(4 * a + b) * pairs + e] = u[b];
    }
}

template <int VEC>
__global__ void __launch_bounds__(WT_THREADS) wino_input_kernel(const float *__restrict__ x, float *__restrict__ V,
                                                                int H, int W, int Cin, int pt, int pl, int TH,
                                                                int TW, int64_t T)
{
    typedef typename VecT<VEC>::type vt;
    const int cv = Cin / VEC;
    const int64_t e = (int64_t)blockIdx.x * WT_THREADS + threadIdx.x;  // t * cv + channel vector
    if (e >= T * cv) return;
    const int64_t t = e / cv;
    const int ci = (int)(e - t * cv) * VEC;
    const int tw = (int)(t % TW);
    const int64_t nt = t / TW;
    const int th = (int)(nt % TH);
    const int64_t n = nt / TH;
    const int ih0 = 2 * th - pt, iw0 = 2 * tw - pl;
    const float *img = x + n * H * (int64_t)W * Cin + ci;
    vt d[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int ih = ih0 + r;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int iw = iw0 + c;
            vt v;
            if constexpr (VEC == 1)
                v = 0.f;
            else
                v = make_float4(0.f, 0.f, 0.f, 0.f);
            if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W)
                v = *(const vt *)(img + ((int64_t)ih * W + iw) * Cin);
            d[r][c] = v;
        }
    }
    vt s[4][4];  // B^T d
#pragma unroll
    for (int c = 0; c < 4; ++c) input_1d(d[0][c], d[1][c], d[2][c], d[3][c], s[0][c], s[1][c], s[2][c], s[3][c]);
    const int64_t plane = T * Cin;
    float *out = V + t * Cin + ci;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        vt v[4];  // (B^T d) B, row a
        input_1d(s[a][0], s[a][1], s[a][2], s[a][3], v[0], v[1], v[2], v[3]);
#pragma unroll
        for (int b = 0; b < 4; ++b) *(vt *)(out + (int64_t)(4 * a + b) * plane) = v[b];
    }
}

template <int VEC>
__global__ void __launch_bounds__(WT_THREADS) wino_output_kernel(const float *__restrict__ M, float *__restrict__ y,
                                                                 int Ho, int Wo, int Cout, int TH, int TW, int64_t T)
{
    typedef typename VecT<VEC>::type vt;
    const int cv = Cout / VEC;
    const int64_t e = (int64_t)blockIdx.x * WT_THREADS + threadIdx.x;  // t * cv + channel vector
    if (e >= T * cv) return;
    const int64_t t = e / cv;
    const int co = (int)(e - t * cv) * VEC;
    const int tw = (int)(t % TW);
    const int64_t nt = t / TW;
    const int th = (int)(nt % TH);
    const int64_t n = nt / TH;
    const int64_t plane = T * Cout;
    const float *in = M + t * Cout + co;
    vt m[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) m[a][b] = *(const vt *)(in + (int64_t)(4 * a + b) * plane);
    vt r[2][4];  // A^T m
#pragma unroll
    for (int b = 0; b < 4; ++b) output_1d(m[0][b], m[1][b], m[2][b], m[3][b], r[0][b], r[1][b]);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int ho = 2 * th + i;
        if (ho >= Ho) continue;
        vt o[2];  // (A^T m) A, row i
        output_1d(r[i][0], r[i][1], r[i][2], r[i][3], o[0], o[1]);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int wo = 2 * tw + j;
            if (wo >= Wo) continue;
            *(vt *)(y + ((n * Ho + ho) * (int64_t)Wo + wo) * Cout + co) = o[j];
        }
    }
}

unsigned blocks_for(int64_t threads) { return (unsigned)((threads + WT_THREADS - 1) / WT_THREADS); }

}  // namespace

hipError_t launch_wino_filter(const float *f, float *U, int64_t Cin, int64_t Cout, hipStream_t stream)
{
    const int64_t pairs = Cin * Cout;
    hipLaunchKernelGGL(wino_filter_kernel, dim3(blocks_for(pairs)), dim3(WT_THREADS), 0, stream, f, U, pairs);
    return hipGetLastError();
}

hipError_t launch_wino_input(const float *x, float *V, int64_t H, int64_t W, int64_t Cin, int64_t pt, int64_t pl,
                             int64_t TH, int64_t TW, int64_t T, bool vec4, hipStream_t stream)
{
    if (vec4)
        hipLaunchKernelGGL(wino_input_kernel<4>, dim3(blocks_for(T * (Cin / 4))), dim3(WT_THREADS), 0, stream, x, V,
                           (int)H, (int)W, (int)Cin, (int)pt, (int)pl, (int)TH, (int)TW, T);
    else
        hipLaunchKernelGGL(wino_input_kernel<1>, dim3(blocks_for(T * Cin)), dim3(WT_THREADS), 0, stream, x, V,
                           (int)H, (int)W, (int)Cin, (int)pt, (int)pl, (int)TH, (int)TW, T);
    return hipGetLastError();
}

hipError_t launch_wino_output(const float *M, float *y, int64_t Ho, int64_t Wo, int64_t Cout, int64_t TH,
                              int64_t TW, int64_t T, bool vec4, hipStream_t stream)
{
    if (vec4)
        hipLaunchKernelGGL(wino_output_kernel<4>, dim3(blocks_for(T * (Cout / 4))), dim3(WT_THREADS), 0, stream, M,
                           y, (int)Ho, (int)Wo, (int)Cout, (int)TH, (int)TW, T);
    else
        hipLaunchKernelGGL(wino_output_kernel<1>, dim3(blocks_for(T * Cout)), dim3(WT_THREADS), 0, stream, M, y,
                           (int)Ho, (int)Wo, (int)Cout, (int)TH, (int)TW, T);
    return hipGetLastError();
}

}  // namespace pk
