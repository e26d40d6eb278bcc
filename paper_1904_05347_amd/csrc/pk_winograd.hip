// pk_winograd.hip -- the transforms of the Winograd convolutions F(2x2, 3x3)
// and F(4x4, 3x3) (Section 4.1.2: the Lavin-Gray minimal-filtering technique
// the paper adopts, whose output-tile size m is the parameter it trades: a
// larger tile needs fewer multiplications per output but has larger transform
// coefficients and smaller batched products), for a 3x3 window at stride 1.
// The product in the middle is the batched contraction of pk_kernel.hpp
// ((m+2)^2 independent Cin-deep products); these kernels are the memory-bound
// steps around it.  With A = m + 2 (the transformed tile's side):
//
//   filter:  U[p][ci][co] = (G g G^T)[p],   g = f[.][.][ci][co]        (3x3 -> AxA)
//   input:   V[p][t][ci]  = (B^T d B)[p],   d = the AxA input tile t   (zero outside)
//   product: M[p] = V[p] U[p]               (T x Cin) (Cin x Cout), p = 0..A*A-1
//   output:  y(m x m block of tile t, co) = A^T mm A,  mm[p] = M[p][t][co]
//
// F(2, 3), interpolation points 0, 1, -1, infinity:
//   G = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1],
//   B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1],  A^T = [1 1 1 0; 0 1 -1 -1].
// F(4, 3), points 0, 1, -1, 2, -2, infinity:
//   G = [1/4 0 0; -1/6 -1/6 -1/6; -1/6 1/6 -1/6; 1/24 1/12 1/6; 1/24 -1/12 1/6; 0 0 1],
//   B^T = [4 0 -5 0 1 0; 0 -4 -4 1 1 0; 0 4 -4 -1 1 0; 0 -2 -1 2 1 0; 0 2 -1 -2 1 0;
//          0 4 0 -5 0 1],
//   A^T = [1 1 1 1 1 0; 0 1 -1 2 -2 0; 0 1 1 4 4 0; 0 1 -1 8 -8 1].
// Tile t = (n, th, tw) covers output rows m*th .. m*th+m-1 and columns
// m*tw .. m*tw+m-1; its input tile starts at row m*th - pt, column
// m*tw - pl.  p = A*a + b for row a, column b of the transformed tile.
//
// Layout (all row-major, in the caller's workspace): U is A*A matrices
// Cin x Cout, V is A*A matrices T x Cin, M is A*A matrices T x Cout, so the
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

template <typename T>
__device__ __forceinline__ T vzero();
template <>
__device__ __forceinline__ float vzero<float>() { return 0.f; }
template <>
__device__ __forceinline__ float4 vzero<float4>() { return make_float4(0.f, 0.f, 0.f, 0.f); }

constexpr int WT_THREADS = 256;

// The 1-D transforms along one axis of a tile (elementwise on vectors):
// e = B^T d (input), r = A^T mm (output), u = G g (filter).
template <int MT>
struct Wino;

template <>
struct Wino<2> {
    static constexpr int A = 4;
    template <typename T>
    __device__ static __forceinline__ void input_1d(const T *d, T *e)
    {
        e[0] = d[0] - d[2];
        e[1] = d[1] + d[2];
        e[2] = d[2] - d[1];
        e[3] = d[1] - d[3];
    }
    template <typename T>
    __device__ static __forceinline__ void output_1d(const T *mm, T *r)
    {
        r[0] = mm[0] + mm[1] + mm[2];
        r[1] = mm[1] - mm[2] - mm[3];
    }
    __device__ static __forceinline__ void filter_1d(const float *g, float *u)
    {
        u[0] = g[0];
        u[1] = 0.5f * (g[0] + g[1] + g[2]);
        u[2] = 0.5f * (g[0] - g[1] + g[2]);
        u[3] = g[2];
    }
};

template <>
struct Wino<4> {
    static constexpr int A = 6;
    template <typename T>
    __device__ static __forceinline__ void input_1d(const T *d, T *e)
    {
        const T a = d[4] - 4.f * d[2];  // shared by rows 1 and 2
        const T b = d[3] - 4.f * d[1];
        const T c = d[4] - d[2];         // shared by rows 3 and 4
        const T s = 2.f * (d[3] - d[1]);
        e[0] = 4.f * d[0] - 5.f * d[2] + d[4];
        e[1] = a + b;
        e[2] = a - b;
        e[3] = c + s;
        e[4] = c - s;
        e[5] = 4.f * d[1] - 5.f * d[3] + d[5];
    }
    template <typename T>
    __device__ static __forceinline__ void output_1d(const T *mm, T *r)
    {
        const T p12 = mm[1] + mm[2], m12 = mm[1] - mm[2];
        const T p34 = mm[3] + mm[4], m34 = mm[3] - mm[4];
        r[0] = mm[0] + p12 + p34;
        r[1] = m12 + 2.f * m34;
        r[2] = p12 + 4.f * p34;
        r[3] = m12 + 8.f * m34 + mm[5];
    }
    __device__ static __forceinline__ void filter_1d(const float *g, float *u)
    {
        const float s = g[0] + g[2];
        u[0] = 0.25f * g[0];
        u[1] = (-1.f / 6.f) * (s + g[1]);
        u[2] = (-1.f / 6.f) * (s - g[1]);
        const float q = (1.f / 24.f) * g[0] + (1.f / 6.f) * g[2];
        u[3] = q + (1.f / 12.f) * g[1];
        u[4] = q - (1.f / 12.f) * g[1];
        u[5] = g[2];
    }
};

template <int MT>
__global__ void __launch_bounds__(WT_THREADS) wino_filter_kernel(const float *__restrict__ f, float *__restrict__ U,
                                                                 int64_t pairs)
{
    constexpr int A = Wino<MT>::A;
    const int64_t e = (int64_t)blockIdx.x * WT_THREADS + threadIdx.x;  // ci * Cout + co
    if (e >= pairs) return;
    float g[3][3];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int c = 0; c < 3; ++c) g[r][c] = f[(int64_t)(r * 3 + c) * pairs + e];
    float t[A][3];  // G g
#pragma unroll
    for (int c = 0; c < 3; ++c) {
        float col[3] = {g[0][c], g[1][c], g[2][c]}, out[A];
        Wino<MT>::filter_1d(col, out);
#pragma unroll
        for (int a = 0; a < A; ++a) t[a][c] = out[a];
    }
#pragma unroll
    for (int a = 0; a < A; ++a) {
        float u[A];  // (G g) G^T, row a
        Wino<MT>::filter_1d(t[a], u);
#pragma unroll
        for (int b = 0; b < A; ++b) U[(int64_t)(A * a + b) * pairs + e] = u[b];
    }
}

template <int MT, int VEC>
__global__ void __launch_bounds__(WT_THREADS) wino_input_kernel(const float *__restrict__ x, float *__restrict__ V,
                                                                int H, int W, int Cin, int pt, int pl, int TH,
                                                                int TW, int64_t T)
{
    constexpr int A = Wino<MT>::A;
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
    const int ih0 = MT * th - pt, iw0 = MT * tw - pl;
    const float *img = x + n * H * (int64_t)W * Cin + ci;
    vt s[A][A];  // B^T d, one input column at a time
#pragma unroll
    for (int c = 0; c < A; ++c) {
        const int iw = iw0 + c;
        vt col[A];
#pragma unroll
        for (int r = 0; r < A; ++r) {
            const int ih = ih0 + r;
            vt v = vzero<vt>();
            if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W)
                v = *(const vt *)(img + ((int64_t)ih * W + iw) * Cin);
            col[r] = v;
        }
        vt out[A];
        Wino<MT>::input_1d(col, out);
#pragma unroll
        for (int a = 0; a < A; ++a) s[a][c] = out[a];
    }
    const int64_t plane = T * Cin;
    float *dst = V + t * Cin + ci;
#pragma unroll
    for (int a = 0; a < A; ++a) {
        vt v[A];  // (B^T d) B, row a
        Wino<MT>::input_1d(s[a], v);
#pragma unroll
        for (int b = 0; b < A; ++b) *(vt *)(dst + (int64_t)(A * a + b) * plane) = v[b];
    }
}

template <int MT, int VEC>
__global__ void __launch_bounds__(WT_THREADS) wino_output_kernel(const float *__restrict__ M, float *__restrict__ y,
                                                                 int Ho, int Wo, int Cout, int TH, int TW, int64_t T)
{
    constexpr int A = Wino<MT>::A;
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
    const float *src = M + t * Cout + co;
    vt r[MT][A];  // A^T mm, one transformed column at a time
#pragma unroll
    for (int b = 0; b < A; ++b) {
        vt col[A], out[MT];
#pragma unroll
        for (int a = 0; a < A; ++a) col[a] = *(const vt *)(src + (int64_t)(A * a + b) * plane);
        Wino<MT>::output_1d(col, out);
#pragma unroll
        for (int i = 0; i < MT; ++i) r[i][b] = out[i];
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        const int ho = MT * th + i;
        if (ho >= Ho) continue;
        vt o[MT];  // (A^T mm) A, row i
        Wino<MT>::output_1d(r[i], o);
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int wo = MT * tw + j;
            if (wo >= Wo) continue;
            *(vt *)(y + ((n * Ho + ho) * (int64_t)Wo + wo) * Cout + co) = o[j];
        }
    }
}

unsigned blocks_for(int64_t threads) { return (unsigned)((threads + WT_THREADS - 1) / WT_THREADS); }

}  // namespace

hipError_t launch_wino_filter(int m, const float *f, float *U, int64_t Cin, int64_t Cout, hipStream_t stream)
{
    const int64_t pairs = Cin * Cout;
    if (m == 4)
        hipLaunchKernelGGL(wino_filter_kernel<4>, dim3(blocks_for(pairs)), dim3(WT_THREADS), 0, stream, f, U, pairs);
    else
        hipLaunchKernelGGL(wino_filter_kernel<2>, dim3(blocks_for(pairs)), dim3(WT_THREADS), 0, stream, f, U, pairs);
    return hipGetLastError();
}

template <int MT>
static void input_launch(const float *x, float *V, int64_t H, int64_t W, int64_t Cin, int64_t pt, int64_t pl,
                         int64_t TH, int64_t TW, int64_t T, bool vec4, hipStream_t stream)
{
    if (vec4)
        hipLaunchKernelGGL((wino_input_kernel<MT, 4>), dim3(blocks_for(T * (Cin / 4))), dim3(WT_THREADS), 0, stream,
                           x, V, (int)H, (int)W, (int)Cin, (int)pt, (int)pl, (int)TH, (int)TW, T);
    else
        hipLaunchKernelGGL((wino_input_kernel<MT, 1>), dim3(blocks_for(T * Cin)), dim3(WT_THREADS), 0, stream, x,
                           V, (int)H, (int)W, (int)Cin, (int)pt, (int)pl, (int)TH, (int)TW, T);
}

hipError_t launch_wino_input(int m, const float *x, float *V, int64_t H, int64_t W, int64_t Cin, int64_t pt,
                             int64_t pl, int64_t TH, int64_t TW, int64_t T, bool vec4, hipStream_t stream)
{
    if (m == 4)
        input_launch<4>(x, V, H, W, Cin, pt, pl, TH, TW, T, vec4, stream);
    else
        input_launch<2>(x, V, H, W, Cin, pt, pl, TH, TW, T, vec4, stream);
    return hipGetLastError();
}

template <int MT>
static void output_launch(const float *M, float *y, int64_t Ho, int64_t Wo, int64_t Cout, int64_t TH, int64_t TW,
                          int64_t T, bool vec4, hipStream_t stream)
{
    if (vec4)
        hipLaunchKernelGGL((wino_output_kernel<MT, 4>), dim3(blocks_for(T * (Cout / 4))), dim3(WT_THREADS), 0,
                           stream, M, y, (int)Ho, (int)Wo, (int)Cout, (int)TH, (int)TW, T);
    else
        hipLaunchKernelGGL((wino_output_kernel<MT, 1>), dim3(blocks_for(T * Cout)), dim3(WT_THREADS), 0, stream, M,
                           y, (int)Ho, (int)Wo, (int)Cout, (int)TH, (int)TW, T);
}

hipError_t launch_wino_output(int m, const float *M, float *y, int64_t Ho, int64_t Wo, int64_t Cout, int64_t TH,
                              int64_t TW, int64_t T, bool vec4, hipStream_t stream)
{
    if (m == 4)
        output_launch<4>(M, y, Ho, Wo, Cout, TH, TW, T, vec4, stream);
    else
        output_launch<2>(M, y, Ho, Wo, Cout, TH, TW, T, vec4, stream);
    return hipGetLastError();
}

}  // namespace pk
