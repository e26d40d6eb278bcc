// pk_direct_tiled.hip -- the tiled direct convolution of Section 4.1.1 with
// its tile and vector widths as compile-time parameters.
//
// The paper's kernel gives each thread a tile of outputs so that the input
// slices of neighbouring outputs, which overlap for windows larger than 1x1,
// are loaded once and reused; the output tile and the vector widths over
// input and output channels are its parameters, and the best choice balances
// reuse against registers (its register and performance heatmaps).  On CDNA
// the unit of work is a 64-lane wave feeding the matrix cores, so the same
// three parameters are set per work-group and per wave:
//   TR x (32*MB)  output tile of a work-group: TR rows, each of MB blocks of
//                 32 consecutive output columns; each of the 4 waves owns
//                 TR/4 rows (the paper's per-thread tile, one level up);
//   NB            output-channel width: each wave computes 32*NB output
//                 channels for its pixels, NB MFMA blocks sharing one input
//                 operand (the paper's output-channel vector);
//   VI            input-channel width: the input patch is staged with loads of
//                 VI consecutive channels (the paper's input-channel vector;
//                 Cin % VI == 0).
// The work-group stages the input patch its tile needs (tile plus halo, all
// input channels) and its block of the filter (every tap, 32*NB output
// channels, zero past Cout and past the reduction) in LDS once.  The
// reduction k = (kh*KW + kw)*Cin + ci runs in steps of two on
// v_mfma_f32_32x32x2_f32: lane l supplies the input value of pixel l % 32 at
// k = 2s + l/32 and the filter value of channel l % 32 at the same k, so each
// step is RW*MB*NB MFMAs fed by RW*MB + NB LDS reads.  The reduction length is
// a run-time value (any window and channel count whose patch and filter block
// fit in LDS), e.g. the 7x7 stride-2 first layer of ResNet-50 (K = 147), which
// the fixed-size direct kernel (K <= 32) does not take.
#include <hip/hip_runtime.h>

#include "pk_configs.hpp"

namespace pk {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int DTT_THREADS = 256;
constexpr int DTT_CHUNK = 4;  // k-steps whose LDS reads are issued together
constexpr int DTT_BATCH = 8;  // staging loads per thread issued before their LDS writes

template <int VI>
struct ChanVec;
template <>
struct ChanVec<1> {
    typedef float type;
};
template <>
struct ChanVec<2> {
    typedef float2 type;
};
template <>
struct ChanVec<4> {
    typedef float4 type;
};

// LDS layout, in floats: the filter block (2*KSP rows of 32*NB), the patch
// offsets of every k (two rows of KSP ints: k = 2s and k = 2s + 1), then the
// patch.  KSP = k-steps rounded up to a multiple of DTT_CHUNK (4): the
// offsets of a chunk of steps are read as one 16-byte vector, the filter rows
// past the reduction are zero, and the patch stays 16-byte aligned.
struct TiledLayout {
    int tc, ksp, filt, koff, patch, total;
};

__host__ __device__ inline TiledLayout tiled_layout(int TR, int TC, int CHB, int K, int KH, int KW, int Cin, int sh,
                                                    int sw)
{
    TiledLayout l;
    l.tc = TC;
    const int ks = (K + 1) / 2;
    l.ksp = (ks + DTT_CHUNK - 1) / DTT_CHUNK * DTT_CHUNK;
    l.filt = 2 * l.ksp * CHB;
    l.koff = 2 * l.ksp;
    const int PH = (TR - 1) * sh + KH, PW = (TC - 1) * sw + KW;
    l.patch = PH * PW * Cin;
    l.total = l.filt + l.koff + l.patch;
    return l;
}

// The work-group's filter block and patch-offset table into LDS (once per
// work-group).  The loads go out in batches of DTT_BATCH per thread before
// any of them is written to LDS, so a work-group waits for about one memory
// round trip per batch, not one per element.
template <int NB>
__device__ __forceinline__ void stage_filter(const KernelArgs &p, float *fl, int *koff, const TiledLayout &L, int c0)
{
    constexpr int CHB = 32 * NB;
    const float *f = p.B;
    const int Cin = p.Cin, KW = p.KW, Cout = p.N, K = p.K;
    const int PW = (L.tc - 1) * p.sw + KW;
    const int tid = threadIdx.x;
    // fl[k][c] = f[k][c0 + c], zero past the reduction and Cout
    for (int e0 = tid; e0 < L.filt; e0 += DTT_THREADS * DTT_BATCH) {
        float v[DTT_BATCH];
#pragma unroll
        for (int u = 0; u < DTT_BATCH; ++u) {
            const int e = e0 + u * DTT_THREADS;
            const int k = e / CHB, c = e - k * CHB;
            v[u] = (e < L.filt && k < K && c0 + c < Cout) ? f[(int64_t)k * Cout + c0 + c] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < DTT_BATCH; ++u)
            if (e0 + u * DTT_THREADS < L.filt) fl[e0 + u * DTT_THREADS] = v[u];
    }
    // koff[h * KSP + s]: patch offset of k = 2s + h from a pixel's window origin
    for (int e = tid; e < L.koff; e += DTT_THREADS) {
        const int hh = e / L.ksp, s = e - hh * L.ksp, k = 2 * s + hh;
        int o = 0;
        if (k < K) {
            const int tap = k / Cin, ci = k - tap * Cin;
            const int kh = tap / KW, kw = tap - kh * KW;
            o = (kh * PW + kw) * Cin + ci;
        }
        koff[e] = o;
    }
}

// The MFMA walk over one output tile (its patch and the filter block in LDS)
// and the stores of its results; shared by both forms of the kernel.
template <int TR, int MB, int NB>
__device__ __forceinline__ void tile_mma_store(const KernelArgs &p, const float *fl, const int *koff,
                                               const float *patch, const TiledLayout &L, int n, int ho0, int wo0,
                                               int c0)
{
    constexpr int TC = 32 * MB, CHB = 32 * NB, RW = TR / 4;
    float *y = p.C;
    const int Cin = p.Cin, KW = p.KW, sh = p.sh, sw = p.sw;
    const int Ho = p.Ho, Wo = p.Wo, Cout = p.N, K = p.K;
    const int row_len = ((TC - 1) * sw + KW) * Cin;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, h = lane >> 5;
    // the lane's window origin in the patch for each of its rows and column blocks
    int base[RW][MB];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) base[r][mb] = (wave * RW + r) * sh * row_len + (32 * mb + l32) * sw * Cin;
    const int *kh_off = koff + h * L.ksp;
    const float *fb = fl + h * CHB + l32;  // filter value of k = 2s + h, channel 32j + l32: fb[2s*CHB + 32j]

    f32x16 acc[RW][MB][NB];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int j = 0; j < NB; ++j) acc[r][mb][j] = f32x16{};

    // The k-steps run in chunks of DTT_CHUNK up to KSP (the steps past the
    // reduction multiply zero filter rows by zero inputs).  The LDS reads of
    // chunk c + 1 (its patch offsets, filter values and then input values)
    // are issued around the MFMAs of chunk c, so each MFMA finds its operands
    // in registers.  A lane past the reduction multiplies a zero filter value
    // by a zero input value (an infinite input would otherwise give
    // 0 * inf = NaN; the read is unconditional and the select follows it).
    constexpr int U = DTT_CHUNK;
    int ko[U];
    float av[U][RW][MB], bv[U][NB];
    auto read_offsets = [&](int s0) {
        const int4 o = *reinterpret_cast<const int4 *>(kh_off + s0);
        ko[0] = o.x, ko[1] = o.y, ko[2] = o.z, ko[3] = o.w;
    };
    auto read_filter = [&](int s0) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < NB; ++j) bv[u][j] = fb[2 * (s0 + u) * CHB + 32 * j];
    };
    auto read_inputs = [&]() {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < RW; ++r)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) av[u][r][mb] = patch[base[r][mb] + ko[u]];
    };
    read_offsets(0);
    read_filter(0);
    read_inputs();
    for (int s0 = 0; s0 < L.ksp; s0 += U) {
        float a_cur[U][RW][MB], b_cur[U][NB];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int j = 0; j < NB; ++j) b_cur[u][j] = bv[u][j];
#pragma unroll
            for (int r = 0; r < RW; ++r)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) a_cur[u][r][mb] = av[u][r][mb];
        }
        const bool more = s0 + U < L.ksp;
        if (more) {
            read_offsets(s0 + U);
            read_filter(s0 + U);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool valid = 2 * (s0 + u) + h < K;
#pragma unroll
            for (int r = 0; r < RW; ++r)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const float a = valid ? a_cur[u][r][mb] : 0.f;
#pragma unroll
                    for (int j = 0; j < NB; ++j)
                        acc[r][mb][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b_cur[u][j], acc[r][mb][j], 0, 0, 0);
                }
            if (u == U / 2 - 1 && more) read_inputs();
        }
    }

    // acc[r][mb][j][i]: row wave*RW + r, column 32*mb + 8*(i/4) + 4*h + i%4,
    // channel c0 + 32*j + l32 of the tile
#pragma unroll
    for (int r = 0; r < RW; ++r) {
        const int ho = ho0 + wave * RW + r;
        if (ho >= Ho) continue;
        float *yrow = y + ((int64_t)n * Ho + ho) * Wo * (int64_t)Cout;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int wo = wo0 + 32 * mb + 8 * (i >> 2) + 4 * h + (i & 3);
                if (wo >= Wo) continue;
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    const int co = c0 + 32 * j + l32;
                    if (co < Cout) yrow[(int64_t)wo * Cout + co] = acc[r][mb][j][i];
                }
            }
    }
}

template <int TR, int MB, int NB, int VI>
__global__ void __launch_bounds__(DTT_THREADS) direct_tiled_kernel(KernelArgs p)
{
    extern __shared__ float smem[];
    constexpr int TC = 32 * MB, CHB = 32 * NB;
    typedef typename ChanVec<VI>::type cvec;
    const float *x = p.A;
    const int H = p.H, W = p.W, Cin = p.Cin, KH = p.KH, KW = p.KW, sh = p.sh, sw = p.sw;
    const int Ho = p.Ho, Wo = p.Wo, K = p.K;
    const TiledLayout L = tiled_layout(TR, TC, CHB, K, KH, KW, Cin, sh, sw);
    const int PW = (TC - 1) * sw + KW;
    const int row_len = PW * Cin;
    float *fl = smem;
    int *koff = reinterpret_cast<int *>(smem + L.filt);
    float *patch = smem + L.filt + L.koff;

    const int tiles_w = (Wo + TC - 1) / TC, tiles_h = (Ho + TR - 1) / TR;
    int b = blockIdx.x;
    const int tx = b % tiles_w;
    b /= tiles_w;
    const int ty = b % tiles_h;
    const int n = b / tiles_h;
    const int ho0 = ty * TR, wo0 = tx * TC, c0 = blockIdx.y * CHB;
    const int tid = threadIdx.x;

    stage_filter<NB>(p, fl, koff, L, c0);
    // The patch staging issues its global loads in batches of DTT_BATCH per
    // thread before writing any of them to LDS (one memory round trip per batch).
    // the input patch, VI channels per load, zero outside the image
    const int ih0 = ho0 * sh - p.pt, iw0 = wo0 * sw - p.pl;
    const float *img = x + (int64_t)n * H * W * Cin;
    for (int q0 = tid * VI; q0 < L.patch; q0 += DTT_THREADS * VI * DTT_BATCH) {
        cvec v[DTT_BATCH];
#pragma unroll
        for (int u = 0; u < DTT_BATCH; ++u) {
            const int q = q0 + u * DTT_THREADS * VI;
            const int r = q / row_len;
            const int rem = q - r * row_len;
            const int col = rem / Cin, ci = rem - col * Cin;
            const int ih = ih0 + r, iw = iw0 + col;
            if (q < L.patch && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W)
                v[u] = *reinterpret_cast<const cvec *>(img + ((int64_t)ih * W + iw) * Cin + ci);
            else
                v[u] = cvec{};
        }
#pragma unroll
        for (int u = 0; u < DTT_BATCH; ++u) {
            const int q = q0 + u * DTT_THREADS * VI;
            if (q < L.patch) *reinterpret_cast<cvec *>(patch + q) = v[u];
        }
    }
    __syncthreads();

    tile_mma_store<TR, MB, NB>(p, fl, koff, patch, L, n, ho0, wo0, c0);
}

// Persistent form: the grid is the work-groups the CUs hold at once; each
// serves one channel block and walks a contiguous run of its output tiles.
// The filter block and the offset table are staged once per work-group, and
// the input patch is double-buffered: the patch of tile t+1 is copied
// straight from global memory into the other LDS buffer (buffer_load ...
// lds, 4 bytes a lane, elements outside the image read as zero through an
// offset past the buffer's range) while tile t is multiplied, so the copy's
// latency hides under the MFMAs.  A work-group walks the patch elements it
// copies incrementally (row, column, channel carried from one copy to the
// next) rather than dividing for each.
template <int TR, int MB, int NB>
__global__ void __launch_bounds__(DTT_THREADS) direct_tiled_persistent_kernel(KernelArgs p)
{
    extern __shared__ float smem[];
    constexpr int TC = 32 * MB, CHB = 32 * NB;
    const float *x = p.A;
    const int H = p.H, W = p.W, Cin = p.Cin, KW = p.KW, sh = p.sh, sw = p.sw;
    const int Ho = p.Ho, Wo = p.Wo, Cout = p.N;
    const TiledLayout L = tiled_layout(TR, TC, CHB, p.K, p.KH, KW, Cin, sh, sw);
    const int PW = (TC - 1) * sw + KW;
    const int pstr = (L.patch + 255) / 256 * 256;  // a patch buffer: whole 256-float copy passes
    float *fl = smem;
    int *koff = reinterpret_cast<int *>(smem + L.filt);
    float *pbuf = smem + L.filt + L.koff;

    const int tiles_w = (Wo + TC - 1) / TC, tiles_h = (Ho + TR - 1) / TR;
    const int per_img = tiles_w * tiles_h, per_cb = per_img * p.batch;
    const int CB = (Cout + CHB - 1) / CHB;
    const int cb = blockIdx.x % CB;
    const int g = blockIdx.x / CB, G = gridDim.x / CB;  // the launch makes gridDim.x a multiple of CB
    const int t0 = (int)((int64_t)g * per_cb / G);
    const int t1 = (int)((int64_t)(g + 1) * per_cb / G);
    if (t0 >= t1) return;  // uniform over the work-group, before any barrier
    const int c0 = cb * CHB;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

    // copy the patch of tile t into dst: this lane's elements are
    // q = (4i + wave) * 64 + lane, i = 0 .. pstr/256 - 1
    const int dcol = 256 / Cin, dci = 256 - dcol * Cin;
    const int q_first = wave * 64 + lane;
    const int row_len = PW * Cin;
    const int r_first = q_first / row_len;
    const int rem_first = q_first - r_first * row_len;
    const int col_first = rem_first / Cin, ci_first = rem_first - col_first * Cin;
    auto copy_patch = [&](int t, float *dst) {
        const int n = t / per_img, rt = t - n * per_img;
        const int ty = rt / tiles_w, tx = rt - ty * tiles_w;
        const int ih0 = ty * TR * sh - p.pt, iw0 = tx * TC * sw - p.pl;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(x + (int64_t)n * H * W * Cin), 0, 0x7fffffff, 0x00020000);
        int q = q_first, r = r_first, col = col_first, ci = ci_first;
        for (int i = 0; i < pstr / 256; ++i) {
            const int ih = ih0 + r, iw = iw0 + col;
            const bool ok = q < L.patch && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W;
            const int off = ok ? ((ih * W + iw) * Cin + ci) * 4 : (int)0x80000000;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs, (__attribute__((address_space(3))) void *)(dst + (4 * i + wave) * 64), 4, off, 0, 0, 0);
            q += 256;
            ci += dci;
            col += dcol;
            if (ci >= Cin) {
                ci -= Cin;
                ++col;
            }
            while (col >= PW) {
                col -= PW;
                ++r;
            }
        }
    };

    copy_patch(t0, pbuf);
    stage_filter<NB>(p, fl, koff, L, c0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    for (int t = t0; t < t1; ++t) {
        const int cur = (t - t0) & 1;
        // the other buffer was last read in the previous tile, before the barrier
        if (t + 1 < t1) copy_patch(t + 1, pbuf + (cur ^ 1) * pstr);
        const int n = t / per_img, rt = t - n * per_img;
        const int ty = rt / tiles_w, tx = rt - ty * tiles_w;
        tile_mma_store<TR, MB, NB>(p, fl, koff, pbuf + cur * pstr, L, n, ty * TR, tx * TC, c0);
        // this wave's copies have landed (and its stores drained); the barrier
        // makes every wave's copies visible and ends the reads of this buffer
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }
}

template <int TR, int MB, int NB>
hipError_t launch_direct_tiled_persistent(const KernelArgs &a, hipStream_t stream)
{
    constexpr int TC = 32 * MB, CHB = 32 * NB;
    const TiledLayout L = tiled_layout(TR, TC, CHB, a.K, a.KH, a.KW, a.Cin, a.sh, a.sw);
    const size_t lds = (size_t)(L.filt + L.koff + 2 * ((L.patch + 255) / 256 * 256)) * sizeof(float);
    if (lds > (size_t)kDirectTiledMaxLds) return hipErrorInvalidValue;
    const int64_t per_cb = (int64_t)((a.Ho + TR - 1) / TR) * ((a.Wo + TC - 1) / TC) * a.batch;
    const int64_t cbs = (a.N + CHB - 1) / CHB;
    if (per_cb >= ((int64_t)1 << 31) || cbs > 65535) return hipErrorInvalidValue;
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, direct_tiled_persistent_kernel<TR, MB, NB>,
                                                     DTT_THREADS, lds) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    int64_t groups = ((int64_t)per_cu * device_cu_count()) / cbs;  // work-groups per channel block
    if (groups < 1) groups = 1;
    if (groups > per_cb) groups = per_cb;
    if (groups * cbs >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    hipLaunchKernelGGL((direct_tiled_persistent_kernel<TR, MB, NB>), dim3((unsigned)(groups * cbs)),
                       dim3(DTT_THREADS), lds, stream, a);
    return hipGetLastError();
}

template <int TR, int MB, int NB, int VI>
hipError_t launch_direct_tiled(const KernelArgs &a, hipStream_t stream)
{
    constexpr int TC = 32 * MB, CHB = 32 * NB;
    const TiledLayout L = tiled_layout(TR, TC, CHB, a.K, a.KH, a.KW, a.Cin, a.sh, a.sw);
    const size_t lds = (size_t)L.total * sizeof(float);
    if (lds > (size_t)kDirectTiledMaxLds || a.Cin % VI != 0) return hipErrorInvalidValue;
    const int64_t tiles = (int64_t)((a.Ho + TR - 1) / TR) * ((a.Wo + TC - 1) / TC) * a.batch;
    const int64_t cbs = (a.N + CHB - 1) / CHB;
    if (tiles >= ((int64_t)1 << 31) || cbs > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL((direct_tiled_kernel<TR, MB, NB, VI>), dim3((unsigned)tiles, (unsigned)cbs),
                       dim3(DTT_THREADS), lds, stream, a);
    return hipGetLastError();
}

}  // namespace

size_t direct_tiled_lds_bytes(const Config *c, int64_t KH, int64_t KW, int64_t Cin, int64_t sh, int64_t sw)
{
    const int64_t K = KH * KW * Cin;
    if (!c || c->tile_rows < 1 || K < 1 || K > (1 << 20) || KH > 4096 || KW > 4096 || sh > 4096 || sw > 4096)
        return (size_t)-1;
    const int TR = c->tile_rows, TC = c->bm / c->tile_rows;
    // in 64-bit: the same arithmetic as tiled_layout, which the kernel runs in 32 bits once this bound holds
    const int64_t ks = (K + 1) / 2, ksp = (ks + DTT_CHUNK - 1) / DTT_CHUNK * DTT_CHUNK;
    const int64_t PH = (TR - 1) * sh + KH, PW = (TC - 1) * sw + KW;
    const int64_t patch = PH * PW * Cin;
    const int64_t floats = 2 * ksp * c->bn + 2 * ksp + (c->persistent ? 2 * ((patch + 255) / 256 * 256) : patch);
    return (size_t)floats * sizeof(float);
}

// name: direct_<rows>x<columns>x<channels>_v<input-channel width>
#define PK_DTT(TR, TC, CHB, VI)                                                                                \
    {"direct_" #TR "x" #TC "x" #CHB "_v" #VI, KIND_DIRECT, TR * TC, CHB, 2, 4, 1, 0, 0, VI, 1, 1, 0,          \
     kDirectTiledMaxLds, &launch_direct_tiled<TR, TC / 32, CHB / 32, VI>, 0, 0, nullptr, 0, 1, 0, TR}

// persistent form: direct_<rows>x<columns>x<channels>_tp (4-byte patch copies)
#define PK_DTP(TR, TC, CHB)                                                                                  \
    {"direct_" #TR "x" #TC "x" #CHB "_tp", KIND_DIRECT, TR * TC, CHB, 2, 4, 1, 0, 0, 1, 1, 1, 1,            \
     kDirectTiledMaxLds, &launch_direct_tiled_persistent<TR, TC / 32, CHB / 32>, 0, 0, nullptr, 0, 1, 0, TR}

const Config *configs_direct_tiled(int *count)
{
    // output tiles of 4, 8, 16 rows x 32, 64 columns; 32 or 64 output
    // channels; input channels loaded 1 or 4 at a time (at most 8 MFMA
    // blocks of accumulators per wave)
    static const Config kTable[] = {
        PK_DTT(4, 32, 32, 1), PK_DTT(4, 32, 64, 1), PK_DTT(4, 64, 32, 1), PK_DTT(4, 64, 64, 1),
        PK_DTT(8, 32, 32, 1), PK_DTT(8, 32, 64, 1), PK_DTT(8, 64, 32, 1), PK_DTT(8, 64, 64, 1),
        PK_DTT(16, 32, 32, 1), PK_DTT(16, 32, 64, 1), PK_DTT(16, 64, 32, 1),
        PK_DTT(4, 32, 32, 4), PK_DTT(4, 32, 64, 4), PK_DTT(4, 64, 32, 4), PK_DTT(4, 64, 64, 4),
        PK_DTT(8, 32, 32, 4), PK_DTT(8, 32, 64, 4), PK_DTT(8, 64, 32, 4), PK_DTT(8, 64, 64, 4),
        PK_DTT(16, 32, 32, 4), PK_DTT(16, 32, 64, 4), PK_DTT(16, 64, 32, 4),
        PK_DTP(4, 32, 32), PK_DTP(4, 32, 64), PK_DTP(4, 64, 32), PK_DTP(4, 64, 64),
        PK_DTP(8, 32, 32), PK_DTP(8, 32, 64), PK_DTP(8, 64, 32), PK_DTP(8, 64, 64),
        PK_DTP(16, 32, 32), PK_DTP(16, 32, 64), PK_DTP(16, 64, 32),
    };
    *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
    return kTable;
}

}  // namespace pk
