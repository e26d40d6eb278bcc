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

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

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

// Persistent form: a grid of the work-groups the CUs hold at once.  The
// layer is bound by writing its output, so the point is to keep those writes
// streaming under the MFMAs:
//   - work-group b serves channel block b % CB only (CB = ceil(Cout / 64))
//     and walks a contiguous run of that block's pixel tiles; its filter
//     values (registers) and each lane's patch offsets are set up once;
//   - the input patch is staged in LDS (three stages); the patch of tile t+2
//     is fetched into registers before tile t's output stores are issued.
//     The vector-memory counter orders loads and stores together, so the
//     wait for a patch never includes the stores issued after it;
//   - each wave computes its two output rows one after the other, so the
//     first row's stores drain while the second row multiplies, and the
//     second row's while the next tile's first row does;
//   - the k-step count KS is a compile-time constant: the MFMA sequence is
//     one straight block, so no wait on the stores is placed inside it.
// Each thread fetches E patch elements (E * 256 >= the patch size).
constexpr int DP_MAX_PATCH = 2048;  // floats of the largest patch this form stages

// OCC: waves per SIMD the registers are allotted for (3 fits every form but
// the largest patch with the longest reduction without spilling).
// V4: 16-byte output stores (Cout % 4 == 0 and a 16-byte aligned output):
// each wave passes its row of results through its own LDS buffer, so that a
// lane stores 4 consecutive channels of one pixel and a store instruction
// writes 4 whole 256-byte pixel rows.  A wave can have 63 memory operations
// in flight, so 16-byte stores keep four times the bytes in flight that
// 4-byte stores do.
constexpr int DP_LDP = DT_CH + 4;  // floats per pixel in a wave's row buffer (rows stay 16-byte aligned)

template <int E, int KS, bool V4, int OCC = (E == 8 && KS == 16) ? 2 : 3>
__global__ void __launch_bounds__(64 * DT_WAVES) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
direct_conv_persistent_kernel(KernelArgs p)
{
    extern __shared__ float smem[];  // three stages of the patch, then (V4) the waves' row buffers
    constexpr int NT = 64 * DT_WAVES;
    const float *x = p.A;
    const float *f = p.B;
    float *y = p.C;
    const int H = p.H, W = p.W, Cin = p.Cin, KW = p.KW, sh = p.sh, sw = p.sw;
    const int Ho = p.Ho, Wo = p.Wo, Cout = p.N, K = p.K;
    const int PH = (DT_ROWS - 1) * sh + p.KH;
    const int PW = (DT_COLS - 1) * sw + KW;
    const int row_len = PW * Cin;
    const int PF = PH * row_len;
    constexpr int STAGE = E * NT;  // floats per LDS stage: every thread writes all E of its slots

    const int tiles_w = (Wo + DT_COLS - 1) / DT_COLS;
    const int per_img = ((Ho + DT_ROWS - 1) / DT_ROWS) * tiles_w;
    const int per_cb = per_img * p.batch;
    const int CB = (Cout + DT_CH - 1) / DT_CH;
    const int cb = blockIdx.x % CB;
    const int g = blockIdx.x / CB, G = gridDim.x / CB;  // the launch makes gridDim.x a multiple of CB
    const int t0 = (int)((int64_t)g * per_cb / G);
    const int t1 = (int)((int64_t)(g + 1) * per_cb / G);
    if (t0 >= t1) return;  // uniform over the work-group, before any barrier
    const int c0 = cb * DT_CH;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wave_s = __builtin_amdgcn_readfirstlane(wave);  // the same value, known uniform
    const int l32 = lane & 31, h = lane >> 5;
    const unsigned y_lane = 4u * (unsigned)h * (unsigned)Cout + (unsigned)l32;  // lane offset in a wave block

    // this thread's patch elements e = tid + i*NT: (row, column) in the patch
    // and the offset from the patch origin in the image (tile independent)
    int rc[E], rel[E];
#pragma unroll
    for (int i = 0; i < E; ++i) {
        const int e = tid + i * NT;
        if (e < PF) {
            const int r = e / row_len;
            const int q = e - r * row_len;
            const int col = q / Cin, ci = q - col * Cin;
            rc[i] = (r << 16) | col;
            rel[i] = (r * W + col) * Cin + ci;
        } else {
            rc[i] = -1;
            rel[i] = 0;
        }
    }
    // per k-step s this lane supplies k = 2s + h: its offset in the patch and
    // the filter values of its two output channels (0 past the window)
    int off[KS];
    float bv[2][KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int k = 2 * s + h;
        int o = 0;
        float b0 = 0.f, b1 = 0.f;
        if (k < K) {
            const int tap = k / Cin, ci = k - tap * Cin;
            const int kh = tap / KW, kw = tap - kh * KW;
            o = (kh * PW + kw) * Cin + ci;
            const int co0 = c0 + l32, co1 = c0 + 32 + l32;
            b0 = co0 < Cout ? f[(int64_t)k * Cout + co0] : 0.f;
            b1 = co1 < Cout ? f[(int64_t)k * Cout + co1] : 0.f;
        }
        off[s] = o;
        bv[0][s] = b0;
        bv[1][s] = b1;
    }

    struct Tile {
        int n, ho0, wo0;
    };
    auto decode = [&](int t) {
        Tile d;
        d.n = t / per_img;
        const int rem = t - d.n * per_img;
        const int ty = rem / tiles_w;
        d.ho0 = ty * DT_ROWS;
        d.wo0 = (rem - ty * tiles_w) * DT_COLS;
        return d;
    };
    // Every load and LDS store below is unconditional (out-of-image and
    // past-the-patch slots load the image's first element, and bit i of
    // `inside` turns slot i into 0 when it is stored to LDS): with no branch
    // around them, and nothing computed from a loaded value before that LDS
    // store, the compiler's wait before it counts only the loads, not the
    // output stores issued after them.
    float v[E];
    unsigned inside = 0;
    auto load_patch = [&](const Tile &d) {
        const int ih0 = d.ho0 * sh - p.pt, iw0 = d.wo0 * sw - p.pl;
        const float *img = x + (int64_t)d.n * H * W * Cin;
        const int64_t origin = ((int64_t)ih0 * W + iw0) * Cin;
        inside = 0;
#pragma unroll
        for (int i = 0; i < E; ++i) {
            const int ih = ih0 + (rc[i] >> 16), iw = iw0 + (rc[i] & 0xffff);
            const bool ok = rc[i] >= 0 && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W;
            v[i] = img[ok ? origin + rel[i] : 0];
            inside |= (unsigned)ok << i;
        }
    };
    auto write_patch = [&](float *stage) {
#pragma unroll
        for (int i = 0; i < E; ++i) stage[tid + i * NT] = ((inside >> i) & 1u) ? v[i] : 0.f;
    };

    Tile cur = decode(t0);
    load_patch(cur);
    write_patch(smem);
    if (t0 + 1 < t1) load_patch(decode(t0 + 1));
    // nothing of the set-up stays in flight into the loop: the loop then only
    // ever waits for the patch loads it issued itself, which precede its stores
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // One output row of the tile for this wave: 32 pixels x 64 channels.
    auto mfma_row = [&](const float *patch, int r, f32x16 (&acc)[2]) {
        const f32x16 zero = {};
        const int prow = (wave * DT_ROWS_PER_WAVE + r) * sh;  // patch row of tap kh = 0
        int lane_off = prow * row_len + l32 * sw * Cin;
        // the offsets lane_off + off[s] are the same for every tile; without
        // this the compiler keeps all of them in registers across the tile loop
        asm volatile("" : "+v"(lane_off));
        const float *base = patch + lane_off;
        // every read is unconditional (off[s] is in the patch for every k): a
        // read under a condition becomes a masked read that the MFMAs wait for
        // one at a time
        float av[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) av[s] = base[off[s]];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            // past the window the filter value is 0; the input value must be
            // 0 too (an infinite input would otherwise give 0 * inf = NaN)
            const float a = 2 * s + h < K ? av[s] : 0.f;
            // the first step starts from zero (an operand, not 32 register moves)
            acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv[0][s], s == 0 ? zero : acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv[1][s], s == 0 ? zero : acc[1], 0, 0, 0);
        }
    };
    // acc[j][i]: pixel column 8*(i/4) + 4*h + i%4 of row r, channel c0 + 32*j + l32.
    // Buffer stores from the row's base (column wo0, channel c0): every store
    // instruction issues, an element outside the output taking an offset past
    // the buffer's range, which the hardware drops.  So the memory operations
    // issued after each patch load are the same on every path, and the wait
    // before its LDS store never covers these stores.
    float *rowbuf = smem + 3 * STAGE + wave * (DT_COLS * DP_LDP);  // V4 only
    auto store_row = [&](const Tile &d, int r, const f32x16 (&acc)[2]) {
        const int ho = d.ho0 + wave_s * DT_ROWS_PER_WAVE + r;
        const bool rows_ok = ho < Ho;
        const bool interior = rows_ok && d.wo0 + DT_COLS <= Wo && c0 + DT_CH <= Cout;
        float *yrow = y + (((int64_t)d.n * Ho + ho) * Wo + d.wo0) * Cout + c0;
        const __amdgpu_buffer_rsrc_t yres = __builtin_amdgcn_make_buffer_rsrc(yrow, (short)0, 0x7fffffff, 0x00020000);
        if constexpr (V4) {
            // results to the wave's buffer as [pixel][channel] (LDS operations of
            // one wave run in order, so the reads below see these writes and the
            // next row's writes follow these reads)
#pragma unroll
            for (int i = 0; i < 16; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    rowbuf[(8 * (i >> 2) + 4 * h + (i & 3)) * DP_LDP + 32 * j + l32] = acc[j][i];
            // lane q: pixel 4m + q/16, channels 4*(q%16) .. +3
            const int px = lane >> 4, ch = (lane & 15) * 4;
#pragma unroll
            for (int m = 0; m < DT_COLS / 4; ++m) {
                const int pm = 4 * m + px;
                const f32x4 v = *reinterpret_cast<const f32x4 *>(rowbuf + pm * DP_LDP + ch);
                const bool ok = interior || (rows_ok && d.wo0 + pm < Wo && c0 + ch < Cout);
                const unsigned e = (unsigned)(pm * Cout + ch);
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), yres, ok ? 4u * e : 0x80000000u,
                                                       0, 0);
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < 16; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int dw = 8 * (i >> 2) + (i & 3);
                const bool ok = interior || (rows_ok && d.wo0 + 4 * h + dw < Wo && c0 + 32 * j + l32 < Cout);
                const unsigned e = (unsigned)(dw * Cout + 32 * j) + y_lane;
                // the builtin's data operand is a 32-bit integer: pass the float's
                // bits (copied out of the vector first: this compiler's bit_cast of a
                // vector element reads element 0)
                const float val = acc[j][i];
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, val), yres,
                                                      ok ? 4u * e : 0x80000000u, 0, 0);
            }
    };

    // Three patch stages: tile t reads stage t % 3.  The patch of tile t+1 is
    // written after the first row of tile t is computed, into the stage tile
    // t-2 read; every wave finished tile t-2 before it reached the previous
    // iteration's barrier.  Row 0's stores drain while row 1 is multiplied.
    f32x16 acc[2];
    int st = 0;
    for (int t = t0;; ++t) {
        const float *patch = smem + st * STAGE;
        const int st1 = st == 2 ? 0 : st + 1;
        mfma_row(patch, 0, acc);
        const bool more = t + 1 < t1;
        if (more) write_patch(smem + st1 * STAGE);  // the patch of tile t+1
        __syncthreads();
        const Tile done = cur;
        if (more) {
            // the patch of tile t+2, fetched before the stores of tile t
            if (t + 2 < t1) load_patch(decode(t + 2));
            cur = decode(t + 1);
        }
        store_row(done, 0, acc);
        mfma_row(patch, 1, acc);
        store_row(done, 1, acc);
        if (!more) break;
        st = st1;
    }
}

int64_t direct_tiles(const KernelArgs &a)
{
    return (int64_t)((a.Ho + DT_ROWS - 1) / DT_ROWS) * ((a.Wo + DT_COLS - 1) / DT_COLS) * a.batch *
           ((a.N + DT_CH - 1) / DT_CH);
}

// three patch stages of E floats per thread, then (V4) a row buffer per wave
template <int E, bool V4>
constexpr size_t direct_persistent_lds()
{
    return (3 * (size_t)E * 64 * DT_WAVES + (V4 ? (size_t)DT_WAVES * DT_COLS * DP_LDP : 0)) * sizeof(float);
}

template <int E, int KS, bool V4>
hipError_t launch_direct_persistent_k(const KernelArgs &a, int64_t pf, hipStream_t stream)
{
    static int per_cu = 0;  // resident work-groups per CU (the same on every MI355X)
    if (per_cu == 0) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, direct_conv_persistent_kernel<E, KS, V4>, 64 * DT_WAVES,
                                                         direct_persistent_lds<E, V4>()) != hipSuccess ||
            n < 1)
            n = 1;
        per_cu = n;
    }
    // CB channel blocks, each served by the same number of work-groups
    const int64_t cbs = (a.N + DT_CH - 1) / DT_CH;
    const int64_t per_cb = direct_tiles(a) / cbs;
    int64_t groups = ((int64_t)per_cu * device_cu_count()) / cbs;
    if (groups < 1) groups = 1;
    if (groups > per_cb) groups = per_cb;
    (void)pf;
    const auto kernel = direct_conv_persistent_kernel<E, KS, V4>;
    const size_t lds = direct_persistent_lds<E, V4>();
    hipLaunchKernelGGL(kernel, dim3((unsigned)(groups * cbs)), dim3(64 * DT_WAVES), lds, stream, a);
    return hipGetLastError();
}

template <int E, bool V4>
hipError_t launch_direct_persistent_v(const KernelArgs &a, int64_t pf, hipStream_t stream)
{
    const int ks = (a.K + 1) / 2;  // k-steps of two
    if (ks <= 4) return launch_direct_persistent_k<E, 4, V4>(a, pf, stream);
    if (ks <= 8) return launch_direct_persistent_k<E, 8, V4>(a, pf, stream);
    if (ks <= 14) return launch_direct_persistent_k<E, 14, V4>(a, pf, stream);
    return launch_direct_persistent_k<E, DT_KMAX / 2, V4>(a, pf, stream);
}

template <int E>
hipError_t launch_direct_persistent_e(const KernelArgs &a, int64_t pf, hipStream_t stream)
{
    if (a.N % 4 == 0 && ((uintptr_t)a.C & 15) == 0) return launch_direct_persistent_v<E, true>(a, pf, stream);
    return launch_direct_persistent_v<E, false>(a, pf, stream);
}

hipError_t launch_direct_persistent(const KernelArgs &a, hipStream_t stream)
{
    const int64_t pf = direct_patch_floats(a.KH, a.KW, a.Cin, a.sh, a.sw);
    if (pf > DP_MAX_PATCH || a.K > DT_KMAX || direct_tiles(a) >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    if (pf <= 4 * 64 * DT_WAVES) return launch_direct_persistent_e<4>(a, pf, stream);
    return launch_direct_persistent_e<8>(a, pf, stream);
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

bool direct_conv_fits(const Config *c, int64_t W, int64_t Wo, int64_t Cout, int64_t KH, int64_t KW, int64_t Cin,
                      int64_t sh, int64_t sw)
{
    if (c && c->tile_rows > 0) {
        // the tiled instances: patch and filter block within their LDS, whole
        // input-channel vectors, grid dimensions in range (the batch is the
        // caller's check); patch offsets are 32-bit, image and output offsets 64-bit
        const size_t lds = direct_tiled_lds_bytes(c, KH, KW, Cin, sh, sw);
        const int64_t tc = c->bm / c->tile_rows;
        return lds <= (size_t)kDirectTiledMaxLds && Cin % c->vec_a == 0 && (Cout + c->bn - 1) / c->bn <= 65535 &&
               (Wo + tc - 1) / tc < ((int64_t)1 << 20) && W < ((int64_t)1 << 30);
    }
    if (KH > DT_KMAX || KW > DT_KMAX || Cin > DT_KMAX || sh > 64 || sw > 64) return false;
    if (KH * KW * Cin > DT_KMAX) return false;
    const int64_t pf = direct_patch_floats(KH, KW, Cin, sh, sw);
    if (!(c && c->persistent)) return pf <= DT_LDS_FLOATS;
    // the persistent form keeps patch offsets in 32 bits (a band of
    // patch-height input rows) and output offsets from a wave's first output
    // (two rows plus a tile) below 2^31 bytes
    const int64_t band = ((DT_ROWS - 1) * sh + KH) * (W + (DT_COLS - 1) * sw + KW) * Cin;
    const int64_t out_span = (DT_ROWS_PER_WAVE * Wo + DT_COLS) * (Cout + DT_CH) * (int64_t)sizeof(float);
    return pf <= DP_MAX_PATCH && band < ((int64_t)1 << 31) && out_span < ((int64_t)1 << 31);
}

const Config *configs_direct(int *count)
{
    static const Config kTable[] = {
        {"direct_8x32x64_k32", KIND_DIRECT, DT_ROWS * DT_COLS, DT_CH, DT_KMAX, DT_WAVES, 1, 0, 0, 1, 1, 1, 0,
         (int)(DT_LDS_FLOATS * sizeof(float)), &launch_direct},
        {"direct_8x32x64_k32_p", KIND_DIRECT, DT_ROWS * DT_COLS, DT_CH, DT_KMAX, DT_WAVES, 1, 0, 0, 1, 1, 1, 1,
         (int)(2 * DP_MAX_PATCH * sizeof(float)), &launch_direct_persistent},
    };
    *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
    return kTable;
}

}  // namespace pk
