// pk_kernel.hpp -- the parameterized fp32 contraction for gfx950.
//
// One template computes a BM x BN block of C = alpha * op(A) * op(B) (+ beta C)
// per work-group, the panel-times-panel decomposition of the blocked GEMM in
// Section 3.1: C is cut into blocks, each block C_ij is the product of the row
// panel A_i and the column panel B_j, and the K dimension is walked in blocks
// of BK (the blocked identity over a partition of K).  The levels of the
// paper's memory hierarchy map onto CDNA4 as
//   global (HBM / L2)  ->  LDS (the paper's local memory), double buffered
//                      ->  VGPRs (private memory)  ->  fp32 MFMA accumulators.
//
// Tile parameters (compile time, as the paper's template parameters):
//   BM, BN      work-group tile of C
//   BK          K-block depth staged in LDS per step
//   WAVES_M/N   wave grid; each 64-lane wave owns a (BM/WAVES_M) x (BN/WAVES_N)
//               sub-tile built from 32 x 32 MFMA blocks
//   VA, VB      elements per global load (1 or 4: 4 = 16-byte loads)
//   AMODE       how op(A) is read: dense k-contiguous ('N'), dense
//               m-contiguous ('T'), or gathered from an NHWC image (implicit
//               GEMM convolution, k = (kh*KW + kw)*Cin + ci)
//   B_KCONTIG   op(B) read from N x K storage ('T') instead of K x N ('N')
//
// Matrix instruction: v_mfma_f32_32x32x2_f32 (full fp32 products and sums).
// For one instruction, lane l supplies A(row l%32, k-slot l/32) and
// B(k-slot l/32, col l%32) and holds 16 results: C(8*(r/4) + 4*(l/32) + r%4,
// l%32) for r = 0..15.  The two k-slots of the instruction are given the
// k-indices h*BK/2 + s (h = l/32, s = 0..BK/2-1) of the current K-block, so
// each lane walks BK/2 consecutive k of its own row: a permutation of the
// K-block that the sum does not see, but one that lets an A row stored
// k-contiguous in LDS be read with 16-byte LDS loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "pk_args.hpp"
#include "pk_partition.hpp"

namespace pk {

// f(std::integral_constant<int, I>{}) for I = 0 .. N-1: a loop whose index
// is a compile-time constant in the body
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>)
{
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F &&f)
{
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

enum AMode { A_KCONTIG = 0, A_MCONTIG = 1, A_CONV = 2 };


// Tile (tm, tn) of logical tile index t, in column strips of group_m tile-rows.
__device__ __forceinline__ void tile_of(const KernelArgs &p, int t, int &tm, int &tn)
{
    tile_of_ints(p.tiles_m, p.tiles_n, p.group_m, t, tm, tn);
}

// Maps the linear work-group id to a C tile.  Work-groups are handed to the
// 8 XCDs round-robin (id % 8); renumbering them so that each XCD receives a
// contiguous run of logical tiles keeps the A and B panels those tiles share
// in that XCD's own L2.  Logical tiles are then ordered in column strips of
// group_m tile-rows so that concurrently running tiles reuse panels.
__device__ __forceinline__ void tile_coords(const KernelArgs &p, int &tm, int &tn)
{
    tile_of(p, xcd_tile(blockIdx.x, p.tiles_m * p.tiles_n, p.xcds), tm, tn);
}

template <int V>
struct Vec;
template <>
struct Vec<1> {
    typedef float T;
    static __device__ __forceinline__ T zero() { return 0.f; }
    static __device__ __forceinline__ T load(const float *p) { return *p; }
    static __device__ __forceinline__ void store(float *p, T v) { *p = v; }
};
template <>
struct Vec<2> {
    typedef f32x2 T;
    static __device__ __forceinline__ T zero() { return f32x2{0.f, 0.f}; }
    static __device__ __forceinline__ T load(const float *p) { return *reinterpret_cast<const f32x2 *>(p); }
    static __device__ __forceinline__ void store(float *p, T v) { *reinterpret_cast<f32x2 *>(p) = v; }
};
template <>
struct Vec<4> {
    typedef f32x4 T;
    static __device__ __forceinline__ T zero() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
    static __device__ __forceinline__ T load(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }
    static __device__ __forceinline__ void store(float *p, T v) { *reinterpret_cast<f32x4 *>(p) = v; }
};

// ----------------------------------------------------------------------------
// Tile loaders: global -> registers (issued one K-block ahead) -> LDS.
// A loader stages ROWS x COLS of a row-major global panel whose COLS are
// contiguous.  Thread t owns chunks c = t + i*NT (VEC elements each); since
// NT is a multiple of the chunks per row, every chunk of a thread sits in the
// same column, and its row pointer is fixed for the whole K loop.
// ----------------------------------------------------------------------------

// Dense operand, k along the contiguous columns (A 'N', B 'T').
// Rows are m (or n); the panel advances along its columns by BK per step.
template <int ROWS, int BK, int VEC, int NT>
struct KContigLoader {
    static constexpr int CPR = BK / VEC;
    static constexpr int LOADS = ROWS * BK / (VEC * NT);
    static_assert(NT % CPR == 0, "threads must cover whole rows");
    static_assert(LOADS >= 1 && ROWS * BK % (VEC * NT) == 0, "tile not divisible");
    typedef typename Vec<VEC>::T VT;
    const float *ptr[LOADS];
    bool row_ok[LOADS];
    int col;  // k offset of this thread's chunks inside the K-block

    __device__ __forceinline__ void init(const float *base, int64_t ld, int row0, int rows, int kbeg, int tid)
    {
        col = (tid % CPR) * VEC;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int r = (tid + i * NT) / CPR;
            row_ok[i] = row0 + r < rows;
            const int rr = row_ok[i] ? row0 + r : 0;
            ptr[i] = base + (int64_t)rr * ld + (int64_t)kbeg * BK + col;
        }
    }
    __device__ __forceinline__ void load(VT *v, int k0, int K) const
    {
        const bool k_ok = k0 + col < K;  // VEC divides K whenever VEC > 1
#pragma unroll
        for (int i = 0; i < LOADS; ++i)
            v[i] = (row_ok[i] && k_ok) ? Vec<VEC>::load(ptr[i]) : Vec<VEC>::zero();
    }
    // the thread's offsets were fixed by init
    __device__ __forceinline__ void load(VT *v, int k0, int K, int) const { load(v, k0, K); }
    __device__ __forceinline__ void advance()
    {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) ptr[i] += BK;
    }
    __device__ __forceinline__ void advance_by(int blocks)
    {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) ptr[i] += (int64_t)BK * blocks;
    }
    // LDS tile [ROWS][BK + PAD]
    template <int LD>
    __device__ __forceinline__ void store(float *lds, const VT *v, int tid) const
    {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int r = (tid + i * NT) / CPR;
            Vec<VEC>::store(lds + r * LD + col, v[i]);
        }
    }
};

// Dense operand whose m (or n) runs along the contiguous columns (A 'T', B 'N').
// Rows are k; the panel advances by BK rows per step.
template <int COLS, int BK, int VEC, int NT>
struct MContigLoader {
    static constexpr int CPR = COLS / VEC;
    static constexpr int LOADS = COLS * BK / (VEC * NT);
    static_assert(NT % CPR == 0 || CPR % NT == 0, "thread/column mapping");
    static_assert(LOADS >= 1 && COLS * BK % (VEC * NT) == 0, "tile not divisible");
    typedef typename Vec<VEC>::T VT;
    const float *ptr;
    int64_t ld;
    bool col_ok[LOADS];

    __device__ __forceinline__ void init(const float *base, int64_t ld_, int col0, int cols, int kbeg, int tid)
    {
        ld = ld_;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int c = ((tid + i * NT) % CPR) * VEC;
            col_ok[i] = col0 + c < cols;  // VEC divides cols whenever VEC > 1
        }
        ptr = base + (int64_t)kbeg * BK * ld + col0;
    }
    // tid is the thread's index within the NT threads that share the panel
    __device__ __forceinline__ void load(VT *v, int k0, int K, int tid) const
    {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int c = (tid + i * NT) % CPR * VEC;
            const int r = (tid + i * NT) / CPR;
            const bool ok = col_ok[i] && (k0 + r < K);
            v[i] = ok ? Vec<VEC>::load(ptr + (int64_t)r * ld + c) : Vec<VEC>::zero();
        }
    }
    __device__ __forceinline__ void load(VT *v, int k0, int K) const { load(v, k0, K, (int)threadIdx.x); }
    __device__ __forceinline__ void advance() { ptr += (int64_t)BK * ld; }
    __device__ __forceinline__ void advance_by(int blocks) { ptr += (int64_t)BK * ld * blocks; }
    // LDS tile [BK][COLS + PAD]
    template <int LD>
    __device__ __forceinline__ void store(float *lds, const VT *v, int tid) const
    {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int c = (tid + i * NT) % CPR * VEC;
            const int r = (tid + i * NT) / CPR;
            Vec<VEC>::store(lds + r * LD + c, v[i]);
        }
    }
};

// Implicit-GEMM gather of A from an NHWC image: row m is the output pixel
// (n, ho, wo), column k is the filter tap (kh, kw) and input channel ci.
// Out-of-image taps read as zero (the zero padding).  With VEC = 4, Cin is a
// multiple of 4 so a chunk never straddles two taps.
template <int ROWS, int BK, int VEC, int NT>
struct ConvGatherLoader {
    static constexpr int CPR = BK / VEC;
    static constexpr int LOADS = ROWS * BK / (VEC * NT);
    static_assert(NT % CPR == 0, "threads must cover whole rows");
    static_assert(LOADS >= 1 && ROWS * BK % (VEC * NT) == 0, "tile not divisible");
    typedef typename Vec<VEC>::T VT;
    const float *img[LOADS];  // start of image n
    int ih0[LOADS], iw0[LOADS];
    int col;
    int ci, kw, kh;  // decomposition of this thread's current k
    int H, W, Cin, KW;

    __device__ __forceinline__ void init(const KernelArgs &p, int row0, int kbeg, int tid)
    {
        H = p.H; W = p.W; Cin = p.Cin; KW = p.KW;
        col = (tid % CPR) * VEC;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int m = row0 + (tid + i * NT) / CPR;
            if (m < p.M) {
                const int wo = m % p.Wo;
                const int t = m / p.Wo;
                const int ho = t % p.Ho;
                const int n = t / p.Ho;
                img[i] = p.A + (int64_t)n * H * W * Cin;
                ih0[i] = ho * p.sh - p.pt;
                iw0[i] = wo * p.sw - p.pl;
            } else {
                img[i] = p.A;
                ih0[i] = -(1 << 28);  // every tap falls outside the image
                iw0[i] = 0;
            }
        }
        const int k = kbeg * BK + col;
        const int tap = k / Cin;
        ci = k - tap * Cin;
        kh = tap / KW;
        kw = tap - kh * KW;
    }
    __device__ __forceinline__ void load(VT *v, int k0, int K) const
    {
        const bool k_ok = k0 + col < K;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int ih = ih0[i] + kh, iw = iw0[i] + kw;
            const bool ok = k_ok && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W;
            v[i] = ok ? Vec<VEC>::load(img[i] + ((int64_t)(ih * W + iw) * Cin + ci)) : Vec<VEC>::zero();
        }
    }
    __device__ __forceinline__ void advance()
    {
        ci += BK;
        while (ci >= Cin) {
            ci -= Cin;
            if (++kw == KW) { kw = 0; ++kh; }
        }
    }
    template <int LD>
    __device__ __forceinline__ void store(float *lds, const VT *v, int tid) const
    {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int r = (tid + i * NT) / CPR;
            Vec<VEC>::store(lds + r * LD + col, v[i]);
        }
    }
};

template <int AMODE, int BM, int BK, int VA, int NT>
struct ALoaderSel;
template <int BM, int BK, int VA, int NT>
struct ALoaderSel<A_KCONTIG, BM, BK, VA, NT> { typedef KContigLoader<BM, BK, VA, NT> T; };
template <int BM, int BK, int VA, int NT>
struct ALoaderSel<A_MCONTIG, BM, BK, VA, NT> { typedef MContigLoader<BM, BK, VA, NT> T; };
template <int BM, int BK, int VA, int NT>
struct ALoaderSel<A_CONV, BM, BK, VA, NT> { typedef ConvGatherLoader<BM, BK, VA, NT> T; };

// LDS padding (floats) appended to each LDS row: keeps rows 16-byte aligned
// and staggers banks between the two k-halves and between rows.
constexpr int LDS_PAD = 4;

template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB>
struct GemmTile {
    static constexpr int NT = 64 * WAVES_M * WAVES_N;
    static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    static constexpr int RM = WM / 32, RN = WN / 32;
    static constexpr bool A_K = AMODE != A_MCONTIG;  // A staged k-contiguous
    static constexpr bool B_K = B_KCONTIG;           // B staged k-contiguous
    static constexpr int LDA_S = A_K ? BK + LDS_PAD : BM + LDS_PAD;
    static constexpr int LDB_S = B_KCONTIG ? BK + LDS_PAD : BN + LDS_PAD;
    static constexpr int A_STAGE = A_K ? BM * LDA_S : BK * LDA_S;
    static constexpr int B_STAGE = B_KCONTIG ? BN * LDB_S : BK * LDB_S;
    static constexpr int LDS_FLOATS = 2 * (A_STAGE + B_STAGE);
    static constexpr int HALF = BK / 2;
    static constexpr int NG = HALF / 4;  // 4-step groups per K-block
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile is made of 32x32 blocks");
    static_assert(BK % 16 == 0, "BK must be a multiple of 16 (an even number of 4-step groups per half)");

    typedef typename ALoaderSel<AMODE, BM, BK, VA, NT>::T ALoader;
    typedef typename std::conditional<B_KCONTIG, KContigLoader<BN, BK, VB, NT>,
                                      MContigLoader<BN, BK, VB, NT>>::type BLoader;
    typedef f32x16 Acc[RM][RN];
    typedef float FragA[RM][4];
    typedef float FragB[RN][4];

    // Operands of one group (4 k-steps) for this lane, from one LDS stage.
    // a_row / b_row: the lane's row of the wave's first 32-row (-column) block.
    static __device__ __forceinline__ void read_group(const float *as, const float *bs, int a_row, int b_row,
                                                      int h, int g, FragA &xa, FragB &xb)
    {
        const int k0 = h * HALF + 4 * g;
#pragma unroll
        for (int i = 0; i < RM; ++i) {
            if constexpr (A_K) {
                const f32x4 v = *reinterpret_cast<const f32x4 *>(as + (a_row + i * 32) * LDA_S + k0);
                xa[i][0] = v[0]; xa[i][1] = v[1]; xa[i][2] = v[2]; xa[i][3] = v[3];
            } else {
#pragma unroll
                for (int t = 0; t < 4; ++t) xa[i][t] = as[(k0 + t) * LDA_S + a_row + i * 32];
            }
        }
#pragma unroll
        for (int j = 0; j < RN; ++j) {
            if constexpr (B_K) {
                const f32x4 v = *reinterpret_cast<const f32x4 *>(bs + (b_row + j * 32) * LDB_S + k0);
                xb[j][0] = v[0]; xb[j][1] = v[1]; xb[j][2] = v[2]; xb[j][3] = v[3];
            } else {
#pragma unroll
                for (int t = 0; t < 4; ++t) xb[j][t] = bs[(k0 + t) * LDB_S + b_row + j * 32];
            }
        }
    }

    // the MFMAs of k-step t of a group
    static __device__ __forceinline__ void mma_step(Acc &acc, const FragA &xa, const FragB &xb, int t)
    {
#pragma unroll
        for (int i = 0; i < RM; ++i)
#pragma unroll
            for (int j = 0; j < RN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(xa[i][t], xb[j][t], acc[i][j], 0, 0, 0);
    }

    static __device__ __forceinline__ void mma_group(Acc &acc, const FragA &xa, const FragB &xb)
    {
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < RM; ++i)
#pragma unroll
                for (int j = 0; j < RN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(xa[i][t], xb[j][t], acc[i][j], 0, 0, 0);
    }

    static __device__ __forceinline__ void zero(Acc &acc)
    {
#pragma unroll
        for (int i = 0; i < RM; ++i)
#pragma unroll
            for (int j = 0; j < RN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    }

    // Row of C that acc[i][*][r] of a lane holds.  The MFMA puts row slot
    // 8*(r/4) + r%4 + 4h of block i's A operand in register r of lane
    // (l32, h).  Blocked rows (ILV false): block i is rows 32i .. 32i+31 of
    // the wave tile, row_base = the wave's first row + 4h.  Interleaved rows
    // (ILV true): slot s of block i is row RM*s + i, so a lane's RM blocks
    // read RM adjacent rows (one 16-byte LDS read for RM = 4 where A is
    // m-contiguous), row_base = the wave's first row + RM*4h.
    template <bool ILV>
    static __device__ __forceinline__ int row_of(int row_base, int i, int r)
    {
        return ILV ? row_base + RM * (8 * (r >> 2) + (r & 3)) + i : row_base + i * 32 + 8 * (r >> 2) + (r & 3);
    }

    // Epilogue of one tile: C = alpha * acc (+ beta * C when BETA), or split
    // z's partial sum alpha * acc into the workspace.  Lane (l32, h) of the
    // wave holds C(row_of<ILV>(row_base, i, r), col_base + j*32) in
    // acc[i][j][r].  BETA = false never reads C (beta == 0).  C is written
    // with non-temporal stores (this launch does not read it again): 2-4 %
    // faster on the HBM-bound ResNet-50 1x1 layers, no change on the others.
    template <bool BETA, bool ILV = false>
    static __device__ __forceinline__ void store(const KernelArgs &p, const Acc &acc, int row_base, int col_base,
                                                 int z)
    {
        if (p.splits > 1) {
            float *out = p.ws + (int64_t)z * p.M * p.N;
#pragma unroll
            for (int i = 0; i < RM; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = row_of<ILV>(row_base, i, r);
                    if (row < p.M) {
#pragma unroll
                        for (int j = 0; j < RN; ++j) {
                            const int col = col_base + j * 32;
                            if (col < p.N) out[(int64_t)row * p.N + col] = p.alpha * acc[i][j][r];
                        }
                    }
                }
            return;
        }
        if constexpr (!BETA) {
#pragma unroll
            for (int i = 0; i < RM; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = row_of<ILV>(row_base, i, r);
                    if (row < p.M) {
                        float *crow = p.C + (int64_t)row * p.ldc;
#pragma unroll
                        for (int j = 0; j < RN; ++j) {
                            const int col = col_base + j * 32;
                            if (col < p.N) __builtin_nontemporal_store(p.alpha * acc[i][j][r], crow + col);
                        }
                    }
                }
        } else {
            // C = alpha * acc + beta * C.  The C values of one 32-row block are
            // all loaded, and the block's results computed, before its first
            // store: the memory counter also counts stores, so a result
            // computed next to its own store makes every store wait for the
            // one before it (a load that follows a store to C cannot be moved
            // above it by the compiler).  Interior lanes skip the bounds tests.
            const bool interior = row_of<ILV>(row_base, RM - 1, 15) < p.M && col_base + (RN - 1) * 32 < p.N;
            const float alpha = p.alpha, beta = p.beta;
#pragma unroll
            for (int i = 0; i < RM; ++i) {
                float v[16][RN];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = row_of<ILV>(row_base, i, r);
                    const float *crow = p.C + (int64_t)row * p.ldc;
#pragma unroll
                    for (int j = 0; j < RN; ++j) {
                        const int col = col_base + j * 32;
                        v[r][j] = (interior || (row < p.M && col < p.N)) ? crow[col] : 0.f;
                    }
                }
#pragma unroll
                for (int r = 0; r < 16; ++r)
#pragma unroll
                    for (int j = 0; j < RN; ++j) {
                        v[r][j] = fmaf(beta, v[r][j], alpha * acc[i][j][r]);
                        asm volatile("" : "+v"(v[r][j]));  // materialise here, before the stores
                    }
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = row_of<ILV>(row_base, i, r);
                    float *crow = p.C + (int64_t)row * p.ldc;
#pragma unroll
                    for (int j = 0; j < RN; ++j) {
                        const int col = col_base + j * 32;
                        if (interior || (row < p.M && col < p.N)) __builtin_nontemporal_store(v[r][j], crow + col);
                    }
                }
            }
        }
    }
};

// K range [kbeg, kend) of split z.
__device__ __forceinline__ void split_range(const KernelArgs &p, int bk, int z, int &kbeg, int &kend)
{
    const int nkb = (p.K + bk - 1) / bk;
    kbeg = z * p.kblocks_per_split;
    kend = min(nkb, kbeg + p.kblocks_per_split);
}

// OCC: the waves per SIMD the register allocation must leave room for
// (1 = no constraint beyond the work-group size).  BETA: the epilogue reads
// C (beta != 0); the beta == 0 form never touches C before writing it and
// carries none of the registers that reading it takes.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB> G;
    typedef typename G::ALoader ALoader;
    typedef typename G::BLoader BLoader;

    __shared__ __attribute__((aligned(16))) float smem[G::LDS_FLOATS];
    float *As = smem;                      // [2][A_STAGE]
    float *Bs = smem + 2 * G::A_STAGE;     // [2][B_STAGE]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;

    if constexpr (AMODE != A_CONV) {  // product blockIdx.y of a batch
        const int64_t bz = blockIdx.y;
        p.A += bz * p.stride_a;
        p.B += bz * p.stride_b;
        p.C += bz * p.stride_c;
    }
    int tm, tn;
    tile_coords(p, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    int kbeg, kend;
    split_range(p, BK, blockIdx.z, kbeg, kend);

    ALoader la;
    BLoader lb;
    if constexpr (AMODE == A_CONV)
        la.init(p, m0, kbeg, tid);
    else
        la.init(p.A, p.lda, m0, p.M, kbeg, tid);
    lb.init(p.B, p.ldb, n0, p.N, kbeg, tid);

    typename G::Acc acc;
    G::zero(acc);
    typename ALoader::VT ra[ALoader::LOADS];
    typename BLoader::VT rb[BLoader::LOADS];

    if (kbeg < kend) {
        la.load(ra, kbeg * BK, p.K);
        lb.load(rb, kbeg * BK, p.K);
        la.advance();
        lb.advance();
        la.template store<G::LDA_S>(As, ra, tid);
        lb.template store<G::LDB_S>(Bs, rb, tid);
    }
    __syncthreads();

    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;

    // Operand registers hold two groups: the one being multiplied and the
    // next one, read from LDS while the current MFMAs run.
    typename G::FragA fa[2];
    typename G::FragB fb[2];

    // Software pipeline over K-blocks (two LDS stages):
    //   issue the global loads of block kb+1;
    //   groups 0..NG-2 of block kb, each overlapping the LDS read of the next group;
    //   store block kb+1 into the other stage, barrier;
    //   read group 0 of block kb+1 while the MFMAs of the last group of kb run.
    // Every read of a stage precedes the barrier that follows it, and every
    // write of a stage follows the barrier that ends the reads of its previous
    // contents, so one barrier per K-block orders both.
    constexpr int NG = G::NG;
    int stage = 0;
    if (kbeg < kend) G::read_group(As, Bs, a_row, b_row, h, 0, fa[0], fb[0]);
    for (int kb = kbeg; kb < kend; ++kb) {
        const bool more = kb + 1 < kend;
        if (more) {
            la.load(ra, (kb + 1) * BK, p.K);
            lb.load(rb, (kb + 1) * BK, p.K);
            la.advance();
            lb.advance();
        }
        const float *as = As + stage * G::A_STAGE;
        const float *bs = Bs + stage * G::B_STAGE;
#pragma unroll
        for (int g = 0; g < NG - 1; ++g) {
            G::read_group(as, bs, a_row, b_row, h, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of these MFMAs
            G::mma_group(acc, fa[g & 1], fb[g & 1]);
        }
        if (more) {
            la.template store<G::LDA_S>(As + (stage ^ 1) * G::A_STAGE, ra, tid);
            lb.template store<G::LDB_S>(Bs + (stage ^ 1) * G::B_STAGE, rb, tid);
        }
        __syncthreads();
        // unconditional (after the last block it reads stale LDS that is never
        // used): a conditional read would make the compiler copy registers
        // between the read and the MFMAs below
        G::read_group(As + (stage ^ 1) * G::A_STAGE, Bs + (stage ^ 1) * G::B_STAGE, a_row, b_row, h, 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NG - 1) & 1], fb[(NG - 1) & 1]);
        stage ^= 1;
    }

    G::template store<BETA>(p, acc, m0 + wm * G::WM + 4 * h, n0 + wn * G::WN + l32, blockIdx.z);
}

// One operand tile copied straight from global memory into LDS by
// buffer_load_dwordx4 ... lds (no staging registers, no LDS write
// instructions).  One such instruction fills 1 KiB of LDS contiguously (lane
// i at base + 16 i), so the tile cannot carry the row padding the
// register-staged loaders use against bank conflicts; chunk positions are
// XOR-swizzled instead.
//   KROWS (A 'N', B 'T'): R x BK, rows of contiguous k, CPR 16-byte chunks
//     per row; chunk c of row r sits at position c ^ ((r / (16 / CPR)) %
//     CPR), so the 16 rows one ds_read_b128 pass touches fall in 16
//     distinct bank quads.
//   k-major (A 'T', B 'N'): BK x R, rows of contiguous m (n); the second
//     half of the K-block (read by lanes 32..63) has its chunks XOR 8, i.e.
//     column x sits at x ^ 32, so the two half-waves' 128-byte reads use
//     opposite halves of the 64 banks.
// Elements past the operand's rows or K get an offset past the buffer's
// range, which the hardware answers with zeros.  Offsets count from a
// per-tile, per-K-block base, so they stay below 2^31 whenever R (KROWS) or
// BK (k-major) rows of the operand do (checked by the host).
template <int R, int BK, int NW, bool KROWS>
struct DmaOperand {
    static constexpr int CPR = KROWS ? BK / 4 : R / 4;  // 16-byte chunks per LDS row
    static constexpr int RPS = KROWS ? 16 / CPR : 1;    // rows per step of the KROWS swizzle
    static constexpr int FLOATS = R * BK;
    static constexpr int L = FLOATS / 256 / NW;  // instructions per lane per K-block
    static_assert(FLOATS % (256 * NW) == 0, "whole 1 KiB pieces per wave");
    static_assert(KROWS ? (CPR <= 16 && 16 % CPR == 0) : (R % 64 == 0), "swizzle geometry");
    int off[L], kk[L];
    bool ok[L];

    // ld: the operand's leading dimension; r0 / rlim: its first row (m or
    // n) of this tile and the row count
    __device__ __forceinline__ void init(int64_t ld, int r0, int rlim, int wave, int lane)
    {
#pragma unroll
        for (int i = 0; i < L; ++i) {
            const int q = (i * NW + wave) * 64 + lane;  // chunk position in the tile
            if constexpr (KROWS) {
                const int r = q / CPR;
                const int c = (q % CPR) ^ ((r / RPS) % CPR);
                off[i] = (r * (int)ld + 4 * c) * 4;
                kk[i] = 4 * c;
                ok[i] = r0 + r < rlim;
            } else {
                const int k = q / CPR;
                const int c = (q % CPR) ^ (k >= BK / 2 ? 8 : 0);
                off[i] = (k * (int)ld + 4 * c) * 4;
                kk[i] = k;
                ok[i] = r0 + 4 * c < rlim;
            }
        }
    }
    // copy K-block k0 of the tile whose rows start at r0 into `tile` (the
    // copy slots I0 .. I1-1 of this lane; the whole block by default)
    template <int I0 = 0, int I1 = L>
    __device__ __forceinline__ void issue(const float *base, int64_t ld, int r0, int k0, int K, float *tile,
                                          int wave) const
    {
        const float *b = KROWS ? base + (int64_t)r0 * ld + k0 : base + (int64_t)k0 * ld + r0;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void *)b, 0, 0x7fffffff, 0x00020000);
#pragma unroll
        for (int i = I0; i < I1; ++i) {
            const int o = (ok[i] && k0 + kk[i] < K) ? off[i] : (int)0x80000000;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs, (__attribute__((address_space(3))) void *)(tile + (i * NW + wave) * 256), 16, o, 0, 0, 0);
        }
    }
    // the four k (h*BK/2 + 4g + t, t = 0..3) of row `row` for MFMA group g
    __device__ __forceinline__ static void read4(const float *tile, int row, int h, int g, float *v)
    {
        if constexpr (KROWS) {
            const int c = h * (BK / 8) + g;
            const f32x4 x = *reinterpret_cast<const f32x4 *>(tile + row * BK + 4 * (c ^ ((row / RPS) % CPR)));
            v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
        } else {
            const int k = h * (BK / 2) + 4 * g;
            const int col = row ^ (32 * h);
#pragma unroll
            for (int t = 0; t < 4; ++t) v[t] = tile[(k + t) * R + col];
        }
    }
    // m-contiguous layout: the same four k of the four adjacent rows row ..
    // row+3 (row a multiple of 4, so they are one 16-byte chunk, which the
    // swizzle moves whole), one 16-byte read per k: v[i][t] is row row+i
    template <typename Frag>
    __device__ __forceinline__ static void read4_rows4(const float *tile, int row, int h, int g, Frag &v)
    {
        static_assert(!KROWS, "adjacent rows share a chunk only in the m-contiguous layout");
        const int k = h * (BK / 2) + 4 * g;
        const int col = row ^ (32 * h);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const f32x4 x = *reinterpret_cast<const f32x4 *>(tile + (k + t) * R + col);
            v[0][t] = x[0]; v[1][t] = x[1]; v[2][t] = x[2]; v[3][t] = x[3];
        }
    }
};

// The implicit-GEMM gather of A (NHWC image, Cin % 4 == 0) copied straight
// into LDS in DmaOperand's KROWS layout: row m of the tile is output pixel
// (n, ho, wo), chunk c its taps' channels 4c .. 4c+3 of the current
// K-block.  With 4 * NW a multiple of CPR every copy slot of a lane has the
// same chunk c, so one (kh, kw, ci) walk per lane serves all of them.  Taps
// outside the image, rows past M and k past K read as zero (offset past the
// buffer's range); offsets count from the image base, so the host checks
// that the input spans less than 2 GiB.
template <int BM, int BK, int NW>
struct DmaConvA {
    typedef DmaOperand<BM, BK, NW, true> Layout;
    static constexpr int CPR = Layout::CPR, RPS = Layout::RPS, L = Layout::L, FLOATS = Layout::FLOATS;
    static_assert((4 * NW) % CPR == 0, "one chunk per lane across the copy slots");
    int nb[L], ih0[L], iw0[L];  // image row base n*H and window origin of each slot's pixel
    int col;                    // this lane's k offset inside the K-block
    int ci, kw, kh;             // decomposition of the lane's current k
    int H, W, Cin, KW;

    __device__ __forceinline__ void init(const KernelArgs &p, int m0, int kbeg, int wave, int lane)
    {
        H = p.H; W = p.W; Cin = p.Cin; KW = p.KW;
        const int r_first = ((wave * 64) + lane) / CPR;
        col = 4 * ((lane % CPR) ^ ((r_first / RPS) % CPR));
#pragma unroll
        for (int i = 0; i < L; ++i) {
            const int m = m0 + ((i * NW + wave) * 64 + lane) / CPR;
            if (m < p.M) {
                const int wo = m % p.Wo;
                const int t = m / p.Wo;
                const int ho = t % p.Ho;
                nb[i] = (t / p.Ho) * H;
                ih0[i] = ho * p.sh - p.pt;
                iw0[i] = wo * p.sw - p.pl;
            } else {
                nb[i] = 0;
                ih0[i] = -(1 << 28);  // every tap falls outside the image
                iw0[i] = 0;
            }
        }
        const int k = kbeg * BK + col;
        const int tap = k / Cin;
        ci = k - tap * Cin;
        kh = tap / KW;
        kw = tap - kh * KW;
    }
    // copy K-block k0 (the one the walk stands at) into `tile` (copy slots
    // I0 .. I1-1 of this lane; the whole block by default), then, once the
    // block's last slot is issued, step the walk `blocks` K-blocks on
    template <int I0 = 0, int I1 = L>
    __device__ __forceinline__ void issue(const float *x, int k0, int K, float *tile, int wave, int blocks = 1)
    {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void *)x, 0, 0x7fffffff, 0x00020000);
        const bool k_ok = k0 + col < K;
#pragma unroll
        for (int i = I0; i < I1; ++i) {
            const int ih = ih0[i] + kh, iw = iw0[i] + kw;
            const bool ok = k_ok && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W;
            const int o = ok ? (((nb[i] + ih) * W + iw) * Cin + ci) * 4 : (int)0x80000000;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs, (__attribute__((address_space(3))) void *)(tile + (i * NW + wave) * 256), 16, o, 0, 0, 0);
        }
        if constexpr (I1 == L) {
            ci += BK * blocks;
            while (ci >= Cin) {
                ci -= Cin;
                if (++kw == KW) { kw = 0; ++kh; }
            }
        }
    }
    __device__ __forceinline__ static void read4(const float *tile, int row, int h, int g, float *v)
    {
        Layout::read4(tile, row, h, g, v);
    }
};

// The contraction (dense operands in any of the four layouts, or the
// convolution's implicit-GEMM gather) with both operand tiles copied
// straight into STAGES LDS stages (DmaOperand, DmaConvA): S-1
// K-blocks are in flight at no register cost.  The compiler does not see
// these writes to LDS, so every wait for them is explicit and followed by a
// compiler memory barrier, and the work-group barrier is issued without
// __syncthreads()'s fence (which would also wait for the copies in flight
// for later blocks).  Same MFMA group pipeline as gemm_kernel.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int AMODE, bool TB, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_dma_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, A_KCONTIG, false, 4, 4> G;  // MFMA and epilogue only
    constexpr int NW = G::NT / 64;
    typedef typename std::conditional<AMODE == A_CONV, DmaConvA<BM, BK, NW>,
                                      DmaOperand<BM, BK, NW, AMODE == A_KCONTIG>>::type OpA;
    typedef DmaOperand<BN, BK, NW, TB> OpB;
    constexpr int A_ST = OpA::FLOATS, B_ST = OpB::FLOATS;  // floats per stage
    constexpr int LPB = OpA::L + OpB::L;                    // copies per lane per K-block
    static_assert(STAGES >= 2 && STAGES <= 4, "two to four LDS stages");
    static_assert((STAGES - 2) * LPB <= 63, "vmcnt range");

    __shared__ __attribute__((aligned(16))) float smem[STAGES * (A_ST + B_ST)];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;

    if constexpr (AMODE != A_CONV) {  // product blockIdx.y of a batch
        const int64_t bz = blockIdx.y;
        p.A += bz * p.stride_a;
        p.B += bz * p.stride_b;
        p.C += bz * p.stride_c;
    }
    int tm, tn;
    tile_coords(p, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    int kbeg, kend;
    split_range(p, BK, blockIdx.z, kbeg, kend);

    OpA oa;
    OpB ob;
    if constexpr (AMODE == A_CONV)
        oa.init(p, m0, kbeg, wave, lane);
    else
        oa.init(p.lda, m0, p.M, wave, lane);
    ob.init(p.ldb, n0, p.N, wave, lane);
    // blocks are issued in K order (the gather's walk steps once per issue)
    auto issue = [&](int kb, int s) {
        float *as = smem + s * (A_ST + B_ST);
        if constexpr (AMODE == A_CONV)
            oa.issue(p.A, kb * BK, p.K, as, wave);
        else
            oa.issue(p.A, p.lda, m0, kb * BK, p.K, as, wave);
        ob.issue(p.B, p.ldb, n0, kb * BK, p.K, as + A_ST, wave);
    };
    // wait until this lane's copies of every issued block but the newest
    // `later` ones (0 .. STAGES-2) have landed in LDS
    auto wait_blocks = [&](int later) {
        if (STAGES >= 4 && later >= 2)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPB) : "memory");
        else if (STAGES >= 3 && later >= 1)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPB) : "memory");
        else
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    // this wave's LDS reads are complete (no copy issued after the barrier
    // can overwrite what they still fetch) and its copies for the block about
    // to be read have landed (wait_blocks), so the barrier alone publishes
    // the stage
    auto barrier = [] {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // an m-contiguous A tile with four 32-row blocks per wave takes them
    // interleaved (GemmTile::row_of): one 16-byte LDS read per k for all four
    // blocks instead of a read of two k per block
    constexpr bool ILV = AMODE == A_MCONTIG && G::RM == 4;
    const int a_row = wm * G::WM + (ILV ? 4 * l32 : l32);
    const int b_row = wn * G::WN + l32;
    auto read_group = [&](const float *as, int g, typename G::FragA &xa, typename G::FragB &xb) {
        if constexpr (ILV) {
            OpA::read4_rows4(as, a_row, h, g, xa);
        } else {
#pragma unroll
            for (int i = 0; i < G::RM; ++i) OpA::read4(as, a_row + i * 32, h, g, xa[i]);
        }
#pragma unroll
        for (int j = 0; j < G::RN; ++j) OpB::read4(as + A_ST, b_row + j * 32, h, g, xb[j]);
    };

    typename G::Acc acc;
    G::zero(acc);
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NG = G::NG;

#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (kbeg + s < kend) issue(kbeg + s, s);
    wait_blocks(min(STAGES - 2, kend - kbeg - 1));
    barrier();
    if (kbeg < kend) read_group(smem, 0, fa[0], fb[0]);

    // Block kb sits in stage s.  At the top the copy of block kb+S-1 goes
    // into the stage block kb-1 used (all of its reads are behind the
    // barrier that ended block kb-1); block kb+1 is waited for before the
    // barrier that ends block kb.
    // A's copies of the next block go out before group 0's MFMAs and B's
    // after its second k-step: the copies of all the waves then reach the
    // memory pipeline in two bursts instead of one (measured in the benchmark
    // step: the 4096^3 GEMMs 0.4-1.3 % faster, the step 0.6 %; spreading the
    // copies over every k-step, or into group 1, was slower)
    auto issue_a = [&](int kb, int st) {
        float *as = smem + st * (A_ST + B_ST);
        if constexpr (AMODE == A_CONV)
            oa.issue(p.A, kb * BK, p.K, as, wave);
        else
            oa.issue(p.A, p.lda, m0, kb * BK, p.K, as, wave);
    };
    auto issue_b = [&](int kb, int st) {
        float *as = smem + st * (A_ST + B_ST);
        ob.issue(p.B, p.ldb, n0, kb * BK, p.K, as + A_ST, wave);
    };
    int s = 0;
    for (int kb = kbeg; kb < kend; ++kb) {
        const int s_next = s + 1 == STAGES ? 0 : s + 1;
        const bool more = kb + STAGES - 1 < kend;
        const int s_fill = s == 0 ? STAGES - 1 : s - 1;
        const float *as = smem + s * (A_ST + B_ST);
        if (more) issue_a(kb + STAGES - 1, s_fill);
        static_for<NG - 1>([&](auto gc) {
            constexpr int g = decltype(gc)::value;
            read_group(as, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (g == 0) {
                G::mma_step(acc, fa[0], fb[0], 0);
                G::mma_step(acc, fa[0], fb[0], 1);
                if (more) issue_b(kb + STAGES - 1, s_fill);
                G::mma_step(acc, fa[0], fb[0], 2);
                G::mma_step(acc, fa[0], fb[0], 3);
            } else {
                G::mma_group(acc, fa[g & 1], fb[g & 1]);
            }
        });
        wait_blocks(min(STAGES - 2, kend - kb - 2));
        barrier();
        // unconditional (stale after the last block, never used)
        read_group(smem + s_next * (A_ST + B_ST), 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NG - 1) & 1], fb[(NG - 1) & 1]);
        s = s_next;
    }

    G::template store<BETA, ILV>(p, acc, m0 + wm * G::WM + (ILV ? 16 * h : 4 * h), n0 + b_row, blockIdx.z);
}

// The same contraction with the global loads TWO K-blocks ahead: two
// register sets alternate, so the loads of block kb+2 are issued while block
// kb multiplies and are stored to LDS only at the end of block kb+1.  Each
// load then has two blocks' MFMAs to arrive in instead of one -- what a small
// tile with a short K-block (64 x 64 x 32: about a thousand MFMA cycles per
// wave) needs to cover the global-load latency when only a few work-groups
// share a CU.  Same LDS stages, barrier and group pipeline as gemm_kernel.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_deep_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB> G;
    typedef typename G::ALoader ALoader;
    typedef typename G::BLoader BLoader;

    __shared__ __attribute__((aligned(16))) float smem[G::LDS_FLOATS];
    float *As = smem;                      // [2][A_STAGE]
    float *Bs = smem + 2 * G::A_STAGE;     // [2][B_STAGE]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;

    if constexpr (AMODE != A_CONV) {  // product blockIdx.y of a batch
        const int64_t bz = blockIdx.y;
        p.A += bz * p.stride_a;
        p.B += bz * p.stride_b;
        p.C += bz * p.stride_c;
    }
    int tm, tn;
    tile_coords(p, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    int kbeg, kend;
    split_range(p, BK, blockIdx.z, kbeg, kend);

    ALoader la;
    BLoader lb;
    if constexpr (AMODE == A_CONV)
        la.init(p, m0, kbeg, tid);
    else
        la.init(p.A, p.lda, m0, p.M, kbeg, tid);
    lb.init(p.B, p.ldb, n0, p.N, kbeg, tid);

    typename G::Acc acc;
    G::zero(acc);
    typename ALoader::VT ra0[ALoader::LOADS], ra1[ALoader::LOADS];
    typename BLoader::VT rb0[BLoader::LOADS], rb1[BLoader::LOADS];

    auto fetch = [&](typename ALoader::VT *ra, typename BLoader::VT *rb, int kb) {
        la.load(ra, kb * BK, p.K);
        lb.load(rb, kb * BK, p.K);
        la.advance();
        lb.advance();
    };
    if (kbeg < kend) fetch(ra0, rb0, kbeg);
    if (kbeg + 1 < kend) fetch(ra1, rb1, kbeg + 1);
    if (kbeg < kend) {
        la.template store<G::LDA_S>(As, ra0, tid);
        lb.template store<G::LDB_S>(Bs, rb0, tid);
    }
    __syncthreads();

    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NG = G::NG;
    if (kbeg < kend) G::read_group(As, Bs, a_row, b_row, h, 0, fa[0], fb[0]);

    // Block kb sits in LDS stage s; the registers `cur` hold block kb+1 and
    // `nxt` (free) receives block kb+2.
    auto block = [&](int kb, int s, typename ALoader::VT *cur_a, typename BLoader::VT *cur_b,
                     typename ALoader::VT *nxt_a, typename BLoader::VT *nxt_b) {
        if (kb + 2 < kend) fetch(nxt_a, nxt_b, kb + 2);
        const float *as = As + s * G::A_STAGE;
        const float *bs = Bs + s * G::B_STAGE;
#pragma unroll
        for (int g = 0; g < NG - 1; ++g) {
            G::read_group(as, bs, a_row, b_row, h, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of these MFMAs
            G::mma_group(acc, fa[g & 1], fb[g & 1]);
        }
        if (kb + 1 < kend) {
            la.template store<G::LDA_S>(As + (s ^ 1) * G::A_STAGE, cur_a, tid);
            lb.template store<G::LDB_S>(Bs + (s ^ 1) * G::B_STAGE, cur_b, tid);
        }
        __syncthreads();
        // unconditional, as in gemm_kernel (after the last block it reads a
        // stage that is never used)
        G::read_group(As + (s ^ 1) * G::A_STAGE, Bs + (s ^ 1) * G::B_STAGE, a_row, b_row, h, 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NG - 1) & 1], fb[(NG - 1) & 1]);
    };
    // two blocks per trip so that each register set keeps one name
    for (int kb = kbeg; kb < kend; kb += 2) {
        block(kb, 0, ra1, rb1, ra0, rb0);
        if (kb + 1 >= kend) break;
        block(kb + 1, 1, ra0, rb0, ra1, rb1);
    }

    G::template store<BETA>(p, acc, m0 + wm * G::WM + 4 * h, n0 + wn * G::WN + l32, blockIdx.z);
}

// The same contraction with the K dimension split INSIDE the work-group,
// for products with few C tiles and a long reduction (the paper's GEMM sweep:
// M, N <= 1024 with K up to 1024 gives 1-256 tiles of 64 x 64, so one
// work-group per tile walks 16-32 K-blocks one after the other, each paying
// the global-load latency).  The work-group holds KS groups of
// WAVES_M x WAVES_N waves; group g multiplies the K-blocks g, g + KS,
// g + 2 KS, ... of the tile through its own two LDS stages (the blocked
// identity over a partition of K, Section 3.1.1), so the chain of dependent
// K-blocks is KS times shorter and KS times more waves work on each tile.
// At the end the groups' partial tiles are added through LDS in group order
// (deterministic; no workspace, no atomics) and group 0 writes C.  Every
// group runs the same number of K-block steps (a group past the last block
// loads zeros), so the work-group's barriers line up.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int KS, int AHEAD, int AMODE, bool B_KCONTIG, int VA, int VB,
          int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N * KS) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_ksplit_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB> G;
    typedef typename G::ALoader ALoader;
    typedef typename G::BLoader BLoader;
    static_assert(AMODE != A_CONV, "dense operands only");
    static_assert(AHEAD == 1 || AHEAD == 2, "loads one or two steps ahead");
    constexpr int GT = G::NT;                      // threads per group
    constexpr int ACCF = G::RM * G::RN * 16;       // accumulator floats per lane
    static_assert((KS - 1) * GT * ACCF <= KS * G::LDS_FLOATS, "partial tiles fit in the stages");

    __shared__ __attribute__((aligned(16))) float smem[KS * G::LDS_FLOATS];

    const int grp = threadIdx.x / GT;
    const int tid = threadIdx.x - grp * GT;
    float *As = smem + grp * G::LDS_FLOATS;        // [2][A_STAGE] of this group
    float *Bs = As + 2 * G::A_STAGE;               // [2][B_STAGE]
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;

    if (p.nbatch > 1) {  // product blockIdx.y of a batch
        const int64_t bz = blockIdx.y;
        p.A += bz * p.stride_a;
        p.B += bz * p.stride_b;
        p.C += bz * p.stride_c;
    }
    int tm, tn;
    tile_coords(p, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    int kbeg, kend;  // K-blocks of this work-group's split
    split_range(p, BK, blockIdx.z, kbeg, kend);
    const int steps = (kend - kbeg + KS - 1) / KS;  // K-block steps of every group
    const int klim = min(p.K, kend * BK);          // k past the split reads as zero

    ALoader la;
    BLoader lb;
    la.init(p.A, p.lda, m0, p.M, kbeg + grp, tid);
    lb.init(p.B, p.ldb, n0, p.N, kbeg + grp, tid);

    typename G::Acc acc;
    G::zero(acc);
    typename ALoader::VT ra0[ALoader::LOADS], ra1[AHEAD == 2 ? ALoader::LOADS : 1];
    typename BLoader::VT rb0[BLoader::LOADS], rb1[AHEAD == 2 ? BLoader::LOADS : 1];

    // step st of group g multiplies K-block kbeg + st*KS + g (zeros past the
    // split: the loaders read nothing at k >= klim); steps are fetched in order
    auto fetch = [&](typename ALoader::VT *ra, typename BLoader::VT *rb, int st) {
        const int k0 = (kbeg + st * KS + grp) * BK;
        la.load(ra, k0, klim, tid);
        lb.load(rb, k0, klim, tid);
        la.advance_by(KS);
        lb.advance_by(KS);
    };
    fetch(ra0, rb0, 0);
    if constexpr (AHEAD == 2) {
        if (1 < steps) fetch(ra1, rb1, 1);
    }
    la.template store<G::LDA_S>(As, ra0, tid);
    lb.template store<G::LDB_S>(Bs, rb0, tid);
    __syncthreads();

    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NG = G::NG;
    G::read_group(As, Bs, a_row, b_row, h, 0, fa[0], fb[0]);

    // Step st sits in LDS stage s.  With AHEAD = 1 the registers `nxt`
    // receive step st+1 and are stored at the end of this step; with
    // AHEAD = 2 `cur` already holds step st+1 (stored at the end of this
    // step) and `nxt` receives step st+2.  Every condition is the same in
    // all groups, so the work-group's barriers line up.
    auto step = [&](int st, int s, typename ALoader::VT *cur_a, typename BLoader::VT *cur_b,
                    typename ALoader::VT *nxt_a, typename BLoader::VT *nxt_b) {
        if (st + AHEAD < steps) fetch(nxt_a, nxt_b, st + AHEAD);
        const float *as = As + s * G::A_STAGE;
        const float *bs = Bs + s * G::B_STAGE;
#pragma unroll
        for (int g = 0; g < NG - 1; ++g) {
            G::read_group(as, bs, a_row, b_row, h, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            G::mma_group(acc, fa[g & 1], fb[g & 1]);
        }
        if (st + 1 < steps) {
            la.template store<G::LDA_S>(As + (s ^ 1) * G::A_STAGE, cur_a, tid);
            lb.template store<G::LDB_S>(Bs + (s ^ 1) * G::B_STAGE, cur_b, tid);
        }
        __syncthreads();
        G::read_group(As + (s ^ 1) * G::A_STAGE, Bs + (s ^ 1) * G::B_STAGE, a_row, b_row, h, 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NG - 1) & 1], fb[(NG - 1) & 1]);
    };
    if constexpr (AHEAD == 1) {
        for (int st = 0, s = 0; st < steps; ++st, s ^= 1) step(st, s, ra0, rb0, ra0, rb0);
    } else {
        // two steps per trip so that each register set keeps one name
        for (int st = 0; st < steps; st += 2) {
            step(st, 0, ra1, rb1, ra0, rb0);
            if (st + 1 >= steps) break;
            step(st + 1, 1, ra0, rb0, ra1, rb1);
        }
    }

    // groups 1..KS-1 leave their partial tiles in LDS, group 0 adds them in
    // group order.  Every stage read that feeds an MFMA is behind the last
    // barrier; the one read after it (group 0 of the next stage, into fa[0])
    // is never used, since NG is even and the last mma_group takes fa[1].
    if (grp > 0) {
        float *slot = smem + (grp - 1) * GT * ACCF + tid;
#pragma unroll
        for (int i = 0; i < G::RM; ++i)
#pragma unroll
            for (int j = 0; j < G::RN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) slot[((i * G::RN + j) * 16 + r) * GT] = acc[i][j][r];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
        for (int q = 1; q < KS; ++q) {
            const float *slot = smem + (q - 1) * GT * ACCF + tid;
#pragma unroll
            for (int i = 0; i < G::RM; ++i)
#pragma unroll
                for (int j = 0; j < G::RN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[i][j][r] += slot[((i * G::RN + j) * 16 + r) * GT];
        }
        G::template store<BETA>(p, acc, m0 + wm * G::WM + 4 * h, n0 + wn * G::WN + l32, blockIdx.z);
    }
}

// The same contraction with ONE LDS stage: every K-block is loaded, stored
// to LDS and multiplied in turn, with a barrier before the store (the last
// block's reads are done) and one after it.  Nothing overlaps the global
// loads inside a work-group; only other resident work-groups hide them.  It
// exists to measure what double buffering (the two-stage pipeline above,
// Section 3.1.2) buys on this hardware.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_single_stage_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB> G;
    typedef typename G::ALoader ALoader;
    typedef typename G::BLoader BLoader;

    __shared__ __attribute__((aligned(16))) float smem[G::A_STAGE + G::B_STAGE];
    float *As = smem;
    float *Bs = smem + G::A_STAGE;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;

    if constexpr (AMODE != A_CONV) {
        const int64_t bz = blockIdx.y;
        p.A += bz * p.stride_a;
        p.B += bz * p.stride_b;
        p.C += bz * p.stride_c;
    }
    int tm, tn;
    tile_coords(p, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    int kbeg, kend;
    split_range(p, BK, blockIdx.z, kbeg, kend);

    ALoader la;
    BLoader lb;
    if constexpr (AMODE == A_CONV)
        la.init(p, m0, kbeg, tid);
    else
        la.init(p.A, p.lda, m0, p.M, kbeg, tid);
    lb.init(p.B, p.ldb, n0, p.N, kbeg, tid);

    typename G::Acc acc;
    G::zero(acc);
    typename ALoader::VT ra[ALoader::LOADS];
    typename BLoader::VT rb[BLoader::LOADS];
    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    typename G::FragA fa;
    typename G::FragB fb;

    for (int kb = kbeg; kb < kend; ++kb) {
        la.load(ra, kb * BK, p.K);
        lb.load(rb, kb * BK, p.K);
        la.advance();
        lb.advance();
        __syncthreads();  // the previous block's LDS reads are done
        la.template store<G::LDA_S>(As, ra, tid);
        lb.template store<G::LDB_S>(Bs, rb, tid);
        __syncthreads();
#pragma unroll
        for (int g = 0; g < G::NG; ++g) {
            G::read_group(As, Bs, a_row, b_row, h, g, fa, fb);
            G::mma_group(acc, fa, fb);
        }
    }

    G::template store<BETA>(p, acc, m0 + wm * G::WM + 4 * h, n0 + wn * G::WN + l32, blockIdx.z);
}

// The items (split z, tile) of a persistent launch: item = z * tiles + tile.
// Each XCD owns a contiguous share of the items (split as evenly as the item
// count allows) and the work-groups resident on it walk that share with a
// stride equal to their number, so at any time an XCD's L2 serves
// neighbouring tiles.  Work-group b runs on XCD b % xcds; the share is only
// used when the grid divides evenly among the XCDs.
struct ItemWalk {
    int cur, end, stride;

    __device__ __forceinline__ void init(int items, int xcds)
    {
        const int G = gridDim.x, b = blockIdx.x;
        const int X = (xcds > 1 && G % xcds == 0) ? xcds : 1;
        const int x = b % X, w = b / X;
        const int q = items / X, r = items % X;
        const int start = x * q + min(x, r);
        end = start + q + (x < r ? 1 : 0);
        stride = G / X;
        cur = start + w;
    }
    __device__ __forceinline__ bool valid() const { return cur < end; }
    __device__ __forceinline__ void next() { cur += stride; }
};


// Persistent form of gemm_kernel: a grid sized to what the CUs hold at once,
// each work-group looping over its items.  The K-block pipeline runs across
// item boundaries: the first block of the next item is loaded and staged
// while the last block of the current one computes, and the epilogue's stores
// overlap the next item's MFMAs, so short reductions (K of one to a few
// blocks) no longer pay a load latency per tile.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_persistent_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB> G;
    typedef typename G::ALoader ALoader;
    typedef typename G::BLoader BLoader;

    __shared__ __attribute__((aligned(16))) float smem[G::LDS_FLOATS];
    float *As = smem;
    float *Bs = smem + 2 * G::A_STAGE;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;
    const int tiles = p.tiles_m * p.tiles_n;

    ItemWalk walk;
    walk.init(tiles * p.splits, p.xcds);
    if (!walk.valid()) return;  // uniform over the work-group, before any barrier

    int m0, n0, z, kb, kend;
    auto decode = [&](int item, int &m0_, int &n0_, int &z_, int &kbeg_, int &kend_) {
        z_ = item / tiles;
        int tm, tn;
        tile_of(p, item - z_ * tiles, tm, tn);
        m0_ = tm * BM;
        n0_ = tn * BN;
        split_range(p, BK, z_, kbeg_, kend_);
    };
    decode(walk.cur, m0, n0, z, kb, kend);

    ALoader la;
    BLoader lb;
    auto init_loaders = [&](int m0_, int n0_, int kbeg_) {
        if constexpr (AMODE == A_CONV)
            la.init(p, m0_, kbeg_, tid);
        else
            la.init(p.A, p.lda, m0_, p.M, kbeg_, tid);
        lb.init(p.B, p.ldb, n0_, p.N, kbeg_, tid);
    };
    init_loaders(m0, n0, kb);

    typename G::Acc acc;
    G::zero(acc);
    typename ALoader::VT ra[ALoader::LOADS];
    typename BLoader::VT rb[BLoader::LOADS];

    la.load(ra, kb * BK, p.K);
    lb.load(rb, kb * BK, p.K);
    la.advance();
    lb.advance();
    la.template store<G::LDA_S>(As, ra, tid);
    lb.template store<G::LDB_S>(Bs, rb, tid);
    __syncthreads();

    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NG = G::NG;
    int stage = 0;
    G::read_group(As, Bs, a_row, b_row, h, 0, fa[0], fb[0]);

    // The same one-barrier pipeline as gemm_kernel, over the sequence of
    // (item, K-block) pairs this work-group owns.
    for (;;) {
        const bool last_block = kb + 1 >= kend;
        int nm0 = m0, nn0 = n0, nz = z, nkb = kb + 1, nkend = kend;
        bool more = true;
        if (last_block) {
            walk.next();
            more = walk.valid();
            if (more) decode(walk.cur, nm0, nn0, nz, nkb, nkend);
        }
        if (more) {
            if (last_block) init_loaders(nm0, nn0, nkb);
            la.load(ra, nkb * BK, p.K);
            lb.load(rb, nkb * BK, p.K);
            la.advance();
            lb.advance();
        }
        const float *as = As + stage * G::A_STAGE;
        const float *bs = Bs + stage * G::B_STAGE;
#pragma unroll
        for (int g = 0; g < NG - 1; ++g) {
            G::read_group(as, bs, a_row, b_row, h, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            G::mma_group(acc, fa[g & 1], fb[g & 1]);
        }
        if (more) {
            la.template store<G::LDA_S>(As + (stage ^ 1) * G::A_STAGE, ra, tid);
            lb.template store<G::LDB_S>(Bs + (stage ^ 1) * G::B_STAGE, rb, tid);
        }
        __syncthreads();
        G::read_group(As + (stage ^ 1) * G::A_STAGE, Bs + (stage ^ 1) * G::B_STAGE, a_row, b_row, h, 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NG - 1) & 1], fb[(NG - 1) & 1]);
        if (last_block) {
            G::template store<BETA>(p, acc, m0 + wm * G::WM + 4 * h, n0 + wn * G::WN + l32, z);
            G::zero(acc);
        }
        if (!more) break;
        m0 = nm0;
        n0 = nn0;
        z = nz;
        kb = nkb;
        kend = nkend;
        stage ^= 1;
    }
}


// Stream-K partition of a product's T = tiles * nkb (tile, K-block)
// iterations over G work-groups: logical work-group g owns the contiguous
// iterations [start(g), start(g+1)) with start(g) = floor(g*T/G), so every
// work-group does the same amount of MFMA work to within one K-block,
// whatever the tile count.  Tile t (iterations [t*nkb, (t+1)*nkb)) is
// computed by the work-groups owner(t*nkb) .. owner((t+1)*nkb - 1), each
// summing a contiguous run of its K-blocks (the blocked identity over a
// partition of K, Section 3.1.1).  A work-group's first and last tile may be
// such partial tiles; their partial sums go to slot 2g and 2g+1.
// Stream-K form of the persistent contraction.  The grid is the resident
// work-groups; each runs the one-barrier K pipeline over its iteration range,
// across tile boundaries.  A tile whose K-blocks all fall in one range is
// finished as usual.  A partial tile's sum is written to the range's slot;
// the work-group that arrives last at the tile's counter (agent-scope atomic)
// adds the partial sums of all its contributors in the order of their K-blocks
// and writes C, so the result does not depend on which one finishes last and
// no work-group ever waits for another.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int AMODE, bool B_KCONTIG, int VA, int VB, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_streamk_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, AMODE, B_KCONTIG, VA, VB> G;
    typedef typename G::ALoader ALoader;
    typedef typename G::BLoader BLoader;
    constexpr int NT = G::NT;

    __shared__ __attribute__((aligned(16))) float smem[G::LDS_FLOATS];
    __shared__ int s_arrival;
    float *As = smem;
    float *Bs = smem + 2 * G::A_STAGE;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;
    const int nkb = p.sk_nkb;
    const StreamK sk{p.tiles_m * p.tiles_n * nkb, (int)gridDim.x, nkb};

    // work-group b runs on XCD b % xcds: give each XCD a contiguous share of
    // the logical ranges, so the tiles an XCD works on are neighbours
    const int lg = sk_logical(blockIdx.x, sk.G, p.xcds);
    const int end = sk.start(lg + 1);
    int seg = sk.start(lg);  // first iteration of the current segment
    if (seg >= end) return;  // uniform over the work-group, before any barrier

    int tile = seg / nkb;
    int kbeg = seg - tile * nkb;
    int kend = min(nkb, kbeg + (end - seg));
    int m0, n0;
    auto decode_tile = [&](int t, int &m0_, int &n0_) {
        int tm, tn;
        tile_of(p, t, tm, tn);
        m0_ = tm * BM;
        n0_ = tn * BN;
    };
    decode_tile(tile, m0, n0);
    int kb = kbeg;

    ALoader la;
    BLoader lb;
    auto init_loaders = [&](int m0_, int n0_, int kbeg_) {
        if constexpr (AMODE == A_CONV)
            la.init(p, m0_, kbeg_, tid);
        else
            la.init(p.A, p.lda, m0_, p.M, kbeg_, tid);
        lb.init(p.B, p.ldb, n0_, p.N, kbeg_, tid);
    };
    init_loaders(m0, n0, kb);

    typename G::Acc acc;
    G::zero(acc);
    typename ALoader::VT ra[ALoader::LOADS];
    typename BLoader::VT rb[BLoader::LOADS];

    la.load(ra, kb * BK, p.K);
    lb.load(rb, kb * BK, p.K);
    la.advance();
    lb.advance();
    la.template store<G::LDA_S>(As, ra, tid);
    lb.template store<G::LDB_S>(Bs, rb, tid);
    __syncthreads();

    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NGR = G::NG;
    int stage = 0;
    G::read_group(As, Bs, a_row, b_row, h, 0, fa[0], fb[0]);

    for (;;) {
        const bool last_block = kb + 1 >= kend;
        int ntile = tile, nm0 = m0, nn0 = n0, nkbeg = kbeg, nkend = kend, nkb1 = kb + 1, nseg = seg;
        bool more = true;
        if (last_block) {
            nseg = seg + (kend - kbeg);
            more = nseg < end;
            if (more) {
                ntile = nseg / nkb;
                nkbeg = nseg - ntile * nkb;
                nkend = min(nkb, nkbeg + (end - nseg));
                decode_tile(ntile, nm0, nn0);
                nkb1 = nkbeg;
            }
        }
        if (more) {
            if (last_block) init_loaders(nm0, nn0, nkb1);
            la.load(ra, nkb1 * BK, p.K);
            lb.load(rb, nkb1 * BK, p.K);
            la.advance();
            lb.advance();
        }
        const float *as = As + stage * G::A_STAGE;
        const float *bs = Bs + stage * G::B_STAGE;
#pragma unroll
        for (int g = 0; g < NGR - 1; ++g) {
            G::read_group(as, bs, a_row, b_row, h, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            G::mma_group(acc, fa[g & 1], fb[g & 1]);
        }
        if (more) {
            la.template store<G::LDA_S>(As + (stage ^ 1) * G::A_STAGE, ra, tid);
            lb.template store<G::LDB_S>(Bs + (stage ^ 1) * G::B_STAGE, rb, tid);
        }
        __syncthreads();
        G::read_group(As + (stage ^ 1) * G::A_STAGE, Bs + (stage ^ 1) * G::B_STAGE, a_row, b_row, h, 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NGR - 1) & 1], fb[(NGR - 1) & 1]);
        if (last_block) {
            const int row_base = m0 + wm * G::WM + 4 * h, col_base = n0 + wn * G::WN + l32;
            bool write = true;  // this work-group writes the tile's C block
            if (kbeg != 0 || kend != nkb) {
                // partial tile: publish this range's sum.  Value r of block
                // (i, j) of thread t sits at float ((i*RN + j)*16 + r)*NT + t
                // of the slot (each store instruction of a wave writes 256
                // contiguous bytes).  The partial sums are written and read
                // with agent-scope atomic accesses, which the hardware keeps
                // coherent across the XCDs' L2 caches, so no cache-wide
                // write-back or invalidation is needed; each wave waits for
                // its stores to complete before the work-group counts itself
                // in.
                float *mine = p.sk_part + (int64_t)sk.slot(lg, tile) * (BM * BN) + tid;
                // the per-element offsets below are constants; without this the
                // compiler hoists all RM*RN*16 addresses out of the tile loop
                // and keeps them in registers
                asm volatile("" : "+v"(mine));
#pragma unroll
                for (int i = 0; i < G::RM; ++i)
#pragma unroll
                    for (int j = 0; j < G::RN; ++j)
#pragma unroll
                        for (int r = 0; r < 16; ++r)
                            __hip_atomic_store(mine + ((i * G::RN + j) * 16 + r) * NT, acc[i][j][r],
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores are complete
                __syncthreads();
                if (tid == 0)
                    s_arrival = __hip_atomic_fetch_add(p.sk_cnt + tile, 1, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                __syncthreads();
                const int lo = sk.owner(tile * nkb), hi = sk.owner(tile * nkb + nkb - 1);
                write = s_arrival == hi - lo;  // the last contributor: uniform over the work-group
                if (write) {
                    // sum the contributors' partial sums in K-block order (its own
                    // re-read like the others), so the bits do not depend on
                    // which contributor adds them
                    // (the first contributor's load redefines acc whole, so the
                    // values the MFMAs left there are dead from here on)
                    auto gather = [&](int g, bool first) {
                        const float *src = p.sk_part + (int64_t)sk.slot(g, tile) * (BM * BN) + tid;
                        asm volatile("" : "+v"(src));
#pragma unroll
                        for (int i = 0; i < G::RM; ++i)
#pragma unroll
                            for (int j = 0; j < G::RN; ++j)
#pragma unroll
                                for (int r = 0; r < 16; ++r) {
                                    const float v = __hip_atomic_load(src + ((i * G::RN + j) * 16 + r) * NT,
                                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                                    acc[i][j][r] = first ? v : acc[i][j][r] + v;
                                }
                    };
                    gather(lo, true);
                    for (int g = lo + 1; g <= hi; ++g) gather(g, false);
                }
            }
            if (write) G::template store<BETA>(p, acc, row_base, col_base, 0);
            G::zero(acc);
        }
        if (!more) break;
        tile = ntile;
        m0 = nm0;
        n0 = nn0;
        kbeg = nkbeg;
        kend = nkend;
        kb = nkb1;
        seg = nseg;
        stage ^= 1;
    }
}


// The K-split contraction (groups of waves splitting each tile's K-blocks,
// as gemm_ksplit_kernel) with every group's operand tiles copied straight
// into its own STAGES LDS stages (DmaOperand), so each group has S-1 of its
// K-blocks in flight at no register cost -- for products with few tiles and
// a long reduction, whose time is the chain of a group's K-blocks.  A group
// past the split's last K-block copies zeros (k bounded by the split).  All
// groups take the same number of steps, so the work-group's barriers line
// up; at the end the partial tiles are added through LDS in group order.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int KS, int STAGES, int AMODE, bool TB, int OCC,
          bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N * KS) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_dma_ksplit_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, A_KCONTIG, false, 4, 4> G;  // MFMA and epilogue only
    constexpr int GT = G::NT, NW = GT / 64;  // threads and waves per group
    typedef typename std::conditional<AMODE == A_CONV, DmaConvA<BM, BK, NW>,
                                      DmaOperand<BM, BK, NW, AMODE == A_KCONTIG>>::type OpA;
    typedef DmaOperand<BN, BK, NW, TB> OpB;
    constexpr int A_ST = OpA::FLOATS, B_ST = OpB::FLOATS;
    constexpr int GSTAGES = STAGES * (A_ST + B_ST);  // floats of one group's stages
    constexpr int LPB = OpA::L + OpB::L;
    constexpr int ACCF = G::RM * G::RN * 16;  // accumulator floats per lane
    static_assert(STAGES >= 2 && STAGES <= 4, "two to four LDS stages");
    static_assert((STAGES - 2) * LPB <= 63, "vmcnt range");
    static_assert((KS - 1) * GT * ACCF <= KS * GSTAGES, "partial tiles fit in the stages");

    __shared__ __attribute__((aligned(16))) float smem[KS * GSTAGES];

    const int grp = __builtin_amdgcn_readfirstlane(threadIdx.x / GT);
    const int tid = threadIdx.x - grp * GT;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // within the group
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;
    float *gs = smem + grp * GSTAGES;

    if constexpr (AMODE != A_CONV) {
        if (p.nbatch > 1) {  // product blockIdx.y of a batch
            const int64_t bz = blockIdx.y;
            p.A += bz * p.stride_a;
            p.B += bz * p.stride_b;
            p.C += bz * p.stride_c;
        }
    }
    int tm, tn;
    tile_coords(p, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    int kbeg, kend;  // K-blocks of this work-group's split
    split_range(p, BK, blockIdx.z, kbeg, kend);
    const int steps = (kend - kbeg + KS - 1) / KS;  // K-block steps of every group
    const int klim = min(p.K, kend * BK);          // k past the split reads as zero

    OpA oa;
    OpB ob;
    if constexpr (AMODE == A_CONV)
        oa.init(p, m0, kbeg + grp, wave, lane);  // the gather walks this group's K-blocks, KS apart
    else
        oa.init(p.lda, m0, p.M, wave, lane);
    ob.init(p.ldb, n0, p.N, wave, lane);
    // step st of group g is K-block kbeg + st*KS + g; steps are issued in order
    auto issue = [&](int st, int s) {
        const int k0 = (kbeg + st * KS + grp) * BK;
        float *as = gs + s * (A_ST + B_ST);
        if constexpr (AMODE == A_CONV)
            oa.issue(p.A, k0, klim, as, wave, KS);
        else
            oa.issue(p.A, p.lda, m0, k0, klim, as, wave);
        ob.issue(p.B, p.ldb, n0, k0, klim, as + A_ST, wave);
    };
    auto wait_blocks = [&](int later) {
        if (STAGES >= 4 && later >= 2)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPB) : "memory");
        else if (STAGES >= 3 && later >= 1)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPB) : "memory");
        else
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    auto barrier = [] {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    auto read_group = [&](const float *as, int g, typename G::FragA &xa, typename G::FragB &xb) {
#pragma unroll
        for (int i = 0; i < G::RM; ++i) OpA::read4(as, a_row + i * 32, h, g, xa[i]);
#pragma unroll
        for (int j = 0; j < G::RN; ++j) OpB::read4(as + A_ST, b_row + j * 32, h, g, xb[j]);
    };

    typename G::Acc acc;
    G::zero(acc);
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NG = G::NG;

#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < steps) issue(s, s);
    wait_blocks(min(STAGES - 2, steps - 1));
    barrier();
    if (steps > 0) read_group(gs, 0, fa[0], fb[0]);

    int s = 0;
    for (int st = 0; st < steps; ++st) {
        const int s_next = s + 1 == STAGES ? 0 : s + 1;
        if (st + STAGES - 1 < steps) issue(st + STAGES - 1, s == 0 ? STAGES - 1 : s - 1);
        const float *as = gs + s * (A_ST + B_ST);
#pragma unroll
        for (int g = 0; g < NG - 1; ++g) {
            read_group(as, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            G::mma_group(acc, fa[g & 1], fb[g & 1]);
        }
        wait_blocks(min(STAGES - 2, steps - st - 2));
        barrier();
        // unconditional (stale after the last step, never used)
        read_group(gs + s_next * (A_ST + B_ST), 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NG - 1) & 1], fb[(NG - 1) & 1]);
        s = s_next;
    }

    // every copy has landed and every stage read is done before the partial
    // tiles of groups 1..KS-1 overwrite the stages; group 0 adds them in
    // group order and writes C
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    barrier();
    if (grp > 0) {
        float *slot = smem + (grp - 1) * GT * ACCF + tid;
#pragma unroll
        for (int i = 0; i < G::RM; ++i)
#pragma unroll
            for (int j = 0; j < G::RN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) slot[((i * G::RN + j) * 16 + r) * GT] = acc[i][j][r];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
        for (int q = 1; q < KS; ++q) {
            const float *slot = smem + (q - 1) * GT * ACCF + tid;
#pragma unroll
            for (int i = 0; i < G::RM; ++i)
#pragma unroll
                for (int j = 0; j < G::RN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[i][j][r] += slot[((i * G::RN + j) * 16 + r) * GT];
        }
        G::template store<BETA>(p, acc, m0 + wm * G::WM + 4 * h, n0 + wn * G::WN + l32, blockIdx.z);
    }
}

// Stream-K form of the direct-to-LDS contraction: the grid is the resident
// work-groups and each walks its share of the (tile, K-block) iterations as
// gemm_streamk_kernel does, with the copies issued STAGES-1 iterations ahead
// across tile boundaries (the operand helpers are set up again whenever the
// copies enter a new tile; the LDS stage ring runs on unbroken).  Partial
// tiles are published and finished by their last contributor in K order, as
// there.  The epilogue's stores count on the same vector-memory counter as
// the copies and retire in order, so a wait issued after them only waits
// longer, never too little.
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int AMODE, bool TB, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_dma_streamk_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, A_KCONTIG, false, 4, 4> G;  // MFMA and epilogue only
    constexpr int NT = G::NT, NW = NT / 64;
    typedef typename std::conditional<AMODE == A_CONV, DmaConvA<BM, BK, NW>,
                                      DmaOperand<BM, BK, NW, AMODE == A_KCONTIG>>::type OpA;
    typedef DmaOperand<BN, BK, NW, TB> OpB;
    constexpr int A_ST = OpA::FLOATS, B_ST = OpB::FLOATS;
    constexpr int LPB = OpA::L + OpB::L;
    static_assert(STAGES >= 2 && STAGES <= 4, "two to four LDS stages");
    static_assert((STAGES - 2) * LPB <= 63, "vmcnt range");

    __shared__ __attribute__((aligned(16))) float smem[STAGES * (A_ST + B_ST)];
    __shared__ int s_arrival;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;
    const int nkb = p.sk_nkb;
    const StreamK sk{p.tiles_m * p.tiles_n * nkb, (int)gridDim.x, nkb};

    // work-group b runs on XCD b % xcds: give each XCD a contiguous share of
    // the logical ranges, so the tiles an XCD works on are neighbours
    const int lg = sk_logical(blockIdx.x, sk.G, p.xcds);
    const int beg = sk.start(lg), end = sk.start(lg + 1);
    if (beg >= end) return;  // uniform over the work-group, before any barrier

    auto decode_tile = [&](int t, int &m0_, int &n0_) {
        int tm, tn;
        tile_of(p, t, tm, tn);
        m0_ = tm * BM;
        n0_ = tn * BN;
    };

    // producer: the next iteration to copy, its stage, and the tile the
    // operand helpers are set up for
    OpA oa;
    OpB ob;
    int pj = beg, ps = 0, p_tile = -1, pm0 = 0, pn0 = 0;
    // A's copies of iteration pj (setting the operand helpers up again when
    // it starts a new tile), then B's, which move the producer on
    auto issue_next_a = [&]() {
        const int t = pj / nkb, kb = pj - t * nkb;
        if (t != p_tile) {
            p_tile = t;
            decode_tile(t, pm0, pn0);
            if constexpr (AMODE == A_CONV)
                oa.init(p, pm0, kb, wave, lane);
            else
                oa.init(p.lda, pm0, p.M, wave, lane);
            ob.init(p.ldb, pn0, p.N, wave, lane);
        }
        float *as = smem + ps * (A_ST + B_ST);
        if constexpr (AMODE == A_CONV)
            oa.issue(p.A, kb * BK, p.K, as, wave);
        else
            oa.issue(p.A, p.lda, pm0, kb * BK, p.K, as, wave);
    };
    auto issue_next_b = [&]() {
        const int kb = pj - p_tile * nkb;
        float *as = smem + ps * (A_ST + B_ST);
        ob.issue(p.B, p.ldb, pn0, kb * BK, p.K, as + A_ST, wave);
        ++pj;
        ps = ps + 1 == STAGES ? 0 : ps + 1;
    };
    auto issue_next = [&]() {
        issue_next_a();
        issue_next_b();
    };
    auto wait_blocks = [&](int later) {
        if (STAGES >= 4 && later >= 2)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPB) : "memory");
        else if (STAGES >= 3 && later >= 1)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPB) : "memory");
        else
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    auto barrier = [] {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    auto read_group = [&](const float *as, int g, typename G::FragA &xa, typename G::FragB &xb) {
#pragma unroll
        for (int i = 0; i < G::RM; ++i) OpA::read4(as, a_row + i * 32, h, g, xa[i]);
#pragma unroll
        for (int j = 0; j < G::RN; ++j) OpB::read4(as + A_ST, b_row + j * 32, h, g, xb[j]);
    };

    typename G::Acc acc;
    G::zero(acc);
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NGR = G::NG;

    for (int i = 0; i < STAGES - 1 && pj < end; ++i) issue_next();
    int cj = beg, cs = 0;  // consumer: the iteration being multiplied and its stage
    wait_blocks(min(STAGES - 2, pj - cj - 1));
    barrier();
    read_group(smem, 0, fa[0], fb[0]);

    int tile = beg / nkb;
    int kbeg = beg - tile * nkb;
    int m0, n0;
    decode_tile(tile, m0, n0);
    for (;;) {
        // the copies of the next iteration in two bursts, as in gemm_dma_kernel
        const bool more = pj < end;
        if (more) issue_next_a();
        const float *as = smem + cs * (A_ST + B_ST);
        static_for<NGR - 1>([&](auto gc) {
            constexpr int g = decltype(gc)::value;
            read_group(as, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (g == 0) {
                G::mma_step(acc, fa[0], fb[0], 0);
                G::mma_step(acc, fa[0], fb[0], 1);
                if (more) issue_next_b();
                G::mma_step(acc, fa[0], fb[0], 2);
                G::mma_step(acc, fa[0], fb[0], 3);
            } else {
                G::mma_group(acc, fa[g & 1], fb[g & 1]);
            }
        });
        const int cs_next = cs + 1 == STAGES ? 0 : cs + 1;
        wait_blocks(min(STAGES - 2, pj - cj - 2));
        barrier();
        // unconditional (stale after the last iteration, never used)
        read_group(smem + cs_next * (A_ST + B_ST), 0, fa[0], fb[0]);
        __builtin_amdgcn_sched_barrier(0);
        G::mma_group(acc, fa[(NGR - 1) & 1], fb[(NGR - 1) & 1]);

        const int kb = cj - tile * nkb;
        if (kb == nkb - 1 || cj + 1 == end) {
            const int kend = kb + 1;
            const int row_base = m0 + wm * G::WM + 4 * h, col_base = n0 + wn * G::WN + l32;
            bool write = true;  // this work-group writes the tile's C block
            if (kbeg != 0 || kend != nkb) {
                // partial tile: publish this range's sum (layout and coherence
                // as in gemm_streamk_kernel), then the last contributor adds
                // all of them in K-block order
                float *mine = p.sk_part + (int64_t)sk.slot(lg, tile) * (BM * BN) + tid;
                asm volatile("" : "+v"(mine));
#pragma unroll
                for (int i = 0; i < G::RM; ++i)
#pragma unroll
                    for (int j = 0; j < G::RN; ++j)
#pragma unroll
                        for (int r = 0; r < 16; ++r)
                            __hip_atomic_store(mine + ((i * G::RN + j) * 16 + r) * NT, acc[i][j][r],
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores are complete
                __syncthreads();
                if (tid == 0)
                    s_arrival = __hip_atomic_fetch_add(p.sk_cnt + tile, 1, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                __syncthreads();
                const int lo = sk.owner(tile * nkb), hi = sk.owner(tile * nkb + nkb - 1);
                write = s_arrival == hi - lo;  // the last contributor: uniform over the work-group
                if (write) {
                    auto gather = [&](int g, bool first) {
                        const float *src = p.sk_part + (int64_t)sk.slot(g, tile) * (BM * BN) + tid;
                        asm volatile("" : "+v"(src));
#pragma unroll
                        for (int i = 0; i < G::RM; ++i)
#pragma unroll
                            for (int j = 0; j < G::RN; ++j)
#pragma unroll
                                for (int r = 0; r < 16; ++r) {
                                    const float v = __hip_atomic_load(src + ((i * G::RN + j) * 16 + r) * NT,
                                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                                    acc[i][j][r] = first ? v : acc[i][j][r] + v;
                                }
                    };
                    gather(lo, true);
                    for (int g = lo + 1; g <= hi; ++g) gather(g, false);
                }
            }
            if (write) G::template store<BETA>(p, acc, row_base, col_base, 0);
            G::zero(acc);
            if (cj + 1 < end) {
                tile = (cj + 1) / nkb;
                kbeg = 0;
                decode_tile(tile, m0, n0);
            }
        }
        if (cj + 1 == end) break;
        ++cj;
        cs = cs_next;
    }
}

// Contraction with op(B) resident in LDS, for short reductions (the 1x1
// convolutions of ResNet-50's bottlenecks: K = 64 input channels, N = 64 or
// 256 output channels).  There the whole of B is one K-block and at most
// 64 KB, while A and C stream through HBM once (8-16 flop per byte), so the
// time goes to memory, not to the MFMAs.  A persistent work-group loads one
// BN-column block of B once (stored n-major, k contiguous, for 16-byte
// operand reads), then walks a contiguous range of BM-row tiles of A.
// K == BK and N a multiple of BN (the launcher checks); M is arbitrary.
//
// Per tile t the A rows of tile t+2 are fetched into registers before tile
// t's C stores are issued, and stored to LDS only after tile t+1 has been
// multiplied.  The vector-memory counter orders loads and stores together,
// so that wait covers the loads alone, never the stores behind them: tile t's
// stores drain while tile t+1 multiplies.  For that count to be exact on
// every path nothing around the loads and stores is conditional: rows past M
// are fetched from row M-1 and zeroed on their way into LDS, and C is written
// with buffer stores whose out-of-range offset (rows past M) the hardware
// drops.  (beta != 0 keeps the generic epilogue, which reads C.)
template <int BM, int BN, int BK, int WAVES_M, int WAVES_N, int OCC, bool BETA>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(OCC, 8)))
gemm_bres_kernel(KernelArgs p)
{
    typedef GemmTile<BM, BN, BK, WAVES_M, WAVES_N, A_KCONTIG, true, 4, 4> G;
    constexpr int NT = G::NT;
    constexpr int CPR = BK / 4;              // 16-byte chunks per A row
    constexpr int AL = BM * BK / (4 * NT);   // A chunks per thread per tile
    static_assert(BN % 4 == 0 && (BK * BN / 4) % NT == 0, "B staging");
    static_assert(NT % CPR == 0 && AL >= 1 && AL <= 32 && (BM * BK) % (4 * NT) == 0, "A staging");

    __shared__ __attribute__((aligned(16))) float smem[2 * G::A_STAGE + G::B_STAGE];
    float *As = smem;                   // [2][BM][BK + PAD]
    float *Bs = smem + 2 * G::A_STAGE;  // [BN][BK + PAD]: B transposed

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int l32 = lane & 31, h = lane >> 5;

    // N = NCB column blocks of BN, each served by gridDim.x / NCB work-groups.
    // Work-group b serves block (b / X) % NCB (X = XCD count, a divisor of the
    // grid per block): the work-groups that walk the same rows for the other
    // blocks run on the same XCD, so A is fetched into its L2 once.
    const int ncb = p.N / BN;
    const int X = p.xcds > 1 ? p.xcds : 1;
    const int cb = (int)(blockIdx.x / X) % ncb;
    const int rg = (int)(blockIdx.x / (X * ncb)) * X + (int)(blockIdx.x % X);
    const int groups = (int)gridDim.x / ncb;
    const int n0 = cb * BN;
    const int tiles = (p.M + BM - 1) / BM;
    const int t0 = (int)(((int64_t)rg * tiles) / groups);
    const int t1 = (int)(((int64_t)(rg + 1) * tiles) / groups);
    if (t0 >= t1) return;  // uniform over the work-group, before any barrier

    // B: BK x BN row-major in global memory -> Bs[n][k].  Chunk c (4 columns
    // of one row) goes to a lane so that a wave covers 16 consecutive k of 4
    // adjacent column chunks: its transposed writes then fall in 64 distinct
    // banks (4 columns apart is 4 * (BK + 4) = 16 mod 64 banks), and its
    // global reads are 64-byte runs of 16 rows.  (Consecutive lanes on
    // consecutive column chunks would land a wave's writes in 4 banks.)
    static_assert(BK % 16 == 0 && BN % 16 == 0, "B staging by 16 k x 4 chunks");
#pragma unroll
    for (int i = 0; i < BK * BN / 4 / NT; ++i) {
        const int c = tid + i * NT;
        const int rest = c / 64;
        const int k = (rest % (BK / 16)) * 16 + c % 16;
        const int n = ((rest / (BK / 16)) * 4 + (c / 16) % 4) * 4;
        const f32x4 v = *reinterpret_cast<const f32x4 *>(p.B + (int64_t)k * p.ldb + n0 + n);
        Bs[(n + 0) * G::LDB_S + k] = v[0];
        Bs[(n + 1) * G::LDB_S + k] = v[1];
        Bs[(n + 2) * G::LDB_S + k] = v[2];
        Bs[(n + 3) * G::LDB_S + k] = v[3];
    }

    // this thread's A chunks: row (tid + i*NT) / CPR of the tile, columns col .. col+3
    const int col = (tid % CPR) * 4;
    f32x4 ra[AL];
    unsigned inside = 0;  // bit i: chunk i's row is below M
    auto load_a = [&](int t) {
        inside = 0;
#pragma unroll
        for (int i = 0; i < AL; ++i) {
            const int row = t * BM + (tid + i * NT) / CPR;
            const bool ok = row < p.M;
            ra[i] = *reinterpret_cast<const f32x4 *>(p.A + (int64_t)(ok ? row : p.M - 1) * p.lda + col);
            inside |= (unsigned)ok << i;
        }
    };
    auto write_a = [&](float *stage) {
#pragma unroll
        for (int i = 0; i < AL; ++i) {
            const f32x4 v = ((inside >> i) & 1u) ? ra[i] : f32x4{0.f, 0.f, 0.f, 0.f};
            *reinterpret_cast<f32x4 *>(stage + ((tid + i * NT) / CPR) * G::LDA_S + col) = v;
        }
    };

    load_a(t0);
    write_a(As);
    if (t0 + 1 < t1) load_a(t0 + 1);
    // nothing of the set-up stays in flight into the loop: the loop then only
    // ever waits for the loads it issued itself, which precede its stores
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    const int a_row = wm * G::WM + l32;
    const int b_row = wn * G::WN + l32;
    typename G::FragA fa[2];
    typename G::FragB fb[2];
    constexpr int NGR = G::NG;
    // C(t*BM + wm*WM + 4h + i*32 + 8*(r/4) + r%4, wn*WN + l32 + 32j) = acc[i][j][r]: a
    // wave-uniform part plus this lane's offset
    const unsigned c_lane = 4u * (unsigned)h * (unsigned)p.ldc + (unsigned)(n0 + wn * G::WN + l32);
    const float alpha = p.alpha;

    // Stores q = [Q0, Q1) of tile t's results: q = (i*16 + r)*RN + j.
    constexpr int NQ = G::RM * 16 * G::RN;
    auto store_range = [&](const typename G::Acc &acc, int t, auto q0_c, auto q1_c) {
        constexpr int Q0 = decltype(q0_c)::value, Q1 = decltype(q1_c)::value;
        const __amdgpu_buffer_rsrc_t cres =
            __builtin_amdgcn_make_buffer_rsrc(p.C + (int64_t)t * BM * p.ldc, (short)0, 0x7fffffff, 0x00020000);
#pragma unroll
        for (int q = Q0; q < Q1; ++q) {
            const int j = q % G::RN, r = (q / G::RN) % 16, i = q / (16 * G::RN);
            const int dr = wm * G::WM + i * 32 + 8 * (r >> 2) + (r & 3);  // row in the tile, less 4h
            const bool ok = t * BM + dr + 4 * h < p.M;
            const unsigned e = (unsigned)(dr * p.ldc + 32 * j) + c_lane;
            // the builtin's data operand is a 32-bit integer: pass the float's bits
            const float val = alpha * acc[i][j][r];
            // non-temporal (cache policy 2): C is not read again by this launch
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, val), cres, ok ? 4u * e : 0x80000000u,
                                                  0, 2);
        }
    };
    // The MFMAs of one tile (A from stage `as`) into acc; with PREV, the
    // stores of the previous tile's results (prev) are issued in slices
    // between the MFMA groups, so no wave ever waits at a barrier or issues
    // its stores while its SIMD's matrix pipe has nothing to do.
    auto mma_tile = [&](const float *as, typename G::Acc &acc, const typename G::Acc &prev, int tprev, auto with_prev) {
        constexpr bool PREV = decltype(with_prev)::value;
        G::read_group(as, Bs, a_row, b_row, h, 0, fa[0], fb[0]);
        G::zero(acc);
        constexpr int SPG = (NQ + NGR - 1) / NGR;  // stores per group
        [&]<int... G_>(std::integer_sequence<int, G_...>) {
            (
                [&] {
                    constexpr int g = G_;
                    if (g + 1 < NGR) G::read_group(as, Bs, a_row, b_row, h, g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
                    __builtin_amdgcn_sched_barrier(0);
                    G::mma_group(acc, fa[g & 1], fb[g & 1]);
                    if constexpr (PREV) {
                        constexpr int q0 = g * SPG < NQ ? g * SPG : NQ;
                        constexpr int q1 = (g + 1) * SPG < NQ ? (g + 1) * SPG : NQ;
                        store_range(prev, tprev, std::integral_constant<int, q0>{}, std::integral_constant<int, q1>{});
                    }
                }(),
                ...);
        }(std::make_integer_sequence<int, NGR>{});
    };
    auto store_all = [&](const typename G::Acc &acc, int t) {
        if constexpr (BETA)
            G::template store<true>(p, acc, t * BM + wm * G::WM + 4 * h, n0 + wn * G::WN + l32, 0);
        else
            store_range(acc, t, std::integral_constant<int, 0>{}, std::integral_constant<int, NQ>{});
    };
    // After tile t: its successor's A rows into the other stage, the barrier
    // that also ends every wave's reads of tile t's stage, then the loads of
    // tile t+2 (issued before any store of tile t).
    auto advance = [&](int t, int stage) {
        if (t + 1 < t1) write_a(As + (stage ^ 1) * G::A_STAGE);
        __syncthreads();
        if (t + 2 < t1) load_a(t + 2);
    };

    typename G::Acc acc0, acc1;
    if constexpr (BETA) {
        // beta != 0 reads C in its epilogue: tiles one after the other
        int stage = 0;
        for (int t = t0; t < t1; ++t) {
            mma_tile(As + stage * G::A_STAGE, acc0, acc1, 0, std::false_type{});
            advance(t, stage);
            store_all(acc0, t);
            stage ^= 1;
        }
    } else {
        mma_tile(As, acc0, acc1, 0, std::false_type{});
        advance(t0, 0);
        int t = t0 + 1, stage = 1;
        // tiles in pairs so that each accumulator set has a fixed name
        for (;;) {
            if (t >= t1) {
                store_all(acc0, t - 1);
                break;
            }
            mma_tile(As + stage * G::A_STAGE, acc1, acc0, t - 1, std::true_type{});
            advance(t, stage);
            ++t;
            stage ^= 1;
            if (t >= t1) {
                store_all(acc1, t - 1);
                break;
            }
            mma_tile(As + stage * G::A_STAGE, acc0, acc1, t - 1, std::true_type{});
            advance(t, stage);
            ++t;
            stage ^= 1;
        }
    }
}

}  // namespace pk
