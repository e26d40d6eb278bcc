/*
 * pk.h -- parameterized fp32 GEMM and 2-D convolution forward for AMD
 * Instinct MI355X (gfx950).
 *
 * The operations are those of "Cross-Platform Performance Portability Using
 * Highly Parametrized SYCL Kernels" (Lawson et al., arXiv 1904.05347):
 *   - GEMM, Section 3.1: C = alpha * op(A) * op(B) + beta * C, with op the
 *     identity or the transpose;
 *   - convolution forward, Section 4.1 (Algorithm 1 and the centred-window
 *     formula after it): an NHWC input, an HWIO filter (the paper's
 *     H x W x C input, R x S x C x K filter), cross-correlation (no filter
 *     flip), with the stride and window of the paper's layer tables and
 *     explicit zero padding.
 *
 * Conventions shared by every call:
 *   - Every tensor pointer is a DEVICE pointer to fp32 data.  The caller owns
 *     all memory; the library allocates no device memory and keeps no pointer
 *     after a call returns.
 *   - Storage is row-major (C order).  A column-major caller maps onto the
 *     same call by swapping the operands: the column-major product
 *     C = alpha op(A) op(B) + beta C is pk_sgemm(transB, transA, N, M, K,
 *     alpha, B, ldb, A, lda, beta, C, ldc).
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls are
 *     asynchronous and ordered on that stream; results are valid once it
 *     has synchronised.  No call synchronises the device.
 *   - Outputs must not overlap inputs.
 *   - Every call returns a pk_status.  Invalid arguments are detected before
 *     any work is queued; pk_last_invalid_param() then names the 1-based
 *     position of the offending argument.  Nothing aborts and no C++
 *     exception crosses this interface.
 *   - Thread safety: calls may come from several host threads at once.  The
 *     "last" queries below report the calling thread's most recent call.
 */
#ifndef PK_H
#define PK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PK_OK = 0,
    PK_ERR_INVALID_VALUE = 1, /* an argument is out of range; see pk_last_invalid_param() */
    PK_ERR_NOT_SUPPORTED = 2, /* a well-formed request this library does not implement */
    PK_ERR_WORKSPACE = 3,     /* a forced split-K or stream-K configuration lacks workspace */
    PK_ERR_LAUNCH = 4,        /* the HIP runtime refused a kernel launch */
    PK_ERR_SCRATCH_LIMIT = 5  /* pk_conv2d_fwd_noalloc: the call needs more scratch than the
                                 library's static buffer holds (PK_NOALLOC_SCRATCH_BYTES) */
} pk_status;

/*
 * Single-precision GEMM (Section 3.1):  C <- alpha * op(A) * op(B) + beta * C.
 *
 *   transA, transB  'N'/'n' (op = identity) or 'T'/'t'/'C'/'c' (op = transpose;
 *                   'C' equals 'T' for real data).
 *   M, N, K         op(A) is M x K, op(B) is K x N, C is M x N.  Each >= 0.
 *   A, lda          row-major; M x K with lda >= max(1, K) for 'N',
 *                   K x M with lda >= max(1, M) for 'T'.
 *   B, ldb          row-major; K x N with ldb >= max(1, N) for 'N',
 *                   N x K with ldb >= max(1, K) for 'T'.
 *   C, ldc          row-major M x N, ldc >= max(1, N).  Read only if beta != 0.
 *
 * Quick returns (netlib BLAS semantics): M == 0 or N == 0 does nothing;
 * alpha == 0 or K == 0 sets C <- beta * C without reading A or B;
 * beta == 0 writes C without reading it, so NaN or Inf in C is not propagated.
 * A and B may be NULL only when they are not read.
 * Results are deterministic: the same call on the same device gives the same
 * bits (no atomics; any split of K is reduced in a fixed order).
 */
int pk_sgemm(char transA, char transB, int64_t M, int64_t N, int64_t K,
             float alpha, const float *A, int64_t lda,
             const float *B, int64_t ldb,
             float beta, float *C, int64_t ldc, void *stream);

/*
 * Bytes of device workspace that lets pk_sgemm_ws split the reduction K of
 * this product across work-groups, for the configuration the next
 * pk_sgemm_ws call on this thread would choose with 16-byte aligned, tightly
 * packed operands (a forced one included); 0 when that configuration needs
 * none.  A split keeps one M x N partial sum per slice of K; a stream-K
 * configuration two partial tiles per resident work-group and one arrival
 * counter per tile of C.  Products whose tiles fill the CUs take no split.
 * Host-only apart from an occupancy query of the kernel.
 */
size_t pk_sgemm_workspace_bytes(char transA, char transB, int64_t M, int64_t N, int64_t K);

/*
 * pk_sgemm with a workspace (the same operation, arguments, quick returns
 * and determinism; error positions as there, then 14 = workspace).
 *   workspace    optional device buffer of workspace_bytes; with at least
 *                pk_sgemm_workspace_bytes() a product with few tiles of C
 *                and a long K may split K across work-groups (the partial
 *                products, each alpha-scaled, are added in slice order by a
 *                second kernel that also applies beta * C) or run stream-K
 *                (16-byte alignment needed).  NULL / too small selects a
 *                configuration and split that need none.  It must not
 *                overlap A, B or C.  Contents on return are unspecified.
 *                Two calls that overlap in time must not share a workspace.
 */
int pk_sgemm_ws(char transA, char transB, int64_t M, int64_t N, int64_t K,
                float alpha, const float *A, int64_t lda,
                const float *B, int64_t ldb,
                float beta, float *C, int64_t ldc,
                void *workspace, size_t workspace_bytes, void *stream);

/*
 * Output size of a convolution window (the stride S and window W columns of
 * the paper's layer tables): Ho = floor((H + pt + pb - KH) / sh) + 1, and the
 * same for Wo.  Pads >= 0, strides >= 1, window >= 1 and not larger than the
 * padded image.  Host-only; touches no GPU.
 */
int pk_conv2d_out_dims(int64_t H, int64_t W, int64_t KH, int64_t KW,
                       int64_t sh, int64_t sw, int64_t pt, int64_t pl,
                       int64_t pb, int64_t pr, int64_t *Ho, int64_t *Wo);

/*
 * "SAME" padding: the output keeps ceil(H / sh) x ceil(W / sw) pixels and the
 * least total padding that gives it is split with the odd pixel at the
 * bottom/right.  pads_tlbr receives {top, left, bottom, right}.  Host-only.
 */
int pk_conv2d_same_pads(int64_t H, int64_t W, int64_t KH, int64_t KW,
                        int64_t sh, int64_t sw, int64_t pads_tlbr[4]);

/*
 * Bytes of device workspace that lets pk_conv2d_fwd split the reduction
 * (KH * KW * Cin) of this problem across work-groups, for the configuration
 * the next pk_conv2d_fwd call on this thread would choose (a forced one
 * included); 0 when that configuration needs none.  A split-K configuration
 * keeps one partial sum of y per slice of the reduction; a stream-K one keeps
 * two partial tiles per resident work-group and one arrival counter per tile
 * of y.  Host-only apart from an occupancy query of the kernel.
 */
size_t pk_conv2d_workspace_bytes(int64_t N, int64_t H, int64_t W, int64_t Cin,
                                 int64_t KH, int64_t KW, int64_t Cout,
                                 int64_t sh, int64_t sw, int64_t pt, int64_t pl,
                                 int64_t pb, int64_t pr);

/*
 * 2-D convolution forward (Section 4.1, Algorithm 1 with a centred, zero-
 * padded window):
 *   y[n][ho][wo][co] = sum_{kh, kw, ci} x~[n][ho*sh - pt + kh][wo*sw - pl + kw][ci]
 *                                       * f[kh][kw][ci][co]
 * where x~ is x inside the H x W image and 0 outside.
 *
 *   x            N x H x W x Cin, contiguous (NHWC).
 *   f            KH x KW x Cin x Cout, contiguous (HWIO).
 *   sh, sw       strides >= 1.  pt, pl, pb, pr: zero padding >= 0.
 *   y            N x Ho x Wo x Cout, contiguous (NHWC).  Ho, Wo must equal
 *                pk_conv2d_out_dims() of the geometry (else INVALID_VALUE).
 *   workspace    optional device buffer of workspace_bytes, 16-byte aligned;
 *                with at least pk_conv2d_workspace_bytes() the reduction may
 *                be split across work-groups (split-K, or stream-K: equal
 *                shares of the (tile, K-block) iterations per resident
 *                work-group, partial tiles finished by their last
 *                contributor).  NULL / too small selects a configuration
 *                that needs none.  Contents on return are unspecified.  Two
 *                calls that overlap in time must not share a workspace.
 * N == 0 does nothing.  Dilation, groups, bias and activation are not part
 * of this operation.
 */
int pk_conv2d_fwd(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                  const float *f, int64_t KH, int64_t KW, int64_t Cout,
                  int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb, int64_t pr,
                  float *y, int64_t Ho, int64_t Wo,
                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * pk_conv2d_fwd for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * It runs exactly what pk_conv2d_fwd runs when given the workspace that
 * pk_conv2d_workspace_bytes() asks for (same configuration, split and
 * results, bit for bit), with that workspace taken from a static device
 * buffer of PK_NOALLOC_SCRATCH_BYTES that the library holds on every device
 * it runs on until the process ends.  It calls no hipMalloc, hipFree or
 * other allocating routine.
 *
 * Arguments, layouts, quick returns and argument positions of errors are
 * those of pk_conv2d_fwd without the workspace pair.  A call whose
 * workspace would exceed PK_NOALLOC_SCRATCH_BYTES returns
 * PK_ERR_SCRATCH_LIMIT before any work is queued (pass a workspace to
 * pk_conv2d_fwd instead).  The first call on a device looks up that device's
 * copy of the buffer (no allocation, no stream work).
 * Every call on one device shares that device's buffer: calls that overlap
 * in time on one device (two streams, two host threads) race on it and must
 * be serialised by the caller.  The buffer keeps the last call's contents;
 * each call clears what it needs zeroed with a kernel on `stream`.
 */
#define PK_NOALLOC_SCRATCH_BYTES ((size_t)80 << 20)
int pk_conv2d_fwd_noalloc(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                          const float *f, int64_t KH, int64_t KW, int64_t Cout,
                          int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb, int64_t pr,
                          float *y, int64_t Ho, int64_t Wo, void *stream);

/*
 * Winograd convolution F(2x2, 3x3) (Section 4.1.2, the transform technique
 * the paper takes from Lavin and Gray): the same operation as pk_conv2d_fwd
 * for a 3 x 3 window at stride 1, computed as
 *   U = G g G^T per (ci, co) filter,  V = B^T d B per 4 x 4 input tile d and
 *   channel,  M[p] = V[p] U[p] for the 16 positions p of the transformed
 *   tile (one batched product, Cin deep),  y = A^T m A per 2 x 2 output block,
 * with 2.25x fewer multiplications than the direct sum.  Its fp32 rounding
 * differs from the direct sum's: each output is accurate to 1e-5 times the
 * same chain evaluated on absolute values (matrix entries and operands).
 *
 * Arguments, layouts and argument positions of errors are those of
 * pk_conv2d_fwd.  KH = KW = 3 and sh = sw = 1 are required (else
 * PK_ERR_NOT_SUPPORTED); any padding >= 0.
 *   workspace    REQUIRED device buffer, 16-byte aligned, of at least
 *                pk_conv2d_winograd_workspace_bytes() bytes (else
 *                PK_ERR_WORKSPACE; misaligned: PK_ERR_INVALID_VALUE at 19).
 *                It holds the transformed filter, input and products;
 *                contents on return are unspecified.  It must not overlap
 *                x, f or y.
 * pk_last_config_name() names the contraction configuration of the product.
 */
size_t pk_conv2d_winograd_workspace_bytes(int64_t N, int64_t H, int64_t W, int64_t Cin,
                                          int64_t Cout, int64_t pt, int64_t pl,
                                          int64_t pb, int64_t pr);
int pk_conv2d_winograd_fwd(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                           const float *f, int64_t KH, int64_t KW, int64_t Cout,
                           int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb, int64_t pr,
                           float *y, int64_t Ho, int64_t Wo,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * Winograd convolution F(m x m, 3x3) with the output-tile size m as a
 * parameter (Section 4.1.2: the tile size trades fewer multiplications for
 * larger transform coefficients and smaller batched products), m = 2 or 4.
 * m = 2 is pk_conv2d_winograd_fwd.  m = 4 uses the published Lavin-Gray
 * F(4, 3) matrices (interpolation points 0, 1, -1, 2, -2 and infinity):
 * 6 x 6 input tiles, 36 batched products of (T x Cin)(Cin x Cout) with
 * T = N * ceil(Ho/4) * ceil(Wo/4), 4x fewer multiplications than the
 * direct sum.  Accuracy: 1e-5 times the transform chain evaluated on
 * absolute values (larger for m = 4: its matrices have entries up to 8 and
 * the non-dyadic 1/6, 1/12, 1/24).
 *
 * Arguments and error positions are those of pk_conv2d_winograd_fwd with m
 * inserted at position 19 (m not 2 or 4: PK_ERR_INVALID_VALUE at 19), so
 * the workspace is argument 20 (misaligned: PK_ERR_INVALID_VALUE at 20).
 * pk_conv2d_winograd_tile_workspace_bytes returns 0 for an m other than 2, 4.
 */
size_t pk_conv2d_winograd_tile_workspace_bytes(int64_t m, int64_t N, int64_t H, int64_t W,
                                               int64_t Cin, int64_t Cout, int64_t pt,
                                               int64_t pl, int64_t pb, int64_t pr);
int pk_conv2d_winograd_tile_fwd(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                                const float *f, int64_t KH, int64_t KW, int64_t Cout,
                                int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb,
                                int64_t pr, float *y, int64_t Ho, int64_t Wo, int64_t m,
                                void *workspace, size_t workspace_bytes, void *stream);

/*
 * Automated parameter search: the measured, per-device choice of a compiled
 * configuration that the paper makes by hand for each of its devices
 * (Section 5) and plans to automate (Section 7).  Every compiled
 * configuration that takes the problem (the single-LDS-stage ablation forms
 * excepted) -- with each split of the reduction in {1, 2, 3, 4, 6, 8, 12,
 * 16} and the configuration's own rule split that the workspace holds (none
 * for stream-K, B-resident and direct forms) -- runs one untimed call and then three
 * timed runs of `iters` calls (more for short calls: up to about 1 ms per
 * run) on the caller's operands, on `stream` (HIP events; the median run
 * counts); the fastest is recorded in a process-wide
 * table that later calls with the same key consult before the built-in
 * choices:
 *   GEMM: (transA, transB, M, N, K);
 *   convolution: (N*Ho*Wo, Cout, KH*KW*Cin, window, stride), KH == KW and
 *   sh == sw only (else PK_ERR_NOT_SUPPORTED after validation).
 * The call synchronizes the stream.  C (y) is written many times: with
 * beta != 0 its final contents are unspecified, so pass a scratch C.
 * Arguments and error positions are those of pk_sgemm_ws / pk_conv2d_fwd, then
 * iters (>= 1), stream, result (non-NULL).  An empty problem records
 * nothing (result->config is "").  The table holds 256 entries (else
 * PK_ERR_NOT_SUPPORTED); pk_tune_reset() empties it.
 */
typedef struct {
    char config[64];   /* fastest configuration's name */
    int splits;        /* split of the reduction it ran with (1 = none) */
    float ms;          /* its mean time per call */
    int candidates;    /* (configuration, split) pairs timed */
} pk_tune_result;

int pk_tune_sgemm(char transA, char transB, int64_t M, int64_t N, int64_t K,
                  float alpha, const float *A, int64_t lda, const float *B, int64_t ldb,
                  float beta, float *C, int64_t ldc,
                  void *workspace, size_t workspace_bytes,
                  int iters, void *stream, pk_tune_result *result);
int pk_tune_conv2d_fwd(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                       const float *f, int64_t KH, int64_t KW, int64_t Cout,
                       int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb, int64_t pr,
                       float *y, int64_t Ho, int64_t Wo,
                       void *workspace, size_t workspace_bytes,
                       int iters, void *stream, pk_tune_result *result);
int pk_tune_reset(void);

/* Static text for a status code. */
const char *pk_status_string(int status);

/* 1-based argument position of this thread's last PK_ERR_INVALID_VALUE, 0 if none. */
int pk_last_invalid_param(void);

/* Name of the compiled configuration this thread's last pk_sgemm or
 * pk_conv2d_fwd call ran ("" after an error or an empty problem, "scale" for
 * C <- beta * C).  Static storage. */
const char *pk_last_config_name(void);

/*
 * The compiled tile-parameter space.  Each configuration is one kernel
 * instance: work-group tile BM x BN, K-block depth BK, a wave grid, the
 * operand layouts it reads, its vector load widths and its LDS footprint.
 */
typedef struct {
    const char *name;
    int kind;        /* 0 = GEMM, 1 = implicit-GEMM convolution, 2 = tiled direct convolution */
    int bm, bn, bk;  /* work-group tile and K-block depth */
    int waves_m, waves_n; /* wave grid; each wave owns (bm/waves_m) x (bn/waves_n) */
    int threads;     /* work-group size */
    int trans_a, trans_b; /* operand layouts read (1 = transposed storage) */
    int vec_a, vec_b; /* elements per global load */
    int stages;      /* LDS buffers (2 = double buffered, 3 = two K-blocks in flight) */
    int lds_bytes;   /* LDS per work-group */
    int occupancy;   /* waves per SIMD its registers are allotted for (1 = unconstrained) */
    int persistent;  /* 1 = one work-group per resident slot, each looping over tiles */
    int streamk;     /* 1 = stream-K: resident work-groups share the (tile, K-block) iterations
                        evenly; convolution calls only (it needs the workspace) */
    int bres;        /* 1 = op(B) held whole in LDS while row tiles of A stream past; runs
                        only products with K == bk and N == bn (op(A) = A, op(B) = B) */
    int kgroups;     /* groups of waves splitting K inside one work-group (1 = none); their
                        partial tiles are added through LDS in group order */
    int dma;         /* 1 = operands copied straight from global memory into LDS (no
                        staging registers, unpadded swizzled tiles, `stages` of them) */
} pk_config_info;

int pk_num_configs(void);
/* Fills *info for configuration idx (0 <= idx < pk_num_configs()). */
int pk_get_config(int idx, pk_config_info *info);

/*
 * Forces every later call on this thread to use the named configuration
 * (NULL or "" restores the selector).  A forced configuration that cannot run
 * a given call (wrong layout, alignment, kind) makes that call return
 * PK_ERR_NOT_SUPPORTED.  Unknown names give PK_ERR_INVALID_VALUE.  The
 * environment variable PK_FORCE_CONFIG, read at first use, sets the same
 * override for threads that never call this; if it names no configuration,
 * every pk_sgemm(_ws) / pk_conv2d_fwd call returns PK_ERR_INVALID_VALUE with
 * pk_last_invalid_param() == 0.
 */
int pk_force_config(const char *name);

/* Forces the split of the reduction across work-groups of later
 * pk_sgemm_ws and convolution calls on this thread (0 restores the
 * selector's choice; 1 = no split).  A forced split needs workspace for
 * every slice (else PK_ERR_WORKSPACE); B-resident configurations take none
 * (PK_ERR_NOT_SUPPORTED); stream-K configurations ignore it. */
int pk_force_splits(int splits);

/*
 * Measurement probes (not part of the operations above): they give the
 * denominators against which the kernels are judged.
 *
 * pk_probe_mfma_peak: `blocks` work-groups of 256 threads, each wave issuing
 * `iters` x 4 independent v_mfma_f32_32x32x2_f32 (4096 flops each) with no
 * memory traffic; one float per thread is written to out (blocks * 256
 * floats, device memory).  Flops = blocks * 4 * iters * 4 * 4096.
 * pk_probe_mfma_data: the same with operands that differ on every MFMA
 * (random values read once from src, which holds at least 2^20 floats):
 * blocks * 4 * iters * 16 MFMAs of 4096 flops.
 * pk_probe_copy: dst[0:n] = src[0:n] with 16-byte accesses; n a multiple of 4,
 * both pointers 16-byte aligned device memory.  Bytes moved = 8 * n.
 * Both are asynchronous on `stream` and return PK_ERR_INVALID_VALUE on bad
 * arguments (without setting pk_last_invalid_param).
 */
int pk_probe_mfma_peak(int blocks, int iters, float *out, void *stream);
int pk_probe_mfma_data(int blocks, int iters, const float *src, float *out, void *stream);
int pk_probe_copy(const float *src, float *dst, int64_t n, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PK_H */
