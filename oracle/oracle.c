/*
 * oracle.c -- plain CPU reference for the fp32 GEMM and the NHWC/HWIO 2-D
 * convolution forward of "Cross-Platform Performance Portability Using Highly
 * Parametrized SYCL Kernels" (Lawson et al., arXiv 1904.05347).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this file; only the tests, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no code with the HIP kernels.
 *
 * Everything here is the plain definition written out, one output element at
 * a time, accumulated in double precision:
 *   - GEMM (Section 3.1, the displayed definition of C = alpha op(A) op(B) +
 *     beta C): ref(i,j) = alpha * sum_k opA(i,k) * opB(k,j) + beta * C(i,j).
 *   - Convolution (Section 4.1, Algorithm 1 and the centred-window formula
 *     that follows it): out(n,ho,wo,co) = sum_{kh,kw,ci} X~(n, ho*sh - pt + kh,
 *     wo*sw - pl + kw, ci) * F(kh,kw,ci,co), where X~ is zero outside the
 *     image.  No filter flip (cross-correlation, as the formula pairs input
 *     tap (x,y) with filter tap (x,y)).
 * Alongside each value it returns scale = sum |product|, the magnitude against
 * which an fp32 result is judged (|gpu - ref| <= 1e-5 * scale).
 * The Winograd F(2x2, 3x3) and F(4x4, 3x3) steps of Section 4.1.2 follow at
 * the end of the file, with their own scale (the same steps on absolute
 * values).
 *
 * Storage is row-major (C order).  For GEMM: A is M x K (lda >= K) when
 * transA is 'N', K x M (lda >= M) when 'T'; B is K x N (ldb >= N) or N x K
 * (ldb >= K); C is M x N (ldc >= N).  'C' is read as 'T' (real data).
 * netlib conventions: alpha == 0 or K == 0 leaves beta * C and reads neither
 * A nor B; beta == 0 does not read C.
 *
 * Products of two fp32 values are exact in double (48 significant bits), so
 * the only rounding is the double-precision summation.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_BAD_ARG 1

static int trans_flag(char t)
{
    if (t == 'N' || t == 'n') return 0;
    if (t == 'T' || t == 't' || t == 'C' || t == 'c') return 1;
    return -1;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------ GEMM */

/* op(A)(i,k): A itself when not transposed, else A stored K x M. */
static double op_a(const float *A, int64_t lda, int ta, int64_t i, int64_t k)
{
    return ta ? (double)A[k * lda + i] : (double)A[i * lda + k];
}

/* op(B)(k,j): B itself when not transposed, else B stored N x K. */
static double op_b(const float *B, int64_t ldb, int tb, int64_t k, int64_t j)
{
    return tb ? (double)B[j * ldb + k] : (double)B[k * ldb + j];
}

static void gemm_element(int ta, int tb, int64_t K, double alpha,
                         const float *A, int64_t lda, const float *B, int64_t ldb,
                         double beta, const float *C, int64_t ldc,
                         int64_t i, int64_t j, double *ref, double *scale)
{
    double s = 0.0, t = 0.0;
    if (alpha != 0.0) {
        for (int64_t k = 0; k < K; ++k) {
            double p = op_a(A, lda, ta, i, k) * op_b(B, ldb, tb, k, j);
            s += p;
            t += fabs(p);
        }
    }
    double r = alpha * s;
    if (beta != 0.0) r += beta * (double)C[i * ldc + j];
    *ref = r;
    *scale = t;
}

static int gemm_args_ok(int ta, int tb, int64_t M, int64_t N, int64_t K,
                        int64_t lda, int64_t ldb, int64_t ldc)
{
    if (ta < 0 || tb < 0 || M < 0 || N < 0 || K < 0) return 0;
    int64_t a_cols = ta ? M : K, b_cols = tb ? K : N;
    if (lda < (a_cols > 1 ? a_cols : 1)) return 0;
    if (ldb < (b_cols > 1 ? b_cols : 1)) return 0;
    if (ldc < (N > 1 ? N : 1)) return 0;
    return 1;
}

/* Full product: ref and scale are M x N, row-major, leading dimension N. */
int oracle_sgemm(char transA, char transB, int64_t M, int64_t N, int64_t K,
                 float alpha, const float *A, int64_t lda,
                 const float *B, int64_t ldb,
                 float beta, const float *C, int64_t ldc,
                 double *ref, double *scale)
{
    int ta = trans_flag(transA), tb = trans_flag(transB);
    if (!gemm_args_ok(ta, tb, M, N, K, lda, ldb, ldc)) return ORACLE_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            gemm_element(ta, tb, K, (double)alpha, A, lda, B, ldb, (double)beta,
                         C, ldc, i, j, &ref[i * N + j], &scale[i * N + j]);
    return ORACLE_OK;
}

/* Selected elements (rows[s], cols[s]) only, for sizes too large to do whole. */
int oracle_sgemm_at(char transA, char transB, int64_t M, int64_t N, int64_t K,
                    float alpha, const float *A, int64_t lda,
                    const float *B, int64_t ldb,
                    float beta, const float *C, int64_t ldc,
                    int64_t count, const int64_t *rows, const int64_t *cols,
                    double *ref, double *scale)
{
    int ta = trans_flag(transA), tb = trans_flag(transB);
    if (!gemm_args_ok(ta, tb, M, N, K, lda, ldb, ldc)) return ORACLE_BAD_ARG;
    for (int64_t s = 0; s < count; ++s)
        if (rows[s] < 0 || rows[s] >= M || cols[s] < 0 || cols[s] >= N) return ORACLE_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t s = 0; s < count; ++s)
        gemm_element(ta, tb, K, (double)alpha, A, lda, B, ldb, (double)beta,
                     C, ldc, rows[s], cols[s], &ref[s], &scale[s]);
    return ORACLE_OK;
}

/* ----------------------------------------------------------- convolution */

/* Output size of a window KH x KW moved with stride sh x sw over an image
 * zero-padded by pt/pb rows and pl/pr columns: floor((H + pt + pb - KH)/sh)+1.
 * The layer tables of Section 5 fix this reading: 3x3 stride 1 keeps the
 * size with one pixel of padding, 7x7 stride 2 maps 230 to 112 unpadded. */
int oracle_conv2d_out_dims(int64_t H, int64_t W, int64_t KH, int64_t KW,
                           int64_t sh, int64_t sw, int64_t pt, int64_t pl,
                           int64_t pb, int64_t pr, int64_t *Ho, int64_t *Wo)
{
    if (H < 0 || W < 0 || KH < 1 || KW < 1 || sh < 1 || sw < 1 ||
        pt < 0 || pl < 0 || pb < 0 || pr < 0)
        return ORACLE_BAD_ARG;
    int64_t hspan = H + pt + pb - KH, wspan = W + pl + pr - KW;
    if (hspan < 0 || wspan < 0) return ORACLE_BAD_ARG;
    *Ho = hspan / sh + 1;
    *Wo = wspan / sw + 1;
    return ORACLE_OK;
}

/* "SAME" padding: output size ceil(H/s); the total padding
 * max((Ho-1)*s + KH - H, 0) is split with the smaller half on top/left. */
int oracle_same_pads(int64_t H, int64_t W, int64_t KH, int64_t KW,
                     int64_t sh, int64_t sw, int64_t pads_tlbr[4])
{
    if (H < 1 || W < 1 || KH < 1 || KW < 1 || sh < 1 || sw < 1) return ORACLE_BAD_ARG;
    int64_t ho = (H + sh - 1) / sh, wo = (W + sw - 1) / sw;
    int64_t ph = (ho - 1) * sh + KH - H, pw = (wo - 1) * sw + KW - W;
    if (ph < 0) ph = 0;
    if (pw < 0) pw = 0;
    pads_tlbr[0] = ph / 2;
    pads_tlbr[1] = pw / 2;
    pads_tlbr[2] = ph - ph / 2;
    pads_tlbr[3] = pw - pw / 2;
    return ORACLE_OK;
}

typedef struct {
    const float *x;
    int64_t N, H, W, C;
    const float *f;
    int64_t KH, KW, K;
    int64_t sh, sw, pt, pl;
} conv_problem;

static void conv_element(const conv_problem *p, int64_t n, int64_t ho, int64_t wo,
                         int64_t co, double *ref, double *scale)
{
    double s = 0.0, t = 0.0;
    for (int64_t kh = 0; kh < p->KH; ++kh) {
        int64_t ih = ho * p->sh - p->pt + kh;
        for (int64_t kw = 0; kw < p->KW; ++kw) {
            int64_t iw = wo * p->sw - p->pl + kw;
            int inside = ih >= 0 && ih < p->H && iw >= 0 && iw < p->W;
            for (int64_t ci = 0; ci < p->C; ++ci) {
                double xv = inside ? (double)p->x[((n * p->H + ih) * p->W + iw) * p->C + ci] : 0.0;
                double fv = (double)p->f[((kh * p->KW + kw) * p->C + ci) * p->K + co];
                double prod = xv * fv;
                s += prod;
                t += fabs(prod);
            }
        }
    }
    *ref = s;
    *scale = t;
}

static int conv_setup(conv_problem *p, const float *x, int64_t N, int64_t H, int64_t W,
                      int64_t Cin, const float *f, int64_t KH, int64_t KW, int64_t Cout,
                      int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb, int64_t pr,
                      int64_t Ho, int64_t Wo)
{
    int64_t ho, wo;
    if (N < 0 || Cin < 1 || Cout < 1) return ORACLE_BAD_ARG;
    if (oracle_conv2d_out_dims(H, W, KH, KW, sh, sw, pt, pl, pb, pr, &ho, &wo) != ORACLE_OK)
        return ORACLE_BAD_ARG;
    if (ho != Ho || wo != Wo) return ORACLE_BAD_ARG;
    p->x = x; p->N = N; p->H = H; p->W = W; p->C = Cin;
    p->f = f; p->KH = KH; p->KW = KW; p->K = Cout;
    p->sh = sh; p->sw = sw; p->pt = pt; p->pl = pl;
    return ORACLE_OK;
}

/* Whole output: ref and scale are N x Ho x Wo x Cout (NHWC). */
int oracle_conv2d(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                  const float *f, int64_t KH, int64_t KW, int64_t Cout,
                  int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb, int64_t pr,
                  int64_t Ho, int64_t Wo, double *ref, double *scale)
{
    conv_problem p;
    if (conv_setup(&p, x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr, Ho, Wo))
        return ORACLE_BAD_ARG;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t ho = 0; ho < Ho; ++ho)
            for (int64_t wo = 0; wo < Wo; ++wo)
                for (int64_t co = 0; co < Cout; ++co) {
                    int64_t o = ((n * Ho + ho) * Wo + wo) * Cout + co;
                    conv_element(&p, n, ho, wo, co, &ref[o], &scale[o]);
                }
    return ORACLE_OK;
}

/* Selected outputs, by flat NHWC index into the N x Ho x Wo x Cout result. */
int oracle_conv2d_at(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                     const float *f, int64_t KH, int64_t KW, int64_t Cout,
                     int64_t sh, int64_t sw, int64_t pt, int64_t pl, int64_t pb, int64_t pr,
                     int64_t Ho, int64_t Wo, int64_t count, const int64_t *flat,
                     double *ref, double *scale)
{
    conv_problem p;
    if (conv_setup(&p, x, N, H, W, Cin, f, KH, KW, Cout, sh, sw, pt, pl, pb, pr, Ho, Wo))
        return ORACLE_BAD_ARG;
    int64_t total = N * Ho * Wo * Cout;
    for (int64_t s = 0; s < count; ++s)
        if (flat[s] < 0 || flat[s] >= total) return ORACLE_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t s = 0; s < count; ++s) {
        int64_t o = flat[s];
        int64_t co = o % Cout, pix = o / Cout;
        int64_t wo = pix % Wo, nh = pix / Wo;
        int64_t ho = nh % Ho, n = nh / Ho;
        conv_element(&p, n, ho, wo, co, &ref[s], &scale[s]);
    }
    return ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * Winograd convolution F(m x m, 3 x 3) (Section 4.1.2, the minimal-filtering
 * technique of Lavin and Gray that the paper adopts), for a 3x3 window at
 * stride 1, with output tiles of m x m, m = 2 or 4.  Every m x m block of
 * outputs (tile th, tw) is computed from the (m+2) x (m+2) input tile d that
 * starts at row m*th - pt, column m*tw - pl (zero outside the image), in the
 * paper's order of steps:
 *   V = BT d BT^T          input transform, per channel
 *   U = G g G^T            filter transform of the 3x3 filter g, per (ci, co)
 *   M = sum_ci U (.) V     (m+2)^2 independent sums over the channels -- the
 *                          batched matrix multiply of the description
 *   Y = AT M AT^T          output transform to the m x m outputs
 * The matrices are the published ones of Lavin and Gray: for F(2, 3) the
 * interpolation points 0, 1, -1 and infinity,
 *   BT = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1],
 *   G  = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1],
 *   AT = [1 1 1 0; 0 1 -1 -1];
 * for F(4, 3) the points 0, 1, -1, 2, -2 and infinity (below).  The paper's
 * trade-off is the tile size: F(4, 3) needs 36 products per 16 outputs per
 * channel pair against F(2, 3)'s 16 per 4, at the price of larger transform
 * coefficients (more rounding) and smaller batched products.
 * In exact arithmetic Y is the convolution.  The scale returned with each
 * output is the same chain with every matrix entry and operand replaced by
 * its absolute value: the magnitude that bounds the rounding error of the
 * transformed computation, as sum |a*b| does for the direct sum.
 * ------------------------------------------------------------------------- */
typedef struct {
    int m;            /* outputs per tile side; the input tile is m + 2 */
    double BT[6][6];  /* (m+2) x (m+2) input transform */
    double G[6][3];   /* (m+2) x 3 filter transform */
    double AT[4][6];  /* m x (m+2) output transform */
} wino_matrices;

static const wino_matrices WINO_F2 = {
    2,
    {{1, 0, -1, 0}, {0, 1, 1, 0}, {0, -1, 1, 0}, {0, 1, 0, -1}},
    {{1, 0, 0}, {0.5, 0.5, 0.5}, {0.5, -0.5, 0.5}, {0, 0, 1}},
    {{1, 1, 1, 0}, {0, 1, -1, -1}}};

static const wino_matrices WINO_F4 = {
    4,
    {{4, 0, -5, 0, 1, 0}, {0, -4, -4, 1, 1, 0}, {0, 4, -4, -1, 1, 0},
     {0, -2, -1, 2, 1, 0}, {0, 2, -1, -2, 1, 0}, {0, 4, 0, -5, 0, 1}},
    {{1.0 / 4, 0, 0}, {-1.0 / 6, -1.0 / 6, -1.0 / 6}, {-1.0 / 6, 1.0 / 6, -1.0 / 6},
     {1.0 / 24, 1.0 / 12, 1.0 / 6}, {1.0 / 24, -1.0 / 12, 1.0 / 6}, {0, 0, 1}},
    {{1, 1, 1, 1, 1, 0}, {0, 1, -1, 2, -2, 0}, {0, 1, 1, 4, 4, 0}, {0, 1, -1, 8, -8, 1}}};

static void winograd_element(const conv_problem *p, const wino_matrices *w, int64_t n,
                             int64_t ho, int64_t wo, int64_t co, double *ref, double *scale)
{
    const int m = w->m, t = m + 2;
    const int64_t th = ho / m, tw = wo / m;
    const int i = (int)(ho % m), j = (int)(wo % m);
    const int64_t ih0 = m * th - p->pt, iw0 = m * tw - p->pl;
    double acc[6][6] = {{0}}, acc_abs[6][6] = {{0}};
    for (int64_t ch = 0; ch < p->C; ++ch) {
        double d[6][6], g[3][3];
        for (int r = 0; r < t; ++r)
            for (int c = 0; c < t; ++c) {
                int64_t ih = ih0 + r, iw = iw0 + c;
                const int in_image = (ih >= 0 && ih < p->H) && (iw >= 0 && iw < p->W);
                d[r][c] = in_image ? (double)p->x[((n * p->H + ih) * p->W + iw) * p->C + ch] : 0.0;
            }
        for (int r = 0; r < 3; ++r)
            for (int c = 0; c < 3; ++c)
                g[r][c] = (double)p->f[((r * 3 + c) * p->C + ch) * p->K + co];
        for (int a = 0; a < t; ++a)
            for (int b = 0; b < t; ++b) {
                double v = 0.0, va = 0.0, u = 0.0, ua = 0.0;
                for (int r = 0; r < t; ++r)
                    for (int c = 0; c < t; ++c) {
                        v += w->BT[a][r] * d[r][c] * w->BT[b][c];
                        va += fabs(w->BT[a][r]) * fabs(d[r][c]) * fabs(w->BT[b][c]);
                    }
                for (int r = 0; r < 3; ++r)
                    for (int c = 0; c < 3; ++c) {
                        u += w->G[a][r] * g[r][c] * w->G[b][c];
                        ua += fabs(w->G[a][r]) * fabs(g[r][c]) * fabs(w->G[b][c]);
                    }
                acc[a][b] += u * v;
                acc_abs[a][b] += ua * va;
            }
    }
    double y = 0.0, ya = 0.0;
    for (int a = 0; a < t; ++a)
        for (int b = 0; b < t; ++b) {
            y += w->AT[i][a] * acc[a][b] * w->AT[j][b];
            ya += fabs(w->AT[i][a]) * acc_abs[a][b] * fabs(w->AT[j][b]);
        }
    *ref = y;
    *scale = ya;
}

static int winograd_setup(conv_problem *p, const float *x, int64_t N, int64_t H, int64_t W,
                          int64_t Cin, const float *f, int64_t Cout, int64_t pt, int64_t pl,
                          int64_t pb, int64_t pr, int64_t Ho, int64_t Wo)
{
    return conv_setup(p, x, N, H, W, Cin, f, 3, 3, Cout, 1, 1, pt, pl, pb, pr, Ho, Wo);
}

static int winograd_whole(const wino_matrices *w, const float *x, int64_t N, int64_t H,
                          int64_t W, int64_t Cin, const float *f, int64_t Cout, int64_t pt,
                          int64_t pl, int64_t pb, int64_t pr, int64_t Ho, int64_t Wo,
                          double *ref, double *scale)
{
    conv_problem p;
    if (winograd_setup(&p, x, N, H, W, Cin, f, Cout, pt, pl, pb, pr, Ho, Wo)) return ORACLE_BAD_ARG;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t ho = 0; ho < Ho; ++ho)
            for (int64_t wo = 0; wo < Wo; ++wo)
                for (int64_t co = 0; co < Cout; ++co) {
                    int64_t o = ((n * Ho + ho) * Wo + wo) * Cout + co;
                    winograd_element(&p, w, n, ho, wo, co, &ref[o], &scale[o]);
                }
    return ORACLE_OK;
}

static int winograd_sampled(const wino_matrices *w, const float *x, int64_t N, int64_t H,
                            int64_t W, int64_t Cin, const float *f, int64_t Cout, int64_t pt,
                            int64_t pl, int64_t pb, int64_t pr, int64_t Ho, int64_t Wo,
                            int64_t count, const int64_t *flat, double *ref, double *scale)
{
    conv_problem p;
    if (winograd_setup(&p, x, N, H, W, Cin, f, Cout, pt, pl, pb, pr, Ho, Wo)) return ORACLE_BAD_ARG;
    int64_t total = N * Ho * Wo * Cout;
    for (int64_t s = 0; s < count; ++s)
        if (flat[s] < 0 || flat[s] >= total) return ORACLE_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t s = 0; s < count; ++s) {
        int64_t o = flat[s];
        int64_t c_out = o % Cout, pixel = o / Cout;
        int64_t w_out = pixel % Wo, image_row = pixel / Wo;
        int64_t h_out = image_row % Ho, img = image_row / Ho;
        winograd_element(&p, w, img, h_out, w_out, c_out, &ref[s], &scale[s]);
    }
    return ORACLE_OK;
}

/* Whole output of the F(2x2, 3x3) computation: ref and scale are N x Ho x Wo x Cout. */
int oracle_winograd_f2x3(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                         const float *f, int64_t Cout, int64_t pt, int64_t pl, int64_t pb,
                         int64_t pr, int64_t Ho, int64_t Wo, double *ref, double *scale)
{
    return winograd_whole(&WINO_F2, x, N, H, W, Cin, f, Cout, pt, pl, pb, pr, Ho, Wo, ref, scale);
}

/* Selected outputs of the F(2x2, 3x3) computation, by flat NHWC index. */
int oracle_winograd_f2x3_at(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                            const float *f, int64_t Cout, int64_t pt, int64_t pl, int64_t pb,
                            int64_t pr, int64_t Ho, int64_t Wo, int64_t count,
                            const int64_t *flat, double *ref, double *scale)
{
    return winograd_sampled(&WINO_F2, x, N, H, W, Cin, f, Cout, pt, pl, pb, pr, Ho, Wo, count, flat,
                            ref, scale);
}

/* Whole output of the F(4x4, 3x3) computation: ref and scale are N x Ho x Wo x Cout. */
int oracle_winograd_f4x3(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                         const float *f, int64_t Cout, int64_t pt, int64_t pl, int64_t pb,
                         int64_t pr, int64_t Ho, int64_t Wo, double *ref, double *scale)
{
    return winograd_whole(&WINO_F4, x, N, H, W, Cin, f, Cout, pt, pl, pb, pr, Ho, Wo, ref, scale);
}

/* Selected outputs of the F(4x4, 3x3) computation, by flat NHWC index. */
int oracle_winograd_f4x3_at(const float *x, int64_t N, int64_t H, int64_t W, int64_t Cin,
                            const float *f, int64_t Cout, int64_t pt, int64_t pl, int64_t pb,
                            int64_t pr, int64_t Ho, int64_t Wo, int64_t count,
                            const int64_t *flat, double *ref, double *scale)
{
    return winograd_sampled(&WINO_F4, x, N, H, W, Cin, f, Cout, pt, pl, pb, pr, Ho, Wo, count, flat,
                            ref, scale);
}
