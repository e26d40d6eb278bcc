// pk_args.hpp -- the argument block every contraction kernel receives.
#pragma once

#include <stdint.h>

namespace pk {

struct KernelArgs {
    const float *A;  // dense A, or the NHWC image for A_CONV
    const float *B;  // dense B (for the convolution: the HWIO filter, K x Cout)
    float *C;
    float *ws;       // split-K partial sums, splits x M x N (NULL when splits == 1)
    int M, N, K;
    int64_t lda, ldb, ldc;
    float alpha, beta;
    int tiles_m, tiles_n;
    int splits, kblocks_per_split;
    int xcds, group_m;
    // implicit-GEMM geometry: A(m, k) = x[n][ho*sh - pt + kh][wo*sw - pl + kw][ci]
    // with m = (n*Ho + ho)*Wo + wo and k = (kh*KW + kw)*Cin + ci.
    int H, W, Cin, KW, sh, sw, pt, pl, Ho, Wo;
    int KH, batch;  // used by the direct convolution only
    // batched products (non-persistent GEMM instances): grid.y = nbatch
    // independent products, matrix b at A + b*stride_a, B + b*stride_b,
    // C + b*stride_c (elements).  0 = one product.
    int nbatch;
    int64_t stride_a, stride_b, stride_c;
    // stream-K launches: K-blocks per tile, partial-tile slots (2 per
    // work-group, BM x BN floats each) and one arrival counter per tile, both
    // in the caller's workspace; the counters are zeroed before each launch.
    int sk_nkb, sk_groups;  // sk_groups: the launch's work-groups (host side)
    float *sk_part;
    int *sk_cnt;
};

}  // namespace pk
