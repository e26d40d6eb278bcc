"""Checks that pin the CPU oracle to facts other than itself.

Each ``pin_*`` function takes an oracle object (``oracle.Oracle``) and raises
AssertionError when that oracle disagrees with what the paper or plain
mathematics fixes.  ``test_oracle.py`` runs them against the real oracle;
``test_oracle_mutations.py`` runs them against copies of the oracle with a
planted mistake and requires at least one of them to fail for each mistake.

What pins what:
  - brute force: exact rational arithmetic (``fractions.Fraction``) over
    explicitly materialised matrices and zero-padded images, with window
    positions found by enumeration rather than by a size formula;
  - identity and permutation matrices, delta filters (no flip, pad offset);
  - closed forms for all-ones data (K; KH*KW*Cin inside the image, 6*Cin on
    an edge and 4*Cin at a corner of a 3x3 stride-1 "same" convolution);
  - invariants (1x1 convolution == GEMM, im2col product, (AB)^T = B^T A^T);
  - a textbook routine: torch's CPU float64 matmul and conv2d;
  - the paper's layer tables (output sizes from window and stride);
  - Winograd F(2x2, 3x3) (Section 4.1.2): its value against the exact
    brute-force convolution (it is the same function in exact arithmetic),
    bit-equality with the direct sum on small integers, and its error scale
    against a hand-derived closed form and the direct scale it must bound.
"""
from __future__ import annotations

import csv
import itertools
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_golden(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        rows = [line for line in fh if not line.startswith("#")]
    return list(csv.DictReader(rows))


def _rng(seed):
    return np.random.default_rng(seed)


def _nan(M, N):
    # C for beta == 0: never read, so NaN there must not reach the result
    return np.full((M, N), np.nan, np.float32)


def _grid_uniform(rng, shape):
    # values on a 2**-23 grid in [-1, 1), as the workload generator draws them
    return (rng.random(int(np.prod(shape)), dtype=np.float32) * np.float32(2) - np.float32(1)).reshape(shape)


# ------------------------------------------------------- brute force (P2)

def _frac_matrix(a2d):
    return [[Fraction(float(v)) for v in row] for row in a2d]


def brute_gemm(op_a, op_b, alpha, beta, c):
    """Exact alpha*op_a@op_b + beta*c on explicit (already transposed) matrices."""
    A = _frac_matrix(op_a)
    B = _frac_matrix(op_b)
    M, K = len(A), len(A[0]) if A else 0
    N = len(B[0]) if B else c.shape[1]
    out = np.empty((M, N), dtype=np.float64)
    mag = np.empty((M, N), dtype=np.float64)
    fa, fb = Fraction(float(alpha)), Fraction(float(beta))
    for i in range(M):
        for j in range(N):
            terms = [A[i][k] * B[k][j] for k in range(K)]
            v = fa * sum(terms, Fraction(0))
            if beta != 0:
                v += fb * Fraction(float(c[i, j]))
            out[i, j] = float(v)
            mag[i, j] = float(sum((abs(t) for t in terms), Fraction(0)))
    return out, mag


def brute_conv(x, f, stride, pads):
    """Exact convolution by sliding the window over an explicitly padded image."""
    pt, pl, pb, pr = pads
    sh, sw = stride
    xp = np.pad(x, ((0, 0), (pt, pb), (pl, pr), (0, 0)))
    N, Hp, Wp, C = xp.shape
    KH, KW, _, K = f.shape
    tops = list(range(0, Hp - KH + 1, sh))
    lefts = list(range(0, Wp - KW + 1, sw))
    out = np.empty((N, len(tops), len(lefts), K), dtype=np.float64)
    mag = np.empty_like(out)
    F = [[[[Fraction(float(f[a, b, c, k])) for k in range(K)] for c in range(C)]
          for b in range(KW)] for a in range(KH)]
    for n in range(N):
        for oi, top in enumerate(tops):
            for oj, left in enumerate(lefts):
                win = xp[n, top:top + KH, left:left + KW, :]
                for k in range(K):
                    terms = [Fraction(float(win[a, b, c])) * F[a][b][c][k]
                             for a in range(KH) for b in range(KW) for c in range(C)]
                    out[n, oi, oj, k] = float(sum(terms, Fraction(0)))
                    mag[n, oi, oj, k] = float(sum((abs(t) for t in terms), Fraction(0)))
    return out, mag


def _storage(rng, rows, cols, slack):
    """A rows x cols matrix stored with leading dimension cols + slack (junk in the slack)."""
    full = _grid_uniform(rng, (rows, cols + slack))
    if slack:
        full[:, cols:] = np.float32(1e30)  # must never be read
    return full


def pin_gemm_brute_force(orc):
    rng = _rng(7)
    for (M, N, K), ta, tb, slack in itertools.product(
            [(1, 1, 1), (2, 3, 5), (5, 2, 3), (7, 5, 2), (3, 7, 7)], "NT", "NT", (0, 2)):
        a_st = _storage(rng, K if ta == "T" else M, M if ta == "T" else K, slack)
        b_st = _storage(rng, N if tb == "T" else K, K if tb == "T" else N, slack)
        c = _grid_uniform(rng, (M, N + slack))
        op_a = (a_st[:, :M].T if ta == "T" else a_st[:, :K])
        op_b = (b_st[:, :K].T if tb == "T" else b_st[:, :N])
        for alpha, beta in [(1.0, 0.0), (1.5, -0.75), (-2.0, 0.5)]:
            exp, mag = brute_gemm(op_a, op_b, alpha, beta, c[:, :N])
            ref, scale = orc.sgemm(ta, tb, M, N, K, alpha, a_st, a_st.shape[1],
                                   b_st, b_st.shape[1], beta, c, c.shape[1])
            # dyadic alpha/beta and at most 7 grid products: fp64 sums are exact
            assert np.array_equal(ref, exp), (M, N, K, ta, tb, slack, alpha, beta)
            assert np.array_equal(scale, mag), (M, N, K, ta, tb, slack)


def pin_conv_brute_force(orc):
    rng = _rng(11)
    cases = []
    for H, W in [(1, 1), (3, 4), (5, 5)]:
        for KH, KW in [(1, 1), (2, 3), (3, 3)]:
            for s in (1, 2, 3):
                for pads in [(0, 0, 0, 0), (1, 1, 1, 1), (2, 0, 1, 2), (0, 2, 2, 1)]:
                    if H + pads[0] + pads[2] < KH or W + pads[1] + pads[3] < KW:
                        continue
                    cases.append((H, W, KH, KW, s, pads))
    for idx, (H, W, KH, KW, s, pads) in enumerate(cases):
        N, C, K = (2, 2, 3) if idx % 3 == 0 else (1, 3, 2)
        sh, sw = (s, s) if idx % 2 else (s, 1)
        x = _grid_uniform(rng, (N, H, W, C))
        f = _grid_uniform(rng, (KH, KW, C, K))
        exp, mag = brute_conv(x, f, (sh, sw), pads)
        ref, scale = orc.conv2d(x, f, (sh, sw), pads)
        assert ref.shape == exp.shape, (H, W, KH, KW, (sh, sw), pads, ref.shape, exp.shape)
        np.testing.assert_array_equal(ref, exp, err_msg=str((H, W, KH, KW, (sh, sw), pads)))
        np.testing.assert_array_equal(scale, mag)


# -------------------------------------------- identity, permutation (P3)

def pin_gemm_identity_permutation(orc):
    rng = _rng(3)
    M, N = 6, 5
    b = _grid_uniform(rng, (M, N))
    c = _grid_uniform(rng, (M, N))
    eye = np.eye(M, dtype=np.float32)
    ref, _ = orc.sgemm("N", "N", M, N, M, 1.0, eye, M, b, N, 0.0, _nan(M, N), N)
    assert np.array_equal(ref, b.astype(np.float64))
    ref, _ = orc.sgemm("N", "N", M, N, M, 2.0, eye, M, b, N, 0.5, c, N)
    assert np.array_equal(ref, 2.0 * b.astype(np.float64) + 0.5 * c.astype(np.float64))
    perm = np.array([3, 0, 5, 1, 4, 2])
    P = np.zeros((M, M), dtype=np.float32)
    P[np.arange(M), perm] = 1.0  # row i of P picks row perm[i] of b
    ref, _ = orc.sgemm("N", "N", M, N, M, 1.0, P, M, b, N, 0.0, _nan(M, N), N)
    assert np.array_equal(ref, b[perm].astype(np.float64))
    # the permutation applied from the right permutes columns; B = P^T given as 'T'
    a = _grid_uniform(rng, (N, M))
    ref, _ = orc.sgemm("N", "T", N, M, M, 1.0, a, M, P, M, 0.0, _nan(N, M), M)
    assert np.array_equal(ref, a[:, perm].astype(np.float64))


def pin_conv_delta_filters(orc):
    rng = _rng(5)
    N, H, W, C = 2, 6, 5, 3
    x = _grid_uniform(rng, (N, H, W, C))
    xd = x.astype(np.float64)
    ident = np.zeros((1, 1, C, C), dtype=np.float32)
    ident[0, 0] = np.eye(C)
    ref, _ = orc.conv2d(x, ident, (1, 1), (0, 0, 0, 0))
    assert np.array_equal(ref, xd)
    ref, _ = orc.conv2d(x, ident, (2, 2), (0, 0, 0, 0))
    assert np.array_equal(ref, xd[:, ::2, ::2, :])
    centre = np.zeros((3, 3, C, C), dtype=np.float32)
    centre[1, 1] = np.eye(C)
    ref, _ = orc.conv2d(x, centre, (1, 1), (1, 1, 1, 1))
    assert np.array_equal(ref, xd)
    corner = np.zeros((3, 3, C, C), dtype=np.float32)
    corner[0, 0] = np.eye(C)  # tap (0,0) reads the pixel one up and one left
    ref, _ = orc.conv2d(x, corner, (1, 1), (1, 1, 1, 1))
    exp = np.zeros_like(xd)
    exp[:, 1:, 1:, :] = xd[:, :-1, :-1, :]
    assert np.array_equal(ref, exp)
    last = np.zeros((3, 3, C, C), dtype=np.float32)
    last[2, 1] = np.eye(C)  # tap (2,1) reads the pixel one down
    ref, _ = orc.conv2d(x, last, (1, 1), (1, 1, 1, 1))
    exp = np.zeros_like(xd)
    exp[:, :-1, :, :] = xd[:, 1:, :, :]
    assert np.array_equal(ref, exp)
    # channel mixing: output k takes input channel (k + 1) % C
    mix = np.zeros((1, 1, C, C), dtype=np.float32)
    for k in range(C):
        mix[0, 0, (k + 1) % C, k] = 1.0
    ref, _ = orc.conv2d(x, mix, (1, 1), (0, 0, 0, 0))
    assert np.array_equal(ref, xd[..., [(k + 1) % C for k in range(C)]])


# --------------------------------------------------- closed forms (P4)

def pin_all_ones_closed_forms(orc):
    M, N, K = 9, 7, 13
    ones_a = np.ones((M, K), np.float32)
    ones_b = np.ones((K, N), np.float32)
    c = np.full((M, N), 3.0, np.float32)
    ref, scale = orc.sgemm("N", "N", M, N, K, 1.0, ones_a, K, ones_b, N, 0.5, c, N)
    assert np.all(ref == K + 1.5) and np.all(scale == K)
    ref, scale = orc.sgemm("N", "N", M, N, K, 1.0, -ones_a, K, ones_b, N, 0.0, _nan(M, N), N)
    assert np.all(ref == -K) and np.all(scale == K)
    # K = 0 and alpha = 0 leave beta*C; beta = 0 never reads C (NaN there is harmless)
    ref, _ = orc.sgemm("N", "N", M, N, 0, 1.0, ones_a, 1, ones_b, N, 0.5, c, N)
    assert np.all(ref == 1.5)
    nan_a = np.full((M, K), np.nan, np.float32)
    ref, _ = orc.sgemm("N", "N", M, N, K, 0.0, nan_a, K, ones_b, N, 2.0, c, N)
    assert np.all(ref == 6.0)
    nan_c = np.full((M, N), np.nan, np.float32)
    ref, _ = orc.sgemm("N", "N", M, N, K, 2.0, ones_a, K, ones_b, N, 0.0, nan_c, N)
    assert np.all(ref == 2 * K)
    # 3x3 stride 1 "same": 9*Cin inside, 6*Cin on an edge, 4*Cin at a corner
    Cin, Cout = 5, 2
    x = np.ones((2, 6, 7, Cin), np.float32)
    f = np.ones((3, 3, Cin, Cout), np.float32)
    ref, scale = orc.conv2d(x, f, (1, 1), (1, 1, 1, 1))
    exp = np.full(ref.shape, 9.0 * Cin)
    exp[:, 0, :, :] = exp[:, -1, :, :] = 6.0 * Cin
    exp[:, :, 0, :] = exp[:, :, -1, :] = 6.0 * Cin
    for r in (0, -1):
        for q in (0, -1):
            exp[:, r, q, :] = 4.0 * Cin
    assert np.array_equal(ref, exp) and np.array_equal(scale, exp)
    # without padding every window is full: KH*KW*Cin everywhere
    ref, _ = orc.conv2d(x, f, (2, 2), (0, 0, 0, 0))
    assert ref.shape == (2, 2, 3, Cout) and np.all(ref == 9.0 * Cin)


# ----------------------------------------------------- invariants (P6)

def _im2col(x, KH, KW, stride, pads):
    pt, pl, pb, pr = pads
    xp = np.pad(x.astype(np.float64), ((0, 0), (pt, pb), (pl, pr), (0, 0)))
    N, Hp, Wp, C = xp.shape
    sh, sw = stride
    Ho = (Hp - KH) // sh + 1
    Wo = (Wp - KW) // sw + 1
    cols = np.empty((N, Ho, Wo, KH, KW, C))
    for a in range(KH):
        for b in range(KW):
            cols[:, :, :, a, b, :] = xp[:, a:a + sh * (Ho - 1) + 1:sh, b:b + sw * (Wo - 1) + 1:sw, :]
    return cols.reshape(N * Ho * Wo, KH * KW * C), (N, Ho, Wo)


def pin_invariants(orc):
    rng = _rng(13)
    # 1x1 stride-1 convolution is the GEMM of the reshaped tensors
    x = _grid_uniform(rng, (2, 5, 6, 8))
    f = _grid_uniform(rng, (1, 1, 8, 4))
    ref_c, sc_c = orc.conv2d(x, f, (1, 1), (0, 0, 0, 0))
    ref_g, sc_g = orc.sgemm("N", "N", 60, 4, 8, 1.0, x.reshape(60, 8), 8, f.reshape(8, 4), 4, 0.0, _nan(60, 4), 4)
    assert np.array_equal(ref_c.reshape(60, 4), ref_g) and np.array_equal(sc_c.reshape(60, 4), sc_g)
    # any convolution is im2col(x) @ f viewed as (KH*KW*Cin) x Cout
    for KH, KW, stride, pads in [(3, 3, (1, 1), (1, 1, 1, 1)), (3, 2, (2, 1), (0, 1, 2, 0)),
                                 (2, 2, (2, 2), (0, 0, 1, 1))]:
        x = _grid_uniform(rng, (2, 7, 6, 3))
        f = _grid_uniform(rng, (KH, KW, 3, 5))
        cols, shp = _im2col(x, KH, KW, stride, pads)
        exp = (cols @ f.reshape(-1, 5).astype(np.float64)).reshape(shp + (5,))
        ref, _ = orc.conv2d(x, f, stride, pads)
        np.testing.assert_allclose(ref, exp, rtol=0, atol=1e-12)
    # (A B)^T = B^T A^T through the transpose flags
    M, N, K = 6, 9, 5
    a = _grid_uniform(rng, (M, K))
    b = _grid_uniform(rng, (K, N))
    ref_nn, _ = orc.sgemm("N", "N", M, N, K, 1.0, a, K, b, N, 0.0, _nan(M, N), N)
    ref_tt, _ = orc.sgemm("T", "T", N, M, K, 1.0, b, N, a, K, 0.0, _nan(N, M), M)
    np.testing.assert_allclose(ref_tt, ref_nn.T, rtol=0, atol=1e-12)
    # a stored transpose with the 'T' flag gives the same product as 'N'
    at = np.ascontiguousarray(a.T)
    bt = np.ascontiguousarray(b.T)
    for ta, tb, A_, B_, lda, ldb in [("T", "N", at, b, M, N), ("N", "T", a, bt, K, K), ("T", "T", at, bt, M, K)]:
        ref, _ = orc.sgemm(ta, tb, M, N, K, 1.0, A_, lda, B_, ldb, 0.0, _nan(M, N), N)
        np.testing.assert_allclose(ref, ref_nn, rtol=0, atol=1e-12)
    # linearity in the input, exact on integers
    xi = rng.integers(-8, 9, (1, 5, 5, 4)).astype(np.float32)
    yi = rng.integers(-8, 9, (1, 5, 5, 4)).astype(np.float32)
    fi = rng.integers(-8, 9, (3, 3, 4, 3)).astype(np.float32)
    r1, _ = orc.conv2d(xi, fi, (1, 1), (1, 1, 1, 1))
    r2, _ = orc.conv2d(yi, fi, (1, 1), (1, 1, 1, 1))
    r3, _ = orc.conv2d(xi + yi, fi, (1, 1), (1, 1, 1, 1))
    assert np.array_equal(r1 + r2, r3)
    # translation: shifting the input by (1, 2) shifts the interior outputs
    big = rng.integers(-8, 9, (1, 9, 9, 2)).astype(np.float32)
    fs = rng.integers(-8, 9, (3, 3, 2, 2)).astype(np.float32)
    shifted = np.zeros_like(big)
    shifted[:, 1:, 2:, :] = big[:, :-1, :-2, :]
    ra, _ = orc.conv2d(big, fs, (1, 1), (1, 1, 1, 1))
    rb, _ = orc.conv2d(shifted, fs, (1, 1), (1, 1, 1, 1))
    assert np.array_equal(rb[:, 2:-1, 3:-1], ra[:, 1:-2, 1:-3])


# -------------------------------------------- textbook routine (P7)

def pin_torch_float64(orc):
    import torch
    import torch.nn.functional as F
    rng = _rng(17)
    for ta, tb in itertools.product("NT", "NT"):
        M, N, K = 37, 29, 41
        a_st = _grid_uniform(rng, (K, M) if ta == "T" else (M, K))
        b_st = _grid_uniform(rng, (N, K) if tb == "T" else (K, N))
        c = _grid_uniform(rng, (M, N))
        ta_t = torch.from_numpy(a_st).double()
        tb_t = torch.from_numpy(b_st).double()
        opa = ta_t.t() if ta == "T" else ta_t
        opb = tb_t.t() if tb == "T" else tb_t
        exp = (1.25 * (opa @ opb) - 0.5 * torch.from_numpy(c).double()).numpy()
        ref, _ = orc.sgemm(ta, tb, M, N, K, 1.25, a_st, a_st.shape[1], b_st, b_st.shape[1], -0.5, c, N)
        np.testing.assert_allclose(ref, exp, rtol=1e-13, atol=1e-13)
    for (N, H, W, C, K), (KH, KW), stride, pads in [
            ((2, 9, 8, 6, 5), (3, 3), (1, 1), (1, 1, 1, 1)),
            ((1, 10, 11, 4, 3), (3, 3), (2, 2), (0, 0, 1, 1)),
            ((2, 8, 8, 3, 4), (7, 7), (2, 2), (3, 3, 3, 3)),
            ((1, 6, 7, 5, 6), (1, 1), (2, 2), (0, 0, 0, 0)),
            ((1, 6, 7, 2, 3), (2, 3), (1, 2), (1, 0, 0, 2))]:
        x = _grid_uniform(rng, (N, H, W, C))
        f = _grid_uniform(rng, (KH, KW, C, K))
        xt = torch.from_numpy(x).double().permute(0, 3, 1, 2)
        ft = torch.from_numpy(f).double().permute(3, 2, 0, 1)
        pt, pl, pb, pr = pads
        y = F.conv2d(F.pad(xt, (pl, pr, pt, pb)), ft, stride=stride)
        exp = y.permute(0, 2, 3, 1).numpy()
        ref, _ = orc.conv2d(x, f, stride, pads)
        assert ref.shape == exp.shape
        np.testing.assert_allclose(ref, exp, rtol=1e-13, atol=1e-13)
    # torch's stride-1 "same" for an even window puts the extra row/column
    # at the bottom/right, as the oracle's split does
    x = _grid_uniform(rng, (1, 6, 5, 2))
    f = _grid_uniform(rng, (2, 4, 2, 3))
    pads = orc.same_pads(6, 5, 2, 4, 1, 1)
    y = F.conv2d(torch.from_numpy(x).double().permute(0, 3, 1, 2),
                 torch.from_numpy(f).double().permute(3, 2, 0, 1), padding="same")
    ref, _ = orc.conv2d(x, f, (1, 1), pads)
    np.testing.assert_allclose(ref, y.permute(0, 2, 3, 1).numpy(), rtol=1e-13, atol=1e-13)


# --------------------------------------------- the paper's tables

def pin_layer_tables(orc):
    """Output sizes of every distinct VGG-16 and ResNet-50 layer in the paper.

    Windows of 1 or 3 use "same" padding; the 7x7 stride-2 first ResNet layer
    reads an input that is already padded (230 = 224 + 6) and uses none.
    """
    for name in ("vgg16_layers.csv", "resnet50_layers.csv"):
        for row in read_golden(name):
            k, s = int(row["window"]), int(row["stride"])
            H, W = int(row["in_h"]), int(row["in_w"])
            if k == 7:
                pads = (0, 0, 0, 0)
            else:
                pads = orc.same_pads(H, W, k, k, s, s)
            ho, wo = orc.conv2d_out_dims(H, W, k, k, s, s, *pads)
            assert (ho, wo) == (int(row["out_h"]), int(row["out_w"])), (name, row["layer"], pads)
    # the odd split of a stride-2 3x3 "same" layer: nothing on top/left, one at the bottom/right
    assert orc.same_pads(56, 56, 3, 3, 2, 2) == (0, 0, 1, 1)
    assert orc.same_pads(56, 56, 3, 3, 1, 1) == (1, 1, 1, 1)
    assert orc.same_pads(7, 7, 1, 1, 1, 1) == (0, 0, 0, 0)


def pin_same_padding_property(orc):
    """"Same" padding: the output has ceil(H/s) rows, the total padding is the
    least that gives it, and any odd pixel goes to the bottom/right."""
    for H in range(1, 12):
        for k in range(1, 8):
            for s in range(1, 5):
                pt, pl, pb, pr = orc.same_pads(H, H + 1, k, k, s, s)
                want_h, want_w = -(-H // s), -(-(H + 1) // s)
                assert orc.conv2d_out_dims(H, H + 1, k, k, s, s, pt, pl, pb, pr) == (want_h, want_w)
                for a, b, n in ((pt, pb, H), (pl, pr, H + 1)):
                    assert 0 <= a <= b <= a + 1
                    total = a + b
                    if total > 0:  # one pixel less padding loses an output (or the window no longer fits)
                        span = n + total - 1 - k
                        assert span < 0 or span // s + 1 < -(-n // s)


# -------------------------------------------- Winograd F(2x2, 3x3) (Section 4.1.2)

def pin_winograd_brute_force(orc):
    """The transformed computation is the convolution: equal to the exact
    brute-force result up to fp64 rounding, with ragged 2x2 tiles (odd output
    sizes) and asymmetric padding."""
    rng = _rng(17)
    for H, W in [(3, 3), (4, 5), (5, 4), (6, 7)]:
        for pads in [(0, 0, 0, 0), (1, 1, 1, 1), (2, 0, 1, 2), (0, 2, 2, 1)]:
            if H + pads[0] + pads[2] < 3 or W + pads[1] + pads[3] < 3:
                continue
            x = _grid_uniform(rng, (2, H, W, 3))
            f = _grid_uniform(rng, (3, 3, 3, 2))
            exp, _ = brute_conv(x, f, (1, 1), pads)
            ref, scale = orc.winograd_f2x3(x, f, pads)
            assert ref.shape == exp.shape, (H, W, pads, ref.shape, exp.shape)
            err = np.abs(ref - exp)
            assert np.all(err <= 1e-13 * scale), (H, W, pads, float(np.max(err)))


def pin_winograd_integer_exact(orc):
    """On small integers every intermediate of the transformed computation is
    a multiple of 1/4 far below 2^53: it must equal the direct sum exactly."""
    rng = _rng(19)
    x = rng.integers(-8, 9, size=(2, 7, 6, 5)).astype(np.float32)
    f = rng.integers(-8, 9, size=(3, 3, 5, 4)).astype(np.float32)
    for pads in [(1, 1, 1, 1), (0, 0, 0, 0), (2, 1, 0, 2)]:
        ref_d, _ = orc.conv2d(x, f, (1, 1), pads)
        ref_w, _ = orc.winograd_f2x3(x, f, pads)
        assert np.array_equal(ref_w, ref_d), pads


def pin_winograd_scale(orc):
    """The error scale: on all-ones data without padding every output is
    (4 Cin) * (sum of |G| row sums over the three rows |AT| selects)^2 =
    4 Cin * (1 + 3/2 + 3/2)^2 = 64 Cin (|BT| rows each sum to 2, the rows of
    |G| to 1, 3/2, 3/2, 1); on random data it bounds the direct sum |a*b|
    from above, as every product of the direct sum appears in its expansion
    with total coefficient at least 1."""
    for C in (1, 3, 8):
        x = np.ones((1, 6, 8, C), dtype=np.float32)
        f = np.ones((3, 3, C, 2), dtype=np.float32)
        ref, scale = orc.winograd_f2x3(x, f, (0, 0, 0, 0))
        assert np.all(ref == 9 * C) and np.all(scale == 64 * C), C
    rng = _rng(23)
    x = _grid_uniform(rng, (2, 9, 7, 4))
    f = _grid_uniform(rng, (3, 3, 4, 3))
    for pads in [(1, 1, 1, 1), (0, 0, 0, 0), (2, 0, 1, 2)]:
        _, t = orc.conv2d(x, f, (1, 1), pads)
        _, tw = orc.winograd_f2x3(x, f, pads)
        assert np.all(tw >= t * (1 - 1e-12)), pads


# -------------------------------------------- Winograd F(4x4, 3x3) (Section 4.1.2)

def pin_winograd_f4_brute_force(orc):
    """The F(4x4, 3x3) computation is the convolution: equal to the exact
    brute-force result up to fp64 rounding (its filter transform has the
    non-dyadic entries 1/6, 1/12, 1/24, so equality is within rounding, not
    exact), with ragged 4x4 tiles and asymmetric padding."""
    rng = _rng(29)
    for H, W in [(3, 3), (5, 7), (6, 6), (9, 4), (10, 11)]:
        for pads in [(0, 0, 0, 0), (1, 1, 1, 1), (2, 0, 1, 2), (0, 2, 2, 1)]:
            if H + pads[0] + pads[2] < 3 or W + pads[1] + pads[3] < 3:
                continue
            x = _grid_uniform(rng, (2, H, W, 3))
            f = _grid_uniform(rng, (3, 3, 3, 2))
            exp, _ = brute_conv(x, f, (1, 1), pads)
            ref, scale = orc.winograd_f4x3(x, f, pads)
            assert ref.shape == exp.shape, (H, W, pads, ref.shape, exp.shape)
            err = np.abs(ref - exp)
            assert np.all(err <= 1e-12 * scale), (H, W, pads, float(np.max(err / scale)))


def pin_winograd_f4_scale(orc):
    """The F(4x4, 3x3) error scale in closed form.  On all-ones data without
    padding and with whole tiles, the absolute chain factors per dimension:
    the rows of |BT| sum to 10, 10, 10, 6, 6, 10 and those of |G| to 1/4,
    1/2, 1/2, 7/24, 7/24, 1, so the products per transform row are
    h = (5/2, 5, 5, 7/4, 7/4, 10); the rows of |AT| select
    s = (16, 17, 24, 48) from them, and the output at position (i, j) of
    its tile has scale Cin * s_i * s_j (value 9 Cin).  On random data the
    scale bounds the direct sum of |products| from above."""
    s = np.array([16.0, 17.0, 24.0, 48.0])
    for C in (1, 3, 8):
        x = np.ones((1, 10, 6, C), dtype=np.float32)   # 8 x 4 outputs: whole tiles
        f = np.ones((3, 3, C, 2), dtype=np.float32)
        ref, scale = orc.winograd_f4x3(x, f, (0, 0, 0, 0))
        assert ref.shape == (1, 8, 4, 2)
        assert np.allclose(ref, 9 * C, rtol=1e-13, atol=0), C
        i = np.arange(8) % 4
        j = np.arange(4) % 4
        want = C * np.outer(s[i], s[j])[None, :, :, None]
        assert np.allclose(scale, np.broadcast_to(want, scale.shape), rtol=1e-13, atol=0), C
    rng = _rng(31)
    x = _grid_uniform(rng, (2, 9, 7, 4))
    f = _grid_uniform(rng, (3, 3, 4, 3))
    for pads in [(1, 1, 1, 1), (0, 0, 0, 0), (2, 0, 1, 2)]:
        _, t = orc.conv2d(x, f, (1, 1), pads)
        _, tw = orc.winograd_f4x3(x, f, pads)
        assert np.all(tw >= t * (1 - 1e-12)), pads


def pin_winograd_tile_sizes_agree(orc):
    """F(2x2, 3x3) and F(4x4, 3x3) compute the same convolution: on small
    integers F(2x2) is exact and F(4x4) within its fp64 rounding of it."""
    rng = _rng(37)
    x = rng.integers(-8, 9, size=(2, 11, 9, 6)).astype(np.float32)
    f = rng.integers(-8, 9, size=(3, 3, 6, 5)).astype(np.float32)
    for pads in [(1, 1, 1, 1), (0, 0, 0, 0), (2, 1, 0, 2)]:
        r2, _ = orc.winograd_f2x3(x, f, pads)
        r4, s4 = orc.winograd_f4x3(x, f, pads)
        assert np.all(np.abs(r4 - r2) <= 1e-12 * s4), pads
        assert np.array_equal(np.rint(r4), r2), pads


# -------------------------------------------- sampled entry points

def pin_sampled_equals_whole(orc):
    """Each sampled entry point returns, at every requested flat index, the
    value and scale of the (separately pinned) whole-output function: the
    flat-index decomposition n, ho, wo, co is checked on outputs with
    N > 1, Ho != Wo and Cout > 1, and every index is requested."""
    rng = _rng(41)
    A = _grid_uniform(rng, (33, 47))
    B = _grid_uniform(rng, (47, 21))
    C = _grid_uniform(rng, (33, 21))
    ref, scale = orc.sgemm("N", "N", 33, 21, 47, 0.7, A, 47, B, 21, 0.3, C, 21)
    rows, cols = np.divmod(np.arange(33 * 21), 21)
    r2, s2 = orc.sgemm_at("N", "N", 33, 21, 47, 0.7, A, 47, B, 21, 0.3, C, 21, rows, cols)
    assert np.array_equal(r2, ref.reshape(-1)) and np.array_equal(s2, scale.reshape(-1))
    x = _grid_uniform(rng, (2, 9, 8, 5))
    f = _grid_uniform(rng, (3, 3, 5, 4))
    ref, scale = orc.conv2d(x, f, (2, 1), (1, 0, 1, 2))
    flat = rng.permutation(ref.size)
    r2, s2 = orc.conv2d_at(x, f, (2, 1), (1, 0, 1, 2), flat)
    assert np.array_equal(r2, ref.reshape(-1)[flat]) and np.array_equal(s2, scale.reshape(-1)[flat])
    x = _grid_uniform(rng, (3, 11, 6, 4))
    f = _grid_uniform(rng, (3, 3, 4, 3))
    for m in (2, 4):
        ref, scale = orc.winograd(m, x, f, (1, 0, 2, 1))
        assert ref.shape[1] != ref.shape[2]
        flat = rng.permutation(ref.size)
        r2, s2 = orc.winograd_at(m, x, f, (1, 0, 2, 1), flat)
        assert np.array_equal(r2, ref.reshape(-1)[flat]), m
        assert np.array_equal(s2, scale.reshape(-1)[flat]), m


ALL_PINS = [pin_gemm_brute_force, pin_conv_brute_force, pin_gemm_identity_permutation,
            pin_conv_delta_filters, pin_all_ones_closed_forms, pin_invariants,
            pin_torch_float64, pin_layer_tables, pin_same_padding_property,
            pin_winograd_brute_force, pin_winograd_integer_exact, pin_winograd_scale,
            pin_winograd_f4_brute_force, pin_winograd_f4_scale, pin_winograd_tile_sizes_agree,
            pin_sampled_equals_whole]
