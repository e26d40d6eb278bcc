"""Full-size parity of every benchmark operation, in the launch configuration
the benchmark times (the default selection, with the workspace the library
asks for), checking every output tile.

Section 3.1.1 decomposes C into independent blocks, each a panel product, so
a wrong, lost or misplaced block leaves the others intact: every block has to
be looked at.  Two checks per operation:
  - integer inputs in [-8, 8]: every partial sum is an integer (a half-integer
    with beta = 0.5) far below 2^23, exact in fp32 and in the oracle's fp64 in
    any order, so the WHOLE output must equal the oracle bit for bit.  Outputs
    start as NaN (beta = 0) or hold integer C (beta = 0.5), so an unwritten
    element cannot pass; the GEMMs with beta = 0.5 are also run once with
    beta = 0 into a NaN-filled C.
  - uniform inputs on [-1, 1): the four corners of every output tile of the
    configuration that ran (and random outputs) within the 1e-5 bound.
The GEMM oracle is fed op(A) as an M x K and op(B) as an N x K row-major
matrix (its 'N', 'T' layout), which gives the same k-ordered sums as the
stored layouts with unit-stride reads.
"""
import re

import numpy as np
import pytest

import oracle
from paper_1904_05347_amd import workloads as wl
from tests.gpu_util import assert_parity, dev, host, require_gpu

pytestmark = pytest.mark.gpu

# configs 1, 3a, 3b and the step's three 4096^3 products
GEMM_CASES = [wl.GEMM_SMALL] + wl.GEMM_SWEEP
# the step's ten layers, the batch-1 parity layer and the alternative reading
CONV_CASES = wl.STEP_CONVS + [wl.CONV_SMALL, wl.RESNET_ALT]


def _config(pk, name):
    return {c["name"]: c for c in pk.configs()}[name]


def _oracle_gemm_whole(case, A, B, C, beta):
    opA = A if case.trans_a == "N" else np.ascontiguousarray(A.T)
    opBt = np.ascontiguousarray(B.T) if case.trans_b == "N" else B
    return oracle.sgemm("N", "T", case.M, case.N, case.K, case.alpha, opA, case.K, opBt, case.K,
                        beta, C, case.N)


def _tile_corners(M, N, bm, bn):
    """(rows, cols) of the four corners of every bm x bn tile of an M x N output."""
    r0 = np.arange(0, M, bm)
    c0 = np.arange(0, N, bn)
    r1 = np.minimum(r0 + bm, M) - 1
    c1 = np.minimum(c0 + bn, N) - 1
    rs = np.concatenate([r0, r1])
    cs = np.concatenate([c0, c1])
    rows = np.repeat(rs, cs.size)
    cols = np.tile(cs, rs.size)
    return rows, cols


@pytest.mark.parametrize("case", GEMM_CASES, ids=lambda c: c.name)
def test_gemm_fullsize_integer_whole_output(case):
    torch, pk = require_gpu()
    A, B, C = case.inputs(kind="int")
    ta, tb = case.trans_a == "T", case.trans_b == "T"
    dA, dB = dev(A), dev(B)
    dC = dev(C) if case.beta != 0.0 else torch.full((case.M, case.N), float("nan"), device="cuda")
    pk.gemm(dA, dB, dC, alpha=case.alpha, beta=case.beta, trans_a=ta, trans_b=tb)
    cfg = pk.last_config_name()
    out = host(dC)
    ref, _ = _oracle_gemm_whole(case, A, B, C if case.beta != 0.0 else None, case.beta)
    bad = np.count_nonzero(out.astype(np.float64) != ref)
    assert bad == 0, "%s %s: %d of %d outputs differ" % (case.name, cfg, bad, out.size)
    if case.beta != 0.0:
        # the same product with beta = 0 into NaN: no tile may keep its NaN
        dC0 = torch.full((case.M, case.N), float("nan"), device="cuda")
        pk.gemm(dA, dB, dC0, alpha=case.alpha, beta=0.0, trans_a=ta, trans_b=tb)
        cfg0 = pk.last_config_name()
        out0 = host(dC0)
        want = ref - case.beta * C.astype(np.float64)   # exact: every term is a small half-integer
        bad = np.count_nonzero(out0.astype(np.float64) != want)
        assert bad == 0, "%s beta=0 %s: %d of %d outputs differ" % (case.name, cfg0, bad, out0.size)


@pytest.mark.parametrize("case", GEMM_CASES, ids=lambda c: c.name)
def test_gemm_fullsize_every_tile_corner(case):
    torch, pk = require_gpu()
    A, B, C = case.inputs()
    dC = dev(C) if case.beta != 0.0 else torch.full((case.M, case.N), float("nan"), device="cuda")
    pk.gemm(dev(A), dev(B), dC, alpha=case.alpha, beta=case.beta,
            trans_a=case.trans_a == "T", trans_b=case.trans_b == "T")
    cfg = _config(pk, pk.last_config_name())
    out = host(dC)
    assert np.all(np.isfinite(out)), cfg["name"]
    rows, cols = _tile_corners(case.M, case.N, cfg["bm"], cfg["bn"])
    rng = np.random.default_rng(case.seed)
    rows = np.concatenate([rows, rng.integers(0, case.M, 1000)])
    cols = np.concatenate([cols, rng.integers(0, case.N, 1000)])
    ref, scale = oracle.sgemm_at(case.trans_a, case.trans_b, case.M, case.N, case.K, case.alpha,
                                 A, case.lda, B, case.ldb, case.beta, C if case.beta != 0.0 else None,
                                 case.ldc, rows, cols)
    mx = assert_parity(out[rows, cols], ref, scale, case.name + " " + cfg["name"])
    assert mx < 1e-6


def _conv_geometry(case):
    N, H, W, Cin = case.x_shape
    KH, KW, _, Cout = case.f_shape
    Ho, Wo = oracle.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
    return N, Ho, Wo, Cout


def _conv_tile_corners(cfg, N, Ho, Wo, Cout):
    """Flat NHWC indices of the corners of every output tile the
    configuration writes: BM rows x BN channels of the (N*Ho*Wo) x Cout
    matrix for the contraction kernels, rows x columns of one image x a
    channel block for the direct kernel (its name carries the tile)."""
    if cfg["kind"] == 2:
        m = re.match(r"direct_(\d+)x(\d+)x(\d+)", cfg["name"])
        tr, tc, tch = (int(v) for v in m.groups())
        h0 = np.arange(0, Ho, tr)
        w0 = np.arange(0, Wo, tc)
        c0 = np.arange(0, Cout, tch)
        hs = np.concatenate([h0, np.minimum(h0 + tr, Ho) - 1])
        ws = np.concatenate([w0, np.minimum(w0 + tc, Wo) - 1])
        cs = np.concatenate([c0, np.minimum(c0 + tch, Cout) - 1])
        n, h, w, c = np.meshgrid(np.arange(N), hs, ws, cs, indexing="ij")
        return (((n * Ho + h) * Wo + w) * Cout + c).reshape(-1)
    rows, cols = _tile_corners(N * Ho * Wo, Cout, cfg["bm"], cfg["bn"])
    return rows.astype(np.int64) * Cout + cols


@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: c.name)
def test_conv_fullsize_integer_whole_output(case):
    torch, pk = require_gpu()
    x, f = case.inputs(kind="int")
    shape = _conv_geometry(case)
    y = torch.full(shape, float("nan"), device="cuda")
    pk.conv2d_fwd(dev(x), dev(f), stride=case.stride, padding=case.pads, out=y)
    cfg = pk.last_config_name()
    out = host(y)
    ref, _ = oracle.conv2d(x, f, case.stride, case.pads)
    bad = np.count_nonzero(out.astype(np.float64) != ref)
    assert bad == 0, "%s %s: %d of %d outputs differ" % (case.name, cfg, bad, out.size)


@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: c.name)
def test_conv_fullsize_every_tile_corner(case):
    torch, pk = require_gpu()
    x, f = case.inputs()
    N, Ho, Wo, Cout = _conv_geometry(case)
    y = torch.full((N, Ho, Wo, Cout), float("nan"), device="cuda")
    pk.conv2d_fwd(dev(x), dev(f), stride=case.stride, padding=case.pads, out=y)
    cfg = _config(pk, pk.last_config_name())
    out = host(y).reshape(-1)
    assert np.all(np.isfinite(out)), cfg["name"]
    idx = _conv_tile_corners(cfg, N, Ho, Wo, Cout)
    rng = np.random.default_rng(case.seed)
    idx = np.concatenate([idx, rng.integers(0, out.size, 1000)])
    ref, scale = oracle.conv2d_at(x, f, case.stride, case.pads, idx)
    mx = assert_parity(out[idx], ref, scale, case.name + " " + cfg["name"])
    assert mx < 1e-6
