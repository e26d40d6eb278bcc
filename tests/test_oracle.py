"""The CPU oracle against its pins (brute force, closed forms, invariants,
torch float64, the paper's layer tables), and the tolerance against
reduced-precision arithmetic."""
import numpy as np
import pytest

import oracle
from tests import pins


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.Oracle(oracle._LIB_PATH)


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_invalid_arguments_rejected(orc):
    a = np.zeros((4, 4), np.float32)
    with pytest.raises(ValueError):
        orc.sgemm("X", "N", 4, 4, 4, 1.0, a, 4, a, 4, 0.0, None, 4)
    with pytest.raises(ValueError):
        orc.sgemm("N", "N", 4, 4, 4, 1.0, a, 3, a, 4, 0.0, None, 4)  # lda < K
    with pytest.raises(ValueError):
        orc.conv2d_out_dims(2, 2, 3, 3, 1, 1, 0, 0, 0, 0)  # window larger than image
    with pytest.raises(ValueError):
        orc.sgemm_at("N", "N", 4, 4, 4, 1.0, a, 4, a, 4, 0.0, None, 4, [4], [0])


# ------------------------------------------- the tolerance has teeth (P8)

def _round_significand(x, bits):
    """Round-to-nearest-even of fp32 values to `bits` significand bits (incl. the implicit one)."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    drop = 24 - bits
    half = np.uint64(1 << (drop - 1))
    lsb = (u >> np.uint64(drop)) & np.uint64(1)
    u = (u + half - np.uint64(1) + lsb) & ~np.uint64((1 << drop) - 1)
    return u.astype(np.uint32).view(np.float32)


@pytest.fixture(scope="module")
def gemm512(orc):
    from paper_1904_05347_amd import workloads as wl
    case = wl.GEMM_SMALL
    A, B, C = case.inputs()
    ref, scale = orc.sgemm("N", "N", 512, 512, 512, 1.0, A, 512, B, 512, 0.0, None, 512)
    return A, B, ref, scale


def test_fp32_accumulation_passes(gemm512):
    A, B, ref, scale = gemm512
    # a sequential fp32 dot product per element: the crudest fp32 summation order
    acc = np.zeros((512, 512), np.float32)
    for k in range(512):
        acc += np.outer(A[:, k], B[k, :]).astype(np.float32)
    ok, mx, _ = oracle.within_tolerance(acc, ref, scale)
    assert ok, mx
    assert mx < 5e-6


@pytest.mark.parametrize("bits,name", [(11, "xf32/tf32 inputs"), (8, "bf16 inputs")])
def test_reduced_precision_fails(gemm512, bits, name):
    A, B, ref, scale = gemm512
    Ar = _round_significand(A, bits).astype(np.float64)
    Br = _round_significand(B, bits).astype(np.float64)
    approx = Ar @ Br
    ok, mx, n_bad = oracle.within_tolerance(approx, ref, scale)
    assert not ok, (name, mx)
    assert n_bad > 1000, (name, n_bad)


def test_tolerance_flags_nan_and_single_error(gemm512):
    A, B, ref, scale = gemm512
    good = ref.astype(np.float32)
    assert oracle.within_tolerance(good, ref, scale)[0]
    bad = good.copy()
    bad[17, 400] = np.nan
    assert oracle.within_tolerance(bad, ref, scale)[2] == 1
    bad = good.copy()
    bad[3, 3] += np.float32(1e-4 * scale[3, 3])
    assert oracle.within_tolerance(bad, ref, scale)[2] == 1


def test_paper_gemm_table_local_memory():
    """Table 2's local-memory column is (h*r + w*c) elements of a 64-byte cache
    line (X = 16 floats, Table 1), 4 bytes each, doubled for double buffering."""
    X = 16
    for row in pins.read_golden("gemm_configs.csv"):
        h, w, r, c = (int(row[k]) for k in "hwrc")
        assert int(row["registers"]) == h * w
        assert int(row["work_group"]) == r * c
        if row["local_kib"]:
            assert (h * r * X + X * w * c) * 4 * 2 == int(row["local_kib"]) * 1024, row["name"]
