"""The automated parameter search on the GPU: the tuner times the compiled
configurations, records the fastest, and later calls with the same key run
it -- with results still matching the oracle.  Shapes here are used by no
other test, and the runtime table is emptied afterwards."""
import numpy as np
import pytest

import oracle
from paper_1904_05347_amd import workloads as wl
from tests.gpu_util import assert_parity, dev, host, require_gpu

pytestmark = pytest.mark.gpu


def test_tune_gemm_records_and_is_used():
    torch, pk = require_gpu()
    rng = np.random.default_rng(301)
    M, N, K = 768, 640, 320
    A = wl.uniform(rng, M * K).reshape(M, K)
    B = wl.uniform(rng, K * N).reshape(K, N)
    dA, dB = dev(A), dev(B)
    try:
        pk.gemm(dA, dB)
        default = pk.last_config_name()
        scratch = torch.empty((M, N), dtype=torch.float32, device="cuda")
        r = pk.tune_gemm(dA, dB, scratch, iters=3)
        assert r["candidates"] >= 20 and r["ms"] > 0 and r["splits"] == 1
        names = {c["name"]: c for c in pk.configs()}
        best = names[r["config"]]
        assert best["kind"] == 0 and not best["trans_a"] and not best["trans_b"]
        C = pk.gemm(dA, dB)
        assert pk.last_config_name() == r["config"]
        ref, scale = oracle.sgemm("N", "N", M, N, K, 1.0, A, K, B, N, 0.0, None, N)
        assert_parity(host(C), ref, scale, "tuned " + r["config"])
        # another shape is untouched; a reset restores the built-in choice
        pk.gemm(dA[:512], dB)
        pk.tune_reset()
        pk.gemm(dA, dB)
        assert pk.last_config_name() == default
    finally:
        pk.tune_reset()


def test_tune_conv_records_config_and_split():
    torch, pk = require_gpu()
    rng = np.random.default_rng(302)
    N, H, W, Cin, Cout = 2, 20, 20, 32, 48
    x = wl.uniform(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.uniform(rng, 9 * Cin * Cout).reshape(3, 3, Cin, Cout)
    dx, df = dev(x), dev(f)
    ws = torch.empty(8 * N * H * W * Cout, dtype=torch.float32, device="cuda")
    try:
        r = pk.tune_conv2d(dx, df, padding=(1, 1, 1, 1), workspace=ws, iters=3)
        assert r["candidates"] >= 20 and 1 <= r["splits"] <= 8
        kind = {c["name"]: c["kind"] for c in pk.configs()}[r["config"]]
        assert kind in (1, 2)
        y = pk.conv2d_fwd(dx, df, padding=(1, 1, 1, 1), workspace=ws)
        assert pk.last_config_name() == r["config"]
        ref, scale = oracle.conv2d(x, f, (1, 1), (1, 1, 1, 1))
        assert_parity(host(y), ref, scale, "tuned conv " + r["config"])
        # the same problem without a workspace falls back to an unsplit run of the same configuration
        y2 = pk.conv2d_fwd(dx, df, padding=(1, 1, 1, 1))
        assert pk.last_config_name() == r["config"]
        assert_parity(host(y2), ref, scale, "tuned conv, no workspace")
    finally:
        pk.tune_reset()


def test_tune_conv_window_key_and_empty():
    torch, pk = require_gpu()
    x = torch.rand((1, 9, 9, 8), device="cuda")
    f = torch.rand((3, 1, 8, 8), device="cuda")
    with pytest.raises(pk.PkError):  # KH != KW: outside the table's key
        pk.tune_conv2d(x, f, padding=(1, 0, 1, 0))
    x0 = torch.rand((0, 9, 9, 8), device="cuda")
    f3 = torch.rand((3, 3, 8, 8), device="cuda")
    assert pk.tune_conv2d(x0, f3)["config"] == ""
    pk.tune_reset()


def test_tuned_padded_1x1_does_not_reach_the_gemm_path():
    """A padded 1x1 window has the (M, K, window, stride) of an unpadded one
    but runs through the gather; the unpadded one runs as a plain GEMM.  The
    search's record for the first must never be taken by the second: each
    keeps a configuration of its own path, with oracle parity."""
    torch, pk = require_gpu()
    rng = np.random.default_rng(303)
    Cin = Cout = 64
    xp = wl.uniform(rng, 54 * 54 * Cin).reshape(1, 54, 54, Cin)    # pad 1 -> 56 x 56 outputs
    xu = wl.uniform(rng, 56 * 56 * Cin).reshape(1, 56, 56, Cin)    # no pad -> 56 x 56 outputs
    f = wl.uniform(rng, Cin * Cout).reshape(1, 1, Cin, Cout)
    dxp, dxu, df = dev(xp), dev(xu), dev(f)
    names = {c["name"]: c for c in pk.configs()}
    try:
        r = pk.tune_conv2d(dxp, df, padding=(1, 1, 1, 1), iters=2)
        assert names[r["config"]]["kind"] in (1, 2)   # a gather (or direct) configuration
        yp = pk.conv2d_fwd(dxp, df, padding=(1, 1, 1, 1))
        assert pk.last_config_name() == r["config"]
        ref, scale = oracle.conv2d(xp, f, (1, 1), (1, 1, 1, 1))
        assert_parity(host(yp), ref, scale, "tuned padded 1x1 " + r["config"])
        yu = pk.conv2d_fwd(dxu, df, padding=(0, 0, 0, 0))
        used = pk.last_config_name()
        assert used.startswith("gemm_") and names[used]["kind"] == 0, used
        ref, scale = oracle.conv2d(xu, f, (1, 1), (0, 0, 0, 0))
        assert_parity(host(yu), ref, scale, "unpadded 1x1 after tuning the padded one " + used)
        assert pk.conv2d_workspace_bytes(1, 56, 56, Cin, 1, 1, Cout, 1, 1, 0, 0, 0, 0) >= 0
    finally:
        pk.tune_reset()
