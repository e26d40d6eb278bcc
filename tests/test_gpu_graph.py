"""The library's calls captured into a HIP graph and replayed.

Every call launches kernels only on the caller's stream (the stream-K arrival
counters are cleared by a kernel, not a memset), so a captured sequence
replays to the same bits as the eager calls: checked on three replays, each
after the outputs are overwritten and other eager work has run, for a
stream-K convolution, a split-K convolution and a beta != 0 GEMM (which
reads C, reset before each replay)."""
import numpy as np
import pytest

from paper_1904_05347_amd import workloads as wl
from tests.gpu_util import dev, host, require_gpu

pytestmark = pytest.mark.gpu


def test_graph_replay_matches_eager():
    torch, pk = require_gpu()
    rng = np.random.default_rng(2026)
    # stream-K convolution (the selector's choice for this layer shape class)
    x1 = dev(wl.uniform(rng, 4 * 28 * 28 * 256).reshape(4, 28, 28, 256))
    f1 = dev(wl.uniform(rng, 9 * 256 * 512).reshape(3, 3, 256, 512))
    sk = next(c["name"] for c in pk.configs() if c["streamk"] and c["kind"] == 1)
    ws1 = torch.empty(64 << 20, dtype=torch.float32, device="cuda")
    y1 = torch.empty((4, 28, 28, 512), dtype=torch.float32, device="cuda")
    # split-K convolution
    x2 = dev(wl.uniform(rng, 2 * 14 * 14 * 128).reshape(2, 14, 14, 128))
    f2 = dev(wl.uniform(rng, 9 * 128 * 96).reshape(3, 3, 128, 96))
    ws2 = torch.empty(8 * 2 * 14 * 14 * 96, dtype=torch.float32, device="cuda")
    y2 = torch.empty((2, 14, 14, 96), dtype=torch.float32, device="cuda")
    # GEMM, beta = 0.5 (reads C)
    A = dev(wl.uniform(rng, 384 * 1024).reshape(384, 1024))
    B = dev(wl.uniform(rng, 1024 * 200).reshape(1024, 200))
    C0 = dev(wl.uniform(rng, 384 * 200).reshape(384, 200))
    C = C0.clone()

    def calls():
        pk.force_config(sk)
        try:
            pk.conv2d_fwd(x1, f1, padding=(1, 1, 1, 1), out=y1, workspace=ws1)
        finally:
            pk.force_config(None)
        pk.force_splits(4)
        try:
            pk.conv2d_fwd(x2, f2, padding=(1, 1, 1, 1), out=y2, workspace=ws2)
        finally:
            pk.force_splits(0)
        pk.gemm(A, B, C, alpha=1.0, beta=0.5)

    calls()
    torch.cuda.synchronize()
    ref = [host(y1).copy(), host(y2).copy(), host(C).copy()]
    C.copy_(C0)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (y1, y2):
            t.fill_(float("nan"))
        C.copy_(C0)
        # other eager work of the program between replays
        pk.conv2d_fwd(x2, f2, padding=(1, 1, 1, 1))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [host(y1), host(y2), host(C)]
        for k, (a, b) in enumerate(zip(got, ref)):
            assert np.array_equal(a, b), (rep, k)
    del g
