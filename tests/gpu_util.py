"""Helpers for the GPU parity tests: device transfer, sampling, comparison."""
from __future__ import annotations

import numpy as np
import pytest

import oracle


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    import paper_1904_05347_amd as pk
    pk.load()  # raises when libpk.so is missing: no fallback path exists
    return torch, pk


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def assert_parity(result, ref, scale, what, extra=None, rtol=oracle.RTOL):
    ok, mx, n_bad = oracle.within_tolerance(result, ref, scale, rtol=rtol, extra=extra)
    if not ok:
        r = np.asarray(result, np.float64).reshape(-1)
        rf = np.asarray(ref).reshape(-1)
        bound = rtol * np.asarray(scale).reshape(-1)
        if extra is not None:
            bound = bound + rtol * np.asarray(extra).reshape(-1)
        bad = np.nonzero(~(np.abs(r - rf) <= bound))[0][:5]
        detail = ", ".join("[%d] got %r want %r bound %.3g" % (i, r[i], rf[i], bound[i]) for i in bad)
        raise AssertionError("%s: %d elements outside |err| <= %g*scale (max ratio %.3g); %s"
                             % (what, n_bad, rtol, mx, detail))
    return mx


def sample_rows_cols(M, N, count, seed, tiles=(64, 128)):
    """Sample (row, col) pairs: corners, tile boundaries, then random."""
    rng = np.random.default_rng(seed)
    special_r = {0, M - 1}
    special_c = {0, N - 1}
    for t in tiles:
        for b in range(t, M, t * max(1, M // (t * 8))):
            special_r.update({b - 1, b})
        for b in range(t, N, t * max(1, N // (t * 8))):
            special_c.update({b - 1, b})
    sr = np.array(sorted(r for r in special_r if 0 <= r < M))
    sc = np.array(sorted(c for c in special_c if 0 <= c < N))
    rr = [np.repeat(sr, len(sc)), np.tile(sc, len(sr))]
    rows = np.concatenate([rr[0], rng.integers(0, M, count)])
    cols = np.concatenate([rr[1], rng.integers(0, N, count)])
    return rows, cols


def sample_conv_outputs(N, Ho, Wo, Cout, count, seed):
    """Flat NHWC output indices: every border pixel class and random interior ones."""
    rng = np.random.default_rng(seed)
    hs = sorted({0, 1, Ho // 2, Ho - 2, Ho - 1} & set(range(Ho)))
    ws = sorted({0, 1, Wo // 2, Wo - 2, Wo - 1} & set(range(Wo)))
    ns = sorted({0, N - 1})
    cs = sorted({0, Cout - 1, Cout // 2} & set(range(Cout)))
    pix = [((n * Ho + h) * Wo + w) * Cout + c for n in ns for h in hs for w in ws for c in cs]
    rnd = rng.integers(0, N * Ho * Wo * Cout, count)
    return np.concatenate([np.array(pix, dtype=np.int64), rnd.astype(np.int64)])
