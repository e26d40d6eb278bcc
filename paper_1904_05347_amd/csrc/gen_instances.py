"""Writes the pk_inst_*.hip files: the compiled tile-parameter space.

Each entry (BM, BN, BK, WAVES_M, WAVES_N, VA, VB, OCC) becomes one kernel
instance per operand layout.  OCC is the number of waves per SIMD the register
allocation must leave room for (1 = no constraint).  Run from this directory:
``python gen_instances.py``; the outputs are committed sources.
"""
import os

HERE = os.path.dirname(os.path.abspath(__file__))

# GEMM tiles for the three layouts the benchmarks use (NN, TN, NT).
GEMM_TILES = [
    (128, 128, 16, 2, 2, 4, 4, 1), (128, 128, 16, 2, 2, 4, 4, 4),
    (128, 128, 16, 4, 1, 4, 4, 1), (128, 128, 16, 4, 1, 4, 4, 4),
    (128, 128, 16, 1, 4, 4, 4, 1), (128, 128, 16, 1, 4, 4, 4, 4),
    (128, 128, 32, 2, 2, 4, 4, 1), (128, 128, 32, 2, 2, 4, 4, 2),
    (256, 128, 16, 2, 2, 4, 4, 1), (256, 128, 16, 2, 2, 4, 4, 2),
    (128, 256, 16, 2, 2, 4, 4, 1), (128, 256, 16, 2, 2, 4, 4, 2),
    (256, 128, 32, 2, 2, 4, 4, 1), (256, 256, 16, 2, 2, 4, 4, 1),
    (256, 256, 16, 2, 4, 4, 4, 2), (256, 256, 16, 4, 2, 4, 4, 2), (256, 256, 32, 2, 4, 4, 4, 2),
    (256, 128, 32, 4, 2, 4, 4, 2), (256, 128, 16, 4, 2, 4, 4, 2),
    (128, 64, 16, 2, 2, 4, 4, 1), (128, 64, 32, 2, 2, 4, 4, 1),
    (64, 64, 16, 2, 2, 4, 4, 1), (64, 64, 32, 2, 2, 4, 4, 1),
    (128, 128, 64, 2, 4, 4, 4, 2),
    (64, 64, 16, 2, 2, 1, 1, 1),
]
# Persistent forms (grid = resident work-groups, each looping over tiles).
GEMM_PERSISTENT = [
    (64, 64, 16, 2, 2, 4, 4, 1), (64, 64, 32, 2, 2, 4, 4, 1), (128, 64, 16, 2, 2, 4, 4, 1),
    (128, 64, 32, 2, 2, 4, 4, 1), (128, 128, 16, 2, 4, 4, 4, 2), (128, 128, 32, 2, 4, 4, 4, 2),
    (256, 128, 16, 4, 2, 4, 4, 2), (256, 256, 16, 2, 4, 4, 4, 2), (256, 256, 32, 2, 4, 4, 4, 2),
]
CONV_PERSISTENT = [
    (64, 64, 16, 2, 2, 4, 4, 1), (64, 64, 32, 2, 2, 4, 4, 1), (128, 64, 16, 2, 2, 4, 4, 1),
    (128, 128, 16, 2, 4, 4, 4, 2), (128, 128, 32, 2, 4, 4, 4, 2), (256, 128, 16, 4, 2, 4, 4, 2),
]
# Stream-K forms (resident work-groups share the (tile, K-block) iterations
# evenly; partial tiles are finished by their last contributor).  They need a
# workspace, so they serve convolutions (the 1x1 stride-1 layers run the NN
# GEMM instances through the convolution call).
GEMM_STREAMK = [
    (64, 64, 32, 2, 2, 4, 4, 1), (128, 64, 32, 2, 2, 4, 4, 1), (128, 128, 32, 2, 4, 4, 4, 2),
    (256, 128, 32, 4, 2, 4, 4, 2),
]
CONV_STREAMK = [
    (64, 64, 32, 2, 2, 4, 4, 1), (128, 64, 32, 2, 2, 4, 4, 1), (128, 128, 32, 2, 4, 4, 4, 2),
    (256, 128, 32, 4, 2, 4, 4, 2), (256, 256, 16, 2, 4, 4, 4, 2),
]
# B-resident streaming forms (NN only; K == BK and N == BN exactly): the
# 1x1 convolutions with 64 input channels and 64 or 256 output channels.
GEMM_BRES = [(64, 64, 64, 2, 2, 1), (128, 64, 64, 4, 1, 1), (64, 256, 64, 2, 4, 2), (32, 256, 64, 1, 8, 2)]
# Ablation forms (NN only): 2-wide and 4-byte loads of a 128 x 128 tile beside
# its 16-byte form, and single-LDS-stage (not double-buffered) twins of
# instances the benchmarks use ("_s1").
ABLATION_TILES = [(128, 128, 16, 2, 2, 2, 2, 1), (128, 128, 16, 2, 2, 1, 1, 1)]
SINGLE_STAGE = [(128, 128, 16, 2, 2, 4, 4, 1), (64, 64, 32, 2, 2, 4, 4, 1), (256, 256, 32, 2, 4, 4, 4, 2)]
# NN-only tiles for short reductions (1x1 layers with K = 64 .. 256): the
# whole reduction in one or few K-blocks, single LDS stage so that more
# work-groups fit on a CU, and full-width tiles for N = 256.
NN_SHORT_K = [(64, 64, 64, 2, 2, 4, 4, 1), (128, 64, 64, 2, 2, 4, 4, 1), (64, 256, 32, 1, 4, 4, 4, 1),
              (128, 256, 32, 2, 4, 4, 4, 2)]
NN_SHORT_K_1S = [(64, 64, 64, 2, 2, 4, 4, 1), (128, 64, 64, 2, 2, 4, 4, 1), (128, 128, 64, 2, 4, 4, 4, 2)]

# Loads two K-blocks ahead ("_d2"): small tiles whose K-block is too short
# to cover the global-load latency (NN GEMM and convolution).
DEEP = [(64, 64, 16, 2, 2, 4, 4, 1), (64, 64, 32, 2, 2, 4, 4, 1), (128, 64, 32, 2, 2, 4, 4, 1),
        (64, 128, 32, 2, 2, 4, 4, 1), (128, 128, 32, 2, 4, 4, 4, 2)]

# K split among groups of waves inside the work-group ("_kN"): products with
# few tiles and a long reduction (the paper's GEMM sweep).  (BM, BN, BK,
# WAVES_M, WAVES_N, groups, steps loaded ahead (2: "_d2"), VA, VB, OCC)
KSPLIT = [(64, 64, 16, 2, 2, 4, 1, 4, 4, 1), (64, 64, 32, 2, 2, 4, 1, 4, 4, 1), (64, 64, 32, 2, 2, 2, 1, 4, 4, 1),
          (128, 64, 16, 2, 2, 4, 1, 4, 4, 1), (128, 128, 16, 2, 2, 2, 1, 4, 4, 1), (32, 64, 32, 1, 2, 4, 1, 4, 4, 1),
          (32, 64, 16, 1, 2, 8, 1, 4, 4, 1),
          (64, 64, 16, 2, 2, 4, 2, 4, 4, 1), (64, 64, 32, 2, 2, 4, 2, 4, 4, 1), (64, 64, 32, 2, 2, 2, 2, 4, 4, 1),
          (32, 64, 32, 1, 2, 4, 2, 4, 4, 1), (32, 64, 16, 1, 2, 8, 2, 4, 4, 1)]

# Direct-to-LDS staging ("_dmaS", S LDS stages; NN, TN, NT): the
# register-staged loader's alternative, beside the same tiles.  (BM, BN, BK, WAVES_M, WAVES_N,
# stages, OCC)
DMA = [(256, 256, 16, 2, 4, 2, 2), (256, 256, 16, 2, 4, 3, 2), (256, 256, 16, 2, 4, 4, 2), (256, 256, 32, 2, 4, 2, 2),
       (128, 128, 32, 2, 4, 2, 2), (128, 128, 32, 2, 4, 3, 2), (128, 128, 32, 2, 4, 4, 2),
       (128, 128, 16, 2, 2, 3, 1), (128, 128, 16, 2, 2, 4, 1), (64, 64, 32, 2, 2, 3, 1),
       (64, 64, 32, 2, 2, 2, 1), (64, 64, 16, 2, 2, 3, 1)]

# K-split forms of the direct-to-LDS contraction ("_kN_..._dmaS"): (BM, BN,
# BK, WAVES_M, WAVES_N, groups, stages, OCC)
DMA_KSPLIT = [(32, 64, 32, 1, 2, 4, 2, 1), (32, 64, 32, 1, 2, 4, 3, 1), (64, 64, 32, 2, 2, 2, 2, 1),
              (64, 64, 32, 2, 2, 2, 3, 1), (32, 64, 16, 1, 2, 8, 3, 1), (64, 64, 32, 2, 2, 4, 2, 1)]

# ... and for the convolution's gather: few output tiles, long reductions
# (deep layers at small batch, strided 1x1 layers).
DMA_KSPLIT_CONV = [(64, 64, 32, 2, 2, 2, 3, 1), (64, 64, 32, 2, 2, 4, 2, 1), (128, 128, 32, 2, 2, 2, 2, 1)]

# Stream-K forms of the direct-to-LDS contraction (NN GEMM and convolution).
DMA_STREAMK = [(128, 128, 32, 2, 4, 2, 2), (128, 128, 16, 2, 2, 3, 1), (128, 128, 32, 2, 4, 3, 2)]

# TT only needs a large, a small and a scalar-load tile.
TT_TILES = [(128, 128, 16, 2, 2, 4, 4, 1), (64, 64, 16, 2, 2, 4, 4, 1), (64, 64, 16, 2, 2, 1, 1, 1)]

CONV_TILES = [
    (128, 128, 16, 2, 2, 4, 4, 1), (128, 128, 16, 2, 2, 4, 4, 4),
    (128, 128, 32, 2, 2, 4, 4, 1), (128, 128, 32, 2, 2, 4, 4, 2),
    (256, 128, 16, 2, 2, 4, 4, 1), (256, 128, 16, 2, 2, 4, 4, 2),
    (128, 256, 16, 2, 2, 4, 4, 1), (128, 256, 16, 2, 2, 4, 4, 2),
    (256, 128, 32, 2, 2, 4, 4, 1),
    (256, 256, 16, 2, 4, 4, 4, 2), (256, 256, 32, 2, 4, 4, 4, 2),
    (256, 128, 16, 4, 2, 4, 4, 2), (256, 128, 32, 4, 2, 4, 4, 2),
    (128, 256, 16, 2, 4, 4, 4, 2), (128, 128, 16, 2, 4, 4, 4, 2), (128, 128, 32, 2, 4, 4, 4, 2),
    (128, 64, 16, 2, 2, 4, 4, 1), (128, 64, 32, 2, 2, 4, 4, 1),
    (256, 64, 16, 4, 1, 4, 4, 1),
    (64, 64, 16, 2, 2, 4, 4, 1), (64, 64, 32, 2, 2, 4, 4, 1),
    (128, 128, 64, 2, 4, 4, 4, 2),
    (128, 64, 16, 2, 2, 1, 4, 1), (256, 64, 16, 4, 1, 1, 4, 1),
    (64, 64, 16, 2, 2, 1, 1, 1),
    (64, 64, 64, 2, 2, 4, 4, 1), (128, 64, 64, 2, 2, 4, 4, 1),
]


def _name(kind, t, layout=None, persistent=False, single=False, streamk=False, deep=False):
    bm, bn, bk, wm, wn, va, vb, occ = t
    s = "%s_%dx%dx%d_w%dx%d" % (kind, bm, bn, bk, wm, wn)
    if layout:
        s += "_" + layout
    s += "_v%d%d" % (va, vb)
    if occ > 1:
        s += "_o%d" % occ
    if persistent:
        s += "_p"
    if single:
        s += "_s1"
    if streamk:
        s += "_sk"
    if deep:
        s += "_d2"
    return s


def _file(fname, header, func, entries):
    body = "\n".join("        %s," % e for e in entries)
    text = '''// %s -- %s
// Generated by gen_instances.py.
#include "pk_instance_common.hpp"

namespace pk {

const Config *%s(int *count)
{
    static const Config kTable[] = {
%s
    };
    *count = (int)(sizeof(kTable) / sizeof(kTable[0]));
    return kTable;
}

}  // namespace pk
''' % (fname, header, func, body)
    with open(os.path.join(HERE, fname), "w") as fh:
        fh.write(text)


def main():
    for layout, ta, tb, tiles in [("nn", 0, 0, GEMM_TILES), ("tn", 1, 0, GEMM_TILES),
                                  ("nt", 0, 1, GEMM_TILES), ("tt", 1, 1, TT_TILES)]:
        entries = []
        for t in tiles:
            bm, bn, bk, wm, wn, va, vb, occ = t
            entries.append("PK_GEMM(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % (_name("gemm", t, layout), bm, bn, bk, wm, wn, ta, tb, va, vb, occ))
        for t in (GEMM_PERSISTENT if layout != "tt" else []):
            bm, bn, bk, wm, wn, va, vb, occ = t
            entries.append("PK_GEMM_P(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % (_name("gemm", t, layout, True), bm, bn, bk, wm, wn, ta, tb, va, vb, occ))
        for t in (GEMM_STREAMK if layout == "nn" else []):
            bm, bn, bk, wm, wn, va, vb, occ = t
            entries.append("PK_GEMM_SK(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % (_name("gemm", t, layout, streamk=True), bm, bn, bk, wm, wn, ta, tb, va, vb, occ))
        for t in (GEMM_BRES if layout == "nn" else []):
            bm, bn, bk, wm, wn, occ = t
            entries.append("PK_GEMM_BRES(%s, %d, %d, %d, %d, %d, %d)"
                           % ("gemm_%dx%dx%d_w%dx%d_nn_v44%s_br" % (bm, bn, bk, wm, wn, "_o%d" % occ if occ > 1 else ""),
                              bm, bn, bk, wm, wn, occ))
        for t in (ABLATION_TILES if layout == "nn" else []):
            bm, bn, bk, wm, wn, va, vb, occ = t
            entries.append("PK_GEMM(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % (_name("gemm", t, layout), bm, bn, bk, wm, wn, ta, tb, va, vb, occ))
        for t in (NN_SHORT_K if layout == "nn" else []):
            bm, bn, bk, wm, wn, va, vb, occ = t
            entries.append("PK_GEMM(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % (_name("gemm", t, layout), bm, bn, bk, wm, wn, ta, tb, va, vb, occ))
        for t in (KSPLIT if layout != "tt" else []):
            bm, bn, bk, wm, wn, ks, ahead, va, vb, occ = t
            entries.append("PK_GEMM_KS(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % ("gemm_%dx%dx%d_w%dx%d_k%d_%s_v%d%d%s" % (bm, bn, bk, wm, wn, ks, layout, va, vb,
                                                                    "_d2" if ahead == 2 else ""),
                              bm, bn, bk, wm, wn, ks, ahead, ta, tb, va, vb, occ))
        for t in (DMA if layout != "tt" else []):
            bm, bn, bk, wm, wn, st, occ = t
            entries.append("PK_GEMM_DMA(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % ("gemm_%dx%dx%d_w%dx%d_%s_v44%s_dma%d" % (bm, bn, bk, wm, wn, layout,
                                                                     "_o%d" % occ if occ > 1 else "", st),
                              bm, bn, bk, wm, wn, st, ta, tb, occ))
        for t in (DMA_KSPLIT if layout != "tt" else []):
            bm, bn, bk, wm, wn, ks, st, occ = t
            if (ta and bm % 64) or (not tb and bn % 64):
                continue  # an m- or n-contiguous tile needs 64 columns for its swizzle
            entries.append("PK_GEMM_DMA_KS(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % ("gemm_%dx%dx%d_w%dx%d_k%d_%s_v44_dma%d" % (bm, bn, bk, wm, wn, ks, layout, st),
                              bm, bn, bk, wm, wn, ks, st, ta, tb, occ))
        for t in (DMA_STREAMK if layout == "nn" else []):
            bm, bn, bk, wm, wn, st, occ = t
            entries.append("PK_GEMM_DMA_SK(%s, %d, %d, %d, %d, %d, %d, %d)"
                           % ("gemm_%dx%dx%d_w%dx%d_nn_v44%s_dma%d_sk" % (bm, bn, bk, wm, wn,
                                                                        "_o%d" % occ if occ > 1 else "", st),
                              bm, bn, bk, wm, wn, st, occ))
        for t in (DEEP if layout == "nn" else []):
            bm, bn, bk, wm, wn, va, vb, occ = t
            entries.append("PK_GEMM_D(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % (_name("gemm", t, layout, deep=True), bm, bn, bk, wm, wn, ta, tb, va, vb, occ))
        for t in (SINGLE_STAGE + NN_SHORT_K_1S if layout == "nn" else []):
            bm, bn, bk, wm, wn, va, vb, occ = t
            entries.append("PK_GEMM_1S(%s, %d, %d, %d, %d, %d, %d, %d, %d, %d, %d)"
                           % (_name("gemm", t, layout, single=True), bm, bn, bk, wm, wn, ta, tb, va, vb, occ))
        desc = "GEMM instances for op(A) = %s, op(B) = %s." % ("A^T" if ta else "A", "B^T" if tb else "B")
        _file("pk_inst_gemm_%s.hip" % layout, desc, "configs_gemm_%s" % layout, entries)
    entries = []
    for t in CONV_TILES:
        bm, bn, bk, wm, wn, va, vb, occ = t
        entries.append("PK_CONV(%s, %d, %d, %d, %d, %d, %d, %d, %d)"
                       % (_name("conv", t), bm, bn, bk, wm, wn, va, vb, occ))
    for t in CONV_PERSISTENT:
        bm, bn, bk, wm, wn, va, vb, occ = t
        entries.append("PK_CONV_P(%s, %d, %d, %d, %d, %d, %d, %d, %d)"
                       % (_name("conv", t, None, True), bm, bn, bk, wm, wn, va, vb, occ))
    for t in DEEP:
        bm, bn, bk, wm, wn, va, vb, occ = t
        entries.append("PK_CONV_D(%s, %d, %d, %d, %d, %d, %d, %d, %d)"
                       % (_name("conv", t, deep=True), bm, bn, bk, wm, wn, va, vb, occ))
    for t in CONV_STREAMK:
        bm, bn, bk, wm, wn, va, vb, occ = t
        entries.append("PK_CONV_SK(%s, %d, %d, %d, %d, %d, %d, %d, %d)"
                       % (_name("conv", t, streamk=True), bm, bn, bk, wm, wn, va, vb, occ))
    for t in DMA:
        bm, bn, bk, wm, wn, st, occ = t
        if (4 * (64 * wm * wn // 64)) % (bk // 4):
            continue  # the gather needs one chunk per lane across its copy slots
        entries.append("PK_CONV_DMA(%s, %d, %d, %d, %d, %d, %d, %d)"
                       % ("conv_%dx%dx%d_w%dx%d_v44%s_dma%d" % (bm, bn, bk, wm, wn, "_o%d" % occ if occ > 1 else "", st),
                          bm, bn, bk, wm, wn, st, occ))
    for t in DMA_KSPLIT_CONV:
        bm, bn, bk, wm, wn, ks, st, occ = t
        entries.append("PK_CONV_DMA_KS(%s, %d, %d, %d, %d, %d, %d, %d, %d)"
                       % ("conv_%dx%dx%d_w%dx%d_k%d_v44_dma%d" % (bm, bn, bk, wm, wn, ks, st),
                          bm, bn, bk, wm, wn, ks, st, occ))
    for t in DMA_STREAMK:
        bm, bn, bk, wm, wn, st, occ = t
        entries.append("PK_CONV_DMA_SK(%s, %d, %d, %d, %d, %d, %d, %d)"
                       % ("conv_%dx%dx%d_w%dx%d_v44%s_dma%d_sk" % (bm, bn, bk, wm, wn, "_o%d" % occ if occ > 1 else "", st),
                          bm, bn, bk, wm, wn, st, occ))
    _file("pk_inst_conv.hip", "implicit-GEMM convolution instances (A gathered from an NHWC "
          "image, B the HWIO filter viewed as (KH*KW*Cin) x Cout).", "configs_conv", entries)


if __name__ == "__main__":
    main()
