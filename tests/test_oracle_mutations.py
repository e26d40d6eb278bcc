"""Each plausible mistake, planted in a copy of the oracle source and built
on the CPU, must make at least one pin fail: the pins have teeth."""
import os
import subprocess
import sys

import pytest

import oracle

MUTATIONS = {
    "pad offset dropped": ("ho * p->sh - p->pt + kh", "ho * p->sh + kh"),
    "left pad used for rows": ("ho * p->sh - p->pt + kh", "ho * p->sh - p->pl + kh"),
    "filter flipped": ("double fv = (double)p->f[((kh * p->KW + kw)",
                       "double fv = (double)p->f[(((p->KH - 1 - kh) * p->KW + (p->KW - 1 - kw))"),
    "filter taps transposed": ("p->f[((kh * p->KW + kw) * p->C + ci)", "p->f[((kw * p->KH + kh) * p->C + ci)"),
    "input channels reversed": ("p->W + iw) * p->C + ci]", "p->W + iw) * p->C + (p->C - 1 - ci)]"),
    "stride ignored on columns": ("int64_t iw = wo * p->sw - p->pl + kw;", "int64_t iw = wo - p->pl + kw;"),
    "no bounds check": ("int inside = ih >= 0 && ih < p->H && iw >= 0 && iw < p->W;",
                        "int inside = ih >= 0 && iw >= 0 && ih * p->W + iw < p->H * p->W;"),
    "op(A) transpose reversed": ("return ta ? (double)A[k * lda + i] : (double)A[i * lda + k];",
                                 "return ta ? (double)A[i * lda + k] : (double)A[k * lda + i];"),
    "op(B) uses K for ld": ("return tb ? (double)B[j * ldb + k] : (double)B[k * ldb + j];",
                            "return tb ? (double)B[j * ldb + k] : (double)B[k * (ldb - (ldb > 1)) + j];"),
    "beta term dropped": ("if (beta != 0.0) r += beta * (double)C[i * ldc + j];", ""),
    "C always read": ("if (beta != 0.0) r += beta", "r += beta"),
    "alpha applied twice": ("double r = alpha * s;", "double r = alpha * alpha * s;"),
    "scale without abs": ("t += fabs(p);", "t += p;"),
    "conv scale without abs": ("t += fabs(prod);", "t += prod;"),
    "last k dropped": ("for (int64_t k = 0; k < K; ++k)", "for (int64_t k = 0; k + 1 < K; ++k)"),
    "last channel dropped": ("for (int64_t ci = 0; ci < p->C; ++ci)", "for (int64_t ci = 0; ci + 1 < p->C; ++ci)"),
    "output size rounds up": ("*Ho = hspan / sh + 1;", "*Ho = (hspan + sh - 1) / sh + 1;"),
    "same pads extra on top": ("pads_tlbr[0] = ph / 2;", "pads_tlbr[0] = ph - ph / 2;"),
    "same size floor": ("int64_t ho = (H + sh - 1) / sh, wo = (W + sw - 1) / sw;",
                        "int64_t ho = H / sh, wo = W / sw;"),
    "winograd BT row sign": ("{0, -1, 1, 0}, {0, 1, 0, -1}}", "{0, 1, -1, 0}, {0, 1, 0, -1}}"),
    "winograd G half dropped": ("{0.5, -0.5, 0.5}", "{1, -1, 1}"),
    "winograd AT last entry": ("{0, 1, -1, -1}}", "{0, 1, -1, 1}}"),
    "winograd tile origin uses left pad": ("ih0 = m * th - p->pt", "ih0 = m * th - p->pl"),
    "winograd tile stride 1": ("iw0 = m * tw - p->pl", "iw0 = tw - p->pl"),
    "winograd last channel dropped": ("for (int64_t ch = 0; ch < p->C; ++ch)", "for (int64_t ch = 0; ch + 1 < p->C; ++ch)"),
    "winograd scale without abs on AT": ("ya += fabs(w->AT[i][a]) * acc_abs[a][b] * fabs(w->AT[j][b]);",
                                          "ya += w->AT[i][a] * acc_abs[a][b] * w->AT[j][b];"),
    "winograd filter scale without abs": ("ua += fabs(w->G[a][r]) * fabs(g[r][c]) * fabs(w->G[b][c]);",
                                          "ua += fabs(w->G[a][r]) * g[r][c] * fabs(w->G[b][c]);"),
    "winograd F4 BT entry sign": ("{0, -2, -1, 2, 1, 0}", "{0, -2, -1, 2, -1, 0}"),
    "winograd F4 G sixth sign": ("{-1.0 / 6, 1.0 / 6, -1.0 / 6}", "{-1.0 / 6, -1.0 / 6, -1.0 / 6}"),
    "winograd F4 G twenty-fourth": ("{1.0 / 24, 1.0 / 12, 1.0 / 6}, {1.0 / 24,", "{1.0 / 12, 1.0 / 12, 1.0 / 6}, {1.0 / 24,"),
    "winograd F4 AT minus eight": ("{0, 1, -1, 8, -8, 1}", "{0, 1, -1, 8, 8, 1}"),
    "winograd F4 tile of 2": ("static const wino_matrices WINO_F4 = {\n    4,", "static const wino_matrices WINO_F4 = {\n    2,"),
    "winograd sampled rows and columns swapped": ("winograd_element(&p, w, img, h_out, w_out, c_out,",
                                                  "winograd_element(&p, w, img, w_out, h_out, c_out,"),
    "winograd sampled channel from the pixel": ("int64_t c_out = o % Cout, pixel = o / Cout;",
                                                "int64_t c_out = (o / Cout) % Cout, pixel = o / Cout;"),
    "conv sampled rows and columns swapped": ("conv_element(&p, n, ho, wo, co, &ref[s], &scale[s]);",
                                              "conv_element(&p, n, wo, ho, co, &ref[s], &scale[s]);"),
    "gemm sampled column for row": ("C, ldc, rows[s], cols[s], &ref[s], &scale[s]);",
                                    "C, ldc, rows[s], rows[s] % N, &ref[s], &scale[s]);"),
}


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, tmp_path):
    oracle.build(force=False)
    proc = subprocess.run([sys.executable, "-m", "tests.mutant_runner", name, str(tmp_path)],
                          cwd=ROOT, capture_output=True, text=True, timeout=300)
    out = proc.stdout.strip().splitlines()
    assert out and out[-1].startswith("CAUGHT"), (name, proc.returncode, proc.stdout[-2000:], proc.stderr[-2000:])
