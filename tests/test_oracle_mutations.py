"""The pins must catch plausible mistakes in the oracle.

Each mutant below is a copy of oracle/isc_oracle.c with one planted mistake
(a dropped term, a wrong sign or index, a transposed operand, the paper's
printed output-size formula taken literally, ...).  It is compiled on the CPU
and the oracle pin tests are run against it in a subprocess; every mutant
must make at least one pin fail.  Nothing here touches a GPU.
"""
import os
import subprocess
import sys
import tempfile

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "isc_oracle.c")

MUTANTS = {
    "tap_sign": ("i * T + r - P, j * T + s - P, C, H, W)", "i * T - r + P, j * T - s + P, C, H, W)"),
    "stride_dropped": ("i * T + r - P, j * T + s - P, C, H, W)", "i + r - P, j + s - P, C, H, W)"),
    "filter_rs_transposed": ("double wv = (double)w[((k * C + c) * R + r) * S + s];",
                             "double wv = (double)w[((k * C + c) * S + s) * R + r];"),
    "input_plane_transposed": ("return (double)x[((n * C + c) * H + y) * W + xx];",
                               "return (double)x[((n * C + c) * W + xx) * H + y];"),
    "last_tap_dropped": ("for (long s = 0; s < S; ++s) {\n                double xv",
                         "for (long s = 1; s < S; ++s) {\n                double xv"),
    "pad_edge_dropped": ("if (y < 0 || y >= H || xx < 0 || xx >= W) return 0.0;",
                         "if (y < 0 || y >= H || xx < 0 || xx >= W - 1) return 0.0;"),
    "printed_out_size": ("return (int)(num / stride) + 1;", "return (int)((num + 1) / stride);"),
    "signed_zero_nonzero": ("return (b & 0x7fffffffu) != 0u;", "return b != 0u;"),
    "compact_xy_swapped": ("ys[p * HW + cnt] = (int32_t)y;", "ys[p * HW + cnt] = (int32_t)xx;"),
    "row_ptr_after_row": ("            row_ptr[p * (H + 1) + y] = cnt;\n            for (long xx",
                          "            for (long xx"),
    "macs_bound_inclusive": ("if (num / t < out) ++cnt;", "if (num / t <= out) ++cnt;"),
    "relu_keeps_negatives": ("        if (y[i] > 0.0)\n            ++nnz;", "        if (y[i] < 0.0)\n            ++nnz;"),
    "relu_counts_zeros": ("        if (y[i] > 0.0)\n            ++nnz;", "        if (y[i] >= 0.0)\n            ++nnz;"),
    "dw_tap_sign": ("double xv = oracle_xhat(x, n, c, i * T + r - P, j * T + s - P, C, H, W);",
                    "double xv = oracle_xhat(x, n, c, i * T - r + P, j * T + s - P, C, H, W);"),
    "dw_map_transposed": ("dw[((k * C + c) * R + r) * S + s] = acc;", "dw[((c * K + k) * R + r) * S + s] = acc;"),
    "im2col_rs_swapped": ("long y = i * T + r - P, xx = j * T + s - P;",
                          "long y = i * T + s - P, xx = j * T + r - P;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation anchor not found: %s" % name
    mutant_src = tmp_path / ("oracle_%s.c" % name)
    mutant_src.write_text(src.replace(old, new, 1))
    lib = oracle.build(force=True, src=str(mutant_src), out=str(tmp_path / ("lib_%s.so" % name)))
    env = dict(os.environ, ISC_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_pins.py")],
                       cwd=os.path.dirname(HERE), env=env, capture_output=True, text=True,
                       timeout=600)
    assert r.returncode != 0, "mutant %s survived every pin:\n%s" % (name, r.stdout[-2000:])
