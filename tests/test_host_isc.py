"""The host-CPU ISC (the paper's three steps on the CPU, for the CPU speedup
trend of Tab. 2) against the oracle: fp32 within the tolerance, integer
inputs bitwise; and the host im2col against the oracle's."""
import numpy as np
import pytest

import oracle
import workloads
from paper_1704_07724_amd import host

TOL = 1e-4

CASES = [
    # N, C, H, W, K, R, S, T, P, sparsity
    (2, 3, 9, 11, 20, 3, 3, 1, 1, 0.9),
    (1, 4, 12, 12, 50, 5, 5, 1, 0, 0.9),
    (2, 5, 13, 13, 17, 3, 3, 2, 1, 0.7),
    (1, 3, 10, 7, 9, 2, 4, 3, 2, 0.5),
    (1, 6, 7, 7, 33, 1, 1, 1, 0, 0.95),
    (1, 2, 6, 6, 8, 7, 7, 1, 3, 0.0),
    (1, 2, 5, 5, 4, 3, 3, 1, 1, 1.0),
]


def close(got, want):
    return bool(np.all(np.abs(got.astype(np.float64) - want) <= TOL * (1.0 + np.abs(want))))


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("threads", [1, 3])
def test_host_isc_matches_oracle(case, threads):
    N, C, H, W, K, R, S, T, P, sp = case
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=7 + sum(case[:9]))
    y = host.conv2d(x, host.repack(w), T, P, threads=threads)
    assert close(y, oracle.conv2d_f64(x, w, T, P))


def test_host_isc_integer_exact():
    x, w = workloads.integer_case(2, 4, 11, 9, 21, 3, 3, seed=3)
    y = host.conv2d(x, host.repack(w), 1, 1)
    assert np.array_equal(y.astype(np.float64), oracle.conv2d_f64(x, w, 1, 1))


@pytest.mark.parametrize("name", ["tab2_lenet_conv2_n1", "tab2_alexnetc_conv3_n1", "tab2_inception5b_5_n1"])
def test_host_isc_tab2_layers(name):
    layer = [l for l in workloads.WORKLOADS["paper_tab2_n1"].layers if l.name == name][0]
    x, w = workloads.make_inputs(layer)
    y = host.conv2d(x, host.repack(w), layer.T, layer.P)
    assert close(y, oracle.conv2d_f64(x, w, layer.T, layer.P))


def test_host_im2col_matches_oracle():
    x, w = workloads.make_case(1, 3, 9, 8, 4, 3, 2, 2, 1, 0.5, seed=11)
    col = host.im2col(x[0], 3, 2, 2, 1)
    want = oracle.im2col(x, 3, 2, 2, 1)
    assert np.array_equal(col, np.asarray(want, dtype=np.float32).reshape(col.shape))


def test_host_isc_rejects_bad_shapes():
    x = np.zeros((1, 3, 5, 5), np.float32)
    with pytest.raises(ValueError):
        host.conv2d(x, np.zeros((2, 3, 3, 4), np.float32))
    with pytest.raises(ValueError):
        host.conv2d(x, np.zeros((3, 7, 7, 4), np.float32))
