"""Parity of the zero-skipping weight gradient (isc_conv2d_dw) with the oracle.

Bars: |gpu - oracle| <= 1e-4 * (1 + |oracle|) elementwise against the fp64
definition; integer-valued inputs and output gradients keep every fp32
partial sum exact, so there the result equals the oracle bitwise; a zero
input gives exactly zero; two runs agree bitwise (fixed summation order).
"""
import sys

import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


@pytest.fixture(scope="module")
def isc(torch):
    import paper_1704_07724_amd as m
    m.lib()
    return m


def note(*parts):
    print("[case]", *parts, flush=True)
    sys.stdout.flush()


def to_dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def assert_close(got, want, what):
    got = got.astype(np.float64)
    bad = np.abs(got - want) > TOL * (1.0 + np.abs(want))
    if bad.any():
        i = np.flatnonzero(bad.ravel())[0]
        raise AssertionError("%s: %d of %d out of tolerance; first at flat %d: gpu %r oracle %r"
                             % (what, int(bad.sum()), bad.size, i, got.ravel()[i], want.ravel()[i]))


# N, C, H, W, K, R, P, sparsity: every kernel variant (filter size, 64 or 128
# maps per lane group, 16- or 28-column tiles) with ragged maps and channels
DW_CASES = [
    (3, 20, 12, 12, 50, 5, 0, 0.9),     # LeNet conv2-like: 5x5, K <= 64, 16-column tiles
    (2, 7, 27, 27, 70, 5, 2, 0.9),      # AlexNet conv2-like: 28-column tiles, ragged map group
    (2, 13, 13, 13, 64, 3, 1, 0.95),    # 3x3, one map per lane
    (2, 23, 13, 13, 200, 3, 1, 0.9),    # 3x3, two maps per lane, ragged
    (1, 9, 20, 30, 130, 3, 1, 0.8),     # 28-column tiles, ragged last tile
    (2, 37, 7, 7, 96, 1, 0, 0.9),       # 1x1, two maps per lane
    (3, 70, 14, 14, 20, 1, 0, 0.9),     # 1x1, one map per lane, many channels
    (1, 2, 5, 5, 3, 5, 2, 0.5),         # tiny, filter wider than the map
    (1, 1, 1, 1, 1, 1, 0, 0.0),         # one element
]


def _dy(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


@pytest.mark.parametrize("case", DW_CASES, ids=lambda c: "N%d-C%d-%dx%d-K%d-R%d-P%d" % c[:7])
def test_dw_matches_oracle(torch, isc, case):
    N, C, H, W, K, R, P, sp = case
    note("dw", case)
    x, _ = workloads.make_case(N, C, H, W, K, R, R, 1, P, sp, seed=41 + sum(case[:7]))
    Ho, Wo = oracle.out_size(H, R, P, 1), oracle.out_size(W, R, P, 1)
    dy = _dy((N, K, Ho, Wo), 43 + sum(case[:7]))
    got = isc.isc_conv2d_dw(to_dev(torch, x), to_dev(torch, dy), R, R, 1, P).cpu().numpy()
    want = oracle.conv2d_dw_f64(x, dy, R, R, 1, P)
    assert got.shape == want.shape
    assert_close(got, want, "dw %s" % (case,))
    # run to run: the same bits
    again = isc.isc_conv2d_dw(to_dev(torch, x), to_dev(torch, dy), R, R, 1, P).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), again.view(np.uint32))


@pytest.mark.parametrize("case", DW_CASES[:7], ids=lambda c: "N%d-C%d-%dx%d-K%d-R%d-P%d" % c[:7])
def test_dw_integer_exact(torch, isc, case):
    N, C, H, W, K, R, P, sp = case
    note("dw integer", case)
    x, _ = workloads.integer_case(N, C, H, W, K, R, R, seed=47 + sum(case[:7]), sparsity=max(sp, 0.5))
    Ho, Wo = oracle.out_size(H, R, P, 1), oracle.out_size(W, R, P, 1)
    dy = np.random.default_rng(48).integers(-4, 5, (N, K, Ho, Wo)).astype(np.float32)
    got = isc.isc_conv2d_dw(to_dev(torch, x), to_dev(torch, dy), R, R, 1, P).cpu().numpy()
    assert np.array_equal(got.astype(np.float64), oracle.conv2d_dw_f64(x, dy, R, R, 1, P))


def test_dw_zero_input_and_rejects(torch, isc):
    note("dw zero input")
    x = torch.zeros((2, 5, 9, 9), device="cuda")
    dy = torch.randn((2, 6, 9, 9), device="cuda")
    dw = isc.isc_conv2d_dw(x, dy, 3, 3, 1, 1)
    assert bool((dw == 0).all()) and not bool(torch.signbit(dw).any())
    with pytest.raises(isc.IscError) as e:        # stride 2: not taken
        isc.isc_conv2d_dw(x, torch.zeros((2, 6, 5, 5), device="cuda"), 3, 3, 2, 1)
    assert e.value.status == 3
    with pytest.raises(isc.IscError) as e:        # 7x7 filter: not taken
        isc.isc_conv2d_dw(x, torch.zeros((2, 6, 9, 9), device="cuda"), 7, 7, 1, 3)
    assert e.value.status == 3


def test_dw_full_size_every_entry(torch, isc):
    """AlexNet conv2 at full size (batch 128, 96 -> 256, 27x27, 5x5, pad 2,
    sparsity 0.9) as the benchmark runs it: every entry of K x C x R x S
    against the oracle's full weight gradient."""
    layer = [l for l in workloads.WORKLOADS["alexnet_conv2"].layers][0]
    note("dw full", layer.x_shape, layer.w_shape)
    x, _ = workloads.make_inputs(layer)
    Ho = oracle.out_size(layer.H, layer.R, layer.P, 1)
    dy = _dy((layer.N, layer.K, Ho, Ho), 49)
    got = isc.isc_conv2d_dw(to_dev(torch, x), to_dev(torch, dy), layer.R, layer.S, 1, layer.P).cpu().numpy()
    want = oracle.conv2d_dw_f64(x, dy, layer.R, layer.S, 1, layer.P)
    assert_close(got, want, "dw full size")


@pytest.mark.parametrize("R,W", [(1, 13), (3, 13), (3, 30), (5, 11), (5, 27)])
def test_dw_every_tile_variant(torch, isc, R, W):
    """Every compiled tile (rows per tile, maps per lane, 16- or 28-column
    tiles), forced through the measurement overrides, against the oracle on
    ragged maps and channels."""
    N, C, H, K, P = 2, 9, 10, 70, R // 2
    x, _ = workloads.make_case(N, C, H, W, K, R, R, 1, P, 0.8, seed=61 + R + W)
    Ho, Wo = oracle.out_size(H, R, P, 1), oracle.out_size(W, R, P, 1)
    dy = _dy((N, K, Ho, Wo), 62 + R + W)
    want = oracle.conv2d_dw_f64(x, dy, R, R, 1, P)
    variants = [(1, 1), (2, 1), (1, 2), (2, 2)] + ([(4, 1)] if Wo <= 16 else [])
    for kpl, th in variants:
        note("dw variant", R, W, "kpl", kpl, "th", th)
        got = isc.isc_conv2d_dw(to_dev(torch, x), to_dev(torch, dy), R, R, 1, P,
                                tuning={"maps_per_lane": kpl, "rows": th}).cpu().numpy()
        assert_close(got, want, "dw R%d W%d kpl%d th%d" % (R, W, kpl, th))
