"""The rectifier of Eq. 2 in the convolution's epilogue, and the census hand-off
between layers (isc_conv2d_relu, isc_census_read), through the C ABI.

Bars (as for the plain convolution):
  - outputs: |gpu - oracle| <= 1e-4 * (1 + |oracle|) elementwise against
    max(0, Eq. 1) in fp64, and every stored value is +0 or positive;
  - the census of y: exactly N*K*Ho*Wo entries covered and exactly the
    number of nonzero values in the y the GPU wrote (the decision of which
    outputs are zero is taken in fp32 on both sides of that comparison);
  - integer-valued inputs: y equals the oracle bitwise and the census count
    equals the oracle's count of positive outputs;
  - a layer given the census of its input decides as if it had counted the
    input itself (nonzero count and path recorded by isc_decision).
"""
import sys

import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu

TOL = 1e-4
THRESHOLD = 0.9


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


@pytest.fixture(scope="module")
def isc(torch):
    import paper_1704_07724_amd as m
    m.lib()  # raises if the library is not built
    return m


def note(*parts):
    print("[case]", *parts, flush=True)
    sys.stdout.flush()


def to_dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def assert_close(got, want, what):
    got = got.astype(np.float64)
    err = np.abs(got - want)
    bad = err > TOL * (1.0 + np.abs(want))
    if bad.any():
        i = np.flatnonzero(bad.ravel())[0]
        raise AssertionError("%s: %d of %d outputs out of tolerance; first at flat %d: gpu %r oracle %r"
                             % (what, int(bad.sum()), bad.size, i, got.ravel()[i], want.ravel()[i]))


def assert_rectified(y, what):
    bits = y.view(np.uint32)
    assert not np.any(bits >> 31), "%s: a stored value has its sign bit set" % what
    assert not np.any(np.isnan(y)), what


def expected_path(nnz, total):
    return "sparse" if 1.0 - nnz / total >= THRESHOLD else "dense"


# N, C, H, W, K, R, S, T, P, sparsity, the sparse kernel the shape runs
RELU_CASES = [
    (3, 20, 12, 12, 50, 5, 5, 1, 0, 0.9, "fused_reg"),      # LeNet conv2-like, weights in registers
    (2, 9, 20, 20, 64, 5, 5, 1, 2, 0.9, "fused"),           # 16-column tiles, several row groups
    (2, 11, 13, 13, 384, 3, 3, 1, 1, 0.95, "fused_reg"),    # conv3/4-like, six groups of 64 maps
    (1, 7, 13, 13, 200, 3, 3, 1, 1, 0.9, "fused_reg"),      # ragged last map group, 16-column tiles
    (1, 7, 20, 20, 200, 3, 3, 1, 1, 0.9, "fused_ring"),     # filter streamed, ragged last map group
    (1, 4, 9, 70, 96, 5, 5, 1, 2, 0.8, "fused_ring"),       # column tiles, ragged last tile
    (2, 4, 11, 11, 64, 5, 5, 2, 1, 0.8, "fused"),           # stride 2, filter resident
    (2, 4, 21, 21, 64, 5, 5, 2, 1, 0.8, "generic"),         # stride 2, 10 columns: lists, then the epilogue pass
    (1, 3, 10, 9, 9, 2, 3, 1, 1, 0.7, "generic"),           # 2 x 3 filter
]


def _relu_layer(torch, isc, x, w, T, P, path, census=True, wt=None):
    desc = isc.make_desc(*x.shape, w.shape[0], w.shape[2], w.shape[3], T, P)
    yc = isc.census(desc) if census else None
    ws = isc.workspace(desc, path)
    y = isc.isc_conv2d_relu(to_dev(torch, x), to_dev(torch, w), T, P, path=path, threshold=THRESHOLD,
                            y_census=yc, ws=ws, wt=wt)
    return desc, y, yc, ws


@pytest.mark.parametrize("path", ["sparse", "dense", "auto"])
@pytest.mark.parametrize("case", RELU_CASES, ids=lambda c: "%s-%dx%d-K%d-T%d" % (c[10], c[2], c[3], c[4], c[7]))
def test_relu_layer(torch, isc, case, path):
    N, C, H, W, K, R, S, T, P, sp, kernel = case
    note("relu layer", case, path)
    desc = isc.make_desc(N, C, H, W, K, R, S, T, P)
    assert isc.isc_sparse_kernel(desc) == kernel
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=31 + sum(case[:9]))
    _, y, yc, ws = _relu_layer(torch, isc, x, w, T, P, path)
    y = y.cpu().numpy()
    want, _ = oracle.relu_conv2d_f64(x, w, T, P)
    assert_close(y, want, "relu %s %s" % (kernel, path))
    assert_rectified(y, "relu %s %s" % (kernel, path))
    elems, nnz = isc.isc_census_read(yc)
    assert elems == y.size
    assert nnz == int(np.count_nonzero(y))
    assert 0 < nnz < y.size  # both signs occur before the rectifier
    nnz_in, taken = isc.isc_decision(desc, ws)
    if path == "auto":
        assert taken == expected_path(nnz_in, x.size)
        assert nnz_in == int(np.count_nonzero(x))
    else:
        assert taken == path


@pytest.mark.parametrize("path", ["sparse", "dense"])
@pytest.mark.parametrize("case", RELU_CASES, ids=lambda c: "%s-%dx%d-K%d-T%d" % (c[10], c[2], c[3], c[4], c[7]))
def test_relu_layer_integer_exact(torch, isc, case, path):
    """Integer-valued inputs: every fp32 partial sum is exact, so the
    rectified output and its nonzero count equal the oracle's exactly."""
    N, C, H, W, K, R, S, T, P, sp, kernel = case
    note("relu integer", case, path)
    x, w = workloads.integer_case(N, C, H, W, K, R, S, seed=7 + sum(case[:9]))
    _, y, yc, _ = _relu_layer(torch, isc, x, w, T, P, path)
    want, nnz_want = oracle.relu_conv2d_f64(x, w, T, P)
    got = y.cpu().numpy()
    assert np.array_equal(got.astype(np.float64), want)
    assert_rectified(got, "relu integer")
    assert isc.isc_census_read(yc) == (want.size, nnz_want)


def test_relu_dense_materialised_im2col(torch, isc):
    """C*R*S >= 2^16: the dense path writes the im2col matrix and the GEMM
    rectifies and counts as it scatters to NCHW."""
    N, C, H, W, K, R, S, T, P = 1, 2624, 6, 6, 8, 5, 5, 1, 0
    note("relu explicit im2col", (N, C, H, W, K, R, S))
    x, w = workloads.integer_case(N, C, H, W, K, R, S, seed=77, sparsity=0.9, wmax=2)
    _, y, yc, _ = _relu_layer(torch, isc, x, w, T, P, "dense")
    want, nnz_want = oracle.relu_conv2d_f64(x, w, T, P)
    assert np.array_equal(y.cpu().numpy().astype(np.float64), want)
    assert isc.isc_census_read(yc) == (want.size, nnz_want)


def test_relu_without_census_and_with_repacked_filter(torch, isc):
    N, C, H, W, K, R, S, T, P = 2, 16, 13, 13, 96, 3, 3, 1, 1
    note("relu no census, repacked filter")
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, 0.9, seed=91)
    wt = isc.isc_repack_filter(to_dev(torch, w))
    want, _ = oracle.relu_conv2d_f64(x, w, T, P)
    for path in ("sparse", "auto"):
        _, y, _, _ = _relu_layer(torch, isc, x, w, T, P, path, census=False, wt=wt)
        assert_close(y.cpu().numpy(), want, "relu repacked %s" % path)


def _chain_on_gpu(torch, isc, x0, ws_list, use_census=True, use_wt=True, path="auto"):
    """conv3 -> ReLU -> conv4 -> ReLU -> conv5 (3x3, pad 1), each layer given
    the census its predecessor wrote.  Returns per layer (input, output,
    decision)."""
    out = []
    x = to_dev(torch, x0)
    xc = None
    for w in ws_list:
        desc = isc.make_desc(*x.shape, w.shape[0], 3, 3, 1, 1)
        wd = to_dev(torch, w)
        wt = isc.isc_repack_filter(wd) if use_wt else None
        yc = isc.census(desc)
        ws = isc.workspace(desc, path)
        y = isc.isc_conv2d_relu(x, wd, 1, 1, path=path, threshold=THRESHOLD, x_census=xc if use_census else None,
                                wt=wt, y_census=yc, ws=ws)
        out.append((x, y, isc.isc_decision(desc, ws), yc))
        x, xc = y, yc
    return out


def test_chain_census_handoff(torch, isc):
    chain = workloads.WORKLOADS["alexnet_chain345"]
    x0, ws_list = workloads.make_chain(chain, N=2)
    note("chain", x0.shape)
    layers = _chain_on_gpu(torch, isc, x0, ws_list)
    for i, ((xd, yd, (nnz_in, taken), yc), w) in enumerate(zip(layers, ws_list)):
        x = xd.cpu().numpy()
        y = yd.cpu().numpy()
        # parity of each layer on the input the GPU gave it
        want, _ = oracle.relu_conv2d_f64(x, w, 1, 1)
        assert_close(y, want, "chain layer %d" % i)
        assert_rectified(y, "chain layer %d" % i)
        # the decision (from the count of x, or from the census of x for the
        # later layers) is the count of x's nonzeros
        assert nnz_in == int(np.count_nonzero(x)), i
        assert taken == expected_path(nnz_in, x.size), i
        assert isc.isc_census_read(yc) == (y.size, int(np.count_nonzero(y)))
    # the recipe's filters keep the rectified outputs sparse: the later layers
    # take the sparse path from the census
    assert [l[2][1] for l in layers] == ["sparse"] * 3
    # the same chain without the census (each layer counts its input) and
    # without the caller's repacked filters gives the same outputs bit for bit
    plain = _chain_on_gpu(torch, isc, x0, ws_list, use_census=False, use_wt=False)
    for a, b in zip(layers, plain):
        assert torch.equal(a[1], b[1])
        assert a[2] == b[2]


def test_stale_or_foreign_census_runs_dense(torch, isc):
    """A census that does not cover the input (another shape's, or never
    written) leaves the count unknown: AUTO runs the dense path and the
    output is still right."""
    N, C, H, W, K = 2, 24, 13, 13, 40
    note("foreign census")
    x, w = workloads.make_case(N, C, H, W, K, 3, 3, 1, 1, 0.95, seed=93)
    want, _ = oracle.relu_conv2d_f64(x, w, 1, 1)
    desc = isc.make_desc(N, C, H, W, K, 3, 3, 1, 1)
    # a census written for an output of another size
    other = isc.make_desc(1, C, H, W, K, 3, 3, 1, 1)
    xo, wo = workloads.make_case(1, C, H, W, K, 3, 3, 1, 1, 0.5, seed=94)
    foreign = isc.census(other)
    isc.isc_conv2d_relu(to_dev(torch, xo), to_dev(torch, wo), 1, 1, y_census=foreign)
    garbage = isc.census(desc)
    garbage.fill_(0xFF)
    for xc in (foreign, garbage):
        ws = isc.workspace(desc, "auto")
        y = isc.isc_conv2d_relu(to_dev(torch, x), to_dev(torch, w), 1, 1, path="auto", threshold=THRESHOLD,
                                x_census=xc, ws=ws)
        assert_close(y.cpu().numpy(), want, "foreign census")
        nnz, taken = isc.isc_decision(desc, ws)
        assert taken == "dense" and nnz == 2 ** 64 - 1
    with pytest.raises(isc.IscError) as e:
        isc.isc_census_read(garbage)
    assert e.value.status == 10


@pytest.mark.parametrize("path", ["auto", "dense"])
def test_chain_full_size_every_output(torch, isc, path):
    """The chain at its full size (batch 128), as the benchmark runs it: every
    output of every layer against the oracle on the GPU's own input of that
    layer, and every census against a count of the output it describes."""
    chain = workloads.WORKLOADS["alexnet_chain345"]
    x0, ws_list = workloads.make_chain(chain)
    note("chain full", path, x0.shape)
    layers = _chain_on_gpu(torch, isc, x0, ws_list, path=path)
    for i, ((xd, yd, (nnz_in, taken), yc), w) in enumerate(zip(layers, ws_list)):
        if path == "auto":
            assert nnz_in == int(torch.count_nonzero(xd).item())
            assert taken == expected_path(nnz_in, xd.numel())
        assert isc.isc_census_read(yc) == (yd.numel(), int(torch.count_nonzero(yd).item()))
        assert not bool(torch.signbit(yd).any())
        want, _ = oracle.relu_conv2d_f64(xd.cpu().numpy(), w, 1, 1)
        assert_close(yd.cpu().numpy(), want, "chain full %s layer %d" % (path, i))
        del want
    del layers
    torch.cuda.empty_cache()
