"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars:
  - compaction (ISC step 1) and im2col: bit-exact;
  - convolution outputs (sparse and dense paths): elementwise
    |gpu - oracle| <= 1e-4 * (1 + |oracle|);
  - integer-valued inputs: every fp32 partial sum is exact, so both paths
    must equal the oracle bitwise;
  - the dispatcher's choice is the sparsity test 1 - nnz/total >= threshold
    evaluated in double, the same as here.
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
    m.lib()  # raises if the library is not built
    return m


def note(*parts):
    print("[case]", *parts, flush=True)
    sys.stdout.flush()


def to_dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def assert_conv_close(got, want, what):
    got = got.astype(np.float64)
    err = np.abs(got - want)
    bound = TOL * (1.0 + np.abs(want))
    bad = err > bound
    if bad.any():
        i = np.flatnonzero(bad.ravel())[0]
        raise AssertionError("%s: %d of %d outputs out of tolerance; first at flat %d: gpu %r "
                             "oracle %r" % (what, int(bad.sum()), bad.size, i, got.ravel()[i],
                                            want.ravel()[i]))


# ------------------------------------------------------------- compaction --

COMPACT_SHAPES = [
    (1, 1, 1, 1), (2, 3, 5, 7), (3, 4, 12, 12), (2, 5, 27, 27), (1, 3, 13, 13),
    (2, 2, 28, 28), (1, 2, 3, 100), (1, 2, 100, 3), (1, 1, 40, 70), (4, 1, 1, 65),
]


@pytest.mark.parametrize("shape", COMPACT_SHAPES)
@pytest.mark.parametrize("sparsity", [0.0, 0.5, 0.9, 1.0])
def test_compact_bitexact(torch, isc, shape, sparsity):
    note("compact", shape, sparsity)
    rng = np.random.default_rng(hash((shape, sparsity)) & 0xFFFF)
    x = np.abs(rng.standard_normal(shape)).astype(np.float32) + np.float32(0.5)
    x[rng.random(shape) < sparsity] = 0.0
    _check_compact(torch, isc, x)


@pytest.mark.parametrize("shape", [(2, 3500, 33, 33), (1, 13000, 5, 5)])
def test_compact_several_planes_per_wavefront(torch, isc, shape):
    """More planes than wavefronts resident at once: each wavefront lists
    several planes, loading the next while it lists the current one (planes
    of two batches each in the first shape)."""
    note("compact planes per wavefront", shape)
    rng = np.random.default_rng(sum(shape))
    x = np.abs(rng.standard_normal(shape)).astype(np.float32) + np.float32(0.5)
    x[rng.random(shape) < 0.7] = 0.0
    _check_compact(torch, isc, x)


def test_compact_special_values(torch, isc):
    rng = np.random.default_rng(5)
    x = np.abs(rng.standard_normal((2, 3, 9, 11))).astype(np.float32)
    x[rng.random(x.shape) < 0.6] = 0.0
    x[0, 0, 0, 0] = -0.0
    x[0, 1, 2, 3] = np.float32(1e-45)
    x[1, 0, 4, 4] = -np.float32(1e-40)
    x[1, 1, 8, 10] = np.inf
    x[1, 2, 5, 0] = np.nan
    x[0, 2, 3, 3] = -2.5
    note("compact special values")
    _check_compact(torch, isc, x)


def _check_compact(torch, isc, x):
    N, C, H, W = x.shape
    row_ptr, nz, total = isc.isc_compact(to_dev(torch, x))
    torch.cuda.synchronize()
    rp_o, v_o, ys_o, xs_o, tot_o = oracle.compact(x)
    assert int(total.item()) == tot_o
    assert np.array_equal(row_ptr.cpu().numpy(), rp_o)
    ent = nz.cpu().numpy().reshape(N * C, H * W, 2)
    for p in range(N * C):
        cnt = rp_o[p, H]
        assert np.array_equal(ent[p, :cnt, 0].view(np.uint32), v_o[p, :cnt].view(np.uint32))
        yx = ent[p, :cnt, 1].view(np.uint32)
        assert np.array_equal(yx >> 16, ys_o[p, :cnt].astype(np.uint32))
        assert np.array_equal(yx & 0xFFFF, xs_o[p, :cnt].astype(np.uint32))


# ----------------------------------------------------------------- im2col --

@pytest.mark.parametrize("case", [
    (2, 3, 8, 7, 3, 3, 1, 1), (1, 4, 12, 12, 5, 5, 1, 0), (2, 2, 11, 11, 5, 5, 2, 1),
    (1, 3, 9, 10, 2, 3, 3, 2), (3, 2, 6, 6, 1, 1, 1, 0), (1, 1, 13, 13, 3, 3, 1, 1),
])
def test_im2col_bitexact(torch, isc, case):
    N, C, H, W, R, S, T, P = case
    note("im2col", case)
    rng = np.random.default_rng(sum(case))
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    x[rng.random(x.shape) < 0.3] = 0.0
    x[0, 0, 0, 0] = -0.0
    ho, wo = oracle.out_size(H, R, P, T), oracle.out_size(W, S, P, T)
    ldc = N * ho * wo + 37
    col = isc.isc_im2col(to_dev(torch, x), R, S, T, P, ldc=ldc).cpu().numpy()
    want = oracle.im2col(x, R, S, T, P, ldc=ldc)
    assert np.array_equal(col.view(np.uint32), want.view(np.uint32))


# ------------------------------------------------------------------- GEMM --

@pytest.mark.parametrize("mnk", [(1, 1, 1), (50, 512, 500), (32, 300, 17), (64, 257, 64),
                                 (128, 1000, 33), (200, 130, 2400), (384, 256, 3)])
def test_gemm_against_fp64(torch, isc, mnk):
    M, N, Kd = mnk
    note("gemm", mnk)
    rng = np.random.default_rng(M * 7 + N * 3 + Kd)
    a = rng.standard_normal((M, Kd)).astype(np.float32)
    b = rng.standard_normal((Kd, N)).astype(np.float32)
    c = isc.isc_gemm_f32(to_dev(torch, a), to_dev(torch, b)).cpu().numpy().astype(np.float64)
    want = a.astype(np.float64) @ b.astype(np.float64)
    # any order of fp32 sums of Kd products: |error| <= gamma_Kd * sum |a||b|,
    # gamma_n = n u / (1 - n u), u = 2^-24 (+1 for the product rounding)
    u = 2.0 ** -24
    gamma = (Kd + 1) * u / (1 - (Kd + 1) * u)
    bound = gamma * (np.abs(a.astype(np.float64)) @ np.abs(b.astype(np.float64)))
    assert np.all(np.abs(c - want) <= bound), mnk


# ------------------------------------------------------------ convolution --

CONV_CASES = [
    # N, C, H, W, K, R, S, T, P, sparsity
    (2, 5, 12, 12, 50, 5, 5, 1, 0, 0.9),      # LeNet-like, K < 64
    (2, 8, 27, 27, 70, 5, 5, 1, 2, 0.9),      # AlexNet conv2-like, ragged k-block
    (2, 16, 13, 13, 130, 3, 3, 1, 1, 0.95),   # conv3-5-like
    (2, 6, 28, 28, 64, 3, 3, 1, 1, 0.9),      # inception 3x3-like
    (1, 4, 28, 28, 32, 5, 5, 1, 2, 0.9),      # inception 5x5-like
    (2, 7, 14, 14, 40, 1, 1, 1, 0, 0.9),      # 1x1
    (1, 3, 17, 15, 20, 7, 7, 1, 3, 0.8),      # 7x7
    (2, 4, 11, 11, 64, 5, 5, 2, 1, 0.95),     # the paper's LeNet-Conv2 shape (T = 2)
    (1, 3, 10, 9, 9, 2, 3, 1, 1, 0.5),        # generic R x S
    (1, 2, 9, 9, 5, 3, 3, 3, 2, 0.7),         # stride 3
    (1, 3, 20, 200, 66, 3, 3, 1, 1, 0.9),     # wide: several column tiles
    (2, 3, 7, 7, 10, 5, 5, 1, 4, 0.6),        # pad larger than filter - 1
    (1, 1, 1, 1, 1, 1, 1, 1, 0, 0.0),         # smallest
    (3, 2, 6, 6, 3, 6, 6, 1, 0, 0.5),         # filter covers the map (Ho = 1), generic
]


@pytest.mark.parametrize("path", ["sparse", "dense", "auto"])
@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_matches_oracle(torch, isc, case, path):
    N, C, H, W, K, R, S, T, P, sp = case
    note("conv", path, case)
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=abs(hash(case)) % 10000)
    y = isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), T, P, path=path).cpu().numpy()
    want = oracle.conv2d_f64(x, w, T, P)
    assert y.shape == want.shape
    assert_conv_close(y, want, "%s %s" % (path, case))


@pytest.mark.parametrize("path", ["dense", "auto"])
def test_conv_dense_with_im2col_matrix(torch, isc, path):
    """C*R*S >= 2^16: the dense path writes the im2col matrix and runs the
    explicit GEMM instead of gathering inside the GEMM."""
    case = (1, 2700, 6, 6, 8, 5, 5, 1, 0, 0.5)
    N, C, H, W, K, R, S, T, P, sp = case
    note("conv explicit im2col", path, case)
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=27)
    y = isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), T, P, path=path).cpu().numpy()
    assert_conv_close(y, oracle.conv2d_f64(x, w, T, P), "%s %s" % (path, case))


@pytest.mark.parametrize("path", ["sparse", "dense"])
@pytest.mark.parametrize("case", [(2, 6, 12, 12, 50, 5, 5, 1, 0), (2, 16, 13, 13, 130, 3, 3, 1, 1),
                                  (1, 5, 11, 11, 20, 5, 5, 2, 1), (2, 3, 9, 9, 7, 2, 4, 1, 1)])
def test_conv_integer_inputs_bitwise(torch, isc, case, path):
    N, C, H, W, K, R, S, T, P = case
    note("conv integer", path, case)
    x, w = workloads.integer_case(N, C, H, W, K, R, S, seed=sum(case))
    y = isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), T, P, path=path).cpu().numpy()
    want = oracle.conv2d_f64(x, w, T, P)
    assert np.array_equal(y.astype(np.float64), want)


@pytest.mark.parametrize("path", ["sparse", "dense", "auto"])
def test_conv_zero_input_exact_zero(torch, isc, path):
    note("conv zero input", path)
    x = torch.zeros((2, 8, 13, 13), device="cuda")
    w = torch.randn((40, 8, 3, 3), device="cuda")
    y = isc.isc_conv2d(x, w, 1, 1, path=path)
    assert bool((y == 0).all())


def test_sparse_run_to_run_bitwise(torch, isc):
    note("determinism")
    x, w = workloads.make_case(2, 8, 27, 27, 70, 5, 5, 1, 2, 0.9, seed=11)
    xd, wd = to_dev(torch, x), to_dev(torch, w)
    a = isc.isc_conv2d(xd, wd, 1, 2, path="sparse").cpu().numpy()
    b = isc.isc_conv2d(xd, wd, 1, 2, path="sparse").cpu().numpy()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_output_redzone_untouched(torch, isc):
    note("redzone")
    x, w = workloads.make_case(2, 4, 12, 12, 50, 5, 5, 1, 0, 0.9, seed=12)
    n_out = 2 * 50 * 8 * 8
    for path in ("sparse", "dense", "auto"):
        buf = torch.full((n_out + 2048,), 1234.5, device="cuda")
        out = buf[1024:1024 + n_out].view(2, 50, 8, 8)
        isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), 1, 0, path=path, out=out)
        b = buf.cpu().numpy()
        assert np.all(b[:1024] == 1234.5) and np.all(b[1024 + n_out:] == 1234.5), path


# ------------------------------------------------------------- dispatcher --

def oracle_choice(x, threshold):
    total = x.size
    nnz = oracle.compact(x)[4]
    return ("sparse" if 1.0 - nnz / total >= float(np.float32(threshold)) else "dense"), nnz


@pytest.mark.parametrize("sparsity", [0.5, 0.85, 0.9, 0.95, 0.99])
def test_auto_dispatch_choice(torch, isc, sparsity):
    note("dispatch", sparsity)
    x, w = workloads.make_case(4, 10, 12, 12, 50, 5, 5, 1, 0, sparsity, seed=int(sparsity * 100))
    desc = isc.make_desc(4, 10, 12, 12, 50, 5, 5, 1, 0)
    ws = isc.workspace(desc, "auto")
    y = isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), 1, 0, path="auto", threshold=0.9, ws=ws)
    nnz, taken = isc.isc_decision(desc, ws)
    torch.cuda.synchronize()
    assert isc.isc_read_decision(ws) == (taken, nnz)
    want_path, want_nnz = oracle_choice(x, 0.9)
    assert nnz == want_nnz
    assert taken == want_path
    assert_conv_close(y.cpu().numpy(), oracle.conv2d_f64(x, w, 1, 0), "auto %g" % sparsity)


def test_dispatch_threshold_boundary(torch, isc):
    # exactly at the threshold the sparse path is taken; one more nonzero
    # flips it to dense
    note("dispatch boundary")
    N, C, H, W = 1, 4, 10, 10   # 400 inputs: sparsity 0.9 <=> 40 nonzeros
    rng = np.random.default_rng(3)
    w = rng.standard_normal((8, C, 3, 3)).astype(np.float32)
    desc = isc.make_desc(N, C, H, W, 8, 3, 3, 1, 1)
    for nnz, want in ((40, "sparse"), (41, "dense")):
        x = np.zeros((N, C, H, W), np.float32)
        idx = rng.choice(x.size, nnz, replace=False)
        x.ravel()[idx] = 1.0 + rng.random(nnz).astype(np.float32)
        assert oracle_choice(x, 0.9)[0] == want
        ws = isc.workspace(desc, "auto")
        y = isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), 1, 1, path="auto", threshold=0.9, ws=ws)
        got_nnz, taken = isc.isc_decision(desc, ws)
        assert (got_nnz, taken) == (nnz, want)
        assert_conv_close(y.cpu().numpy(), oracle.conv2d_f64(x, w, 1, 1), "boundary %d" % nnz)


def test_forced_paths_record_decision(torch, isc):
    note("forced path record")
    x, w = workloads.make_case(2, 4, 12, 12, 50, 5, 5, 1, 0, 0.5, seed=4)
    desc = isc.make_desc(2, 4, 12, 12, 50, 5, 5, 1, 0)
    ws = isc.workspace(desc, "sparse")
    isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), 1, 0, path="sparse", ws=ws)
    nnz, taken = isc.isc_decision(desc, ws)
    assert taken == "sparse" and nnz == oracle.compact(x)[4]
    ws = isc.workspace(desc, "dense")
    isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), 1, 0, path="dense", ws=ws)
    nnz, taken = isc.isc_decision(desc, ws)
    assert taken == "dense" and nnz == 2 ** 64 - 1


def test_gpu_error_codes(torch, isc):
    note("error codes")
    x = torch.zeros((1, 3, 8, 8), device="cuda")
    w = torch.zeros((3, 3, 3, 3), device="cuda")
    with pytest.raises(isc.IscError) as e:
        isc.isc_conv2d(x, w, 1, 1, ws=torch.empty(16, dtype=torch.uint8, device="cuda"))
    assert e.value.status == 4
    with pytest.raises(isc.IscError) as e:
        isc.isc_conv2d(x, w, 1, 1, out=x)          # output overlaps the input
    assert e.value.status == 5
    with pytest.raises(KeyError):
        isc.isc_conv2d(x, w, 1, 1, path="sideways")


@pytest.mark.parametrize("path", ["auto", "sparse", "dense"])
def test_graph_replay_matches_eager(torch, isc, path):
    """isc_conv2d captured into a HIP graph: every replay, with eager work
    in between, equals the eager result bitwise."""
    note("graph replay", path)
    x, w = workloads.make_case(3, 6, 13, 13, 70, 3, 3, 1, 1, 0.9, seed=21)
    xd, wd = to_dev(torch, x), to_dev(torch, w)
    desc = isc.make_desc(3, 6, 13, 13, 70, 3, 3, 1, 1)
    eager = isc.isc_conv2d(xd, wd, 1, 1, path=path).clone()
    y = torch.empty_like(eager)
    ws = isc.workspace(desc, path)
    fn = lambda: isc.isc_conv2d(xd, wd, 1, 1, path=path, out=y, ws=ws)  # noqa: E731
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    other_x, other_w = workloads.make_case(2, 6, 13, 13, 70, 3, 3, 1, 1, 0.5, seed=22)
    for _ in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, eager)
        isc.isc_conv2d(to_dev(torch, other_x), to_dev(torch, other_w), 1, 1, path=path)
        torch.cuda.synchronize()
    assert_conv_close(eager.cpu().numpy(), oracle.conv2d_f64(x, w, 1, 1), "graph %s" % path)


def test_sparse_conv_entry_from_lists(torch, isc):
    """isc_compact + isc_repack_filter + isc_sparse_conv, one compaction
    shared by two convolutions of the same input (inception-style)."""
    note("sparse conv from shared lists")
    x, _ = workloads.make_case(2, 8, 28, 28, 1, 1, 1, 1, 0, 0.9, seed=31)
    rng = np.random.default_rng(32)
    w3 = (rng.standard_normal((40, 8, 3, 3)) * 0.1).astype(np.float32)
    w5 = (rng.standard_normal((20, 8, 5, 5)) * 0.1).astype(np.float32)
    xd = to_dev(torch, x)
    lists = isc.isc_compact(xd)
    for w, P in ((w3, 1), (w5, 2)):
        wt = isc.isc_repack_filter(to_dev(torch, w))
        K, C, R, S = w.shape
        # [c][r][s][k], K contiguous and zero padded to a multiple of 64
        want_wt = np.zeros((C, R, S, (K + 63) // 64 * 64), np.float32)
        want_wt[..., :K] = w.transpose(1, 2, 3, 0)
        assert np.array_equal(wt.dense().cpu().numpy(), want_wt)
        y = isc.isc_sparse_conv(xd.shape, lists, wt, 1, P).cpu().numpy()
        assert_conv_close(y, oracle.conv2d_f64(x, w, 1, P), "lists P=%d" % P)


# ----------------------------------------------- full-size configurations --

def full_layers():
    for wl in workloads.WORKLOADS.values():
        for layer in wl.layers:
            yield pytest.param(layer, id=layer.name)


def _compact_every_plane(ent, rp_o, v_o, ys_o, xs_o, H):
    """Every plane's list against the oracle's, vectorised: values bit for
    bit, rows and columns, and nothing but the plane's own entries."""
    counts = rp_o[:, H]
    slots = np.arange(ent.shape[1])[None, :]
    used = slots < counts[:, None]
    got_v = ent[:, :, 0].view(np.uint32)
    got_yx = ent[:, :, 1].view(np.uint32)
    assert np.array_equal(got_v[used], v_o.view(np.uint32)[used])
    assert np.array_equal((got_yx >> 16)[used], ys_o.astype(np.uint32)[used])
    assert np.array_equal((got_yx & 0xFFFF)[used], xs_o.astype(np.uint32)[used])


@pytest.mark.parametrize("layer", list(full_layers()))
def test_full_size_every_output(torch, isc, layer):
    """Workload shapes at full size, in the launch configuration the benchmark
    times: compaction bit-exact on every plane, and every output of the
    sparse, dense and AUTO paths against the oracle's full convolution."""
    note("full", layer.name, layer.x_shape, layer.w_shape)
    x, w = workloads.make_inputs(layer)
    xd, wd = to_dev(torch, x), to_dev(torch, w)
    T, P = layer.T, layer.P
    row_ptr, nz, total = isc.isc_compact(xd)
    rp_o, v_o, ys_o, xs_o, tot_o = oracle.compact(x)
    assert int(total.item()) == tot_o
    assert np.array_equal(row_ptr.cpu().numpy(), rp_o)
    _compact_every_plane(nz.cpu().numpy(), rp_o, v_o, ys_o, xs_o, layer.H)
    del row_ptr, nz, v_o, ys_o, xs_o
    want = oracle.conv2d_f64(x, w, T, P)
    for path in ("sparse", "dense", "auto"):
        y = isc.isc_conv2d(xd, wd, T, P, path=path)
        assert_conv_close(y.cpu().numpy(), want, "%s %s" % (layer.name, path))
        del y
    del want
    torch.cuda.empty_cache()


FUSED_CASES = [c for c in CONV_CASES if c[7] == 1 and c[5] == c[6] and c[5] in (1, 3, 5)] + [
    # N, C, H, W, K, R, S, T, P, sparsity: the fused kernel's plans
    (3, 20, 12, 12, 50, 5, 5, 1, 0, 0.9),     # LeNet conv2: 8 phases (3 or 2 maps each), one 8 x 8 tile
    (2, 24, 11, 11, 33, 5, 5, 1, 1, 0.85),    # 3 input maps per wavefront, ragged 8 x 8 tile
    (2, 9, 20, 20, 64, 5, 5, 1, 2, 0.9),      # Wo 20: 16-column tiles, several row groups
    (1, 64, 9, 9, 17, 3, 3, 1, 1, 0.9),       # 3x3: 8 maps per wavefront
    (2, 13, 30, 30, 64, 3, 3, 1, 0, 0.8),     # Wo 28: single-row tiles, ragged phases
    (1, 100, 6, 6, 64, 1, 1, 1, 0, 0.9),      # 1x1, many input maps
    (300, 2, 5, 5, 3, 5, 5, 1, 2, 0.5),       # many images, 5 x 5 maps padded
    # filter streamed through LDS (K > 64 or a filter larger than LDS)
    (2, 9, 27, 27, 256, 5, 5, 1, 2, 0.9),     # AlexNet conv2-like: 4 maps per lane
    (2, 11, 13, 13, 384, 3, 3, 1, 1, 0.95),   # conv3/4-like: 6 maps per lane
    (1, 7, 13, 13, 200, 3, 3, 1, 1, 0.9),     # ragged last map group
    (2, 5, 28, 28, 128, 3, 3, 1, 1, 0.9),     # inception 3x3-like
    (1, 4, 9, 70, 96, 5, 5, 1, 2, 0.8),       # column tiles, ragged last tile
    (3, 3, 6, 6, 130, 1, 1, 1, 0, 0.7),       # 1x1
    (1, 300, 5, 5, 20, 5, 5, 1, 2, 0.9),      # filter of 64 maps larger than LDS
    # stride 2 (filter resident, at most 8 output columns)
    (3, 20, 11, 11, 64, 5, 5, 2, 1, 0.95),    # LeNet conv2 of Tab. 2
    (2, 7, 16, 15, 33, 5, 5, 2, 2, 0.8),      # 8 x 8 output, ragged columns
    (2, 9, 12, 9, 40, 3, 3, 2, 1, 0.9),       # 3 x 3, 6 x 5 output
    (1, 3, 4, 4, 5, 3, 3, 2, 0, 0.5),         # 1 x 1 output
]


@pytest.mark.parametrize("case", FUSED_CASES)
def test_sparse_conv_fused_entry(torch, isc, case):
    """The workspace-free entry point (on-the-fly compaction) against the
    oracle, and the AUTO path on the same shape runs it."""
    N, C, H, W, K, R, S, T, P, sp = case
    note("fused entry", case)
    desc = isc.make_desc(N, C, H, W, K, R, S, T, P)
    assert isc.isc_sparse_kernel(desc) in ("fused", "fused_reg", "fused_ring")
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=11 + sum(case[:9]))
    wt = isc.isc_repack_filter(to_dev(torch, w))
    y = isc.isc_sparse_conv_fused(to_dev(torch, x), wt, T, P).cpu().numpy()
    want = oracle.conv2d_f64(x, w, T, P)
    assert_conv_close(y, want, "fused %s" % (case,))
    y2 = isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), T, P, path="sparse").cpu().numpy()
    assert np.array_equal(y, y2), "the sparse path and the fused entry point differ"
    # integer-valued inputs: every fp32 sum is exact, so the result is bitwise
    xi, wi = workloads.integer_case(N, C, H, W, K, R, S, seed=5 + sum(case[:9]))
    yi = isc.isc_sparse_conv_fused(to_dev(torch, xi), isc.isc_repack_filter(to_dev(torch, wi)), T, P)
    assert np.array_equal(yi.cpu().numpy().astype(np.float64), oracle.conv2d_f64(xi, wi, T, P))


def test_sparse_conv_fused_rejects_ineligible(torch, isc):
    note("fused ineligible")
    x = torch.zeros((1, 2, 12, 12), device="cuda")
    w = torch.zeros((65, 2, 7, 7), device="cuda")
    with pytest.raises(isc.IscError) as e:
        isc.isc_sparse_conv_fused(x, isc.isc_repack_filter(w), 1, 0)
    assert e.value.status == 3


@pytest.mark.parametrize("case", [(3, 20, 12, 12, 50, 5, 5, 1, 0, 0.9), (2, 24, 11, 11, 33, 5, 5, 1, 1, 0.85),
                                  (2, 9, 8, 8, 64, 3, 3, 1, 1, 0.9)])
def test_fused_weight_placements_agree(torch, isc, case):
    """Plans whose wavefronts share no channel stream the weights to
    registers by default; the filter-in-LDS kernel (tuning kernel "fused") on the
    same shapes: both against the oracle, and bitwise equal to each other
    (the same channel order per phase and the same pairing of the phases
    per output)."""
    N, C, H, W, K, R, S, T, P, sp = case
    note("fused weight placement", case)
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=71 + sum(case[:9]))
    wt = isc.isc_repack_filter(to_dev(torch, w))
    want = oracle.conv2d_f64(x, w, T, P)
    outs = []
    desc = isc.make_desc(N, C, H, W, K, R, S, T, P)
    assert isc.isc_sparse_kernel(desc, {"kernel": "fused"}) == "fused"
    for tu in (None, {"kernel": "fused"}):
        y = isc.isc_sparse_conv_fused(to_dev(torch, x), wt, T, P, tuning=tu).cpu().numpy()
        assert_conv_close(y, want, "fused %s %s" % (tu, case))
        outs.append(y)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


@pytest.mark.parametrize("case", [(2, 12, 7, 7, 150, 3, 3, 1, 1, 0.9), (3, 9, 8, 8, 128, 5, 5, 1, 2, 0.9),
                                  (1, 5, 5, 6, 65, 3, 3, 1, 1, 0.8), (130, 4, 7, 7, 96, 3, 3, 1, 1, 0.9),
                                  (2, 11, 13, 13, 200, 3, 3, 1, 1, 0.9), (40, 6, 14, 14, 70, 3, 3, 1, 1, 0.9),
                                  (2, 7, 12, 12, 130, 5, 5, 1, 2, 0.9), (2, 40, 9, 9, 100, 1, 1, 1, 0, 0.9),
                                  (3, 33, 16, 16, 80, 1, 1, 1, 0, 0.8)])
def test_register_kernel_map_groups(torch, isc, case):
    """The register-weight kernel (tuning kernel "fused_reg") beyond 64 maps
    (one workgroup per group of 64, ragged last group included) and on
    16-column tiles, every tile height it takes: plain and rectified with the
    census, against the oracle; and the filter-ring kernel (tuning kernel
    "fused_ring") on the same shape."""
    N, C, H, W, K, R, S, T, P, sp = case
    note("register kernel map groups", case)
    desc = isc.make_desc(N, C, H, W, K, R, S, T, P)
    reg = {"kernel": "fused_reg"}
    assert isc.isc_sparse_kernel(desc, reg) == "fused_reg"
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=83 + sum(case[:9]))
    wt = isc.isc_repack_filter(to_dev(torch, w))
    want = oracle.conv2d_f64(x, w, T, P)
    Wo = want.shape[3]
    full = 4 if Wo <= 8 else 2
    for th in (full, full // 2):
        tu = {"kernel": "fused_reg", "rows": th}
        assert isc.isc_sparse_plan(desc, tu)["rows"] == th
        y = isc.isc_sparse_conv_fused(to_dev(torch, x), wt, T, P, tuning=tu).cpu().numpy()
        assert_conv_close(y, want, "register kernel th%d %s" % (th, case))
    yc = isc.census(desc)
    z = isc.isc_conv2d_relu(to_dev(torch, x), to_dev(torch, w), T, P, path="sparse", y_census=yc,
                            ws=isc.workspace(desc, "sparse"), tuning=reg).cpu().numpy()
    want_relu, _ = oracle.relu_conv2d_f64(x, w, T, P)
    assert_conv_close(z, want_relu, "register kernel relu %s" % (case,))
    assert isc.isc_census_read(yc) == (z.size, int(np.count_nonzero(z)))
    ring = {"kernel": "fused_ring"}
    other = isc.isc_sparse_kernel(desc, ring)
    assert other in ("fused", "fused_ring"), other
    y = isc.isc_sparse_conv_fused(to_dev(torch, x), wt, T, P, tuning=ring).cpu().numpy()
    assert_conv_close(y, want, "%s kernel %s" % (other, case))


@pytest.mark.parametrize("case", [(1, 384, 5, 5, 384, 3, 3, 1, 1, 0.9), (1, 100, 9, 7, 70, 3, 3, 1, 1, 0.5),
                                  (2, 48, 7, 7, 128, 5, 5, 1, 2, 0.9), (1, 60, 6, 6, 20, 5, 5, 1, 2, 0.3),
                                  (3, 800, 4, 4, 33, 1, 1, 1, 0, 0.6), (100, 128, 13, 13, 256, 3, 3, 1, 1, 0.5),
                                  (60, 64, 14, 14, 320, 3, 3, 1, 1, 0.5)])
def test_dense_split_reduction(torch, isc, case):
    """The dense path's GEMM with its reduction split over C*R*S (grids of
    fewer than 128 tiles, and the last two shapes: 266 and 276 tiles of
    128 x 128, which the GEMM's model splits into four and two ranges to
    even out the CUs' shares): plain, rectified with the census, and under
    AUTO, against the oracle; and the unsplit GEMM (tuning gemm_split = -1)
    on the same shape with a workspace that has no room for partial sums."""
    N, C, H, W, K, R, S, T, P, sp = case
    note("dense split", case)
    desc = isc.make_desc(N, C, H, W, K, R, S, T, P)
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=91 + sum(case[:9]))
    want = oracle.conv2d_f64(x, w, T, P)
    xd, wd = to_dev(torch, x), to_dev(torch, w)
    ws = isc.workspace(desc, "dense")
    y = isc.isc_conv2d(xd, wd, T, P, path="dense", ws=ws).cpu().numpy()
    assert_conv_close(y, want, "dense split %s" % (case,))
    yc = isc.census(desc)
    z = isc.isc_conv2d_relu(xd, wd, T, P, path="dense", y_census=yc, ws=ws).cpu().numpy()
    want_relu, _ = oracle.relu_conv2d_f64(x, w, T, P)
    assert_conv_close(z, want_relu, "dense split relu %s" % (case,))
    assert isc.isc_census_read(yc) == (z.size, int(np.count_nonzero(z)))
    a = isc.isc_conv2d(xd, wd, T, P, path="auto", threshold=0.99, ws=isc.workspace(desc, "auto")).cpu().numpy()
    assert_conv_close(a, want, "auto (dense) split %s" % (case,))
    u = isc.isc_conv2d(xd, wd, T, P, path="dense", ws=isc.workspace(desc, "dense"),
                       tuning={"gemm_split": -1}).cpu().numpy()
    assert_conv_close(u, want, "dense unsplit %s" % (case,))
    # the same with a workspace too small for the partial sums (the dense
    # path's implicit GEMM, unsplit, needs only its decision record)
    small = torch.empty(4096, dtype=torch.uint8, device="cuda")
    assert small.numel() < isc.isc_workspace_size(desc, "dense")
    with pytest.raises(isc.IscError):
        isc.isc_conv2d(xd, wd, T, P, path="dense", ws=small)
    v = isc.isc_conv2d(xd, wd, T, P, path="dense", ws=small, tuning={"gemm_split": -1}).cpu().numpy()
    assert np.array_equal(v.view(np.uint32), u.view(np.uint32))


def test_side_stream_parity(torch, isc):
    """Calls enqueued on a stream other than the current one: temporaries are
    allocated on that stream, and the results equal the oracle's after the
    stream is synchronised, with other work running on the current stream."""
    note("side stream")
    x, w = workloads.make_case(4, 12, 27, 27, 100, 5, 5, 1, 2, 0.9, seed=44)
    want = oracle.conv2d_f64(x, w, 1, 2)
    xd, wd = to_dev(torch, x), to_dev(torch, w)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    outs = []
    for path in ("sparse", "dense", "auto"):
        outs.append(isc.isc_conv2d(xd, wd, 1, 2, path=path, stream=side))
        junk = torch.empty(1 << 22, device="cuda")          # reuse pressure on the current stream
        junk.fill_(float("nan"))
    side.synchronize()
    for path, y in zip(("sparse", "dense", "auto"), outs):
        assert_conv_close(y.cpu().numpy(), want, "side stream %s" % path)


def _ring_tiles():
    """The filter-ring kernel's compiled tiles, read from its header:
    (R, maps per lane, rows, cols, wavefronts per workgroup)."""
    import os
    import re
    src = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_1704_07724_amd",
                            "csrc", "sparse_fring.hpp")).read()
    out = []
    for r in (1, 3, 5):
        body = re.search(r"kTiles%d\[\] = \{(.*?)\};" % r, src, re.S).group(1)
        for t in re.findall(r"\{(\d+), (\d+), (\d+), (\d+)\}", body):
            out.append((r,) + tuple(int(v) for v in t))
    return out


@pytest.mark.parametrize("tile", _ring_tiles(), ids=lambda t: "R%d-kpl%d-%dx%d-w%d" % t)
def test_every_ring_tile(torch, isc, tile):
    """Every compiled tile of the filter-ring kernel, forced through the
    per-call overrides, against the oracle on maps with ragged row bands and
    column tiles, a ragged last map group and a partly filled last
    workgroup; and bitwise on integer inputs."""
    R, kpl, th, tw, nw = tile
    tu = {"kernel": "fused_ring", "maps_per_lane": kpl, "rows": th, "cols": tw, "waves": nw}
    for case in [(2, 5, 17, 19, 70, R, R, 1, R // 2, 0.85), (1, 3, 11, 30, 200, R, R, 1, R // 2, 0.9)]:
        N, C, H, W, K, _, _, T, P, sp = case
        note("ring tile", tile, case)
        desc = isc.make_desc(N, C, H, W, K, R, R, T, P)
        plan = isc.isc_sparse_plan(desc, tu)
        assert (plan["kernel"], plan["maps_per_lane"], plan["rows"], plan["cols"], plan["waves"]) == \
            ("fused_ring", kpl, th, tw, nw), plan
        x, w = workloads.make_case(N, C, H, W, K, R, R, T, P, sp, seed=101 + sum(case[:5]) + kpl * 7 + th * 3 + tw)
        y = isc.isc_sparse_conv_fused(to_dev(torch, x), isc.isc_repack_filter(to_dev(torch, w)), T, P,
                                      tuning=tu).cpu().numpy()
        assert_conv_close(y, oracle.conv2d_f64(x, w, T, P), "ring tile %s %s" % (tile, case))
        xi, wi = workloads.integer_case(N, C, H, W, K, R, R, seed=5 + kpl + th + tw)
        yi = isc.isc_sparse_conv_fused(to_dev(torch, xi), isc.isc_repack_filter(to_dev(torch, wi)), T, P, tuning=tu)
        assert np.array_equal(yi.cpu().numpy().astype(np.float64), oracle.conv2d_f64(xi, wi, T, P))


def test_auto_crossover_both_sides(torch, isc):
    """AUTO with the per-shape crossover (the library's default threshold):
    on a shape whose modelled crossover lies inside (0, 1), an input below it
    runs the dense path and one above it the sparse path; the decision is the
    integer comparison of the input's nonzero count, and both outputs match
    the oracle."""
    case = (8, 96, 27, 27, 256, 5, 5, 1, 2)
    N, C, H, W, K, R, S, T, P = case
    desc = isc.make_desc(*case)
    s_star = isc.isc_crossover_sparsity(desc)
    assert 0.3 < s_star < 0.95, s_star
    for sp, want in ((s_star - 0.2, "dense"), (min(0.99, s_star + 0.15), "sparse")):
        note("crossover", case, "sparsity", sp, want)
        x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=301 + int(sp * 100))
        measured = 1.0 - np.count_nonzero(x) / x.size
        assert (measured >= s_star) == (want == "sparse")
        ws = isc.workspace(desc, "auto")
        y = isc.isc_conv2d(to_dev(torch, x), to_dev(torch, w), T, P, path="auto", threshold=isc.THRESHOLD_CROSSOVER,
                           ws=ws)
        nnz, taken = isc.isc_decision(desc, ws)
        assert nnz == int(np.count_nonzero(x)) and taken == want
        assert_conv_close(y.cpu().numpy(), oracle.conv2d_f64(x, w, T, P), "crossover %s" % want)
