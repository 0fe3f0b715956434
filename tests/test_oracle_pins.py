"""Pins for the CPU oracle: each check ties it to something other than itself.

- the scatter ("inverse") form of the convolution written as plain Python
  loops, on tiny inputs: every input element adds W * x to the outputs it
  reaches (Sec. "Sparse Convolution", the ISC view), which shares no index
  expression with the oracle's gather loop over Eq. 1;
- torch.nn.functional.conv2d in float64 on the CPU (an independent library);
- closed forms: 1x1 filters are a matrix product, all-ones input and filters
  count the in-bounds taps, a centred delta filter reproduces the input,
  a zero input gives exactly zero, stride T subsamples the stride-1 output;
- exact linearity on dyadic values;
- compaction against numpy's flatnonzero; the nonzero-MAC count against a
  brute-force enumeration and against the dense count for all-nonzero input;
- im2col against a numpy sliding-window construction and the GEMM identity
  of Fig. 3 (M_K x M_I = M_O);
- the rectifier of Eq. 2 against torch.relu, the exact split
  relu(o) - relu(-o) = o, and the identity / all-zero closed forms; its
  nonzero count against numpy's count of positive outputs;
- the weight gradient against its zero-skipping scatter form in plain Python,
  torch's conv2d_weight in float64, the adjoint identity
  <conv(x, w), dy> = <w, dw(x, dy)> (exact on dyadic values, which ties it to
  the pinned forward oracle) and the 1x1 matrix product.
"""
import itertools

import numpy as np
import pytest

import oracle
import workloads


# ---------------------------------------------------------------- helpers ---

def scatter_conv_py(x, w, T, P):
    """Inverse form: loop over inputs, add each one's products to the outputs
    it reaches.  out[n,k,oy,ox] with oy*T = y + P - r."""
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    Ho = (H + 2 * P - R) // T + 1
    Wo = (W + 2 * P - S) // T + 1
    out = [[[[0.0] * Wo for _ in range(Ho)] for _ in range(K)] for _ in range(N)]
    for n in range(N):
        for c in range(C):
            for y in range(H):
                for xx in range(W):
                    v = float(x[n, c, y, xx])
                    for r in range(R):
                        ty = y + P - r
                        if ty < 0 or ty % T:
                            continue
                        oy = ty // T
                        if oy >= Ho:
                            continue
                        for s in range(S):
                            tx = xx + P - s
                            if tx < 0 or tx % T:
                                continue
                            ox = tx // T
                            if ox >= Wo:
                                continue
                            for k in range(K):
                                out[n][k][oy][ox] += float(w[k, c, r, s]) * v
    return np.array(out, dtype=np.float64).reshape(N, K, Ho, Wo)


def rand_case(rng, N, C, H, W, K, R, S, sparsity=0.5):
    x = np.abs(rng.standard_normal((N, C, H, W))).astype(np.float32)
    x[rng.random(x.shape) < sparsity] = 0.0
    w = rng.standard_normal((K, C, R, S)).astype(np.float32)
    return x, w


# ------------------------------------------------------------ output size ---

def test_out_size_standard_formula():
    # floor((H + 2P - R)/T) + 1 for every small combination, against
    # len(range(...)) of the valid window starts
    for H, R, P, T in itertools.product(range(1, 12), range(1, 6), range(0, 3), range(1, 4)):
        starts = [i for i in range(-P, H + P) if i + R <= H + P and (i + P) % T == 0]
        assert oracle.out_size(H, R, P, T) == len(starts), (H, R, P, T)


def test_out_size_matches_printed_formula_at_stride_one():
    # Sec. "Sparsity of ReLUs" prints H_out = (H + 2P - R + 1)/T; at T = 1 it
    # equals the standard formula for every layer of Tab. 2 with T = 1
    import json, os
    tab = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_tables.json")))
    for row in tab["table2_layers"]:
        H, R, P, T = row["H"], row["R"], row["P"], row["T"]
        if T == 1:
            assert oracle.out_size(H, R, P, T) == H + 2 * P - R + 1
        else:
            # LeNet-Conv2 (T = 2): the printed formula gives a non-integer,
            # the floor reading gives the size a strided window count has
            assert (H + 2 * P - R + 1) / T != int((H + 2 * P - R + 1) / T)
            assert oracle.out_size(H, R, P, T) == (H + 2 * P - R) // T + 1


# ------------------------------------------------------------ convolution ---

@pytest.mark.parametrize("seed", range(12))
def test_conv_equals_scatter_form_bruteforce(seed):
    rng = np.random.default_rng(1000 + seed)
    N = int(rng.integers(1, 3)); C = int(rng.integers(1, 4)); K = int(rng.integers(1, 4))
    R = int(rng.integers(1, 4)); S = int(rng.integers(1, 4))
    T = int(rng.integers(1, 4)); P = int(rng.integers(0, 3))
    H = int(rng.integers(max(1, R - 2 * P), 8)); W = int(rng.integers(max(1, S - 2 * P), 8))
    x, w = rand_case(rng, N, C, H, W, K, R, S)
    got = oracle.conv2d_f64(x, w, T, P)
    want = scatter_conv_py(x, w, T, P)
    assert got.shape == want.shape
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(10))
def test_conv_equals_torch_float64(seed):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2000 + seed)
    N = int(rng.integers(1, 4)); C = int(rng.integers(1, 9)); K = int(rng.integers(1, 9))
    R = int(rng.choice([1, 2, 3, 5])); S = int(rng.choice([1, 3, 5]))
    T = int(rng.integers(1, 4)); P = int(rng.integers(0, 3))
    H = int(rng.integers(max(1, R - 2 * P), 17)); W = int(rng.integers(max(1, S - 2 * P), 17))
    x, w = rand_case(rng, N, C, H, W, K, R, S, sparsity=0.7)
    got = oracle.conv2d_f64(x, w, T, P)
    want = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                      stride=T, padding=P).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_one_by_one_is_matmul():
    rng = np.random.default_rng(7)
    x, w = rand_case(rng, 3, 6, 5, 7, 4, 1, 1)
    got = oracle.conv2d_f64(x, w, 1, 0)
    want = np.einsum("kc,nchw->nkhw", w[:, :, 0, 0].astype(np.float64), x.astype(np.float64))
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
    # with stride T the same holds on the subsampled input
    got2 = oracle.conv2d_f64(x, w, 2, 0)
    want2 = np.einsum("kc,nchw->nkhw", w[:, :, 0, 0].astype(np.float64),
                      x[:, :, ::2, ::2].astype(np.float64))
    np.testing.assert_allclose(got2, want2, rtol=1e-13, atol=1e-13)


def test_zero_input_gives_exact_zero():
    rng = np.random.default_rng(8)
    _, w = rand_case(rng, 1, 5, 9, 9, 6, 3, 3)
    x = np.zeros((2, 5, 9, 9), np.float32)
    out = oracle.conv2d_f64(x, w, 1, 1)
    assert out.shape == (2, 6, 9, 9)
    assert np.all(out == 0.0)


@pytest.mark.parametrize("T,P", [(1, 0), (1, 2), (2, 1), (3, 2)])
def test_ones_closed_form(T, P):
    # x = 1, w = 1: O[i, j] = C * (#rows r with 0 <= i*T + r - P < H) * (#cols likewise)
    N, C, H, W, K, R, S = 2, 3, 9, 8, 2, 3, 4
    x = np.ones((N, C, H, W), np.float32)
    w = np.ones((K, C, R, S), np.float32)
    out = oracle.conv2d_f64(x, w, T, P)
    Ho, Wo = out.shape[2:]
    for i in range(Ho):
        cr = min(H, i * T - P + R) - max(0, i * T - P)
        for j in range(Wo):
            cs = min(W, j * T - P + S) - max(0, j * T - P)
            assert np.all(out[:, :, i, j] == C * cr * cs), (i, j)


def test_linearity_exact_on_dyadic_values():
    rng = np.random.default_rng(9)
    shape_x, shape_w = (2, 4, 7, 6), (3, 4, 3, 3)
    # dyadic values: small integers / 8, so every product and sum is exact in fp64
    x1 = (rng.integers(0, 16, shape_x) / 8).astype(np.float32)
    x2 = (rng.integers(0, 16, shape_x) / 8).astype(np.float32)
    w = (rng.integers(-8, 9, shape_w) / 4).astype(np.float32)
    a, b = 3.0, -0.5
    lhs = oracle.conv2d_f64((a * x1 + b * x2).astype(np.float32), w, 1, 1)
    rhs = a * oracle.conv2d_f64(x1, w, 1, 1) + b * oracle.conv2d_f64(x2, w, 1, 1)
    assert np.array_equal(lhs, rhs)


@pytest.mark.parametrize("R", [1, 3, 5])
def test_delta_filter_reproduces_input(R):
    rng = np.random.default_rng(10 + R)
    C = 4
    x, _ = rand_case(rng, 2, C, 7, 9, 1, 1, 1)
    w = np.zeros((C, C, R, R), np.float32)
    for c in range(C):
        w[c, c, (R - 1) // 2, (R - 1) // 2] = 1.0
    out = oracle.conv2d_f64(x, w, 1, (R - 1) // 2)
    assert np.array_equal(out, x.astype(np.float64))
    # a delta at (0, 0) with no padding is a shift: O[i, j] = X[i, j]
    # restricted to the valid window; at (R-1, R-1) it is X[i+R-1, j+R-1]
    w2 = np.zeros((C, C, R, R), np.float32)
    for c in range(C):
        w2[c, c, R - 1, R - 1] = 1.0
    out2 = oracle.conv2d_f64(x, w2, 1, 0)
    assert np.array_equal(out2, x[:, :, R - 1:, R - 1:].astype(np.float64))


@pytest.mark.parametrize("T", [2, 3])
def test_stride_subsamples_stride_one(T):
    rng = np.random.default_rng(20 + T)
    x, w = rand_case(rng, 2, 3, 11, 10, 3, 3, 2)
    full = oracle.conv2d_f64(x, w, 1, 1)
    strided = oracle.conv2d_f64(x, w, T, 1)
    assert np.array_equal(strided, full[:, :, ::T, ::T])


def test_pointwise_matches_full():
    rng = np.random.default_rng(30)
    x, w = rand_case(rng, 3, 5, 10, 9, 7, 3, 5)
    full = oracle.conv2d_f64(x, w, 2, 2)
    idx = rng.choice(full.size, size=200, replace=False)
    pts = oracle.conv2d_f64_at(x, w, 2, 2, idx)
    assert np.array_equal(pts, full.ravel()[idx])


# ------------------------------------------------------------- compaction ---

def test_compaction_against_flatnonzero():
    rng = np.random.default_rng(40)
    x, _ = rand_case(rng, 3, 4, 9, 13, 1, 1, 1, sparsity=0.8)
    x[0, 0, 1, 2] = -0.0          # signed zero counts as zero
    x[0, 1, 3, 3] = np.float32(1e-45)  # a denormal counts as nonzero
    x[1, 2, 0, 0] = np.inf
    x[2, 3, 8, 12] = np.nan
    row_ptr, v, ys, xs, total = oracle.compact(x)
    N, C, H, W = x.shape
    bits = x.view(np.uint32) & np.uint32(0x7FFFFFFF)
    assert total == int(np.count_nonzero(bits))
    for p in range(N * C):
        plane_bits = bits.reshape(N * C, H * W)[p]
        nzi = np.flatnonzero(plane_bits)   # ascending = row-major
        cnt = nzi.size
        assert row_ptr[p, H] == cnt
        assert np.array_equal(ys[p, :cnt], nzi // W)
        assert np.array_equal(xs[p, :cnt], nzi % W)
        assert np.array_equal(v[p, :cnt].view(np.uint32),
                              x.reshape(N * C, H * W)[p, nzi].view(np.uint32))
        assert np.array_equal(row_ptr[p, :H],
                              np.searchsorted(nzi // W, np.arange(H), side="left"))
        assert np.all(np.diff(row_ptr[p]) >= 0)


def test_compaction_scatter_back_reproduces_input():
    rng = np.random.default_rng(41)
    x, _ = rand_case(rng, 2, 3, 6, 5, 1, 1, 1, sparsity=0.6)
    row_ptr, v, ys, xs, total = oracle.compact(x)
    N, C, H, W = x.shape
    rebuilt = np.zeros_like(x).reshape(N * C, H, W)
    for p in range(N * C):
        cnt = row_ptr[p, H]
        rebuilt[p, ys[p, :cnt], xs[p, :cnt]] = v[p, :cnt]
    assert np.array_equal(rebuilt.reshape(x.shape), x)


# -------------------------------------------------------- nonzero MACs ---

def nz_macs_bruteforce(x, K, R, S, T, P):
    N, C, H, W = x.shape
    Ho = (H + 2 * P - R) // T + 1
    Wo = (W + 2 * P - S) // T + 1
    cnt = 0
    # enumerate (output, tap) pairs whose input is a nonzero inside the map
    for n, c, i, j, r, s in itertools.product(range(N), range(C), range(Ho), range(Wo),
                                              range(R), range(S)):
        y, xx = i * T + r - P, j * T + s - P
        if 0 <= y < H and 0 <= xx < W and x[n, c, y, xx] != 0:
            cnt += K
    return cnt


@pytest.mark.parametrize("T,P", [(1, 0), (1, 1), (2, 1), (3, 2)])
def test_nz_macs_bruteforce(T, P):
    rng = np.random.default_rng(50 + T * 10 + P)
    x, _ = rand_case(rng, 2, 3, 7, 8, 1, 1, 1, sparsity=0.6)
    for K, R, S in [(1, 3, 3), (4, 2, 5), (3, 1, 1)]:
        assert oracle.nz_macs(x, K, R, S, T, P) == nz_macs_bruteforce(x, K, R, S, T, P)


def test_nz_macs_dense_input_equals_direct_count():
    # every input nonzero, no padding, stride 1: each (output, tap) pair has an
    # in-map input, so the count is the direct convolution's Ho*Wo*R*S*K*C
    # (Sec. "Sparse Convolution") per image
    x = np.ones((3, 4, 10, 9), np.float32)
    K, R, S = 5, 3, 4
    Ho, Wo = 10 - R + 1, 9 - S + 1
    assert oracle.nz_macs(x, K, R, S, 1, 0) == 3 * Ho * Wo * R * S * K * 4
    assert oracle.nz_macs(np.zeros_like(x), K, R, S, 1, 0) == 0


# ----------------------------------------------------------------- im2col ---

@pytest.mark.parametrize("T,P", [(1, 0), (1, 2), (2, 1)])
def test_im2col_against_sliding_window(T, P):
    rng = np.random.default_rng(60 + T + P)
    x, w = rand_case(rng, 2, 3, 8, 7, 4, 3, 2)
    N, C, H, W = x.shape
    _, _, R, S = w.shape
    col = oracle.im2col(x, R, S, T, P)
    xp = np.pad(x, ((0, 0), (0, 0), (P, P), (P, P)))
    win = np.lib.stride_tricks.sliding_window_view(xp, (R, S), axis=(2, 3))[:, :, ::T, ::T]
    # win[n, c, i, j, r, s] -> rows (c, r, s), columns (n, i, j)
    want = win.transpose(1, 4, 5, 0, 2, 3).reshape(C * R * S, -1)
    assert np.array_equal(col, want)
    # Fig. 3: M_K [K x RSC] times M_I gives M_O [K x HoWo] (per image columns)
    mo = w.reshape(w.shape[0], -1).astype(np.float64) @ col.astype(np.float64)
    Ho, Wo = oracle.out_size(H, R, P, T), oracle.out_size(W, S, P, T)
    mo = mo.reshape(w.shape[0], N, Ho, Wo).transpose(1, 0, 2, 3)
    np.testing.assert_allclose(mo, oracle.conv2d_f64(x, w, T, P), rtol=1e-12, atol=1e-12)


def test_im2col_row_stride_leaves_tail():
    rng = np.random.default_rng(70)
    x, _ = rand_case(rng, 1, 2, 5, 5, 1, 1, 1)
    col = oracle.im2col(x, 3, 3, 1, 1, ldc=40)
    assert col.shape == (18, 40)
    assert np.all(col[:, 25:] == 0)


# ----------------------------------------------- integer-valued exactness ---

def test_integer_inputs_are_exact_in_fp32_order_free():
    # the parity bar for the GPU path on integer inputs is bitwise: check that
    # the oracle's fp64 value is an integer and fits fp32 exactly
    x, w = workloads.integer_case(2, 5, 9, 9, 4, 3, 3, seed=80)
    out = oracle.conv2d_f64(x, w, 1, 1)
    assert np.array_equal(out, np.round(out))
    assert np.max(np.abs(out)) < 2 ** 24
    assert np.array_equal(out.astype(np.float32).astype(np.float64), out)


# ------------------------------------------- rectifier (Eq. 2) and counts ---

def test_relu_conv_against_torch_float64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(4100)
    for T, P in [(1, 0), (1, 1), (2, 2)]:
        x, w = rand_case(rng, 2, 5, 11, 9, 6, 3, 3, sparsity=0.6)
        y, nnz = oracle.relu_conv2d_f64(x, w, T, P)
        want = torch.relu(torch.nn.functional.conv2d(torch.from_numpy(x).double(),
                                                     torch.from_numpy(w).double(),
                                                     stride=T, padding=P)).numpy()
        np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-12)
        assert nnz == int(np.count_nonzero(want))


def test_relu_splits_the_convolution_exactly():
    # conv(-x) = -conv(x) exactly in fp64, so relu(o) - relu(-o) = o: the
    # rectifier keeps the positive part and nothing else; the rectified
    # output is non-negative, equals o or 0 everywhere, and its count is the
    # number of positive outputs
    rng = np.random.default_rng(4101)
    x, w = rand_case(rng, 2, 4, 9, 8, 5, 3, 3, sparsity=0.5)
    x[:, :, :3, :] = 0.0  # exact zero outputs along the top rows
    o = oracle.conv2d_f64(x, w, 1, 1)
    pos, n_pos = oracle.relu_conv2d_f64(x, w, 1, 1)
    neg, n_neg = oracle.relu_conv2d_f64(-x, w, 1, 1)
    assert np.array_equal(pos - neg, o)
    assert np.all(pos >= 0.0) and np.all((pos == o) | (pos == 0.0))
    assert np.any(o == 0.0)
    assert n_pos == int(np.count_nonzero(o > 0.0)) == int(np.count_nonzero(pos))
    assert n_neg == int(np.count_nonzero(o < 0.0))
    assert n_pos + n_neg + int(np.count_nonzero(o == 0.0)) == o.size


def test_relu_closed_forms():
    # non-negative input and filter: the rectifier is the identity; a
    # non-positive filter: every output is rectified to zero
    rng = np.random.default_rng(4102)
    x, w = rand_case(rng, 1, 3, 7, 7, 4, 3, 3, sparsity=0.3)
    w = np.abs(w)
    y, nnz = oracle.relu_conv2d_f64(x, w, 1, 1)
    assert np.array_equal(y, oracle.conv2d_f64(x, w, 1, 1))
    assert nnz == int(np.count_nonzero(y))
    y2, nnz2 = oracle.relu_conv2d_f64(x, -w, 1, 1)
    assert nnz2 == 0 and np.all(y2 == 0.0)


# ------------------------------------------- weight gradient (training) ---

def scatter_dw_py(x, dy, R, S, T, P):
    """Zero-skipping form: every nonzero input adds x * dy at each output it
    reaches to the gradient of the tap that connects them."""
    N, C, H, W = x.shape
    K, Ho, Wo = dy.shape[1], dy.shape[2], dy.shape[3]
    dw = [[[[0.0] * S for _ in range(R)] for _ in range(C)] for _ in range(K)]
    for n in range(N):
        for c in range(C):
            for y in range(H):
                for xx in range(W):
                    v = float(x[n, c, y, xx])
                    if v == 0.0:
                        continue
                    for r in range(R):
                        ty = y + P - r
                        if ty < 0 or ty % T or ty // T >= Ho:
                            continue
                        for s in range(S):
                            tx = xx + P - s
                            if tx < 0 or tx % T or tx // T >= Wo:
                                continue
                            for k in range(K):
                                dw[k][c][r][s] += v * float(dy[n, k, ty // T, tx // T])
    return np.array(dw, dtype=np.float64)


@pytest.mark.parametrize("seed", range(6))
def test_dw_equals_scatter_form_bruteforce(seed):
    rng = np.random.default_rng(5000 + seed)
    N = int(rng.integers(1, 3)); C = int(rng.integers(1, 4)); K = int(rng.integers(1, 4))
    R = int(rng.choice([1, 2, 3])); S = int(rng.choice([1, 3]))
    T = int(rng.integers(1, 4)); P = int(rng.integers(0, 3))
    H = int(rng.integers(max(1, R - 2 * P), 8)); W = int(rng.integers(max(1, S - 2 * P), 8))
    x, _ = rand_case(rng, N, C, H, W, K, R, S)
    Ho, Wo = oracle.out_size(H, R, P, T), oracle.out_size(W, S, P, T)
    dy = rng.standard_normal((N, K, Ho, Wo)).astype(np.float32)
    np.testing.assert_allclose(oracle.conv2d_dw_f64(x, dy, R, S, T, P), scatter_dw_py(x, dy, R, S, T, P),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_dw_against_torch_float64(seed):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5100 + seed)
    N = int(rng.integers(1, 4)); C = int(rng.integers(1, 7)); K = int(rng.integers(1, 7))
    R = int(rng.choice([1, 3, 5])); S = R
    T = int(rng.integers(1, 3)); P = int(rng.integers(0, 3))
    H = int(rng.integers(max(1, R - 2 * P), 14)); W = int(rng.integers(max(1, S - 2 * P), 14))
    x, _ = rand_case(rng, N, C, H, W, K, R, S, sparsity=0.8)
    Ho, Wo = oracle.out_size(H, R, P, T), oracle.out_size(W, S, P, T)
    dy = rng.standard_normal((N, K, Ho, Wo)).astype(np.float32)
    want = torch.nn.grad.conv2d_weight(torch.from_numpy(x).double(), (K, C, R, S), torch.from_numpy(dy).double(),
                                       stride=T, padding=P).numpy()
    np.testing.assert_allclose(oracle.conv2d_dw_f64(x, dy, R, S, T, P), want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("T,P", [(1, 0), (1, 2), (2, 1)])
def test_dw_adjoint_of_the_convolution(T, P):
    # <conv(x, w), dy> = <w, dw(x, dy)> for every w: the gradient is the
    # adjoint of Eq. 1 in w.  Dyadic values keep both sides exact in fp64.
    rng = np.random.default_rng(5200 + T + P)
    N, C, H, W, K, R, S = 2, 3, 8, 7, 4, 3, 3
    x = (rng.integers(0, 8, (N, C, H, W)) / 4).astype(np.float32)
    x[rng.random(x.shape) < 0.6] = 0.0
    w = (rng.integers(-8, 9, (K, C, R, S)) / 8).astype(np.float32)
    o = oracle.conv2d_f64(x, w, T, P)
    dy = (rng.integers(-8, 9, o.shape) / 2).astype(np.float32)
    lhs = float(np.sum(o * dy.astype(np.float64)))
    rhs = float(np.sum(w.astype(np.float64) * oracle.conv2d_dw_f64(x, dy, R, S, T, P)))
    assert lhs == rhs


def test_dw_one_by_one_is_matmul_and_zero_input():
    rng = np.random.default_rng(5300)
    x, _ = rand_case(rng, 3, 5, 6, 4, 2, 1, 1)
    dy = rng.standard_normal((3, 7, 6, 4)).astype(np.float32)
    want = sum(dy[n].reshape(7, -1).astype(np.float64) @ x[n].reshape(5, -1).T.astype(np.float64) for n in range(3))
    np.testing.assert_allclose(oracle.conv2d_dw_f64(x, dy, 1, 1)[:, :, 0, 0], want, rtol=1e-13, atol=1e-13)
    assert np.all(oracle.conv2d_dw_f64(np.zeros_like(x), dy, 1, 1) == 0.0)
