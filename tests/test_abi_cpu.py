"""The C-ABI library on the host: it loads, exports every symbol include/isc.h
declares, and rejects bad arguments before touching any device (these run
without a GPU; no compute call is made)."""
import ctypes
import os
import re

import pytest

import oracle
import paper_1704_07724_amd as isc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "isc.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(isc_[a-z0-9_]+)\s*\(", text)))


def test_library_loads_and_exports_header_symbols():
    L = isc.lib()
    names = header_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(isc.EXPORTS)
    assert "gfx950" in isc.isc_version()


def test_status_strings():
    for code in range(0, 11):
        assert isc.status_str(code)
    assert isc.status_str(99) == "unknown status"


@pytest.mark.parametrize("H,R,P,T", [(12, 5, 0, 1), (27, 5, 2, 1), (13, 3, 1, 1), (11, 5, 1, 2),
                                     (7, 7, 3, 2), (9, 2, 0, 3), (1, 1, 0, 1), (5, 7, 1, 1)])
def test_out_shape_matches_oracle(H, R, P, T):
    d = isc.make_desc(1, 1, H, H + 1, 1, R, R, T, P)
    ho_o = oracle.out_size(H, R, P, T)
    wo_o = oracle.out_size(H + 1, R, P, T)
    if ho_o < 1 or wo_o < 1:
        with pytest.raises(isc.IscError) as e:
            isc.isc_out_shape(d)
        assert e.value.status == 2
    else:
        assert isc.isc_out_shape(d) == (ho_o, wo_o)


def test_workspace_sizes_ordered():
    d = isc.make_desc(8, 20, 12, 12, 50, 5, 5, 1, 0)
    sp = isc.isc_workspace_size(d, "sparse")
    de = isc.isc_workspace_size(d, "dense")
    au = isc.isc_workspace_size(d, "auto")
    assert sp > 0 and de > 0
    assert au >= max(sp, de)
    # the dense path gathers the unrolled matrix inside its GEMM (C*R*S <
    # 2^16): control block only; this shape compacts on the fly (K <= 64, few
    # input maps): control block, per-workgroup counts and the repacked
    # filter (C*R*S x 64 floats) only
    assert de < 4096
    assert 20 * 25 * 64 * 4 <= sp < 20 * 25 * 64 * 4 + 8192
    # more output maps than one pass holds: the filter is streamed, the input
    # still compacted on the fly -- the repacked filter and no lists
    d2 = isc.make_desc(2, 96, 27, 27, 256, 5, 5, 1, 2)
    assert 96 * 25 * 256 * 4 <= isc.isc_workspace_size(d2, "sparse") < 96 * 25 * 256 * 4 + 8192
    # a shape no on-the-fly kernel takes (stride 2): the lists (8 bytes per
    # input element) and the repacked filter
    d3 = isc.make_desc(2, 96, 27, 27, 256, 5, 5, 2, 2)
    assert isc.isc_workspace_size(d3, "sparse") >= 2 * 96 * 27 * 27 * 8 + 96 * 25 * 256 * 4
    # C*R*S >= 2^16: the dense path materialises C*R*S rows of >= N*Ho*Wo floats
    big = isc.make_desc(1, 2700, 6, 6, 8, 5, 5, 1, 0)
    assert isc.isc_workspace_size(big, "dense") >= 2700 * 25 * 2 * 2 * 4


def _conv(desc, x=0x1000, w=0x200000, y=0x400000, ws=0x800000, ws_bytes=1 << 30, path=0,
          th=0.9):
    return isc.lib().isc_conv2d(ctypes.byref(desc) if desc is not None else None, x, w, y, ws,
                                ws_bytes, path, ctypes.c_float(th), None)


def test_conv2d_validation_errors():
    good = isc.make_desc(2, 3, 8, 8, 4, 3, 3, 1, 1)
    assert _conv(None) == 1                                    # NULL desc
    assert _conv(good, x=0) == 1                               # NULL input
    assert _conv(isc.make_desc(0, 3, 8, 8, 4, 3, 3, 1, 1)) == 2
    assert _conv(isc.make_desc(2, 3, 8, 8, 4, 3, 3, 0, 1)) == 2  # stride 0
    assert _conv(isc.make_desc(2, 3, 8, 8, 4, 3, 3, 1, -1)) == 2
    assert _conv(isc.make_desc(2, 3, 2, 2, 4, 5, 5, 1, 0)) == 2  # filter larger than input
    assert _conv(isc.make_desc(1, 1, 70000, 1, 1, 1, 1, 1, 0)) == 3   # H > 65535
    assert _conv(isc.make_desc(4096, 512, 64, 64, 1, 1, 1, 1, 0)) == 3  # > 2^31 elements
    assert _conv(good, path=7) == 6
    assert _conv(good, th=1.5) == 10
    assert _conv(good, th=float("nan")) == 10
    assert _conv(good, x=0x1002) == 9                          # misaligned
    assert _conv(good, ws=0x800010) == 9                       # workspace not 256-aligned
    assert _conv(good, ws_bytes=16) == 4
    assert _conv(good, y=0x1000) == 5                          # y overlaps x
    assert _conv(good, y=0x800000) == 5                        # y overlaps the workspace


def test_conv2d_without_device_reports_device():
    # arguments valid, no GPU in this process -> ISC_ERR_DEVICE, nothing launched
    try:
        import torch
        if torch.cuda.is_available():
            pytest.skip("a GPU is present")
    except Exception:
        pass
    good = isc.make_desc(2, 3, 8, 8, 4, 3, 3, 1, 1)
    assert _conv(good) == 7


def test_compact_im2col_gemm_validation():
    L = isc.lib()
    d = isc.make_desc(2, 3, 8, 8, 1, 1, 1, 1, 0)
    assert L.isc_compact(ctypes.byref(d), 0, 0x1000, 0x2000, 0x3000, None) == 1
    assert L.isc_compact(ctypes.byref(d), 0x100000, 0x100000, 0x200000, 0x300000, None) == 5
    assert L.isc_compact(ctypes.byref(d), 0x100000, 0x200000, 0x300004, 0x400000, None) == 9
    assert L.isc_im2col(ctypes.byref(d), 0x100000, 0x200000, 10, None) == 10  # ldc < N*Ho*Wo
    assert L.isc_im2col(ctypes.byref(d), 0x100000, 0x100000, 128, None) == 5
    assert L.isc_gemm_f32(0, 4, 4, 0x1000, 4, 0x2000, 4, 0x3000, 4, None) == 2
    assert L.isc_gemm_f32(4, 4, 4, 0x1000, 3, 0x2000, 4, 0x3000, 4, None) == 2  # lda < Kd
    assert L.isc_gemm_f32(4, 4, 4, 0x1000, 4, 0x2000, 4, 0x1000, 4, None) == 5  # c overlaps a


def test_dispatch_defaults_from_the_binding(monkeypatch):
    """The path and AUTO's threshold default to ISC_PATH / ISC_SPARSE_THRESHOLD,
    read by the binding (the library reads no environment); unset, AUTO runs
    the library's per-shape crossover and the path is AUTO."""
    monkeypatch.delenv("ISC_PATH", raising=False)
    monkeypatch.delenv("ISC_SPARSE_THRESHOLD", raising=False)
    assert isc.default_path() == "auto"
    assert isc.default_threshold() == isc.THRESHOLD_CROSSOVER == -1.0
    assert isc.default_threshold(0.9) == 0.9
    monkeypatch.setenv("ISC_PATH", "dense")
    monkeypatch.setenv("ISC_SPARSE_THRESHOLD", "0.9")
    assert isc.default_path() == "dense" and isc.default_path("sparse") == "sparse"
    assert isc.default_threshold() == 0.9


def test_library_reads_no_environment():
    """No plan of the library depends on an inherited environment: the
    shared object imports no getenv."""
    import subprocess
    out = subprocess.run(["nm", "-D", "--undefined-only", isc.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    imported = {line.split()[-1].split("@")[0] for line in out.splitlines() if line.strip()}
    assert "getenv" not in imported and "secure_getenv" not in imported


def test_crossover_threshold_accepted():
    # a negative threshold asks for the per-shape crossover; NaN is rejected
    good = isc.make_desc(2, 3, 8, 8, 4, 3, 3, 1, 1)
    assert _conv(good, th=-1.0) in (0, 7)                     # valid (no device here: DEVICE)
    assert _conv(good, th=float("nan")) == 10


def test_sparse_kernel_choice():
    """Host-side choice of the sparse kernel for the workload shapes."""
    d = isc.make_desc
    assert isc.isc_sparse_kernel(d(256, 20, 12, 12, 50, 5, 5, 1, 0)) == "fused_reg"  # LeNet conv2
    assert isc.isc_sparse_kernel(d(128, 16, 28, 28, 32, 5, 5, 1, 2)) == "fused"    # inception 5x5
    assert isc.isc_sparse_kernel(d(128, 96, 27, 27, 256, 5, 5, 1, 2)) == "fused_ring"  # AlexNet conv2
    assert isc.isc_sparse_kernel(d(128, 384, 13, 13, 256, 3, 3, 1, 1)) == "fused_reg"  # AlexNet conv5
    assert isc.isc_sparse_kernel(d(128, 384, 5, 5, 384, 3, 3, 1, 1)) == "fused_reg"   # Tab. 2 AlexNet conv4
    assert isc.isc_sparse_kernel(d(1, 832, 7, 7, 256, 1, 1, 1, 0)) == "fused_reg"     # Tab. 2 inception 5a.1
    assert isc.isc_sparse_kernel(d(128, 16, 17, 17, 32, 5, 5, 1, 2)) == "fused"       # 17 columns: filter in LDS
    assert isc.isc_sparse_kernel(d(128, 16, 17, 17, 96, 5, 5, 1, 2)) == "fused_ring"  # 17 columns, K > 64
    assert isc.isc_sparse_kernel(d(128, 96, 28, 28, 128, 3, 3, 1, 1)) == "fused_ring"  # inception 3x3
    assert isc.isc_sparse_kernel(d(1, 3, 20, 200, 66, 3, 3, 1, 1)) == "fused_ring"     # column tiles
    assert isc.isc_sparse_kernel(d(2, 4, 11, 11, 64, 5, 5, 2, 1)) == "fused"       # stride 2, 5 x 5 output
    assert isc.isc_sparse_kernel(d(128, 20, 11, 11, 64, 5, 5, 2, 1)) == "fused"    # LeNet conv2 of Tab. 2
    assert isc.isc_sparse_kernel(d(2, 4, 21, 21, 64, 5, 5, 2, 1)) == "generic"     # stride 2, 10 columns
    assert isc.isc_sparse_kernel(d(2, 4, 11, 11, 65, 5, 5, 2, 1)) == "generic"     # stride 2, K > 64
    assert isc.isc_sparse_kernel(d(1, 3, 10, 9, 9, 2, 3, 1, 1)) == "generic"       # 2 x 3 filter
    assert isc.isc_sparse_kernel(d(1, 3, 9, 9, 9, 7, 7, 1, 3)) == "generic"        # 7 x 7 filter


def test_fused_entry_validation():
    L = isc.lib()
    ok = isc.make_desc(1, 2, 12, 12, 8, 5, 5, 1, 0)
    big_k = isc.make_desc(1, 2, 12, 12, 65, 7, 7, 1, 0)       # 7 x 7 filter: not taken
    strided = isc.make_desc(1, 2, 24, 24, 8, 5, 5, 2, 0)      # stride 2 with 10 output columns: not taken
    x, w, y = 0x1000, 0x200000, 0x400000
    assert L.isc_sparse_conv_fused(None, x, w, y, None, None) == 1
    assert L.isc_sparse_conv_fused(ctypes.byref(ok), None, w, y, None, None) == 1
    assert L.isc_sparse_conv_fused(ctypes.byref(big_k), x, w, y, None, None) == 3
    assert L.isc_sparse_conv_fused(ctypes.byref(strided), x, w, y, None, None) == 3
    assert L.isc_sparse_conv_fused(ctypes.byref(ok), x, w, x + 4, None, None) == 5   # y overlaps x
    assert L.isc_sparse_conv_fused(ctypes.byref(ok), x + 2, w, y, None, None) == 9   # misaligned
    bad = isc.Tuning(reserved=1)
    assert L.isc_sparse_conv_fused(ctypes.byref(ok), x, w, y, ctypes.byref(bad), None) == 10
    assert L.isc_sparse_conv_fused(ctypes.byref(ok), x, w, y, None, None) == 7       # no gfx950 here


def test_census_size():
    # room for the workgroups of every kernel that may write the output: at
    # least the GEMM's ceil(K/32) * ceil(N*Ho*Wo/64) and the 1024 of the
    # stand-alone epilogue pass, after a 16-byte header; multiple of 16 bytes
    d = isc.make_desc(128, 256, 13, 13, 384, 3, 3, 1, 1)
    n = isc.isc_census_size(d)
    assert n % 16 == 0
    assert n >= 16 + 4 * (384 // 32) * ((128 * 169 + 63) // 64)
    small = isc.isc_census_size(isc.make_desc(1, 1, 3, 3, 1, 3, 3, 1, 0))
    assert small >= 16 + 4 * 1024
    with pytest.raises(isc.IscError) as e:
        isc.isc_census_size(isc.make_desc(0, 1, 3, 3, 1, 3, 3, 1, 0))
    assert e.value.status == 2


def _relu(desc, x=0x1000, xc=None, xcb=0, w=0x200000, wt=None, y=0x400000, yc=None, ycb=0,
          ws=0x800000, ws_bytes=1 << 30, path=0, th=0.9):
    return isc.lib().isc_conv2d_relu(ctypes.byref(desc), x, xc, xcb, w, wt, y, yc, ycb, ws, ws_bytes,
                                     path, ctypes.c_float(th), None, None)


def test_conv2d_relu_validation():
    good = isc.make_desc(2, 3, 8, 8, 4, 3, 3, 1, 1)
    cb = isc.isc_census_size(good)
    yc = 0x10000000
    assert _relu(good, x=0) == 1
    assert _relu(good, yc=yc, ycb=cb - 16) == 4                  # census too small
    assert _relu(good, yc=yc + 8, ycb=cb) == 9                   # census misaligned
    assert _relu(good, xc=0x20000008, xcb=4096) == 9             # input census misaligned
    assert _relu(good, xc=0x20000000, xcb=8) == 4                # input census below its header
    assert _relu(good, wt=0x30000004) == 9                       # repacked filter misaligned
    assert _relu(good, yc=0x400000, ycb=cb) == 5                 # census overlaps y
    assert _relu(good, yc=0x1000, ycb=cb) == 5                   # census overlaps x
    assert _relu(good, yc=yc, ycb=cb, xc=yc, xcb=cb) == 5        # input and output census overlap
    assert _relu(good, wt=0x400000) == 5                         # wt overlaps y
    assert _relu(good, y=0x1000) == 5
    assert _relu(good, path=9) == 6
    try:
        import torch
        if torch.cuda.is_available():
            return
    except Exception:
        pass
    assert _relu(good, yc=yc, ycb=cb, xc=0x20000000, xcb=cb) == 7  # valid; no gfx950 here


def test_census_read_validation():
    L = isc.lib()
    e, n = ctypes.c_uint64(), ctypes.c_uint64()
    assert L.isc_census_read(None, 4096, ctypes.byref(e), ctypes.byref(n), None) == 1
    assert L.isc_census_read(0x1000, 8, ctypes.byref(e), ctypes.byref(n), None) == 4


def test_dw_entry_validation():
    L = isc.lib()
    d = isc.make_desc(2, 3, 9, 9, 8, 3, 3, 1, 1)
    n = isc.isc_conv2d_dw_workspace_size(d)
    assert n > 0 and n % 256 == 0
    with pytest.raises(isc.IscError) as e:                      # stride 2: not taken
        isc.isc_conv2d_dw_workspace_size(isc.make_desc(2, 3, 9, 9, 8, 3, 3, 2, 1))
    assert e.value.status == 3
    with pytest.raises(isc.IscError) as e:                      # 7x7 filter: not taken
        isc.isc_conv2d_dw_workspace_size(isc.make_desc(2, 3, 9, 9, 8, 7, 7, 1, 3))
    assert e.value.status == 3
    x, dy, dw, ws = 0x1000, 0x100000, 0x200000, 0x300000
    assert L.isc_conv2d_dw(ctypes.byref(d), None, dy, dw, ws, n, None, None) == 1
    assert L.isc_conv2d_dw(ctypes.byref(d), x, dy, dw, ws, n - 1, None, None) == 4    # workspace too small
    assert L.isc_conv2d_dw(ctypes.byref(d), x, dy, x, ws, n, None, None) == 5        # dw overlaps x
    assert L.isc_conv2d_dw(ctypes.byref(d), x, dy, dw, ws + 16, n, None, None) == 9  # workspace misaligned
    try:
        import torch
        if torch.cuda.is_available():
            return
    except Exception:
        pass
    assert L.isc_conv2d_dw(ctypes.byref(d), x, dy, dw, ws, n, None, None) == 7       # no gfx950 here


def test_dense_split_workspace():
    """Host plan of the dense GEMM's split reduction: a grid under 128 tiles
    splits C*R*S into ranges of at least 256 (multiples of 32, at most 16)
    and the workspace holds ranges x K x N*Ho*Wo partial sums; short
    reductions do not split; larger grids split only where that evens out
    the CUs' shares enough."""
    d = isc.make_desc(1, 384, 5, 5, 384, 3, 3, 1, 1)     # 3 tiles, C*R*S 3456
    lenet = isc.make_desc(256, 20, 12, 12, 50, 5, 5, 1, 0)  # 256 tiles of 64 x 64: no split
    base = isc.isc_workspace_size(lenet, "dense")          # the control block alone
    split = isc.isc_workspace_size(d, "dense")
    # min(16, ceil(256 / 3), 3456 // 256) = 13 ranges asked -> ranges of 288 -> 12 ranges
    assert split - base == 12 * 384 * 25 * 4
    short = isc.make_desc(3, 500, 4, 4, 33, 1, 1, 1, 0)   # C*R*S 500 < 2 * 256
    assert isc.isc_workspace_size(short, "dense") == base
    # grids of 128 x 128 tiles split where the GEMM's model gains 10 %: AlexNet
    # conv5 at batch 128 (338 tiles, two on 82 CUs) in three ranges of 1152;
    # conv3 (507 tiles, two on almost every CU) and the inception 3x3 branch
    # (784 tiles, a modelled 5 %) not at all
    conv5 = isc.make_desc(128, 384, 13, 13, 256, 3, 3, 1, 1)
    assert isc.isc_workspace_size(conv5, "dense") - base == 3 * 256 * 128 * 169 * 4
    conv3 = isc.make_desc(128, 256, 13, 13, 384, 3, 3, 1, 1)
    inc3 = isc.make_desc(128, 96, 28, 28, 128, 3, 3, 1, 1)
    assert isc.isc_workspace_size(conv3, "dense") == base
    assert isc.isc_workspace_size(inc3, "dense") == base


def test_sparse_plan_and_overrides():
    """The plan query reports the kernel and launch shape, and a per-call
    tuning forces what the shape can take and is ignored otherwise."""
    d = isc.make_desc
    lenet = d(256, 20, 12, 12, 50, 5, 5, 1, 0)
    p = isc.isc_sparse_plan(lenet)
    assert p["kernel"] == "fused_reg" and p["phases"] == 8 and p["waves"] == 8
    assert (p["rows"], p["cols"]) == (4, 8) and p["workgroups"] == 256 * 2
    # the filter in LDS instead of the register-weight kernel
    q = isc.isc_sparse_plan(lenet, {"kernel": "fused"})
    assert q["kernel"] == "fused" and q["rows"] * q["cols"] <= 64
    # the register-weight kernel's two tile heights
    assert isc.isc_sparse_plan(lenet, {"rows": 2})["rows"] == 2
    conv2 = d(128, 96, 27, 27, 256, 5, 5, 1, 2)
    r = isc.isc_sparse_plan(conv2, {"kernel": "fused_ring", "maps_per_lane": 2, "rows": 1})
    assert (r["kernel"], r["maps_per_lane"], r["rows"]) == ("fused_ring", 2, 1)
    assert r["workgroups"] == 128 * 27 // 4 * 2      # 1 x 28 tiles, four to a workgroup, two map groups
    # five maps per lane: no such tile, the library's own choice runs
    assert isc.isc_sparse_plan(conv2, {"kernel": "fused_ring", "maps_per_lane": 5}) == isc.isc_sparse_plan(conv2)
    assert isc.isc_sparse_plan(d(2, 4, 21, 21, 64, 5, 5, 2, 1))["kernel"] == "generic"
    with pytest.raises(isc.IscError) as e:
        isc.isc_sparse_plan(lenet, isc.Tuning(reserved=3))
    assert e.value.status == 10


def test_read_decision_validation():
    L = isc.lib()
    p, n = ctypes.c_int32(), ctypes.c_uint64()
    assert L.isc_read_decision(None, ctypes.byref(p), ctypes.byref(n)) == 1
    assert L.isc_read_decision(0x1000, None, ctypes.byref(n)) == 1


def test_crossover_model_orders_shapes():
    """AUTO's per-shape crossover (host model): the 5x5 layers cross far
    below the paper's 0.9, AlexNet conv3 between 0.3 and 0.85; of Tab. 2's
    1x1 layers at batch 128, inception 4a.1 (14 x 14) goes sparse only past
    0.98 if ever, inception 5a.1 (7 x 7, 832 channels) between 0.85 and 0.97;
    the crossover is a sparsity in [0, 1] or 2.0 (never)."""
    d = isc.make_desc
    lenet = isc.isc_crossover_sparsity(d(256, 20, 12, 12, 50, 5, 5, 1, 0))
    conv2 = isc.isc_crossover_sparsity(d(128, 96, 27, 27, 256, 5, 5, 1, 2))
    conv3 = isc.isc_crossover_sparsity(d(128, 256, 13, 13, 384, 3, 3, 1, 1))
    one = isc.isc_crossover_sparsity(d(128, 480, 14, 14, 192, 1, 1, 1, 0))
    five = isc.isc_crossover_sparsity(d(128, 832, 7, 7, 256, 1, 1, 1, 0))
    assert 0.0 <= lenet < 0.5 and 0.3 < conv2 < 0.7 and 0.3 < conv3 < 0.85
    assert one > 0.98 and 0.85 < five < 0.97
    for s in (lenet, conv2, conv3):
        assert 0.0 <= s <= 1.0
    # a shape only the list kernels take keeps the paper's 0.9
    assert abs(isc.isc_crossover_sparsity(d(2, 4, 21, 21, 64, 5, 5, 2, 1)) - 0.9) < 1e-3
