"""The allocation-free entry point (isc_conv2d_noalloc) through the C ABI:
its output against isc_conv2d's with a caller's workspace (the same kernels,
so bit for bit) and against the oracle, on two calls in a row, the second
with a smaller input, on every path."""
import sys

import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu

TOL = 1e-4


def note(*parts):
    print("[case]", *parts, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("path", ["auto", "sparse", "dense"])
def test_noalloc_matches_workspace_entry(path):
    import torch
    import paper_1704_07724_amd as isc
    assert torch.cuda.is_available()
    isc.lib()
    cases = [(4, 12, 27, 27, 100, 5, 5, 1, 2, 0.9), (2, 5, 12, 12, 50, 5, 5, 1, 0, 0.9)]  # second smaller
    for case in cases:
        N, C, H, W, K, R, S, T, P, sp = case
        note("noalloc", path, case)
        x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=501 + sum(case[:9]))
        xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
        desc = isc.make_desc(N, C, H, W, K, R, S, T, P)
        assert isc.isc_workspace_size(desc, path) <= isc.NOALLOC_SCRATCH_BYTES
        ref = isc.isc_conv2d(xd, wd, T, P, path=path, threshold=0.9, ws=isc.workspace(desc, path))
        out = torch.full_like(ref, float("nan"))
        isc.isc_conv2d_noalloc(xd, wd, out, T, P, path=path, threshold=0.9)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), "noalloc differs from the workspace entry point"
        want = oracle.conv2d_f64(x, w, T, P)
        got = out.cpu().numpy().astype(np.float64)
        assert np.all(np.abs(got - want) <= TOL * (1.0 + np.abs(want)))


def test_noalloc_rejects_workspace_beyond_scratch():
    import torch
    import paper_1704_07724_amd as isc
    assert torch.cuda.is_available()
    note("noalloc limit")
    # stride 2: compacted lists of 8 bytes per input element, 2^21 elements
    desc = isc.make_desc(2, 64, 128, 128, 8, 3, 3, 2, 1)
    assert isc.isc_workspace_size(desc, "sparse") > isc.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((2, 64, 128, 128), device="cuda")
    w = torch.zeros((8, 64, 3, 3), device="cuda")
    out = torch.empty((2, 8, 64, 64), device="cuda")
    with pytest.raises(isc.IscError) as e:
        isc.isc_conv2d_noalloc(x, w, out, 2, 1, path="sparse")
    assert e.value.status == 3


def test_noalloc_runs_the_gemm_unsplit_when_its_partial_sums_do_not_fit():
    """AlexNet conv5 at batch 128 on the dense path: the GEMM's split
    reduction wants 66 MB of partial sums, more than the scratch buffer, so
    the allocation-free entry point runs the GEMM unsplit -- bit for bit the
    output of isc_conv2d with tuning gemm_split = -1 -- and matches the
    oracle."""
    import torch
    import paper_1704_07724_amd as isc
    assert torch.cuda.is_available()
    isc.lib()
    case = (128, 384, 13, 13, 256, 3, 3, 1, 1, 0.5)
    N, C, H, W, K, R, S, T, P, sp = case
    note("noalloc unsplit", case)
    desc = isc.make_desc(N, C, H, W, K, R, S, T, P)
    assert isc.isc_workspace_size(desc, "dense") > isc.NOALLOC_SCRATCH_BYTES
    x, w = workloads.make_case(N, C, H, W, K, R, S, T, P, sp, seed=777)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    ref = isc.isc_conv2d(xd, wd, T, P, path="dense", ws=isc.workspace(desc, "dense"), tuning={"gemm_split": -1})
    out = torch.full_like(ref, float("nan"))
    isc.isc_conv2d_noalloc(xd, wd, out, T, P, path="dense")
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    want = oracle.conv2d_f64(x, w, T, P)
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - want) <= TOL * (1.0 + np.abs(want)))
