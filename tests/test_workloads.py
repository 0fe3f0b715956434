"""Statistics of the seeded synthetic inputs (they stand in for the paper's
ReLU outputs on MNIST / CIFAR-10 / ImageNet, which are not available)."""
import json
import os

import numpy as np
import pytest

import workloads


def test_paper_table_transcription_consistent():
    # Tab. 3's speedup column equals GEMM / ISC to the printed precision
    tab = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_tables.json")))
    assert len(tab["table2_layers"]) == len(tab["table3_cpu_ms"]) == 10
    for row in tab["table3_cpu_ms"]:
        assert abs(row["gemm_ms"] / row["isc_ms"] - row["speedup"]) < 0.03, row
        assert row["sparsity"] >= 0.9   # the paper times only layers at >= 0.9


def test_iid_sparsity_and_values():
    layer = workloads.small_case(4, 8, 12, 12, 6, 3, 3, 1, 1, 0.9, seed=1)
    x, w = workloads.make_inputs(layer, seed=1)
    assert x.dtype == np.float32 and w.dtype == np.float32
    s = np.mean(x == 0)
    assert abs(s - 0.9) < 0.02
    assert np.all(x >= 0)
    assert abs(np.std(w) - 0.1) < 0.02


def test_seeded_reproducible():
    layer = workloads.WORKLOADS["lenet_conv2_tiny"].layers[0]
    x1, w1 = workloads.make_inputs(layer)
    x2, w2 = workloads.make_inputs(layer)
    assert np.array_equal(x1, x2) and np.array_equal(w1, w2)
    assert layer.seed == workloads.BASE_SEED + 1000


def test_clustered_exact_zero_count():
    layer = workloads.small_case(3, 5, 16, 16, 2, 3, 3, 1, 1, 0.9, seed=3, clustered=True)
    x, _ = workloads.make_inputs(layer, seed=3)
    assert int(np.sum(x == 0)) == int(np.ceil(0.9 * x.size))
    # zeros cluster: a zero's 4-neighbours are zero more often than chance
    z = x == 0
    same = np.mean(z[:, :, 1:, :] & z[:, :, :-1, :]) / np.mean(z[:, :, 1:, :])
    assert same > 0.92


def test_workload_shapes():
    names = set(workloads.WORKLOADS)
    assert names == {"lenet_conv2_tiny", "lenet_conv2_batch", "alexnet_conv2",
                     "alexnet_conv345", "inception_28", "alexnet_chain345", "paper_tab2", "paper_tab2_n1"}
    sweep = workloads.WORKLOADS["lenet_conv2_batch"].layers
    assert [l.sparsity for l in sweep] == [0.5, 0.7, 0.9, 0.95, 0.99]
    assert len({l.seed for l in sweep}) == 5


def test_integer_case_bounds():
    x, w = workloads.integer_case(2, 3, 5, 5, 2, 3, 3, seed=4)
    assert set(np.unique(x)).issubset(set(range(0, 8)))
    assert set(np.unique(w)).issubset(set(range(-4, 5)))


def test_chain_weights_and_input():
    chain = workloads.WORKLOADS["alexnet_chain345"]
    x0, ws = workloads.make_chain(chain, N=2)
    assert x0.shape == (2, 256, 13, 13)
    assert [w.shape for w in ws] == [l.w_shape for l in chain.layers]
    # each layer's input channels are the previous layer's output maps
    for a, b in zip(chain.layers, chain.layers[1:]):
        assert b.C == a.K and (b.H, b.W) == (a.H, a.W)
    for w, l in zip(ws, chain.layers):
        assert abs(float(w.mean()) - l.w_mean) < 0.1 * l.sigma
        assert abs(float(w.std()) - l.sigma) < 0.05 * l.sigma
    assert abs((x0 == 0).mean() - 0.95) < 0.01
    # weights drawn again from the same seeds are the same
    _, ws2 = workloads.make_chain(chain, N=1)
    assert all(np.array_equal(a, b) for a, b in zip(ws, ws2))


def test_tab2_layers():
    """The ten layers of the paper's Tab. 2 (C, H_in, K, R x S, P, T,
    sparsity as printed), at batch 128 and batch 1, each with its own seed."""
    for name, n in (("paper_tab2", 128), ("paper_tab2_n1", 1)):
        layers = workloads.WORKLOADS[name].layers
        assert len(layers) == 10 and all(l.N == n for l in layers)
        assert len({l.seed for l in layers}) == 10
        first = layers[0]
        assert (first.C, first.H, first.W, first.K, first.R, first.S, first.P, first.T, first.sparsity) == \
            (20, 11, 11, 64, 5, 5, 1, 2, 0.95)
        last = layers[-1]
        assert (last.C, last.H, last.K, last.R, last.P, last.T, last.sparsity) == (48, 7, 128, 5, 2, 1, 0.95)
        assert sorted({l.sparsity for l in layers}) == [0.9, 0.95]
    x, _ = workloads.make_inputs(workloads.WORKLOADS["paper_tab2_n1"].layers[6])
    assert x.shape == (1, 832, 7, 7) and abs((x == 0).mean() - 0.95) < 0.01
