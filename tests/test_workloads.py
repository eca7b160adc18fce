"""Seeded synthetic inputs: determinism and the structural facts each
generator promises.  CPU only."""
import numpy as np
import torch

import workloads


def test_er_graph_exact_counts_and_determinism():
    rp1, c1 = workloads.er_graph(2000, 10_000, seed=0)
    rp2, c2 = workloads.er_graph(2000, 10_000, seed=0)
    assert torch.equal(rp1, rp2) and torch.equal(c1, c2)
    assert int(rp1[-1]) == 20_000 == c1.numel()
    rows = torch.repeat_interleave(torch.arange(2000), rp1[1:] - rp1[:-1])
    assert not bool((rows == c1).any())                      # no self loops
    key = rows * 2000 + c1
    assert torch.unique(key).numel() == key.numel()          # no duplicate pairs
    # symmetric
    rkey = c1 * 2000 + rows
    assert torch.equal(torch.sort(key).values, torch.sort(rkey).values)
    # rows sorted ascending
    for v in range(0, 2000, 97):
        seg = c1[rp1[v]:rp1[v + 1]]
        assert bool((seg[1:] >= seg[:-1]).all())
    rp3, _ = workloads.er_graph(2000, 10_000, seed=1)
    assert not torch.equal(rp1, rp3)


def test_rmat_graph_structure():
    n, m = 5000, 40_000
    rp, col = workloads.rmat_graph(n, m, seed=0)
    assert int(rp[-1]) == 2 * m and int(col.min()) >= 0 and int(col.max()) < n
    rows = torch.repeat_interleave(torch.arange(n), rp[1:] - rp[:-1])
    assert not bool((rows == col).any())
    st = workloads.graph_stats(rp, col)
    assert st["max_degree"] > 10 * st["mean_degree"]          # skewed degrees
    rp2, col2 = workloads.rmat_graph(n, m, seed=0)
    assert torch.equal(rp, rp2) and torch.equal(col, col2)
    rpd, cold = workloads.rmat_graph(n, m, seed=0, directed=True)
    assert int(rpd[-1]) == m


def test_features_labels_targets_weights():
    x = workloads.features(100, 7, seed=0)
    assert x.dtype == torch.float32 and torch.equal(x, workloads.features(100, 7, seed=0))
    assert abs(float(x.mean())) < 0.2 and abs(float(x.std()) - 1) < 0.2
    h = workloads.features(100, 7, seed=0, dtype=torch.float16)
    assert h.dtype == torch.float16 and torch.equal(h, x.half())
    y = workloads.labels(1000, 47)
    assert int(y.min()) >= 0 and int(y.max()) < 47
    perm = workloads.target_batches(1000, 64)
    assert torch.equal(torch.sort(perm).values, torch.arange(1000))
    t0 = workloads.targets_for_step(perm, 64, 0)
    t1 = workloads.targets_for_step(perm, 64, 1)
    assert t0.numel() == 64 and len(set(t0.tolist()) & set(t1.tolist())) == 0
    w = workloads.glorot(200, 256, 0, 0)
    assert w.shape == (200, 256) and float(w.abs().max()) <= np.sqrt(6 / 456) + 1e-6
