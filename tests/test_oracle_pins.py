"""Pins for the CPU oracle against facts fixed outside it: published test
vectors, library routines, dense brute force, closed forms, invariants,
sampling statistics and finite differences.  CPU only."""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from tests import dense

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


# ---------------------------------------------------------------------------
# random-number draws and conversions
# ---------------------------------------------------------------------------

def test_splitmix64_published_outputs():
    state = 0
    for idx, hexval in _golden_rows("splitmix64_seed0.txt"):
        state = (state + 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF
        assert oracle.mix64(state) == int(hexval, 16), idx


def test_sample_key_is_nested_mix():
    # key = mix(mix(mix(mix(mix(seed)^step)^hop)^v)^t) written out with Python ints
    M = (1 << 64) - 1

    def mix(z):
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
        return z ^ (z >> 31)

    for seed, step, hop, v, t in [(0, 0, 1, 0, 0), (7, 3, 2, 123456789, 24), (2**63 + 5, 2**40, 3, 2**33, 1023)]:
        want = mix(mix(mix(mix(mix(seed) ^ step) ^ hop) ^ v) ^ t)
        assert oracle.sample_key(seed, step, hop, v, t) == want


def test_bounded_range_and_extremes():
    assert oracle.bounded(0, 10) == 0
    assert oracle.bounded((1 << 64) - 1, 10) == 9
    assert oracle.bounded(1 << 63, 10) == 5
    rng = np.random.default_rng(1)
    for key in rng.integers(0, 2**63, size=200, dtype=np.int64).tolist():
        for b in (1, 2, 7, 1000, 2**32):
            x = oracle.bounded(int(key) * 2 + 1, b)
            assert 0 <= x < b


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),        # subnormals
        np.array([0.0, -0.0, np.inf, -np.inf, 3.4e38, -3.4e38], dtype=np.float32),
        # exact ties: lower 16 bits == 0x8000 with even and odd upper halves
        np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x00008000], dtype=np.uint32).view(np.float32),
    ])
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([oracle.lib().orc_f32_to_bf16(float(v)) for v in x], dtype=np.uint16)
    assert np.array_equal(got, want)
    assert np.array_equal(oracle.f32_to_bf16_bits(x), want)
    nan_bits = np.array([0x7FC00001, 0x7F800001, 0xFFC12345], dtype=np.uint32).view(np.float32)
    for v in nan_bits:
        b = oracle.lib().orc_f32_to_bf16(float(v))
        assert math.isnan(oracle.lib().orc_bf16_to_f32(b))


def test_fp16_widening_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want = bits.view(np.float16).astype(np.float32)
    got = np.array([oracle.lib().orc_f16_to_f32(int(b)) for b in bits], dtype=np.float32)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), want[~nan].view(np.uint32))


# ---------------------------------------------------------------------------
# sampler
# ---------------------------------------------------------------------------

def test_sampler_takes_whole_row_when_short():
    for d in range(0, 12):
        for k in (1, 5, 11, 25):
            if d <= k:
                assert oracle.sample_positions(d, k, 0, 0, 1, 17).tolist() == list(range(d))


def test_sampler_invariants():
    for v in range(300):
        d = 5 + v % 200
        k = 1 + v % 30
        p = oracle.sample_positions(d, k, 3, 1, 2, v)
        if d <= k:
            continue
        assert p.size == k
        assert np.all(np.diff(p) > 0)
        assert p[0] >= 0 and p[-1] < d


def test_floyd_subsets_equiprobable_chi2():
    from scipy.stats import chi2
    d, k, trials = 6, 3, 100_000
    counts = {}
    incl = np.zeros(d)
    for v in range(trials):
        p = tuple(oracle.sample_positions(d, k, 0, 0, 1, v).tolist())
        counts[p] = counts.get(p, 0) + 1
        incl[list(p)] += 1
    assert len(counts) == math.comb(d, k) == 20
    exp = trials / 20
    stat = sum((c - exp) ** 2 / exp for c in counts.values())
    assert stat < chi2.ppf(0.999, 19), stat
    # per-position inclusion probability k/d
    assert np.allclose(incl / trials, k / d, atol=0.01)


def test_floyd_large_row_inclusion_uniform():
    d, k, trials = 1000, 25, 8000
    incl = np.zeros(d)
    for v in range(trials):
        incl[oracle.sample_positions(d, k, 5, 2, 1, v)] += 1
    # each position has inclusion probability k/d; check buckets of 100
    buckets = incl.reshape(10, 100).sum(1) / (trials * k / 10)
    assert np.all(np.abs(buckets - 1.0) < 0.05), buckets


def _brute_block(rowptr, col, dst, fanout, seed, step, hop):
    """Relabel with Python sets and sorted(), from the sampled positions."""
    lists = []
    for v in dst:
        d = int(rowptr[v + 1] - rowptr[v])
        pos = oracle.sample_positions(d, fanout, seed, step, hop, int(v))
        lists.append([int(col[rowptr[v] + p]) for p in pos])
    dset = set(int(v) for v in dst)
    new = sorted(set(u for l in lists for u in l) - dset)
    src = [int(v) for v in dst] + new
    index = {u: i for i, u in enumerate(src)}
    brow = [0]
    bcol = []
    for l in lists:
        bcol.extend(index[u] for u in l)
        brow.append(len(bcol))
    # transpose by scanning sources then rows (independent of the oracle's counting method)
    cscptr = [0]
    cscrow = []
    for j in range(len(src)):
        for i in range(len(dst)):
            for e in range(brow[i], brow[i + 1]):
                if bcol[e] == j:
                    cscrow.append(i)
        cscptr.append(len(cscrow))
    return src, brow, bcol, cscptr, cscrow


@pytest.mark.parametrize("seed", range(6))
def test_block_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(8, 64))
    rowptr, col = dense.small_multigraph(rng, n, avg_deg=4, hubs=1, isolated=2, multi=True)
    n_dst = int(rng.integers(1, n))
    dst = rng.choice(n, size=n_dst, replace=False).astype(np.int64)
    for fanout in (1, 3, 25):
        blk = oracle.build_block(rowptr, col, dst, fanout, seed, 4, 2)
        src, brow, bcol, cscptr, cscrow = _brute_block(rowptr, col, dst, fanout, seed, 4, 2)
        assert blk.src_ids.tolist() == src
        assert blk.rowptr.tolist() == brow
        assert blk.col.tolist() == bcol
        assert blk.cscptr.tolist() == cscptr
        assert blk.cscrow.tolist() == cscrow
        # invariants
        assert blk.src_ids[:n_dst].tolist() == dst.tolist()
        assert len(set(blk.src_ids.tolist())) == blk.n_src
        assert blk.n_src <= n_dst + blk.nnz
        assert np.all(blk.col < blk.n_src)


def test_block_relabel_matches_vectorised_numpy():
    rng = np.random.default_rng(11)
    n = 400
    rowptr, col = dense.small_multigraph(rng, n, avg_deg=9, hubs=3, isolated=5)
    dst = rng.choice(n, size=60, replace=False).astype(np.int64)
    blk = oracle.build_block(rowptr, col, dst, 7, 9, 1, 1)
    g = blk.src_ids[blk.col]  # global id of each sampled edge
    new = np.setdiff1d(np.unique(g), dst)
    assert np.array_equal(blk.src_ids[len(dst):], new)
    # stable transpose via numpy's stable argsort
    order = np.argsort(blk.col, kind="stable")
    rows = np.repeat(np.arange(len(dst)), np.diff(blk.rowptr))
    assert np.array_equal(blk.cscrow, rows[order])
    assert np.array_equal(blk.cscptr, np.concatenate([[0], np.cumsum(np.bincount(blk.col, minlength=blk.n_src))]))


def test_block_out_of_range_and_capacity_errors():
    rowptr = np.array([0, 2, 3, 3], dtype=np.int64)
    col = np.array([1, 2, 0], dtype=np.int64)
    with pytest.raises(ValueError):
        oracle.build_block(rowptr, col, np.array([5], dtype=np.int64), 2, 0, 0, 1)


def test_gcn_norm_closed_form():
    rowptr = np.array([0, 0, 1, 4, 12], dtype=np.int64)
    got = oracle.gcn_norm(rowptr)
    want = np.array([1.0, 1 / math.sqrt(2), 0.5, 1 / 3], dtype=np.float32)
    assert np.array_equal(got, want)


# ---------------------------------------------------------------------------
# gather
# ---------------------------------------------------------------------------

def test_gather_is_fancy_indexing_bitwise():
    rng = np.random.default_rng(2)
    table = rng.standard_normal((50, 13)).astype(np.float32)
    table.view(np.uint32)[3, 4] = 0x7FC0BEEF  # NaN with payload
    table.view(np.uint32)[7, 0] = 0xFF80DEAD
    ids = rng.integers(0, 50, size=200).astype(np.int64)
    got = oracle.gather(table, ids, oracle.F32)
    assert np.array_equal(got.view(np.uint32), table[ids].view(np.uint32))
    got16 = oracle.gather(table, ids, oracle.BF16)
    want16 = torch.from_numpy(table[ids]).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    ok = ~np.isnan(table[ids])
    assert np.array_equal(got16[ok], want16[ok])
    h = rng.standard_normal((30, 9)).astype(np.float16)
    ids2 = rng.integers(0, 30, size=40).astype(np.int64)
    assert np.array_equal(oracle.gather(h, ids2, oracle.F32), h[ids2].astype(np.float32))
    want_b = torch.from_numpy(h[ids2].astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.gather(h, ids2, oracle.BF16), want_b)


# ---------------------------------------------------------------------------
# aggregation
# ---------------------------------------------------------------------------

def _random_block(seed, n=80, n_dst=20, fanout=5):
    rng = np.random.default_rng(seed)
    rowptr, col = dense.small_multigraph(rng, n, avg_deg=6, hubs=2, isolated=3)
    dst = rng.choice(n, size=n_dst, replace=False).astype(np.int64)
    blk = oracle.build_block(rowptr, col, dst, fanout, seed, 0, 1)
    nrm = oracle.gcn_norm(rowptr)
    return rng, rowptr, col, blk, nrm[blk.src_ids]


@pytest.mark.parametrize("seed", range(4))
def test_aggregate_fwd_dense_brute_force(seed):
    rng, _, _, blk, sn = _random_block(seed)
    h = rng.standard_normal((blk.n_src, 7))
    got_s = oracle.aggregate_fwd(oracle.SAGE, blk, None, h, oracle.F64)
    np.testing.assert_allclose(got_s, dense.sage_mean_matrix(blk) @ h, rtol=1e-13, atol=1e-13)
    got_g = oracle.aggregate_fwd(oracle.GCN, blk, sn, h, oracle.F64)
    np.testing.assert_allclose(got_g, dense.gcn_matrix(blk, sn) @ h, rtol=1e-13, atol=1e-13)


def test_aggregate_fwd_invariants():
    rng, rowptr, _, blk, sn = _random_block(7, n_dst=30)
    deg = np.diff(blk.rowptr)
    h = np.full((blk.n_src, 5), 2.5)
    got = oracle.aggregate_fwd(oracle.SAGE, blk, None, h, oracle.F64)
    assert np.allclose(got[deg > 0], 2.5) and np.all(got[deg == 0] == 0)
    # linearity
    h1, h2 = rng.standard_normal((2, blk.n_src, 4))
    for kind, s in ((oracle.SAGE, None), (oracle.GCN, sn)):
        a = oracle.aggregate_fwd(kind, blk, s, 2 * h1 - 3 * h2, oracle.F64)
        b = 2 * oracle.aggregate_fwd(kind, blk, s, h1, oracle.F64) - 3 * oracle.aggregate_fwd(kind, blk, s, h2, oracle.F64)
        np.testing.assert_allclose(a, b, atol=1e-12)
    # GCN on ones: nrm_i (nrm_i + sum_e nrm_col)
    ones = np.ones((blk.n_src, 1))
    got = oracle.aggregate_fwd(oracle.GCN, blk, sn, ones, oracle.F64)[:, 0]
    want = [float(np.float32(sn[i] * sn[i])) + sum(float(np.float32(sn[i] * sn[blk.col[e]]))
                                                   for e in range(blk.rowptr[i], blk.rowptr[i + 1]))
            for i in range(blk.n_dst)]
    np.testing.assert_allclose(got, np.array(want, dtype=np.float64), rtol=1e-12)
    # GCN on a row with no sampled neighbour: self term only (isolated dst)
    iso = np.where(deg == 0)[0]
    for i in iso:
        assert got[i] == float(np.float32(sn[i] * sn[i]))


@pytest.mark.parametrize("seed,n_dst", [(0, 30), (1, 30), (2, 30), (3, 80)])
def test_aggregate_fwd_max_is_numpy_max_with_first_argmax(seed, n_dst):
    # small integers force ties; the multigraph repeats edges.  The maximum
    # is numpy's, the argmax the source of numpy's first maximal position
    # in the row's edge order; rows without neighbours (the isolated
    # vertices, all destinations when n_dst = 80) give 0 and -1.
    rng, _, _, blk, _ = _random_block(seed + 40, n_dst=n_dst)
    f = 5
    h = rng.integers(-3, 4, size=(blk.n_src, f)).astype(np.float64)
    out, arg = oracle.aggregate_fwd_max(blk, h, oracle.F64)
    deg = np.diff(blk.rowptr)
    assert (deg > 1).any() and (n_dst < 80 or (deg == 0).any())
    for i in range(blk.n_dst):
        cols = blk.col[blk.rowptr[i]:blk.rowptr[i + 1]]
        if cols.size == 0:
            assert np.all(out[i] == 0) and np.all(arg[i] == -1)
            continue
        np.testing.assert_array_equal(out[i], h[cols].max(axis=0))
        np.testing.assert_array_equal(arg[i], cols[np.argmax(h[cols], axis=0)])
    # bf16 storage: the maximum of the stored values, bit for bit
    hb = oracle.f32_to_bf16_bits(rng.standard_normal((blk.n_src, f)).astype(np.float32))
    outb, argb = oracle.aggregate_fwd_max(blk, hb, oracle.BF16)
    hv = oracle.to_float64(hb)
    for i in np.nonzero(deg)[0]:
        cols = blk.col[blk.rowptr[i]:blk.rowptr[i + 1]]
        best = cols[np.argmax(hv[cols], axis=0)]
        np.testing.assert_array_equal(argb[i], best)
        np.testing.assert_array_equal(outb[i], hb[best, np.arange(f)])


@pytest.mark.parametrize("seed", range(3))
def test_aggregate_bwd_max_adjoint_duplicates_and_mask(seed):
    # With the argmax fixed the forward is the linear map H -> [S H || P H]
    # (P selects the winning source of each element), so the backward must
    # be its transpose: <[S H || P H], dA> = <H, dH>.  Distinct values make
    # the selection stable, so a small step along any source element moves
    # the output by exactly dH's value there.
    rng, _, _, blk, _ = _random_block(seed + 50, n_dst=25)
    f = 6
    h = rng.standard_normal((blk.n_src, f))
    da = rng.standard_normal((blk.n_dst, 2 * f))
    mx, arg = oracle.aggregate_fwd_max(blk, h, oracle.F64)
    fwd = np.concatenate([h[:blk.n_dst], mx], axis=1)
    bwd = oracle.aggregate_bwd_max(blk, arg, da, f, None, oracle.F64)
    assert abs(np.sum(fwd * da) - np.sum(h * bwd)) <= 1e-12 * np.sum(np.abs(fwd * da))
    eps = 1e-7
    for _ in range(10):
        j, c = int(rng.integers(blk.n_src)), int(rng.integers(f))
        h2 = h.copy()
        h2[j, c] += eps
        mx2, _ = oracle.aggregate_fwd_max(blk, h2, oracle.F64)
        fwd2 = np.concatenate([h2[:blk.n_dst], mx2], axis=1)
        assert abs((np.sum(fwd2 * da) - np.sum(fwd * da)) / eps - bwd[j, c]) <= 1e-6
    # a source sampled twice by one row and winning it takes the gradient once
    dup = [(i, v) for i in range(blk.n_dst)
           for v in np.unique(blk.col[blk.rowptr[i]:blk.rowptr[i + 1]], return_counts=True)[0][
               np.unique(blk.col[blk.rowptr[i]:blk.rowptr[i + 1]], return_counts=True)[1] > 1]]
    assert dup, "the block has no repeated edge"
    i, v = dup[0]
    hd = np.zeros((blk.n_src, 1))
    hd[v, 0] = 1.0
    _, ad = oracle.aggregate_fwd_max(blk, hd, oracle.F64)
    assert ad[i, 0] == v
    dd = np.zeros((blk.n_dst, 2))
    dd[i, 1] = 1.0
    got = oracle.aggregate_bwd_max(blk, ad, dd, 1, None, oracle.F64)
    assert got[v, 0] == 1.0 and np.sum(np.abs(got)) == 1.0
    # ReLU mask of the layer below
    hbelow = rng.standard_normal((blk.n_src, f))
    masked = oracle.aggregate_bwd_max(blk, arg, da, f, hbelow, oracle.F64)
    np.testing.assert_array_equal(masked, np.where(hbelow > 0, bwd, 0.0))


def test_full_fanout_equals_textbook_operators():
    rng = np.random.default_rng(3)
    n = 40
    rowptr, col = dense.small_multigraph(rng, n, avg_deg=5, hubs=1, isolated=2)
    dst = np.arange(n, dtype=np.int64)
    blk = oracle.build_block(rowptr, col, dst, 10_000, 0, 0, 1)
    assert blk.n_src == n and np.array_equal(blk.src_ids, dst)
    A = np.zeros((n, n))
    for v in range(n):
        for e in range(rowptr[v], rowptr[v + 1]):
            A[v, col[e]] += 1
    deg = A.sum(1)
    h = rng.standard_normal((n, 6))
    Dinv = np.where(deg > 0, 1 / np.maximum(deg, 1), 0)
    np.testing.assert_allclose(oracle.aggregate_fwd(oracle.SAGE, blk, None, h, oracle.F64), Dinv[:, None] * (A @ h),
                               atol=1e-13)
    Dh = np.diag(1 / np.sqrt(deg + 1))
    want = Dh @ (A + np.eye(n)) @ Dh @ h
    sn = oracle.gcn_norm(rowptr)
    got = oracle.aggregate_fwd(oracle.GCN, blk, sn, h, oracle.F64)
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-6)  # nrm products are fp32


def test_gcn_regular_graph_rows_sum_to_one():
    n, d = 30, 4  # circulant 4-regular graph
    rows = [sorted({(v + s) % n for s in (-2, -1, 1, 2)}) for v in range(n)]
    rowptr = np.array([0] + np.cumsum([len(r) for r in rows]).tolist(), dtype=np.int64)
    col = np.array([u for r in rows for u in r], dtype=np.int64)
    dst = np.arange(0, n, 3, dtype=np.int64)
    blk = oracle.build_block(rowptr, col, dst, d, 0, 0, 1)
    sn = oracle.gcn_norm(rowptr)[blk.src_ids]
    got = oracle.aggregate_fwd(oracle.GCN, blk, sn, np.ones((blk.n_src, 1)), oracle.F64)
    np.testing.assert_allclose(got, 1.0, rtol=1e-6)


@pytest.mark.parametrize("seed", range(3))
def test_aggregate_bwd_adjoint_and_dense_transpose(seed):
    rng, _, _, blk, sn = _random_block(seed + 20)
    f = 6
    h = rng.standard_normal((blk.n_src, f))
    # SAGE: forward operator H -> [S H || M H]
    da = rng.standard_normal((blk.n_dst, 2 * f))
    fwd = np.concatenate([h[:blk.n_dst], oracle.aggregate_fwd(oracle.SAGE, blk, None, h, oracle.F64)], axis=1)
    bwd = oracle.aggregate_bwd(oracle.SAGE, blk, None, da, f, None, oracle.F64)
    assert abs(np.sum(fwd * da) - np.sum(h * bwd)) <= 1e-12 * np.sum(np.abs(fwd * da))
    want = dense.self_select_matrix(blk).T @ da[:, :f] + dense.sage_mean_matrix(blk).T @ da[:, f:]
    np.testing.assert_allclose(bwd, want, atol=1e-13)
    # GCN
    dg = rng.standard_normal((blk.n_dst, f))
    fwd = oracle.aggregate_fwd(oracle.GCN, blk, sn, h, oracle.F64)
    bwd = oracle.aggregate_bwd(oracle.GCN, blk, sn, dg, f, None, oracle.F64)
    assert abs(np.sum(fwd * dg) - np.sum(h * bwd)) <= 1e-12 * np.sum(np.abs(fwd * dg))
    np.testing.assert_allclose(bwd, dense.gcn_matrix(blk, sn).T @ dg, atol=1e-13)
    # ReLU mask of the layer below
    hb = rng.standard_normal((blk.n_src, f))
    masked = oracle.aggregate_bwd(oracle.GCN, blk, sn, dg, f, hb, oracle.F64)
    np.testing.assert_array_equal(masked, np.where(hb > 0, bwd, 0.0))


# ---------------------------------------------------------------------------
# update, loss, optimizer
# ---------------------------------------------------------------------------

def _bf16_round(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def test_update_fwd_bwd_dense():
    rng = np.random.default_rng(4)
    m, ke, n = 37, 9, 11
    a_s = rng.standard_normal((m, ke))
    a_n = rng.standard_normal((m, ke))
    w = rng.standard_normal((2 * ke, n))
    b = rng.standard_normal(n)
    A = np.concatenate([a_s, a_n], 1)
    z = oracle.update_fwd(a_s, a_n, w, b, relu=False, gemm_code=oracle.F64, out_code=oracle.F64)
    np.testing.assert_allclose(z, A @ w + b, rtol=1e-12, atol=1e-12)
    hr = oracle.update_fwd(a_s, a_n, w, b, relu=True, gemm_code=oracle.F64, out_code=oracle.F64)
    np.testing.assert_array_equal(hr, np.where(z > 0, z, 0.0))
    g = rng.standard_normal((m, n))
    dw, db, da = oracle.update_bwd(a_s, a_n, w, g, oracle.F64, want_da=True, out_code=oracle.F64)
    np.testing.assert_allclose(dw, A.T @ g, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, g.sum(0), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(da, g @ w.T, rtol=1e-12, atol=1e-12)


def test_update_bf16_operand_rounding():
    rng = np.random.default_rng(5)
    m, k, n = 50, 24, 16
    a32 = rng.standard_normal((m, k)).astype(np.float32)
    a = oracle.f32_to_bf16_bits(a32)          # stored bf16 activations
    w = rng.standard_normal((k, n)).astype(np.float32)
    b = rng.standard_normal(n).astype(np.float32)
    got = oracle.update_fwd(a, None, w, b, relu=True, gemm_code=oracle.BF16, out_code=oracle.BF16)
    ref = oracle.bf16_bits_to_f32(a).astype(np.float64) @ _bf16_round(w) + b.astype(np.float64)
    ref = np.where(ref > 0, ref, 0)
    want = torch.from_numpy(ref).to(torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    diff = np.abs(got.astype(np.int32) - want.astype(np.int32))
    assert diff.max() <= 1 and (diff > 0).mean() < 0.01
    g = rng.standard_normal((m, n)).astype(np.float32)
    dw, db, da = oracle.update_bwd(a, None, w, g, oracle.BF16, want_da=True)
    A = oracle.bf16_bits_to_f32(a).astype(np.float64)
    np.testing.assert_allclose(dw, A.T @ _bf16_round(g), rtol=1e-6, atol=1e-5)
    np.testing.assert_allclose(db, g.astype(np.float64).sum(0), rtol=1e-6, atol=1e-5)  # bias grad is unrounded
    np.testing.assert_allclose(da, _bf16_round(g) @ _bf16_round(w).T, rtol=1e-6, atol=1e-5)


def test_loss_zero_logits_is_log_c_and_matches_torch():
    for c in (8, 47, 172, 153):
        loss, g = oracle.softmax_ce(np.zeros((4, c), dtype=np.float32), np.arange(4) % c)
        assert abs(loss - math.log(c)) < 1e-12
        np.testing.assert_allclose(g.sum(1), 0, atol=1e-7)
    rng = np.random.default_rng(6)
    z = rng.standard_normal((64, 47)) * 3
    y = rng.integers(0, 47, size=64)
    loss, g = oracle.softmax_ce(z, y, oracle.F64)
    zt = torch.tensor(z, requires_grad=True)
    lt = torch.nn.functional.cross_entropy(zt, torch.tensor(y))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-12
    np.testing.assert_allclose(g, zt.grad.numpy(), atol=1e-14)
    # large logits stay finite
    loss, g = oracle.softmax_ce(np.array([[1e4, 0.0, -1e4]]), np.array([1]), oracle.F64)
    assert abs(loss - 1e4) < 1e-9 and np.isfinite(g).all()


def test_sgd_closed_form():
    w = np.array([1.0, -2.0, 3.5], dtype=np.float32)
    dw = np.array([0.5, 0.25, -1.0], dtype=np.float32)
    np.testing.assert_array_equal(oracle.sgd(w, dw, 0.5), np.array([0.75, -2.125, 4.0], dtype=np.float32))


# ---------------------------------------------------------------------------
# whole step: finite differences and an autograd dense reference
# ---------------------------------------------------------------------------

def _tiny_problem(kind, seed=0, n=60, f=(5, 4, 3), fanouts=(4, 3), batch=8):
    rng = np.random.default_rng(seed)
    rowptr, col = dense.small_multigraph(rng, n, avg_deg=5, hubs=1, isolated=2)
    table = rng.standard_normal((n, f[0])).astype(np.float64)
    labels = rng.integers(0, f[-1], size=n).astype(np.int64)
    targets = rng.choice(n, size=batch, replace=False).astype(np.int64)
    L = len(f) - 1
    ws, bs = [], []
    for l in range(1, L + 1):
        K = f[l - 1] if kind == oracle.GCN else 2 * f[l - 1]
        ws.append(rng.standard_normal((K, f[l])) * 0.7)
        bs.append(rng.standard_normal(f[l]) * 0.1)
    cfg = oracle.StepConfig(kind=kind, dims=f, fanouts=fanouts, precision=oracle.F64, seed=seed, step=3, lr=0.1)
    nrm = oracle.gcn_norm(rowptr)
    return rowptr, col, nrm, table, labels, targets, ws, bs, cfg


def _autograd_reference(kind, blocks, nrm, table, labels, targets, ws, bs):
    L = len(ws)
    layer_block = {l: blocks[L - l] for l in range(1, L + 1)}
    h = torch.tensor(table[blocks[-1].src_ids])
    wt = [torch.tensor(w, requires_grad=True) for w in ws]
    bt = [torch.tensor(b, requires_grad=True) for b in bs]
    for l in range(1, L + 1):
        blk = layer_block[l]
        if kind == oracle.SAGE:
            a = torch.cat([h[:blk.n_dst], torch.tensor(dense.sage_mean_matrix(blk)) @ h], 1)
        elif kind == oracle.SAGE_MAX:
            # torch's max over each row's sampled neighbours (its backward
            # routes the gradient to one maximal entry); zero for empty rows
            rows = []
            for i in range(blk.n_dst):
                cols = torch.tensor(blk.col[blk.rowptr[i]:blk.rowptr[i + 1]].astype(np.int64))
                rows.append(h[cols].max(0).values if cols.numel() else torch.zeros(h.shape[1], dtype=h.dtype))
            a = torch.cat([h[:blk.n_dst], torch.stack(rows)], 1)
        else:
            a = torch.tensor(dense.gcn_matrix(blk, nrm[blk.src_ids])) @ h
        z = a @ wt[l - 1] + bt[l - 1]
        h = torch.relu(z) if l < L else z
    loss = torch.nn.functional.cross_entropy(h, torch.tensor(labels[targets]))
    loss.backward()
    return loss.item(), [w.grad.numpy() for w in wt], [b.grad.numpy() for b in bt]


@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN, oracle.SAGE_MAX])
def test_train_step_matches_autograd_dense(kind):
    rowptr, col, nrm, table, labels, targets, ws, bs, cfg = _tiny_problem(kind, seed=1)
    out = oracle.train_step(rowptr, col, nrm, table, labels, targets, ws, bs, cfg)
    loss, gw, gb = _autograd_reference(kind, out["blocks"], nrm, table, labels, targets, ws, bs)
    assert abs(out["loss"] - loss) < 1e-12
    for l in range(1, len(ws) + 1):
        np.testing.assert_allclose(out["dW"][l], gw[l - 1], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(out["dB"][l], gb[l - 1], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(out["new_w"][l - 1], ws[l - 1] - cfg.lr * gw[l - 1], rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN, oracle.SAGE_MAX])
def test_train_step_three_layers_matches_autograd(kind):
    rowptr, col, nrm, table, labels, targets, ws, bs, cfg = _tiny_problem(kind, seed=2, f=(4, 5, 3, 3),
                                                                         fanouts=(3, 2, 2))
    out = oracle.train_step(rowptr, col, nrm, table, labels, targets, ws, bs, cfg)
    loss, gw, gb = _autograd_reference(kind, out["blocks"], nrm, table, labels, targets, ws, bs)
    assert abs(out["loss"] - loss) < 1e-12
    for l in range(1, 4):
        np.testing.assert_allclose(out["dW"][l], gw[l - 1], rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN, oracle.SAGE_MAX])
def test_train_step_finite_differences(kind):
    rowptr, col, nrm, table, labels, targets, ws, bs, cfg = _tiny_problem(kind, seed=3)
    out = oracle.train_step(rowptr, col, nrm, table, labels, targets, ws, bs, cfg)
    blocks = out["blocks"]
    L = len(ws)
    # stay away from ReLU kinks: every hidden pre-activation is far from 0
    for l in range(1, L):
        blk = blocks[L - l]
        a_self = out["H"][l - 1][:blk.n_dst] if kind != oracle.GCN else out["AGG"][l]
        a_nbr = out["AGG"][l] if kind != oracle.GCN else None
        z = oracle.update_fwd(np.ascontiguousarray(a_self), a_nbr, ws[l - 1], bs[l - 1], relu=False,
                              gemm_code=oracle.F64, out_code=oracle.F64)
        assert np.abs(z).min() > 1e-4
    rng = np.random.default_rng(0)
    h = 1e-6
    for l in range(1, L + 1):
        for _ in range(6):
            k = int(rng.integers(0, ws[l - 1].shape[0]))
            c = int(rng.integers(0, ws[l - 1].shape[1]))
            wp = [w.copy() for w in ws]
            wm = [w.copy() for w in ws]
            wp[l - 1][k, c] += h
            wm[l - 1][k, c] -= h
            lp = oracle.train_step(rowptr, col, nrm, table, labels, targets, wp, bs, cfg, blocks=blocks)["loss"]
            lm = oracle.train_step(rowptr, col, nrm, table, labels, targets, wm, bs, cfg, blocks=blocks)["loss"]
            fd = (lp - lm) / (2 * h)
            an = out["dW"][l][k, c]
            assert abs(fd - an) <= 1e-6 * max(1e-3, abs(an)) + 1e-9, (l, k, c, fd, an)


def test_table3_shapes_pin_workload_presets():
    import workloads
    rows = {r[0]: r for r in _golden_rows("table3_layer_dims.txt")}
    p = rows["ogbn-products"]
    for w in (workloads.RMAT_SAGE, workloads.RMAT_GCN):
        assert (w.n, w.m) == (int(p[1]), int(p[2]))
        assert w.dims == (int(p[3]), int(p[4]), int(p[5]))
        assert w.fanouts == (25, 10) and w.batch == 1024
    q = rows["ogbn-papers100M"]
    assert (workloads.RMAT_SAGE3.n, workloads.RMAT_SAGE3.m) == (int(q[1]), int(q[2]))
    assert workloads.RMAT_SAGE3.dims[0] == int(q[3]) and workloads.RMAT_SAGE3.dims[-1] == int(q[5])


def test_relu_flip_inverts_only_the_marked_backward_decisions():
    # a flipped decision zeroes (or passes) exactly that element of the
    # gradient below, and nothing in the forward pass changes
    rng = np.random.default_rng(3)
    n, f = 60, 6
    rp = np.concatenate([[0], np.cumsum(rng.integers(1, 5, n))]).astype(np.int64)
    col = rng.integers(0, n, rp[-1]).astype(np.int64)
    col = np.concatenate([np.sort(col[rp[i]:rp[i + 1]]) for i in range(n)]).astype(np.int64)
    table = rng.standard_normal((n, f)).astype(np.float32)
    labels = rng.integers(0, 3, n).astype(np.int64)
    targets = np.arange(8, dtype=np.int64)
    dims, fan = (f, 5, 3), (3, 3)
    ws = [rng.standard_normal((2 * dims[l], dims[l + 1])).astype(np.float32) for l in range(2)]
    bs = [np.zeros(dims[l + 1], np.float32) for l in range(2)]
    cfg = oracle.StepConfig(kind=oracle.SAGE, dims=dims, fanouts=fan, precision=oracle.F32, seed=1, step=0)
    ref = oracle.train_step(rp, col, None, table, labels, targets, ws, bs, cfg)
    h1 = ref["H"][1]
    on = np.argwhere(h1 > 0)[0]
    off = np.argwhere(h1 <= 0)[0]
    flip = np.zeros(h1.shape, dtype=bool)
    flip[tuple(on)] = flip[tuple(off)] = True
    alt = oracle.train_step(rp, col, None, table, labels, targets, ws, bs, cfg, blocks=ref["blocks"],
                            relu_flip={1: flip})
    assert alt["loss"] == ref["loss"] and np.array_equal(alt["H"][1], h1)
    g_ref, g_alt = ref["G"][1], alt["G"][1]
    assert g_alt[tuple(on)] == 0.0 and g_ref[tuple(on)] != 0.0
    keep = ~flip
    assert np.array_equal(g_alt[keep], g_ref[keep])
