"""Parity of every C-ABI call against the CPU oracle, on the GPU.

Integer work (sampling, block ids, transposes, gathers) must match bit for
bit.  Floating point is compared normwise, max|x - r| / max|r|, against
1e-4 (fp32 arithmetic) or 2e-2 (bf16 storage / GEMM operands), with the
oracle rounding at the same points as the kernels.
"""

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests import dense

pytestmark = pytest.mark.gpu

gnn = pytest.importorskip("paper_2303_00158_amd.gnn")

DEV = torch.device("cuda:0")
TOL = {oracle.F32: 1e-4, oracle.BF16: 2e-2}


def relerr(got, want):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    den = max(np.abs(want).max() if want.size else 0.0, 1e-30)
    return float(np.abs(got - want).max() / den) if want.size else 0.0


def to_np_act(t: torch.Tensor) -> np.ndarray:
    """Device activation -> oracle array (bf16 as raw uint16 bits)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def from_np_act(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def upload_block(blk: "oracle.Block", src_norm=None) -> "gnn.DeviceBlock":
    """Device copy of an oracle block (capacities = exact sizes)."""
    b = gnn.DeviceBlock.__new__(gnn.DeviceBlock)
    mk = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dtype=dt) if len(a) else np.zeros(1, dt)).to(DEV)  # noqa
    b.counts = torch.tensor([blk.n_dst, blk.n_src, blk.nnz, 0], dtype=torch.int64, device=DEV)
    b.src_ids = mk(blk.src_ids, np.int64)
    b.rowptr = mk(blk.rowptr, np.int64)
    b.col = mk(blk.col, np.int32)
    b.cscptr = mk(blk.cscptr, np.int64)
    b.cscrow = mk(blk.cscrow, np.int32)
    b.src_norm = mk(src_norm, np.float32) if src_norm is not None else None
    b.c = gnn.Block(blk.n_dst, blk.n_src, blk.nnz, b.counts.data_ptr(), b.src_ids.data_ptr(), b.rowptr.data_ptr(),
                    b.col.data_ptr(), b.cscptr.data_ptr(), b.cscrow.data_ptr(),
                    b.src_norm.data_ptr() if b.src_norm is not None else None)
    return b


def test_library_is_the_hip_build():
    assert gnn.lib().gnn_abi_version() == 2
    x = torch.ones(4, device=DEV)
    gnn.sgd(x, torch.ones(4, device=DEV), 0.5)
    torch.cuda.synchronize()
    assert torch.equal(x.cpu(), torch.full((4,), 0.5))


# ---------------------------------------------------------------------------
# GCN norms
# ---------------------------------------------------------------------------

def test_gcn_norm_bitexact():
    deg = np.concatenate([np.arange(0, 5000), np.array([65535, 65536, 999_999, 1_000_000, 123_456_789 // 100])])
    rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    g = gnn.DeviceGraph(torch.from_numpy(rowptr).to(DEV), torch.zeros(1, dtype=torch.int64, device=DEV))
    got = gnn.gcn_norm(g).cpu().numpy()
    want = oracle.gcn_norm(rowptr)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


# ---------------------------------------------------------------------------
# sampler
# ---------------------------------------------------------------------------

def _graph_cases():
    rng = np.random.default_rng(0)
    rp, cl = dense.small_multigraph(rng, 300, avg_deg=8, hubs=3, isolated=10)
    yield "multigraph300", rp, cl
    rp, cl = workloads.rmat_graph(20_000, 150_000, seed=1)
    yield "rmat20k", rp.numpy(), cl.numpy()
    rp, cl = workloads.er_graph(10_000, 50_000, seed=0)
    yield "er10k", rp.numpy(), cl.numpy()


@pytest.mark.parametrize("fanout", [1, 5, 25, 70, 300])
def test_build_block_bitexact(fanout):
    for name, rowptr, col in _graph_cases():
        n = rowptr.size - 1
        g = gnn.DeviceGraph(torch.from_numpy(rowptr).to(DEV), torch.from_numpy(col).to(DEV))
        nrm_d = gnn.gcn_norm(g)
        nrm_h = oracle.gcn_norm(rowptr)
        rng = np.random.default_rng(fanout)
        n_dst = min(n, 257)
        dst = rng.choice(n, size=n_dst, replace=False).astype(np.int64)
        # chain two hops: hop 2 reads hop 1's sources and its device count
        blk1 = gnn.DeviceBlock(n, n_dst, fanout, True, True, DEV)
        ws = gnn.sampler_workspace(n, blk1.c.cap_src, fanout, DEV)
        gnn.build_block(g, torch.from_numpy(dst).to(DEV), fanout, 7, 3, 1, blk1, ws, gcn_norm_t=nrm_d)
        blk2 = gnn.DeviceBlock(n, blk1.c.cap_src, fanout, True, True, DEV)
        gnn.build_block(g, blk1.src_ids, fanout, 7, 3, 2, blk2, ws, n_dst_dev=blk1.counts[1:2], gcn_norm_t=nrm_d)
        torch.cuda.synchronize()
        ref1 = oracle.build_block(rowptr, col, dst, fanout, 7, 3, 1)
        ref2 = oracle.build_block(rowptr, col, ref1.src_ids, fanout, 7, 3, 2)
        for got, ref in ((blk1.host(), ref1), (blk2.host(), ref2)):
            assert got["n_dst"] == ref.n_dst and got["n_src"] == ref.n_src and got["nnz"] == ref.nnz, name
            assert np.array_equal(got["src_ids"], ref.src_ids), name
            assert np.array_equal(got["rowptr"], ref.rowptr), name
            assert np.array_equal(got["col"], ref.col), name
            assert np.array_equal(got["cscptr"], ref.cscptr), name
            assert np.array_equal(got["cscrow"], ref.cscrow), name
            assert np.array_equal(got["src_norm"].view(np.uint32), nrm_h[ref.src_ids].view(np.uint32)), name
        # the workspace is left clean: rebuilding gives the same block
        gnn.build_block(g, torch.from_numpy(dst).to(DEV), fanout, 7, 3, 1, blk1, ws, gcn_norm_t=nrm_d)
        torch.cuda.synchronize()
        again = blk1.host()
        assert np.array_equal(again["col"], ref1.col) and np.array_equal(again["src_ids"], ref1.src_ids)


def test_build_block_flags_a_scan_wait_that_gives_up():
    # The row-pointer scan is single-pass: each row tile waits, boundedly,
    # for the prefix of the tile before it.  The host's test hook makes row
    # tile 1 publish nothing and every wait give up after 64 polls, so tile
    # 2's wait runs out: the build still finishes and flags GNN_DEVERR_WAIT
    # in counts[3], which gnn_check_device_errors reports.  With the hook
    # cleared, the same workspace builds the oracle's block with no flag.
    rowptr, col = workloads.rmat_graph(20_000, 150_000, seed=1)
    rowptr, col = rowptr.numpy(), col.numpy()
    n, n_dst, fanout = 20_000, 1000, 10  # 4 row tiles of 256
    g = gnn.DeviceGraph(torch.from_numpy(rowptr).to(DEV), torch.from_numpy(col).to(DEV))
    dst = np.random.default_rng(4).choice(n, size=n_dst, replace=False).astype(np.int64)
    dst_d = torch.from_numpy(dst).to(DEV)
    blk = gnn.DeviceBlock(n, n_dst, fanout, True, False, DEV)
    ws = gnn.sampler_workspace(n, n_dst, fanout, DEV)
    gnn.build_block(g, dst_d, fanout, 7, 3, 1, blk, ws)
    gnn.check_device_errors(blk.counts[3:4])
    try:
        gnn.debug_sampler_fault(1, 64)
        print("[device errors] build with a silent row tile", flush=True)
        gnn.build_block(g, dst_d, fanout, 7, 3, 1, blk, ws)
        with pytest.raises(gnn.GnnError) as e:
            gnn.check_device_errors(blk.counts[3:4])
        assert e.value.code == gnn.GNN_EDEVICE and "GNN_DEVERR_WAIT" in str(e.value)
        assert int(blk.counts[3].item()) & gnn.GNN_DEVERR_WAIT
    finally:
        gnn.debug_sampler_fault(-1, 0)
    gnn.build_block(g, dst_d, fanout, 7, 3, 1, blk, ws)
    gnn.check_device_errors(blk.counts[3:4])
    got, ref = blk.host(), oracle.build_block(rowptr, col, dst, fanout, 7, 3, 1)
    for key in ("src_ids", "rowptr", "col", "cscptr", "cscrow"):
        assert np.array_equal(got[key], getattr(ref, key)), key


def test_build_block_degenerate_cases():
    # isolated destinations, a destination whose neighbours are all destinations, an empty batch
    rowptr = np.array([0, 0, 2, 4, 4, 5], dtype=np.int64)
    col = np.array([2, 3, 1, 1, 0], dtype=np.int64)
    n = 5
    g = gnn.DeviceGraph(torch.from_numpy(rowptr).to(DEV), torch.from_numpy(col).to(DEV))
    ws = gnn.sampler_workspace(n, 16, 3, DEV)
    for dst in ([0, 3], [1, 2, 3], [4, 0], [2]):
        d = np.array(dst, dtype=np.int64)
        blk = gnn.DeviceBlock(n, len(dst), 3, True, False, DEV)
        gnn.build_block(g, torch.from_numpy(d).to(DEV), 3, 0, 0, 1, blk, ws)
        torch.cuda.synchronize()
        got = blk.host()
        ref = oracle.build_block(rowptr, col, d, 3, 0, 0, 1)
        assert np.array_equal(got["src_ids"], ref.src_ids) and np.array_equal(got["col"], ref.col)
        assert np.array_equal(got["cscptr"], ref.cscptr) and np.array_equal(got["cscrow"], ref.cscrow)
    # n_dst = 0 through a device count
    blk = gnn.DeviceBlock(n, 4, 3, True, False, DEV)
    zero = torch.zeros(1, dtype=torch.int64, device=DEV)
    gnn.build_block(g, torch.zeros(4, dtype=torch.int64, device=DEV), 3, 0, 0, 1, blk, ws, n_dst_dev=zero)
    torch.cuda.synchronize()
    got = blk.host()
    assert got["n_dst"] == 0 and got["n_src"] == 0 and got["nnz"] == 0 and got["cscptr"].tolist() == [0]


def _hub_graph():
    # destinations 1..10000 (more rows than one LDS window of the transpose
    # sort); every one links to hub 0, every 7th twice (a duplicate edge);
    # rows 1..17 link to vertex 11000 (a column just over the one-lane sort
    # limit), rows 18..33 to vertex 11001 (exactly at it); two more random
    # neighbours each.  No degree exceeds the fanout, so all edges are kept.
    rng = np.random.default_rng(11)
    n = 12_000
    nbrs = [[] for _ in range(n)]
    for v in range(1, 10_001):
        nbrs[v].append(0)
        if v % 7 == 0:
            nbrs[v].append(0)
        if v <= 17:
            nbrs[v].append(11_000)
        elif v <= 33:
            nbrs[v].append(11_001)
        nbrs[v] += rng.integers(10_001, n, size=2).tolist()
    rowptr = np.zeros(n + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum([len(x) for x in nbrs])
    col = np.array([u for x in nbrs for u in x], dtype=np.int64)
    return rowptr, col


def test_build_block_transpose_long_columns():
    rowptr, col = _hub_graph()
    n = rowptr.size - 1
    g = gnn.DeviceGraph(torch.from_numpy(rowptr).to(DEV), torch.from_numpy(col).to(DEV))
    fanout = 8
    dst_all = np.random.default_rng(3).permutation(np.arange(1, 10_001)).astype(np.int64)
    ws = gnn.sampler_workspace(n, dst_all.size, fanout, DEV)
    dst_d = torch.from_numpy(dst_all).to(DEV)
    blk = gnn.DeviceBlock(n, dst_all.size, fanout, True, False, DEV)
    for n_dst in (10_000, 4_097, 4_096, 300):  # the same workspace and block, shrinking batches
        dst = dst_all[:n_dst]
        n_dev = torch.tensor([n_dst], dtype=torch.int64, device=DEV)  # the first n_dst ids of dst_d
        print(f"[transpose] hub graph, n_dst={n_dst}", flush=True)
        gnn.build_block(g, dst_d, fanout, 5, 0, 1, blk, ws, n_dst_dev=n_dev)
        torch.cuda.synchronize()
        got = blk.host()
        ref = oracle.build_block(rowptr, col, dst, fanout, 5, 0, 1)
        assert int(blk.counts[3].item()) == 0
        assert np.array_equal(got["col"], ref.col)
        assert np.array_equal(got["cscptr"], ref.cscptr)
        assert np.array_equal(got["cscrow"], ref.cscrow)
        lens = np.diff(ref.cscptr)
        assert lens.max() > n_dst // 2  # the hub's column
        if n_dst == dst_all.size:
            assert (lens == 17).any() and (lens == 16).any()


def test_build_block_rejects_bad_arguments():
    rowptr = torch.tensor([0, 1, 2], dtype=torch.int64, device=DEV)
    col = torch.tensor([1, 0], dtype=torch.int64, device=DEV)
    g = gnn.DeviceGraph(rowptr, col)
    ws = gnn.sampler_workspace(2, 2, 1, DEV)
    blk = gnn.DeviceBlock(2, 2, 1, True, False, DEV)
    with pytest.raises(gnn.GnnError) as e:
        gnn.build_block(g, torch.tensor([0, 1], device=DEV), 0, 0, 0, 1, blk, ws)
    assert e.value.code == gnn.GNN_EINVAL
    small = torch.empty(256, dtype=torch.uint8, device=DEV)
    with pytest.raises(gnn.GnnError) as e:
        gnn.build_block(g, torch.tensor([0, 1], device=DEV), 1, 0, 0, 1, blk, small)
    assert e.value.code == gnn.GNN_ESIZE


# ---------------------------------------------------------------------------
# gather
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dim", [4, 13, 100, 128, 768])
def test_gather_bitexact(dim):
    rng = np.random.default_rng(dim)
    n = 5000
    table = rng.standard_normal((n, dim)).astype(np.float32)
    table.view(np.uint32)[7, 1] = 0x7FC0BEEF
    ids = rng.integers(0, n, size=3001).astype(np.int64)
    ids[:3] = 7
    t_d = torch.from_numpy(table).to(DEV)
    ids_d = torch.from_numpy(ids).to(DEV)
    out = torch.empty((ids.size, dim), dtype=torch.float32, device=DEV)
    gnn.gather_features(t_d, ids_d, out)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), oracle.gather(table, ids, oracle.F32).view(np.uint32))
    out_b = torch.empty((ids.size, dim), dtype=torch.bfloat16, device=DEV)
    gnn.gather_features(t_d, ids_d, out_b)
    assert np.array_equal(to_np_act(out_b), oracle.gather(table, ids, oracle.BF16))
    # fp16 table -> bf16 and -> fp32
    h16 = table.astype(np.float16)
    h_d = torch.from_numpy(h16).to(DEV)
    gnn.gather_features(h_d, ids_d, out_b)
    assert np.array_equal(to_np_act(out_b), oracle.gather(h16, ids, oracle.BF16))
    gnn.gather_features(h_d, ids_d, out)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), oracle.gather(h16, ids, oracle.F32).view(np.uint32))
    # a device count below the capacity leaves the tail untouched
    out.fill_(-5.0)
    n_dev = torch.tensor([1000], dtype=torch.int64, device=DEV)
    gnn.gather_features(t_d, ids_d, out, n_ids_dev=n_dev)
    o = out.cpu().numpy()
    assert np.array_equal(o[:1000].view(np.uint32), table[ids[:1000]].view(np.uint32)) and np.all(o[1000:] == -5.0)


def test_gather_pinned_host_table_zero_copy():
    rng = np.random.default_rng(3)
    n, dim = 4096, 96
    table = torch.from_numpy(rng.standard_normal((n, dim)).astype(np.float16)).pin_memory()
    ids = rng.integers(0, n, size=777).astype(np.int64)
    out = torch.empty((ids.size, dim), dtype=torch.bfloat16, device=DEV)
    gnn.gather_features(table, torch.from_numpy(ids).to(DEV), out, loc=gnn.GNN_LOC_HOST_PINNED)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_act(out), oracle.gather(table.numpy(), ids, oracle.BF16))


# ---------------------------------------------------------------------------
# aggregation with oracle-supplied blocks
# ---------------------------------------------------------------------------

def _oracle_block(seed, n=3000, n_dst=400, fanout=12):
    rp, cl = workloads.rmat_graph(n, n * 6, seed=seed)
    rp, cl = rp.numpy(), cl.numpy()
    rng = np.random.default_rng(seed)
    dst = rng.choice(n, size=n_dst, replace=False).astype(np.int64)
    blk = oracle.build_block(rp, cl, dst, fanout, seed, 0, 1)
    nrm = oracle.gcn_norm(rp)[blk.src_ids]
    return blk, nrm


def _act(rng, rows, f, code):
    x = rng.standard_normal((rows, f)).astype(np.float32)
    return oracle.f32_to_bf16_bits(x) if code == oracle.BF16 else x


@pytest.mark.parametrize("f", [4, 13, 100, 256, 300])
@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN])
@pytest.mark.parametrize("code", [oracle.F32, oracle.BF16])
def test_aggregate_fwd_parity(f, kind, code):
    blk, nrm = _oracle_block(f + 10 * kind)
    rng = np.random.default_rng(f)
    h = _act(rng, blk.n_src, f, code)
    want = oracle.aggregate_fwd(kind, blk, nrm if kind == oracle.GCN else None, h, code)
    db = upload_block(blk, nrm if kind == oracle.GCN else None)
    out = torch.empty((blk.n_dst, f), dtype=torch.bfloat16 if code == oracle.BF16 else torch.float32, device=DEV)
    gnn.aggregate_fwd(db, kind, from_np_act(h), out)
    got = to_np_act(out)
    assert relerr(oracle.to_float64(got), oracle.to_float64(want)) <= (1e-5 if code == oracle.F32 else 8e-3)


def _hub_block(seed, n=6000, hubs=64, n_dst=700, fanout=25, isolated_every=53):
    """A hub-heavy block: every non-hub vertex links to all `hubs` hub
    vertices (plus two random vertices), some vertices are isolated, so the
    destinations of a tile mostly sample the same few sources."""
    rng = np.random.default_rng(seed)
    nbrs = []
    for v in range(n):
        if v < hubs or v % isolated_every == 0:
            nbrs.append(np.zeros(0, np.int64))
        else:
            nbrs.append(np.concatenate([np.arange(hubs), rng.integers(0, n, 2)]).astype(np.int64))
    rp = np.zeros(n + 1, np.int64)
    rp[1:] = np.cumsum([a.size for a in nbrs])
    cl = np.concatenate(nbrs)
    dst = rng.choice(np.arange(hubs, n), size=n_dst, replace=False).astype(np.int64)
    blk = oracle.build_block(rp, cl, dst, fanout, seed, 0, 1)
    nrm = oracle.gcn_norm(rp)[blk.src_ids]
    return blk, nrm


DEDUP_BLOCKS = {
    "rmat": lambda seed: _oracle_block(seed, n_dst=500, fanout=25),
    "hub": lambda seed: _hub_block(seed),
    # 16 rows x 40 edges > the 512 a tile stages: those tiles read directly
    "hub_long_rows": lambda seed: _hub_block(seed, fanout=40),
}


@pytest.mark.parametrize("graph", sorted(DEDUP_BLOCKS))
@pytest.mark.parametrize("f", [4, 13, 100, 256, 300])
@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN])
def test_aggregate_fwd_dedup_equals_pull(graph, f, kind):
    # the tile-deduplicated aggregation sums in the pull kernel's order:
    # bitwise the same output, for every dtype pair
    blk, nrm = DEDUP_BLOCKS[graph](f + 7 * kind)
    assert blk.nnz > 0
    db = upload_block(blk, nrm if kind == oracle.GCN else None)
    rng = np.random.default_rng(f + kind)
    for hc, oc in [(oracle.BF16, oracle.BF16), (oracle.F32, oracle.F32), (oracle.BF16, oracle.F32),
                   (oracle.F32, oracle.BF16)]:
        h = from_np_act(_act(rng, blk.n_src, f, hc))
        odt = torch.bfloat16 if oc == oracle.BF16 else torch.float32
        want = torch.full((blk.n_dst, f), float("nan"), dtype=odt, device=DEV)
        got = torch.full((blk.n_dst, f), float("nan"), dtype=odt, device=DEV)
        print(f"[dedup] {graph} f={f} kind={kind} {hc}->{oc}", flush=True)
        gnn.aggregate_fwd(db, kind, h, want)
        gnn.aggregate_fwd_dedup(db, kind, h, got)
        torch.cuda.synchronize()
        iv = torch.int16 if oc == oracle.BF16 else torch.int32
        assert torch.equal(got.view(iv), want.view(iv)), (graph, f, kind, hc, oc)


def test_aggregate_fwd_dedup_against_oracle():
    blk, nrm = _hub_block(11)
    rng = np.random.default_rng(11)
    for kind in (oracle.SAGE, oracle.GCN):
        h = _act(rng, blk.n_src, 64, oracle.F32)
        want = oracle.aggregate_fwd(kind, blk, nrm if kind == oracle.GCN else None, h, oracle.F32)
        db = upload_block(blk, nrm if kind == oracle.GCN else None)
        out = torch.empty((blk.n_dst, 64), dtype=torch.float32, device=DEV)
        gnn.aggregate_fwd_dedup(db, kind, from_np_act(h), out)
        assert relerr(out.cpu().numpy().astype(np.float64), want) <= 1e-5


@pytest.mark.parametrize("f", [4, 13, 100, 256])
@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN])
@pytest.mark.parametrize("hb_code", [None, oracle.F32, oracle.BF16])
def test_aggregate_bwd_parity(f, kind, hb_code):
    blk, nrm = _oracle_block(3 + f + kind)
    rng = np.random.default_rng(f)
    ka = 2 * f if kind == oracle.SAGE else f
    da = rng.standard_normal((blk.n_dst, ka)).astype(np.float32)
    hb = _act(rng, blk.n_src, f, hb_code) if hb_code is not None else None
    want = oracle.aggregate_bwd(kind, blk, nrm if kind == oracle.GCN else None, da, f, hb, oracle.F32)
    db = upload_block(blk, nrm if kind == oracle.GCN else None)
    out = torch.empty((blk.n_src, f), dtype=torch.float32, device=DEV)
    gnn.aggregate_bwd(db, kind, from_np_act(da), f, out, h_below=from_np_act(hb) if hb is not None else None)
    assert relerr(out.cpu().numpy(), want) <= 1e-5


def test_aggregate_bwd_is_bitwise_reproducible():
    blk, nrm = _oracle_block(99, n_dst=800, fanout=25)
    f = 256
    rng = np.random.default_rng(0)
    da = from_np_act(rng.standard_normal((blk.n_dst, 2 * f)).astype(np.float32))
    db = upload_block(blk)
    a = torch.empty((blk.n_src, f), dtype=torch.float32, device=DEV)
    b = torch.empty_like(a)
    gnn.aggregate_bwd(db, oracle.SAGE, da, f, a)
    gnn.aggregate_bwd(db, oracle.SAGE, da, f, b)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


# ---------------------------------------------------------------------------
# GraphSAGE's max aggregator
# ---------------------------------------------------------------------------

def _multigraph_block(seed, n=1500, n_dst=300, fanout=100):
    """A block of a multigraph: repeated edges, isolated destinations (empty
    rows), hub rows longer than one 64-edge window, and popular sources
    (every vertex also links to three of six, repeats allowed) whose
    transpose columns span several windows and hold repeated rows."""
    rng = np.random.default_rng(seed)
    rowptr, col = dense.small_multigraph(rng, n, avg_deg=12, hubs=4, isolated=25)
    deg = np.diff(rowptr)
    popular = rng.choice(np.nonzero(deg > 0)[0], size=6, replace=False)
    rows = [np.sort(np.concatenate([col[rowptr[v]:rowptr[v + 1]], rng.choice(popular, size=3)])) if deg[v] else
            col[rowptr[v]:rowptr[v + 1]] for v in range(n)]
    rowptr = np.concatenate([[0], np.cumsum([r.size for r in rows])]).astype(np.int64)
    col = np.concatenate(rows).astype(np.int64)
    deg = np.diff(rowptr)
    special = np.concatenate([np.argsort(-deg, kind="stable")[:4], np.nonzero(deg == 0)[0][:3]])
    rest = np.setdiff1d(np.arange(n), special)
    dst = np.concatenate([special, rng.choice(rest, size=n_dst - special.size, replace=False)]).astype(np.int64)
    rng.shuffle(dst)
    blk = oracle.build_block(rowptr, col, dst, fanout, seed, 0, 1)
    assert np.diff(blk.rowptr).max() > 64 and np.diff(blk.cscptr).max() > 96
    return blk


def _max_inputs(rng, blk, f, code, ties):
    if ties:  # small integers: most maxima are tied between several edges
        x = rng.integers(-3, 4, size=(blk.n_src, f)).astype(np.float32)
    else:
        x = rng.standard_normal((blk.n_src, f)).astype(np.float32)
    return oracle.f32_to_bf16_bits(x) if code == oracle.BF16 else x


def _has_repeated_edge(blk):
    for i in range(blk.n_dst):
        c = blk.col[blk.rowptr[i]:blk.rowptr[i + 1]]
        if c.size != np.unique(c).size:
            return True
    return False


@pytest.mark.parametrize("f", [1, 4, 13, 100, 256, 300])
@pytest.mark.parametrize("hc,oc", [(oracle.F32, oracle.F32), (oracle.BF16, oracle.BF16), (oracle.BF16, oracle.F32),
                                   (oracle.F32, oracle.BF16)])
@pytest.mark.parametrize("ties", [False, True])
def test_aggregate_fwd_max_parity(f, hc, oc, ties):
    # exact comparisons: the maximum and its argmax match bit for bit
    blk = _multigraph_block(f + 3 * hc + 11 * oc)
    assert _has_repeated_edge(blk) and (np.diff(blk.rowptr) == 0).any()
    rng = np.random.default_rng(f + hc)
    h = _max_inputs(rng, blk, f, hc, ties)
    want, want_arg = oracle.aggregate_fwd_max(blk, h, oc)
    db = upload_block(blk)
    odt = torch.bfloat16 if oc == oracle.BF16 else torch.float32
    out = torch.full((blk.n_dst, f), float("nan"), dtype=odt, device=DEV)
    arg = torch.full((blk.n_dst, f), -7, dtype=torch.int32, device=DEV)
    print(f"[max fwd] f={f} {hc}->{oc} ties={ties}", flush=True)
    gnn.aggregate_fwd_max(db, from_np_act(h), out, arg)
    assert np.array_equal(arg.cpu().numpy(), want_arg)
    got = to_np_act(out)
    iv = np.uint16 if oc == oracle.BF16 else np.uint32
    assert np.array_equal(got.view(iv), want.view(iv))


def test_aggregate_fwd_max_nan_and_unaligned_rows():
    # A NaN is kept only when it is the row's first edge; f = 13 takes the
    # per-element path.  NaN payloads may differ, so NaN positions and the
    # other values are compared separately.
    blk = _multigraph_block(5)
    f = 13
    rng = np.random.default_rng(5)
    h = rng.standard_normal((blk.n_src, f)).astype(np.float32)
    h[rng.random((blk.n_src, f)) < 0.05] = np.nan
    want, want_arg = oracle.aggregate_fwd_max(blk, h, oracle.F32)
    assert np.isnan(want).any()
    db = upload_block(blk)
    out = torch.empty((blk.n_dst, f), dtype=torch.float32, device=DEV)
    arg = torch.empty((blk.n_dst, f), dtype=torch.int32, device=DEV)
    gnn.aggregate_fwd_max(db, from_np_act(h), out, arg)
    got = out.cpu().numpy()
    assert np.array_equal(arg.cpu().numpy(), want_arg)
    assert np.array_equal(np.isnan(got), np.isnan(want))
    ok = ~np.isnan(want)
    assert np.array_equal(got[ok].view(np.uint32), want[ok].view(np.uint32))


def test_aggregate_fwd_max_device_count_below_capacity():
    # rows from the device count on are left untouched
    blk = _multigraph_block(9)
    f = 64
    rng = np.random.default_rng(9)
    h = _max_inputs(rng, blk, f, oracle.F32, False)
    want, want_arg = oracle.aggregate_fwd_max(blk, h, oracle.F32)
    db = upload_block(blk)
    n = blk.n_dst // 2
    db.counts[0] = n
    out = torch.full((blk.n_dst, f), -5.0, dtype=torch.float32, device=DEV)
    arg = torch.full((blk.n_dst, f), -7, dtype=torch.int32, device=DEV)
    gnn.aggregate_fwd_max(db, from_np_act(h), out, arg)
    o, a = out.cpu().numpy(), arg.cpu().numpy()
    assert np.array_equal(o[:n], want[:n]) and np.array_equal(a[:n], want_arg[:n])
    assert np.all(o[n:] == -5.0) and np.all(a[n:] == -7)
    # a device count of zero writes nothing, forward and backward
    db.counts[0] = 0
    db.counts[1] = 0
    gnn.aggregate_fwd_max(db, from_np_act(h), out, arg)
    d_src = torch.full((blk.n_src, f), -3.0, dtype=torch.float32, device=DEV)
    gnn.aggregate_bwd_max(db, arg, torch.zeros((blk.n_dst, 2 * f), device=DEV), f, d_src)
    torch.cuda.synchronize()
    o, a = out.cpu().numpy(), arg.cpu().numpy()
    assert np.array_equal(o[:n], want[:n]) and np.all(o[n:] == -5.0) and np.all(a[n:] == -7)
    assert torch.all(d_src == -3.0)


@pytest.mark.parametrize("f", [1, 4, 13, 100, 256, 300])
@pytest.mark.parametrize("hb_code", [None, oracle.F32, oracle.BF16])
@pytest.mark.parametrize("ties", [False, True])
def test_aggregate_bwd_max_parity(f, hb_code, ties):
    # argmax from the oracle's forward; a row that sampled a source twice
    # passes its gradient once; with ties one source wins many elements
    blk = _multigraph_block(100 + f + (hb_code or 0))
    rng = np.random.default_rng(f)
    h = _max_inputs(rng, blk, f, oracle.F32, ties)
    _, amax = oracle.aggregate_fwd_max(blk, h, oracle.F32)
    da = rng.standard_normal((blk.n_dst, 2 * f)).astype(np.float32)
    hb = _act(rng, blk.n_src, f, hb_code) if hb_code is not None else None
    want = oracle.aggregate_bwd_max(blk, amax, da, f, hb, oracle.F32)
    db = upload_block(blk)
    out = torch.full((blk.n_src, f), float("nan"), dtype=torch.float32, device=DEV)
    print(f"[max bwd] f={f} hb={hb_code} ties={ties}", flush=True)
    arg_d = torch.from_numpy(amax).to(DEV)
    gnn.aggregate_bwd_max(db, arg_d, from_np_act(da), f, out, h_below=from_np_act(hb) if hb is not None else None)
    got = out.cpu().numpy()
    assert relerr(got, want) <= 1e-6
    # no atomics: a second call gives the same bits
    out2 = torch.empty_like(out)
    gnn.aggregate_bwd_max(db, arg_d, from_np_act(da), f, out2, h_below=from_np_act(hb) if hb is not None else None)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), out2.view(torch.int32))


def test_aggregate_max_round_trip_on_a_sampled_block():
    # forward then backward through the library on a sampled R-MAT block,
    # against the oracle's forward and backward
    blk, _ = _oracle_block(17, n_dst=600, fanout=25)
    f = 128
    rng = np.random.default_rng(17)
    h = oracle.f32_to_bf16_bits(rng.standard_normal((blk.n_src, f)).astype(np.float32))
    want, want_arg = oracle.aggregate_fwd_max(blk, h, oracle.BF16)
    db = upload_block(blk)
    out = torch.empty((blk.n_dst, f), dtype=torch.bfloat16, device=DEV)
    arg = torch.empty((blk.n_dst, f), dtype=torch.int32, device=DEV)
    gnn.aggregate_fwd_max(db, from_np_act(h), out, arg)
    assert np.array_equal(to_np_act(out), want) and np.array_equal(arg.cpu().numpy(), want_arg)
    da = rng.standard_normal((blk.n_dst, 2 * f)).astype(np.float32)
    d_src = torch.empty((blk.n_src, f), dtype=torch.float32, device=DEV)
    gnn.aggregate_bwd_max(db, arg, from_np_act(da), f, d_src, h_below=from_np_act(h))
    assert relerr(d_src.cpu().numpy(), oracle.aggregate_bwd_max(blk, want_arg, da, f, h, oracle.F32)) <= 1e-6


# ---------------------------------------------------------------------------
# one layer's forward in one launch (aggregation + update, loss for the last)
# ---------------------------------------------------------------------------

LAYER_CASES = [
    # f, n_out, n_dst, fanout, last, row-length bound given to the kernel
    (100, 256, 5000, 10, False, 10),   # 16-row tiles, 4-feature chunks, the first layer of the headline model
    (256, 47, 1024, 25, True, 25),     # 4-row tiles, 8-feature chunks, its last layer with the loss
    (32, 64, 301, 5, False, 5),        # ragged last tile
    (64, 8, 77, 3, True, 3),
    (128, 128, 600, 15, False, 15),    # K = 256 (SAGE) on the 2 x 8 register tiles
    (256, 47, 700, 25, True, 1),       # bound far below the real rows: indices read in place
    (256, 47, 9000, 10, True, 10),     # 32-row tiles with the loss epilogue, ragged last tile
]


@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN])
@pytest.mark.parametrize("f,n_out,n_dst,fanout,last,bound", LAYER_CASES)
def test_layer_fwd_parity(kind, f, n_out, n_dst, fanout, last, bound):
    seed = f + n_out + n_dst + kind
    blk, nrm = _oracle_block(seed, n=max(3000, 2 * n_dst), n_dst=n_dst, fanout=fanout)
    rng = np.random.default_rng(seed)
    h = _act(rng, blk.n_src, f, oracle.BF16)
    K = 2 * f if kind == oracle.SAGE else f
    w = (rng.standard_normal((K, n_out)) / np.sqrt(K)).astype(np.float32)
    b = (0.1 * rng.standard_normal(n_out)).astype(np.float32)
    agg = oracle.aggregate_fwd(kind, blk, nrm if kind == oracle.GCN else None, h, oracle.BF16)
    a_self, a_nbr = (h[:blk.n_dst], agg) if kind == oracle.SAGE else (agg, None)
    want = oracle.update_fwd(a_self, a_nbr, w, b, not last, oracle.BF16, oracle.F32 if last else oracle.BF16)

    db = upload_block(blk, nrm if kind == oracle.GCN else None)
    wt = torch.from_numpy(np.ascontiguousarray(w.T)).to(DEV).to(torch.bfloat16)
    agg_out = torch.empty((blk.n_dst, f), dtype=torch.bfloat16, device=DEV)
    out = torch.empty((blk.n_dst, n_out), dtype=torch.float32 if last else torch.bfloat16, device=DEV)
    kw = {}
    if last:
        labels_np = rng.integers(0, n_out, size=max(3000, 2 * n_dst)).astype(np.int64)
        kw = dict(labels=torch.from_numpy(labels_np).to(DEV), batch=blk.n_dst,
                  g_out=torch.empty((blk.n_dst, n_out), dtype=torch.float32, device=DEV),
                  row_loss=torch.empty(blk.n_dst, dtype=torch.float32, device=DEV))
    print(f"[layer_fwd] kind={kind} f={f} n_out={n_out} n_dst={n_dst} last={last} bound={bound}", flush=True)
    gnn.layer_fwd(db, kind, bound, from_np_act(h), wt, torch.from_numpy(b).to(DEV), agg_out, out, **kw)
    torch.cuda.synchronize()
    assert relerr(oracle.to_float64(to_np_act(agg_out)), oracle.to_float64(agg)) <= 8e-3
    assert relerr(oracle.to_float64(to_np_act(out)), oracle.to_float64(want)) <= 8e-3
    if last:
        y = labels_np[blk.src_ids[:blk.n_dst]]
        loss, g = oracle.softmax_ce(want, y)
        assert relerr(kw["g_out"].cpu().numpy(), g) <= 2e-2
        assert abs(float(kw["row_loss"].mean()) - loss) <= 2e-2 * max(1.0, abs(loss))


@pytest.mark.parametrize("sage", [True, False])
@pytest.mark.parametrize("m,cap,ke,n", [(5000, 6000, 100, 256), (301, 301, 32, 64), (1024, 2048, 128, 128),
                                         (77, 77, 64, 47)])
def test_update_fwd_with_shadow_matches_oracle(sage, m, cap, ke, n):
    # gnn_update_fwd given the bf16 W^T: a hidden bf16 layer whose weights fit
    # the fused kernel's register tiles runs it in A-load mode (the layer-1
    # update of the training step); capacity above the device row count
    rng = np.random.default_rng(m + ke + n + sage)
    a_s = oracle.f32_to_bf16_bits(rng.standard_normal((cap, ke)).astype(np.float32))
    a_n = oracle.f32_to_bf16_bits(rng.standard_normal((cap, ke)).astype(np.float32)) if sage else None
    K = (2 if sage else 1) * ke
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    b = (0.1 * rng.standard_normal(n)).astype(np.float32)
    want = oracle.update_fwd(a_s[:m], a_n[:m] if sage else None, w, b, True, oracle.BF16, oracle.BF16)
    wt = torch.from_numpy(np.ascontiguousarray(w.T)).to(DEV).to(torch.bfloat16)
    out = torch.full((cap, n), float("nan"), dtype=torch.bfloat16, device=DEV)
    m_dev = torch.tensor([m], dtype=torch.int64, device=DEV)
    print(f"[update_fwd shadow] sage={sage} m={m} cap={cap} ke={ke} n={n}", flush=True)
    gnn.update_fwd(from_np_act(a_s), from_np_act(a_n) if sage else None, from_np_act(w), from_np_act(b), out, True,
                   gnn.GNN_BF16, m_dev=m_dev, cap_m=cap, wt=wt)
    torch.cuda.synchronize()
    got = to_np_act(out)
    assert relerr(oracle.to_float64(got[:m]), oracle.to_float64(want)) <= 8e-3
    # rows past the device count are not written
    assert torch.isnan(out[m:].float()).all()


def test_layer_fwd_rejects_unsupported_shapes():
    blk, _ = _oracle_block(5, n_dst=50, fanout=4)
    db = upload_block(blk)
    h = torch.zeros((blk.n_src, 512), dtype=torch.bfloat16, device=DEV)
    wt = torch.zeros((256, 1024), dtype=torch.bfloat16, device=DEV)   # K = 1024: beyond the register tiles
    agg = torch.empty((blk.n_dst, 512), dtype=torch.bfloat16, device=DEV)
    out = torch.empty((blk.n_dst, 256), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(gnn.GnnError) as e:
        gnn.layer_fwd(db, oracle.SAGE, 4, h, wt, None, agg, out)
    assert e.value.code == gnn.GNN_EUNSUPPORTED
    # 100 classes: fine for a hidden layer, over the loss epilogue's 64
    h = torch.zeros((blk.n_src, 64), dtype=torch.bfloat16, device=DEV)
    wt = torch.zeros((100, 128), dtype=torch.bfloat16, device=DEV)
    agg = torch.empty((blk.n_dst, 64), dtype=torch.bfloat16, device=DEV)
    gnn.layer_fwd(db, oracle.SAGE, 4, h, wt, None, agg, torch.empty((blk.n_dst, 100), dtype=torch.bfloat16,
                                                                    device=DEV))
    with pytest.raises(gnn.GnnError) as e:
        gnn.layer_fwd(db, oracle.SAGE, 4, h, wt, None, agg, torch.empty((blk.n_dst, 100), device=DEV),
                      labels=torch.zeros(4000, dtype=torch.int64, device=DEV), batch=blk.n_dst,
                      g_out=torch.empty((blk.n_dst, 100), device=DEV), row_loss=torch.empty(blk.n_dst, device=DEV))
    assert e.value.code == gnn.GNN_EUNSUPPORTED


# ---------------------------------------------------------------------------
# both layers of a two-layer model in one launch
# ---------------------------------------------------------------------------

TWO_CASES = [
    # f0, f1, n_out, n_dst, fanout, row-length bound given to the kernel
    (100, 256, 47, 1024, 25, 25),   # the headline model: tiles of up to 104 rows in one pass
    (32, 64, 8, 301, 5, 5),         # ragged last tile, 8-feature A^1 chunks, KSM1 = 4
    (100, 256, 47, 300, 40, 40),    # tiles of more than 112 rows: two passes
    (64, 128, 48, 513, 10, 2),      # bound far below the rows: indices read in place; 48 classes
]


def _two_layer_inputs(kind, f0, f1, n_out, n_dst, fanout, seed, n=None):
    n = n or max(3000, 2 * n_dst)
    blk, nrm = _oracle_block(seed, n=n, n_dst=n_dst, fanout=fanout)
    rng = np.random.default_rng(seed)
    sage = kind == oracle.SAGE
    x_self = _act(rng, blk.n_src, f0, oracle.BF16)
    m1 = _act(rng, blk.n_src, f0, oracle.BF16)
    K1, K2 = (2 if sage else 1) * f0, (2 if sage else 1) * f1
    w1 = (rng.standard_normal((K1, f1)) / np.sqrt(K1)).astype(np.float32)
    w2 = (rng.standard_normal((K2, n_out)) / np.sqrt(K2)).astype(np.float32)
    b1 = (0.1 * rng.standard_normal(f1)).astype(np.float32)
    b2 = (0.1 * rng.standard_normal(n_out)).astype(np.float32)
    labels = rng.integers(0, n_out, size=n).astype(np.int64)  # one per graph vertex (read by vertex id)
    return blk, nrm, x_self, m1, w1, w2, b1, b2, labels


def _shadow(w):
    return torch.from_numpy(np.ascontiguousarray(w.T)).to(DEV).to(torch.bfloat16)


@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN])
@pytest.mark.parametrize("f0,f1,n_out,n_dst,fanout,bound", TWO_CASES)
def test_two_layer_fwd_parity(kind, f0, f1, n_out, n_dst, fanout, bound):
    # gnn_two_layer_fwd against the oracle's composition (update of layer 1,
    # aggregation and update of layer 2, loss, input gradient of layer 2),
    # and bit for bit against the launches it replaces
    seed = f0 + f1 + n_out + n_dst + kind
    sage = kind == oracle.SAGE
    blk, nrm, x_self, m1, w1, w2, b1, b2, labels = _two_layer_inputs(kind, f0, f1, n_out, n_dst, fanout, seed)
    h1 = oracle.update_fwd(x_self if sage else m1, m1 if sage else None, w1, b1, True, oracle.BF16, oracle.BF16)
    agg2 = oracle.aggregate_fwd(kind, blk, nrm if not sage else None, h1, oracle.BF16)
    a_self, a_nbr = (h1[:blk.n_dst], agg2) if sage else (agg2, None)
    logits = oracle.update_fwd(a_self, a_nbr, w2, b2, False, oracle.BF16, oracle.F32)
    loss, g = oracle.softmax_ce(logits, labels[blk.src_ids[:blk.n_dst]])

    db = upload_block(blk, nrm if not sage else None)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)  # noqa
    xs_d, m1_d = from_np_act(x_self), from_np_act(m1)
    wt1, wt2 = _shadow(w1), _shadow(w2)
    out = dict(h1=torch.empty((blk.n_src, f1), dtype=torch.bfloat16, device=DEV),
               agg=torch.empty((blk.n_dst, f1), dtype=torch.bfloat16, device=DEV),
               logits=torch.empty((blk.n_dst, n_out), device=DEV), g=torch.empty((blk.n_dst, n_out), device=DEV),
               rl=torch.empty(blk.n_dst, device=DEV), da=torch.empty((blk.n_dst, w2.shape[0]), device=DEV))
    lab_d = d(labels)
    print(f"[two_layer_fwd] kind={kind} f0={f0} f1={f1} n_out={n_out} n_dst={n_dst} fanout={fanout} bound={bound}",
          flush=True)
    gnn.two_layer_fwd(db, kind, bound, xs_d if sage else None, m1_d, wt1, d(b1), out["h1"], wt2, d(b2), out["agg"],
                      out["logits"], lab_d, blk.n_dst, out["g"], out["rl"], out["da"])
    torch.cuda.synchronize()
    assert relerr(oracle.to_float64(to_np_act(out["h1"])), oracle.to_float64(h1)) <= 8e-3
    assert relerr(oracle.to_float64(to_np_act(out["agg"])), oracle.to_float64(agg2)) <= 8e-3
    assert relerr(out["logits"].cpu().numpy(), logits) <= 8e-3
    assert relerr(out["g"].cpu().numpy(), g) <= 2e-2
    assert abs(float(out["rl"].mean()) - loss) <= 2e-2 * max(1.0, abs(loss))
    # the input gradient from the kernel's own G: bf16 operands, fp32 sums
    g_gpu = out["g"].cpu().numpy()
    a_s_gpu = to_np_act(out["h1"])[:blk.n_dst] if sage else to_np_act(out["agg"])
    _, _, da = oracle.update_bwd(a_s_gpu, to_np_act(out["agg"]) if sage else None, w2, g_gpu, oracle.BF16, True)
    assert relerr(out["da"].cpu().numpy(), da) <= 1e-5

    # the launches it replaces: layer 1's update, the fused last layer, dA
    ref = dict(h1=torch.empty_like(out["h1"]), agg=torch.empty_like(out["agg"]),
               logits=torch.empty_like(out["logits"]), g=torch.empty_like(out["g"]), rl=torch.empty_like(out["rl"]),
               da=torch.empty_like(out["da"]))
    gnn.update_fwd(xs_d if sage else m1_d, m1_d if sage else None, d(w1), d(b1), ref["h1"], True, gnn.GNN_BF16,
                   wt=wt1)
    gnn.layer_fwd(db, kind, bound, ref["h1"], wt2, d(b2), ref["agg"], ref["logits"], labels=lab_d, batch=blk.n_dst,
                  g_out=ref["g"], row_loss=ref["rl"])
    K2 = w2.shape[0]
    dw, dbias = torch.empty((K2, n_out), device=DEV), torch.empty(n_out, device=DEV)
    gnn.update_bwd(ref["h1"][:blk.n_dst] if sage else ref["agg"], ref["agg"] if sage else None, d(w2), ref["g"], dw,
                   dbias, ref["da"], gnn.GNN_BF16)
    torch.cuda.synchronize()
    for k in ("h1", "agg", "logits", "g", "rl", "da"):
        a, b = out[k], ref[k]
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32)), k


@pytest.mark.parametrize("kind", [oracle.SAGE, oracle.GCN])
@pytest.mark.parametrize("f0,f1,n_out,n_dst,fanout,bound,n", [c + (None,) for c in TWO_CASES] +
                         [(100, 256, 47, 2048, 50, 50, 200_000)])
def test_two_layer_bwd_parity(kind, f0, f1, n_out, n_dst, fanout, bound, n):
    # gnn_two_layer_bwd (both layers' dW and db, layer 2's aggregation
    # backward folded into layer 1's dW) from gnn_two_layer_fwd's outputs:
    # against the oracle's composition (aggregation backward with the ReLU
    # mask, then each layer's update backward, bf16 operands) on the GPU's own
    # forward values, and bit for bit against gnn_aggregate_bwd +
    # gnn_update_bwd per layer.  Layers up to 128 wide are rejected (their
    # aggregation backward sums a row in several slots, which the folded job
    # does not repeat).  The last case has layer-1 row splits of two groups
    # (about 9,400 rows over 64 splits of 192).
    seed = 3 * f0 + f1 + n_out + n_dst + kind
    sage = kind == oracle.SAGE
    blk, nrm, x_self, m1, w1, w2, b1, b2, labels = _two_layer_inputs(kind, f0, f1, n_out, n_dst, fanout, seed, n)
    db = upload_block(blk, nrm if not sage else None)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)  # noqa
    xs_d, m1_d = from_np_act(x_self), from_np_act(m1)
    K1, K2 = w1.shape[0], w2.shape[0]
    h1 = torch.empty((blk.n_src, f1), dtype=torch.bfloat16, device=DEV)
    agg = torch.empty((blk.n_dst, f1), dtype=torch.bfloat16, device=DEV)
    g = torch.empty((blk.n_dst, n_out), device=DEV)
    da = torch.empty((blk.n_dst, K2), device=DEV)
    gnn.two_layer_fwd(db, kind, bound, xs_d if sage else None, m1_d, _shadow(w1), d(b1), h1, _shadow(w2), d(b2), agg,
                      torch.empty((blk.n_dst, n_out), device=DEV), d(labels), blk.n_dst, g,
                      torch.empty(blk.n_dst, device=DEV), da)
    m1_rows = torch.tensor([blk.n_src], dtype=torch.int64, device=DEV)
    out = dict(dw1=torch.empty((K1, f1), device=DEV), db1=torch.empty(f1, device=DEV),
               dw2=torch.empty((K2, n_out), device=DEV), db2=torch.empty(n_out, device=DEV))
    print(f"[two_layer_bwd] kind={kind} f0={f0} f1={f1} n_out={n_out} n_dst={n_dst} fanout={fanout}", flush=True)
    if f1 <= 128:
        with pytest.raises(gnn.GnnError) as e:
            gnn.two_layer_bwd(db, kind, xs_d if sage else None, m1_d, m1_rows, blk.n_src, h1, agg, da, g,
                              out["dw1"], out["db1"], out["dw2"], out["db2"])
        assert e.value.code == gnn.GNN_EUNSUPPORTED
        return
    gnn.two_layer_bwd(db, kind, xs_d if sage else None, m1_d, m1_rows, blk.n_src, h1, agg, da, g, out["dw1"],
                      out["db1"], out["dw2"], out["db2"])
    torch.cuda.synchronize()
    # the oracle on the kernel's own forward values
    h1_h, agg_h, g_h, da_h = to_np_act(h1), to_np_act(agg), g.cpu().numpy(), da.cpu().numpy()
    dw2, db2, _ = oracle.update_bwd(h1_h[:blk.n_dst] if sage else agg_h, agg_h if sage else None, w2, g_h,
                                    oracle.BF16, False)
    g1 = oracle.aggregate_bwd(kind, blk, nrm if not sage else None, da_h, f1, h1_h, oracle.F32)
    dw1, db1, _ = oracle.update_bwd(x_self if sage else m1, m1 if sage else None, w1, g1, oracle.BF16, False)
    assert relerr(out["dw2"].cpu().numpy(), dw2) <= 1e-5
    assert relerr(out["db2"].cpu().numpy(), db2) <= 1e-5
    assert relerr(out["dw1"].cpu().numpy(), dw1) <= 2e-3
    assert relerr(out["db1"].cpu().numpy(), db1) <= 1e-5

    # the launches it replaces
    g1_d = torch.empty((blk.n_src, f1), device=DEV)
    gnn.aggregate_bwd(db, kind, da, f1, g1_d, h_below=h1)
    ref = {k: torch.empty_like(v) for k, v in out.items()}
    gnn.update_bwd(xs_d if sage else m1_d, m1_d if sage else None, d(w1), g1_d, ref["dw1"], ref["db1"], None,
                   gnn.GNN_BF16)
    gnn.update_bwd(h1[:blk.n_dst] if sage else agg, agg if sage else None, d(w2), g, ref["dw2"], ref["db2"], None,
                   gnn.GNN_BF16)
    torch.cuda.synchronize()
    for k in out:
        assert torch.equal(out[k].view(torch.int32), ref[k].view(torch.int32)), k


@pytest.mark.parametrize("f0,f1,n_out,n_dst,fanout,bound", TWO_CASES)
def test_two_layer_fwd_max_parity(f0, f1, n_out, n_dst, fanout, bound):
    # gnn_two_layer_fwd_max against the oracle's composition (update of layer
    # 1, max aggregation and update of layer 2, loss), and against the calls
    # it replaces on its own H^1: the maximum and argmax bit for bit
    # (gnn_aggregate_fwd_max), the logits from the same bf16 operands
    seed = 2 * f0 + f1 + n_out + n_dst
    blk, nrm, x_self, m1, w1, w2, b1, b2, labels = _two_layer_inputs(oracle.SAGE, f0, f1, n_out, n_dst, fanout, seed)
    h1 = oracle.update_fwd(x_self, m1, w1, b1, True, oracle.BF16, oracle.BF16)
    agg2, arg2 = oracle.aggregate_fwd_max(blk, h1, oracle.BF16)
    logits = oracle.update_fwd(h1[:blk.n_dst], agg2, w2, b2, False, oracle.BF16, oracle.F32)
    loss, g = oracle.softmax_ce(logits, labels[blk.src_ids[:blk.n_dst]])

    db = upload_block(blk)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)  # noqa
    xs_d, m1_d = from_np_act(x_self), from_np_act(m1)
    wt1, wt2 = _shadow(w1), _shadow(w2)
    out = dict(h1=torch.empty((blk.n_src, f1), dtype=torch.bfloat16, device=DEV),
               agg=torch.empty((blk.n_dst, f1), dtype=torch.bfloat16, device=DEV),
               arg=torch.full((blk.n_dst, f1), -7, dtype=torch.int32, device=DEV),
               logits=torch.empty((blk.n_dst, n_out), device=DEV), g=torch.empty((blk.n_dst, n_out), device=DEV),
               rl=torch.empty(blk.n_dst, device=DEV), da=torch.empty((blk.n_dst, w2.shape[0]), device=DEV))
    lab_d = d(labels)
    print(f"[two_layer_fwd_max] f0={f0} f1={f1} n_out={n_out} n_dst={n_dst} fanout={fanout} bound={bound}",
          flush=True)
    gnn.two_layer_fwd_max(db, bound, xs_d, m1_d, wt1, d(b1), out["h1"], wt2, d(b2), out["agg"], out["arg"],
                          out["logits"], lab_d, blk.n_dst, out["g"], out["rl"], out["da"])
    torch.cuda.synchronize()
    assert relerr(oracle.to_float64(to_np_act(out["h1"])), oracle.to_float64(h1)) <= 8e-3
    assert relerr(oracle.to_float64(to_np_act(out["agg"])), oracle.to_float64(agg2)) <= 8e-3
    agree = float(np.mean(out["arg"].cpu().numpy() == arg2))
    assert agree >= 0.999, agree  # near-ties may fall the other way on H^1's last bits
    assert relerr(out["logits"].cpu().numpy(), logits) <= 8e-3
    assert relerr(out["g"].cpu().numpy(), g) <= 2e-2
    assert abs(float(out["rl"].mean()) - loss) <= 2e-2 * max(1.0, abs(loss))
    # the input gradient from the kernel's own G and operands
    _, _, da = oracle.update_bwd(to_np_act(out["h1"])[:blk.n_dst], to_np_act(out["agg"]), w2,
                                 out["g"].cpu().numpy(), oracle.BF16, True)
    assert relerr(out["da"].cpu().numpy(), da) <= 1e-5

    # the calls it replaces, on its own values where they are inputs
    h1_ref = torch.empty_like(out["h1"])
    gnn.update_fwd(xs_d, m1_d, d(w1), d(b1), h1_ref, True, gnn.GNN_BF16, wt=wt1)
    agg_ref, arg_ref = torch.empty_like(out["agg"]), torch.empty_like(out["arg"])
    gnn.aggregate_fwd_max(db, out["h1"], agg_ref, arg_ref)
    lg_ref = torch.empty_like(out["logits"])
    gnn.update_fwd(out["h1"][:blk.n_dst], out["agg"], d(w2), d(b2), lg_ref, False, gnn.GNN_BF16, wt=wt2)
    torch.cuda.synchronize()
    assert torch.equal(out["h1"].view(torch.int16), h1_ref.view(torch.int16))
    assert torch.equal(out["agg"].view(torch.int16), agg_ref.view(torch.int16))
    assert torch.equal(out["arg"], arg_ref)
    assert torch.equal(out["logits"].view(torch.int32), lg_ref.view(torch.int32))


def test_two_layer_fwd_max_rejects_unsupported():
    blk, nrm, x_self, m1, w1, w2, b1, b2, labels = _two_layer_inputs(oracle.SAGE, 32, 64, 8, 50, 4, 7)
    db = upload_block(blk)
    lab = torch.from_numpy(labels).to(DEV)

    def call(n_out, arg):
        gnn.two_layer_fwd_max(db, 4, from_np_act(x_self), from_np_act(m1),
                              torch.zeros((64, 64), dtype=torch.bfloat16, device=DEV), None,
                              torch.empty((blk.n_src, 64), dtype=torch.bfloat16, device=DEV),
                              torch.zeros((n_out, 128), dtype=torch.bfloat16, device=DEV), None,
                              torch.empty((blk.n_dst, 64), dtype=torch.bfloat16, device=DEV), arg,
                              torch.empty((blk.n_dst, n_out), device=DEV), lab, blk.n_dst,
                              torch.empty((blk.n_dst, n_out), device=DEV), torch.empty(blk.n_dst, device=DEV))

    arg = torch.empty((blk.n_dst * 64 + 4,), dtype=torch.int32, device=DEV)
    call(48, arg[:blk.n_dst * 64].view(blk.n_dst, 64))
    torch.cuda.synchronize()
    for n_out, a in ((49, arg[:blk.n_dst * 64].view(blk.n_dst, 64)),        # classes over 48
                     (8, arg[1:blk.n_dst * 64 + 1].view(blk.n_dst, 64))):   # table not 16-byte aligned
        with pytest.raises(gnn.GnnError) as e:
            call(n_out, a)
        assert e.value.code == gnn.GNN_EUNSUPPORTED


@pytest.mark.parametrize("f0,f1,n_out,n_dst,fanout,bound,n", [c + (None,) for c in TWO_CASES] +
                         [(100, 256, 47, 2048, 50, 50, 200_000)])
def test_two_layer_bwd_max_parity(f0, f1, n_out, n_dst, fanout, bound, n):
    # gnn_two_layer_bwd_max from gnn_two_layer_fwd_max's outputs: against the
    # oracle's own forward and backward chain (update, max aggregation with
    # its argmax, update, loss; then each layer's update backward and the max
    # aggregation backward), and bit for bit against gnn_aggregate_bwd_max +
    # gnn_update_bwd per layer on the same forward values.  Layers up to 128
    # wide are rejected, as for the sums.
    seed = 5 * f0 + f1 + n_out + n_dst
    blk, nrm, x_self, m1, w1, w2, b1, b2, labels = _two_layer_inputs(oracle.SAGE, f0, f1, n_out, n_dst, fanout, seed,
                                                                     n)
    db = upload_block(blk)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)  # noqa
    xs_d, m1_d = from_np_act(x_self), from_np_act(m1)
    K1, K2 = w1.shape[0], w2.shape[0]
    h1 = torch.empty((blk.n_src, f1), dtype=torch.bfloat16, device=DEV)
    agg = torch.empty((blk.n_dst, f1), dtype=torch.bfloat16, device=DEV)
    arg = torch.empty((blk.n_dst, f1), dtype=torch.int32, device=DEV)
    g = torch.empty((blk.n_dst, n_out), device=DEV)
    da = torch.empty((blk.n_dst, K2), device=DEV)
    gnn.two_layer_fwd_max(db, bound, xs_d, m1_d, _shadow(w1), d(b1), h1, _shadow(w2), d(b2), agg, arg,
                          torch.empty((blk.n_dst, n_out), device=DEV), d(labels), blk.n_dst, g,
                          torch.empty(blk.n_dst, device=DEV), da)
    m1_rows = torch.tensor([blk.n_src], dtype=torch.int64, device=DEV)
    out = dict(dw1=torch.empty((K1, f1), device=DEV), db1=torch.empty(f1, device=DEV),
               dw2=torch.empty((K2, n_out), device=DEV), db2=torch.empty(n_out, device=DEV))
    print(f"[two_layer_bwd_max] f0={f0} f1={f1} n_out={n_out} n_dst={n_dst} fanout={fanout}", flush=True)
    args = (db, xs_d, m1_d, m1_rows, blk.n_src, h1, agg, arg, da, g, out["dw1"], out["db1"], out["dw2"], out["db2"])
    if f1 <= 128:
        with pytest.raises(gnn.GnnError) as e:
            gnn.two_layer_bwd_max(*args)
        assert e.value.code == gnn.GNN_EUNSUPPORTED
        return
    gnn.two_layer_bwd_max(*args)
    torch.cuda.synchronize()
    # the oracle's chain from the same inputs
    h1_o = oracle.update_fwd(x_self, m1, w1, b1, True, oracle.BF16, oracle.BF16)
    agg_o, arg_o = oracle.aggregate_fwd_max(blk, h1_o, oracle.BF16)
    lg_o = oracle.update_fwd(h1_o[:blk.n_dst], agg_o, w2, b2, False, oracle.BF16, oracle.F32)
    _, g_o = oracle.softmax_ce(lg_o, labels[blk.src_ids[:blk.n_dst]])
    dw2_o, db2_o, da_o = oracle.update_bwd(h1_o[:blk.n_dst], agg_o, w2, g_o, oracle.BF16, True)
    g1_o = oracle.aggregate_bwd_max(blk, arg_o, da_o, f1, h1_o, oracle.F32)
    dw1_o, db1_o, _ = oracle.update_bwd(x_self, m1, w1, g1_o, oracle.BF16, False)
    assert relerr(out["dw2"].cpu().numpy(), dw2_o) <= 2e-2
    assert relerr(out["db2"].cpu().numpy(), db2_o) <= 2e-2
    assert relerr(out["dw1"].cpu().numpy(), dw1_o) <= 2e-2
    assert relerr(out["db1"].cpu().numpy(), db1_o) <= 2e-2

    # the calls it replaces, on the same forward values
    g1_d = torch.empty((blk.n_src, f1), device=DEV)
    gnn.aggregate_bwd_max(db, arg, da, f1, g1_d, h_below=h1)
    ref = {k: torch.empty_like(v) for k, v in out.items()}
    gnn.update_bwd(xs_d, m1_d, d(w1), g1_d, ref["dw1"], ref["db1"], None, gnn.GNN_BF16)
    gnn.update_bwd(h1[:blk.n_dst], agg, d(w2), g, ref["dw2"], ref["db2"], None, gnn.GNN_BF16)
    torch.cuda.synchronize()
    for k in out:
        assert torch.equal(out[k].view(torch.int32), ref[k].view(torch.int32)), k


def test_two_layer_fwd_rejects_unsupported_shapes():
    blk, nrm, x_self, m1, w1, w2, b1, b2, labels = _two_layer_inputs(oracle.SAGE, 32, 64, 8, 50, 4, 7)
    db = upload_block(blk)
    lab = torch.from_numpy(labels).to(DEV)

    def call(f1, n_out, k1_rows=None):
        wt1 = torch.zeros((f1, 64), dtype=torch.bfloat16, device=DEV)
        wt2 = torch.zeros((n_out, 2 * f1), dtype=torch.bfloat16, device=DEV)
        gnn.two_layer_fwd(db, oracle.SAGE, 4, from_np_act(x_self), from_np_act(m1), wt1, None,
                          torch.empty((blk.n_src, f1), dtype=torch.bfloat16, device=DEV), wt2, None,
                          torch.empty((blk.n_dst, f1), dtype=torch.bfloat16, device=DEV),
                          torch.empty((blk.n_dst, n_out), device=DEV), lab, blk.n_dst,
                          torch.empty((blk.n_dst, n_out), device=DEV), torch.empty(blk.n_dst, device=DEV))

    call(64, 48)  # the largest class count GraphSAGE's staging holds
    torch.cuda.synchronize()
    for f1, n_out in ((512, 8), (64, 49), (60, 8)):  # f1 over 256, classes over 48, f1 % 8 != 0
        with pytest.raises(gnn.GnnError) as e:
            call(f1, n_out)
        assert e.value.code == gnn.GNN_EUNSUPPORTED, (f1, n_out)


# ---------------------------------------------------------------------------
# update GEMMs
# ---------------------------------------------------------------------------

SHAPES = [(1, 4, 1), (77, 3, 47), (300, 100, 256), (1000, 256, 47), (530, 16, 8), (129, 128, 130)]


@pytest.mark.parametrize("sage,m,cap,ke,n,relu", [(True, 700, 1000, 768, 1024, True),
                                                   (False, 513, 513, 512, 520, True),
                                                   (True, 2000, 2048, 256, 512, True),
                                                   (True, 300, 300, 1024, 640, False),
                                                   (False, 1, 256, 1536, 1024, True)])
def test_update_fwd_wide_layer_matches_oracle(sage, m, cap, ke, n, relu):
    # wide layers (K and n_out >= 512) with the bf16 W^T take the 256 x 256
    # matrix-core tiles: ragged rows below the capacity, a last column tile
    # of 8 columns, the fp32 logits epilogue, a single row
    rng = np.random.default_rng(m + ke + n + sage)
    a_s = oracle.f32_to_bf16_bits(rng.standard_normal((cap, ke)).astype(np.float32))
    a_n = oracle.f32_to_bf16_bits(rng.standard_normal((cap, ke)).astype(np.float32)) if sage else None
    K = (2 if sage else 1) * ke
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    b = (0.1 * rng.standard_normal(n)).astype(np.float32)
    ocode = oracle.BF16 if relu else oracle.F32
    want = oracle.update_fwd(a_s[:m], a_n[:m] if sage else None, w, b, relu, oracle.BF16, ocode)
    wt = torch.from_numpy(np.ascontiguousarray(w.T)).to(DEV).to(torch.bfloat16)
    out = torch.full((cap, n), float("nan"), dtype=torch.bfloat16 if relu else torch.float32, device=DEV)
    m_dev = torch.tensor([m], dtype=torch.int64, device=DEV)
    print(f"[update_fwd wide] sage={sage} m={m} cap={cap} ke={ke} n={n} relu={relu}", flush=True)
    gnn.update_fwd(from_np_act(a_s), from_np_act(a_n) if sage else None, from_np_act(w), from_np_act(b), out, relu,
                   gnn.GNN_BF16, m_dev=m_dev, cap_m=cap, wt=wt)
    torch.cuda.synchronize()
    got = oracle.to_float64(to_np_act(out))
    assert relerr(got[:m], oracle.to_float64(want)) <= 8e-3
    assert np.isnan(got[m:]).all()  # rows past the device count are not written


@pytest.mark.parametrize("m,cap,ke", [(16384, 16384, 512), (13300, 13312, 512), (3239, 26624, 768),
                                      (2200, 26624, 768), (1000, 26624, 512), (6000, 26624, 768)])
def test_update_fwd_wide_layer_tile_heights(m, cap, ke):
    # n_out = 1,024.  16,384 rows (K = 1,024) fill exactly one round of 256
    # tiles of 256 rows (taken over 224-row tiles, which would need two);
    # 13,312 rows take 224-row tiles (60 x 4 in one round).  With the row
    # count on the device far below the capacity (26,624 rows: 476 tiles of
    # 224 rows), the few tiles holding rows split their reduction: 60 tiles
    # of K = 1,536 in 4 splits (the host-table model's first layer at 3,239
    # rows), 40 tiles in 6, 20 tiles of K = 1,024 in 8; 6,000 rows (108
    # tiles) do not split, though the summing kernel runs.  The layer is
    # row-wise, so 64 sampled rows and the last rows are checked against
    # the oracle run on just those rows.
    rng = np.random.default_rng(cap + m)
    n = 1024
    a_s = _act(rng, cap, ke, oracle.BF16)
    a_n = _act(rng, cap, ke, oracle.BF16)
    K = 2 * ke
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    b = (0.1 * rng.standard_normal(n)).astype(np.float32)
    wt = torch.from_numpy(np.ascontiguousarray(w.T)).to(DEV).to(torch.bfloat16)
    out = torch.full((cap, n), float("nan"), dtype=torch.bfloat16, device=DEV)
    m_dev = torch.tensor([m], dtype=torch.int64, device=DEV)
    print(f"[update_fwd wide tiles] m={m} cap={cap} k_each={ke}", flush=True)
    gnn.update_fwd(from_np_act(a_s), from_np_act(a_n), from_np_act(w), from_np_act(b), out, True, gnn.GNN_BF16,
                   m_dev=m_dev, cap_m=cap, wt=wt)
    torch.cuda.synchronize()
    got = oracle.to_float64(to_np_act(out))
    rows = np.unique(np.concatenate([rng.choice(m, 64, replace=False), np.arange(m - 40, m)]))
    want = oracle.update_fwd(a_s[rows], a_n[rows], w, b, True, oracle.BF16, oracle.BF16)
    assert relerr(got[rows], oracle.to_float64(want)) <= 8e-3
    assert not np.isnan(got[:m]).any() and np.isnan(got[m:]).all()


@pytest.mark.parametrize("m,ke,n", SHAPES)
@pytest.mark.parametrize("sage", [True, False])
@pytest.mark.parametrize("code", [oracle.F32, oracle.BF16])
def test_update_fwd_parity(m, ke, n, sage, code):
    rng = np.random.default_rng(m + ke + n)
    a_s = _act(rng, m, ke, code)
    a_n = _act(rng, m, ke, code) if sage else None
    K = 2 * ke if sage else ke
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    b = rng.standard_normal(n).astype(np.float32)
    for relu, ocode in ((True, code), (False, oracle.F32)):
        want = oracle.update_fwd(a_s, a_n, w, b, relu, code, ocode)
        out = torch.empty((m, n), dtype=torch.bfloat16 if ocode == oracle.BF16 else torch.float32, device=DEV)
        gnn.update_fwd(from_np_act(a_s), from_np_act(a_n) if sage else None, from_np_act(w), from_np_act(b), out,
                       relu, code)
        err = relerr(oracle.to_float64(to_np_act(out)), oracle.to_float64(want))
        assert err <= (1e-5 if code == oracle.F32 else 8e-3), (relu, err)


@pytest.mark.parametrize("code", [oracle.F32, oracle.BF16])
def test_update_fwd_split_reduction_and_workspace_reuse(code):
    # a long reduction over few output tiles is split across workgroups and
    # finished by a second kernel; a second call on the same workspace
    # (fewer rows, other data) must be as exact as the first
    rng = np.random.default_rng(7)
    ke, n, cap = 1024, 153, 1024
    K = 2 * ke
    nb = gnn._sz()
    gnn._check(gnn.lib().gnn_update_fwd_workspace_size(K, n, cap, code, gnn.ctypes.byref(nb)))
    assert nb.value > 0  # this shape takes the split path
    ws = torch.full((nb.value,), 0xFF, dtype=torch.uint8, device=DEV)  # no zero-fill needed
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    b = rng.standard_normal(n).astype(np.float32)
    tdt = torch.bfloat16 if code == oracle.BF16 else torch.float32
    for m in (1024, 333):
        a_s = _act(rng, m, ke, code)
        a_n = _act(rng, m, ke, code)
        want = oracle.update_fwd(a_s, a_n, w, b, True, code, code)
        out = torch.full((cap, n), 3.0, dtype=tdt, device=DEV)
        m_dev = torch.tensor([m], dtype=torch.int64, device=DEV)
        a_s_d = torch.zeros((cap, ke), dtype=tdt, device=DEV)
        a_n_d = torch.zeros((cap, ke), dtype=tdt, device=DEV)
        a_s_d[:m] = from_np_act(a_s)
        a_n_d[:m] = from_np_act(a_n)
        gnn.update_fwd(a_s_d, a_n_d, from_np_act(w), from_np_act(b), out, True, code, m_dev=m_dev, cap_m=cap, ws=ws)
        got = oracle.to_float64(to_np_act(out))
        assert relerr(got[:m], oracle.to_float64(want)) <= (1e-5 if code == oracle.F32 else 8e-3)
        assert np.all(got[m:] == 3.0)  # rows past the device count untouched


def test_update_workspaces_shared_across_shapes():
    # one forward and one backward workspace serve GEMMs of different shapes
    # in turn (as the layers of a training step do), twice over
    rng = np.random.default_rng(9)
    shapes = [(3000, 100, 256, True), (512, 256, 47, True), (3000, 100, 256, True), (512, 256, 47, True)]
    nb = gnn._sz()
    fw, bw = 0, 0
    for m, ke, n, sage in shapes:
        K = 2 * ke if sage else ke
        gnn._check(gnn.lib().gnn_update_fwd_workspace_size(K, n, m, gnn.GNN_BF16, gnn.ctypes.byref(nb)))
        fw = max(fw, nb.value)
        gnn._check(gnn.lib().gnn_update_bwd_workspace_size(K, n, m, gnn.GNN_BF16, gnn.ctypes.byref(nb)))
        bw = max(bw, nb.value)
    ws_f = torch.zeros(fw, dtype=torch.uint8, device=DEV)
    ws_b = torch.zeros(bw, dtype=torch.uint8, device=DEV)
    for m, ke, n, sage in shapes:
        a_s = _act(rng, m, ke, oracle.BF16)
        a_n = _act(rng, m, ke, oracle.BF16)
        K = 2 * ke
        w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
        g = rng.standard_normal((m, n)).astype(np.float32)
        out = torch.empty((m, n), dtype=torch.float32, device=DEV)
        gnn.update_fwd(from_np_act(a_s), from_np_act(a_n), from_np_act(w), None, out, False, gnn.GNN_BF16, ws=ws_f)
        assert relerr(out.cpu().numpy(), oracle.update_fwd(a_s, a_n, w, None, False, oracle.BF16, oracle.F32)) <= 8e-3
        dw_w, db_w, da_w = oracle.update_bwd(a_s, a_n, w, g, oracle.BF16, want_da=True)
        dw = torch.empty((K, n), device=DEV)
        db = torch.empty(n, device=DEV)
        da = torch.empty((m, K), device=DEV)
        gnn.update_bwd(from_np_act(a_s), from_np_act(a_n), from_np_act(w), from_np_act(g), dw, db, da, gnn.GNN_BF16,
                       ws=ws_b)
        assert relerr(dw.cpu().numpy(), dw_w) <= 8e-3 and relerr(db.cpu().numpy(), db_w) <= 1e-5
        assert relerr(da.cpu().numpy(), da_w) <= 8e-3


@pytest.mark.parametrize("code", [oracle.F32, oracle.BF16])
def test_update_fwd_without_workspace(code):
    rng = np.random.default_rng(8)
    m, ke, n = 700, 100, 256
    a_s = _act(rng, m, ke, code)
    a_n = _act(rng, m, ke, code)
    w = (rng.standard_normal((2 * ke, n)) / 14).astype(np.float32)
    want = oracle.update_fwd(a_s, a_n, w, None, True, code, code)
    out = torch.empty((m, n), dtype=torch.bfloat16 if code == oracle.BF16 else torch.float32, device=DEV)
    gnn.update_fwd(from_np_act(a_s), from_np_act(a_n), from_np_act(w), None, out, True, code, split=False)
    assert relerr(oracle.to_float64(to_np_act(out)), oracle.to_float64(want)) <= (1e-5 if code == oracle.F32 else 8e-3)


def test_update_fwd_device_row_count():
    rng = np.random.default_rng(1)
    m, ke, n = 500, 64, 96
    a = rng.standard_normal((m, ke)).astype(np.float32)
    w = rng.standard_normal((ke, n)).astype(np.float32)
    out = torch.full((m, n), 7.0, device=DEV)
    m_dev = torch.tensor([201], dtype=torch.int64, device=DEV)
    gnn.update_fwd(from_np_act(a), None, from_np_act(w), None, out, False, gnn.GNN_F32, m_dev=m_dev, cap_m=m)
    o = out.cpu().numpy()
    want = oracle.update_fwd(a[:201], None, w, None, False, oracle.F32, oracle.F32)
    assert relerr(o[:201], want) <= 1e-5 and np.all(o[201:] == 7.0)


@pytest.mark.parametrize("m,ke,n", SHAPES + [(26624 // 8, 100, 256), (700, 768, 600)])  # last: the wide-layer dW plan
@pytest.mark.parametrize("sage", [True, False])
@pytest.mark.parametrize("code", [oracle.F32, oracle.BF16])
def test_update_bwd_parity(m, ke, n, sage, code):
    rng = np.random.default_rng(m * 3 + ke + n)
    a_s = _act(rng, m, ke, code)
    a_n = _act(rng, m, ke, code) if sage else None
    K = 2 * ke if sage else ke
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    g = rng.standard_normal((m, n)).astype(np.float32)
    dw_w, db_w, da_w = oracle.update_bwd(a_s, a_n, w, g, code, want_da=True)
    dw = torch.empty((K, n), device=DEV)
    db = torch.empty(n, device=DEV)
    da = torch.empty((m, K), device=DEV)
    gnn.update_bwd(from_np_act(a_s), from_np_act(a_n) if sage else None, from_np_act(w), from_np_act(g), dw, db, da,
                   code)
    tol = 1e-5 if code == oracle.F32 else 8e-3
    assert relerr(dw.cpu().numpy(), dw_w) <= tol
    assert relerr(db.cpu().numpy(), db_w) <= 1e-5
    assert relerr(da.cpu().numpy(), da_w) <= tol


@pytest.mark.parametrize("sage,m,cap,ke,n,want_da,want_db", [
    (True, 1664, 1664, 768, 1024, True, True),   # the host-table first layer at 1/16 of its 26,624 rows
    (True, 1000, 4096, 768, 520, True, True),    # device rows far below capacity (most splits empty); n_out % 32 != 0
    (False, 777, 800, 600, 512, True, False),    # GCN with K = 600: the last K tile runs past K; no db
    (True, 300, 300, 512, 1024, False, True),    # dW alone (a first layer)
    (False, 1, 64, 512, 512, True, True),        # a single row
])
def test_update_bwd_wide_layer_matches_oracle(sage, m, cap, ke, n, want_da, want_db):
    # wide layers (K and n_out >= 512, bf16) take the 256 x 256 matrix-core
    # tiles: dA with G converted on its way to LDS, dW from transposing LDS
    # reads with its rows split across workgroups.  Rows past the device
    # count hold NaN and must reach no output; the workspace starts as NaN
    # bit patterns; a second call must repeat the first bit for bit.
    rng = np.random.default_rng(m + ke + n + sage)
    a_s = _act(rng, cap, ke, oracle.BF16)
    a_n = _act(rng, cap, ke, oracle.BF16) if sage else None
    K = (2 if sage else 1) * ke
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    g = rng.standard_normal((cap, n)).astype(np.float32)
    dw_w, db_w, da_w = oracle.update_bwd(a_s[:m], a_n[:m] if sage else None, w, g[:m], oracle.BF16, want_da=True)
    a_s[m:] = 0x7FC0  # bf16 NaN
    if sage:
        a_n[m:] = 0x7FC0
    g[m:] = np.nan
    nb = gnn._sz()
    gnn._check(gnn.lib().gnn_update_bwd_workspace_size(K, n, cap, gnn.GNN_BF16, gnn.ctypes.byref(nb)))
    ws = torch.full((nb.value,), 0xFF, dtype=torch.uint8, device=DEV)
    m_dev = torch.tensor([m], dtype=torch.int64, device=DEV)
    args = (from_np_act(a_s), from_np_act(a_n) if sage else None, from_np_act(w), from_np_act(g))
    print(f"[update_bwd wide] sage={sage} m={m} cap={cap} ke={ke} n={n} da={want_da} db={want_db}", flush=True)
    outs = []
    for _ in range(2):
        dw = torch.full((K, n), float("nan"), device=DEV)
        db = torch.full((n,), float("nan"), device=DEV) if want_db else None
        da = torch.full((cap, K), 5.0, device=DEV) if want_da else None
        gnn.update_bwd(*args, dw, db, da, gnn.GNN_BF16, m_dev=m_dev, cap_m=cap, ws=ws)
        torch.cuda.synchronize()
        outs.append([t.cpu() for t in (dw, db, da) if t is not None])
    dw, *rest = outs[0]
    assert relerr(dw.numpy(), dw_w) <= 8e-3
    if want_db:
        assert relerr(rest.pop(0).numpy(), db_w) <= 1e-5
    if want_da:
        da = rest.pop(0).numpy()
        assert relerr(da[:m], da_w) <= 8e-3
        assert np.all(da[m:] == 5.0)  # rows past the device count untouched
    for x, y in zip(outs[0], outs[1]):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))


# ---------------------------------------------------------------------------
# loss and optimizer
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("b,c", [(1, 8), (256, 8), (1024, 47), (1000, 172), (33, 153)])
def test_softmax_ce_parity(b, c):
    rng = np.random.default_rng(b + c)
    z = (rng.standard_normal((b, c)) * 4).astype(np.float32)
    labels = rng.integers(0, c, size=5000).astype(np.int64)
    targets = rng.choice(5000, size=b, replace=False).astype(np.int64)
    loss_w, g_w = oracle.softmax_ce(z, labels[targets])
    g = torch.empty((b, c), device=DEV)
    loss = torch.empty(1, device=DEV)
    gnn.softmax_ce(from_np_act(z), from_np_act(labels), from_np_act(targets), g, loss)
    assert abs(loss.item() - loss_w) <= 1e-5 * max(1, abs(loss_w))
    assert relerr(g.cpu().numpy(), g_w) <= 1e-5


def test_sgd_parity():
    rng = np.random.default_rng(0)
    w = rng.standard_normal(10_001).astype(np.float32)
    dw = rng.standard_normal(10_001).astype(np.float32)
    wd = from_np_act(w)
    gnn.sgd(wd, from_np_act(dw), 0.05)
    assert relerr(wd.cpu().numpy(), oracle.sgd(w, dw, 0.05)) <= 1e-7


# ---------------------------------------------------------------------------
# whole training step
# ---------------------------------------------------------------------------

def _step_case(kind, precision, dims, fanouts, n, m, batch, graph="er", steps=1, seed=0):
    if graph == "er":
        rowptr, col = workloads.er_graph(n, m, seed=seed)
    else:
        rowptr, col = workloads.rmat_graph(n, m, seed=seed)
    table = workloads.features(n, dims[0], seed=seed)
    labels = workloads.labels(n, dims[-1], seed=seed)
    perm = workloads.target_batches(n, batch, seed=seed)
    L = len(dims) - 1
    sage = kind != gnn.GNN_AGG_GCN_SYM  # A = [h_self || aggregation]
    ws = [workloads.glorot((2 if sage else 1) * dims[l], dims[l + 1], seed, l) for l in range(L)]
    bs = [torch.zeros(dims[l + 1]) for l in range(L)]
    g = gnn.DeviceGraph(rowptr.to(DEV), col.to(DEV))
    nrm = gnn.gcn_norm(g)
    tr = gnn.Trainer(kind, dims, fanouts, precision, n, batch, ws, bs, device=DEV)
    okind = {gnn.GNN_AGG_SAGE_MEAN: oracle.SAGE, gnn.GNN_AGG_GCN_SYM: oracle.GCN,
             gnn.GNN_AGG_SAGE_MAX: oracle.SAGE_MAX}[kind]
    oprec = oracle.F32 if precision == gnn.GNN_F32 else oracle.BF16
    rp_h, col_h, nrm_h = rowptr.numpy(), col.numpy(), oracle.gcn_norm(rowptr.numpy())
    w_ref = [w.numpy() for w in ws]
    b_ref = [b.numpy() for b in bs]
    t_d, lab_d = table.to(DEV), labels.to(DEV)
    for s in range(steps):
        targets = workloads.targets_for_step(perm, batch, s)
        tr.step(g, t_d, lab_d, targets.to(DEV), seed=seed, step=s, lr=0.05, gcn_norm_t=nrm)
        torch.cuda.synchronize()
        cfg = oracle.StepConfig(kind=okind, dims=dims, fanouts=fanouts, precision=oprec, seed=seed, step=s, lr=0.05)
        ref = oracle.train_step(rp_h, col_h, nrm_h, table.numpy(), labels.numpy(), targets.numpy(), w_ref, b_ref, cfg)
        yield tr, ref, oprec
        w_ref = [w.cpu().numpy() for w in tr.w]   # continue from the GPU's weights
        b_ref = [b.cpu().numpy() for b in tr.b]


def _check_step(tr, ref, oprec, L):
    tol = TOL[oprec]
    for h in range(1, L + 1):
        got = tr.block_view(h)
        want = ref["blocks"][h - 1]
        assert np.array_equal(got["src_ids"], want.src_ids)
        assert np.array_equal(got["rowptr"], want.rowptr)
        assert np.array_equal(got["col"], want.col)
        if h < L:
            assert np.array_equal(got["cscptr"], want.cscptr) and np.array_equal(got["cscrow"], want.cscrow)
    assert int(tr.edges.item()) == ref["edges"]
    assert abs(tr.loss.item() - ref["loss"]) <= tol * max(1.0, abs(ref["loss"]))
    for l in range(1, L + 1):
        assert relerr(tr.dw[l - 1].cpu().numpy(), ref["dW"][l]) <= tol, ("dW", l)
        assert relerr(tr.db[l - 1].cpu().numpy(), ref["dB"][l]) <= tol, ("dB", l)
        assert relerr(tr.w[l - 1].cpu().numpy(), ref["new_w"][l - 1]) <= tol, ("W", l)


def test_train_step_tiny_gcn_fp32():
    dims, fan = (32, 16, 8), (5, 5)
    for tr, ref, oprec in _step_case(gnn.GNN_AGG_GCN_SYM, gnn.GNN_F32, dims, fan, 10_000, 50_000, 256, steps=3):
        _check_step(tr, ref, oprec, 2)
        # the gathered features are bit-exact
        x0 = tr.tensor("x0", 0, ref["x0"].shape[0], 32, torch.float32).cpu().numpy()
        assert np.array_equal(x0, ref["x0"])


@pytest.mark.parametrize("kind", [gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_AGG_GCN_SYM, gnn.GNN_AGG_SAGE_MAX])
def test_train_step_rmat_bf16(kind):
    dims, fan = (100, 256, 47), (25, 10)
    for tr, ref, oprec in _step_case(kind, gnn.GNN_BF16, dims, fan, 30_000, 400_000, 512, graph="rmat", steps=2):
        _check_step(tr, ref, oprec, 2)
        if kind == gnn.GNN_AGG_SAGE_MAX:
            _check_max_tables(tr, ref, 2)


def _check_max_tables(tr, ref, L):
    # the argmax tables the backward reads: each is the oracle's, except
    # where a near-tie falls the other way on activations that differ in
    # their last bit (the oracle sums the update in fp64); those must stay
    # rare
    for l in range(2, L + 1):
        want = ref["ARG"][l]
        got = tr.tensor("argmax", l, want.shape[0], want.shape[1], torch.int32).cpu().numpy()
        agree = float(np.mean(got == want))
        print(f"[max step] layer {l}: argmax agreement {agree:.6f}", flush=True)
        assert agree >= 0.999, (l, agree)
    assert tr.layout.argmax[1] == 0


def test_train_step_max_fp32_three_layers():
    # GraphSAGE-max at depth 3 in fp32: two layers keep argmax tables
    dims, fan = (32, 24, 16, 8), (6, 4, 3)
    for tr, ref, oprec in _step_case(gnn.GNN_AGG_SAGE_MAX, gnn.GNN_F32, dims, fan, 10_000, 60_000, 256, steps=2):
        _check_step(tr, ref, oprec, 3)
        _check_max_tables(tr, ref, 3)


@pytest.mark.parametrize("kind", [gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_AGG_GCN_SYM])
def test_fused_loading_equals_gather_then_aggregate(kind):
    # fp32 table in device memory, bf16 layers: the prepare stage sums layer
    # 1's neighbours straight from the table and gathers X' only for the
    # destination rows.  Its aggregation must equal, bit for bit, a full
    # gather (bf16 round to nearest even) followed by the aggregation kernel
    # over X' on the same block; the gathered destination rows must equal
    # the oracle's X'.
    dims, fan, n, m, batch = (100, 256, 47), (25, 10), 30_000, 400_000, 512
    rowptr, col = workloads.rmat_graph(n, m, seed=3)
    table = workloads.features(n, dims[0], seed=3)
    labels = workloads.labels(n, dims[-1], seed=3)
    targets = workloads.targets_for_step(workloads.target_batches(n, batch, seed=3), batch, 0)
    sage = kind == gnn.GNN_AGG_SAGE_MEAN
    ws = [workloads.glorot((2 if sage else 1) * dims[l], dims[l + 1], 3, l) for l in range(2)]
    bs = [torch.zeros(dims[l + 1]) for l in range(2)]
    g = gnn.DeviceGraph(rowptr.to(DEV), col.to(DEV))
    nrm = gnn.gcn_norm(g)
    tr = gnn.Trainer(kind, dims, fan, gnn.GNN_BF16, n, batch, ws, bs, device=DEV)
    t_d = table.to(DEV)
    print(f"[fused loading] kind={kind}", flush=True)
    tr.step(g, t_d, labels.to(DEV), targets.to(DEV), seed=3, step=0, lr=0.05, gcn_norm_t=nrm)
    torch.cuda.synchronize()
    okind = oracle.GCN if kind == gnn.GNN_AGG_GCN_SYM else oracle.SAGE
    cfg = oracle.StepConfig(kind=okind, dims=dims, fanouts=fan, precision=oracle.BF16, seed=3, step=0, lr=0.05)
    nrm_h = oracle.gcn_norm(rowptr.numpy())
    ref = oracle.train_step(rowptr.numpy(), col.numpy(), nrm_h, table.numpy(), labels.numpy(), targets.numpy(),
                            [w.numpy() for w in ws], [b.numpy() for b in bs], cfg)
    blk = ref["blocks"][1]  # hop 2: layer 1's block
    got_blk = tr.block_view(2)
    assert np.array_equal(got_blk["src_ids"], blk.src_ids) and np.array_equal(got_blk["col"], blk.col)
    x0_dst = tr.tensor("x0", 0, blk.n_dst, dims[0], torch.bfloat16).cpu().view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(x0_dst, ref["x0"][:blk.n_dst])
    db = upload_block(blk, src_norm=nrm_h[blk.src_ids] if not sage else None)
    x0 = torch.empty((blk.n_src, dims[0]), dtype=torch.bfloat16, device=DEV)
    gnn.gather_features(t_d, db.src_ids, x0)
    want = torch.empty((blk.n_dst, dims[0]), dtype=torch.bfloat16, device=DEV)
    gnn.aggregate_fwd(db, kind, x0, want)
    got = tr.tensor("agg", 1, blk.n_dst, dims[0], torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))


def test_train_step_three_layer_sage_bf16():
    dims, fan = (128, 256, 256, 172), (15, 10, 5)
    for tr, ref, oprec in _step_case(gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_BF16, dims, fan, 40_000, 500_000, 256,
                                     graph="rmat"):
        _check_step(tr, ref, oprec, 3)


def test_train_step_is_bitwise_reproducible():
    dims, fan = (100, 256, 47), (25, 10)
    outs = []
    for _ in range(2):
        for tr, ref, _o in _step_case(gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_BF16, dims, fan, 30_000, 400_000, 512,
                                      graph="rmat"):
            outs.append([t.cpu().clone() for t in tr.w + tr.b] + [tr.loss.cpu().clone()])
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))


# ---------------------------------------------------------------------------
# bf16 W^T shadows
# ---------------------------------------------------------------------------

def _shadow_bits(w: torch.Tensor) -> np.ndarray:
    return oracle.f32_to_bf16_bits(np.ascontiguousarray(w.cpu().numpy().T))


def test_model_sync_shadow_is_rne_transpose():
    rng = np.random.default_rng(5)
    dims = (100, 256, 47)
    ws = [torch.from_numpy(rng.standard_normal((2 * dims[l], dims[l + 1])).astype(np.float32)) for l in range(2)]
    ws[0][0, :4] = torch.tensor([float("nan"), float("inf"), -0.0, 1.0 + 2.0 ** -8])  # NaN, inf, sign, tie
    bs = [torch.zeros(dims[l + 1]) for l in range(2)]
    tr = gnn.Trainer(gnn.GNN_AGG_SAGE_MEAN, dims, (25, 10), gnn.GNN_BF16, 1000, 64, ws, bs, device=DEV)
    torch.cuda.synchronize()
    for l in range(2):
        got = tr.wt[l].cpu().view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(got, _shadow_bits(tr.w[l]))


@pytest.mark.parametrize("kind,batch", [(gnn.GNN_AGG_SAGE_MEAN, 512), (gnn.GNN_AGG_SAGE_MEAN, 2048),
                                        (gnn.GNN_AGG_GCN_SYM, 2048)])
def test_train_step_keeps_shadows_and_matches_unshadowed_step(kind, batch):
    # the shadow gives the GEMMs the same bf16 operands as rounding W on load,
    # so a step with shadows is bitwise the step without them; after SGD the
    # shadows equal bf16(W_new^T).  With shadows a two-layer model takes the
    # two-layer forward and the folded backward, without them the per-layer
    # launches, so this also checks those bit for bit against each other; at
    # batch 2048 the folded backward's row splits hold several 128-row groups
    dims, fan, n, m = (100, 256, 47), (25, 10), 30_000, 400_000
    sage = kind == gnn.GNN_AGG_SAGE_MEAN
    rowptr, col = workloads.rmat_graph(n, m, seed=0)
    table = workloads.features(n, dims[0], seed=0).to(DEV)
    labels = workloads.labels(n, dims[-1], seed=0).to(DEV)
    perm = workloads.target_batches(n, batch, seed=0)
    ws = [workloads.glorot((2 if sage else 1) * dims[l], dims[l + 1], 0, l) for l in range(2)]
    bs = [torch.zeros(dims[l + 1]) for l in range(2)]
    g = gnn.DeviceGraph(rowptr.to(DEV), col.to(DEV))
    nrm = None if sage else gnn.gcn_norm(g)
    runs = []
    print(f"[shadows vs none] kind={kind} batch={batch}", flush=True)
    for shadows in (True, False):
        tr = gnn.Trainer(kind, dims, fan, gnn.GNN_BF16, n, batch, ws, bs, device=DEV, shadows=shadows)
        assert bool(tr.wt) == shadows
        for s in range(3):
            tr.step(g, table, labels, workloads.targets_for_step(perm, batch, s).to(DEV), seed=0, step=s, lr=0.05,
                    gcn_norm_t=nrm)
        torch.cuda.synchronize()
        if shadows:
            for l in range(2):
                got = tr.wt[l].cpu().view(torch.int16).numpy().view(np.uint16)
                assert np.array_equal(got, _shadow_bits(tr.w[l])), l
        runs.append([t.cpu().clone() for t in tr.w + tr.b + tr.dw] + [tr.loss.cpu().clone()])
    for a, b in zip(runs[0], runs[1]):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))


# ---------------------------------------------------------------------------
# two-stage step: prepare / compute, pipelined
# ---------------------------------------------------------------------------

def _pipeline_inputs(kind, dims, fanouts, n, m, batch, table_dtype=torch.float32, seed=0):
    rowptr, col = workloads.rmat_graph(n, m, seed=seed)
    table = workloads.features(n, dims[0], seed=seed, dtype=table_dtype)
    labels = workloads.labels(n, dims[-1], seed=seed).to(DEV)
    perm = workloads.target_batches(n, batch, seed=seed)
    L = len(dims) - 1
    sage = kind != gnn.GNN_AGG_GCN_SYM  # A = [h_self || aggregation]
    ws = [workloads.glorot((2 if sage else 1) * dims[l], dims[l + 1], seed, l) for l in range(L)]
    bs = [torch.zeros(dims[l + 1]) for l in range(L)]
    g = gnn.DeviceGraph(rowptr.to(DEV), col.to(DEV))
    targets = [workloads.targets_for_step(perm, batch, s).to(DEV) for s in range(n // batch)]
    return rowptr, col, table, labels, ws, bs, g, targets


def _state(tr):
    return [t.cpu().clone() for t in tr.w + tr.b + tr.dw + tr.db] + [tr.loss.cpu().clone()]


@pytest.mark.parametrize("kind,precision,nslot,steps", [(gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_BF16, 2, 5),
                                                          (gnn.GNN_AGG_GCN_SYM, gnn.GNN_F32, 2, 5),
                                                          (gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_BF16, 3, 7),
                                                          (gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_BF16, 3, 1),
                                                          (gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_BF16, 3, 6),
                                                          (gnn.GNN_AGG_GCN_SYM, gnn.GNN_BF16, 4, 2),
                                                          (gnn.GNN_AGG_SAGE_MEAN, gnn.GNN_BF16, 8, 11),
                                                          (gnn.GNN_AGG_GCN_SYM, gnn.GNN_F32, 8, 3),
                                                          (gnn.GNN_AGG_SAGE_MAX, gnn.GNN_BF16, 4, 6)])
def test_pipelined_two_stage_steps_equal_one_call_steps(kind, precision, nslot, steps):
    # gnn_train_steps: steps in groups of n_prep // 2 through rotating
    # prepare slots (each refilled after the computes that read it; partial
    # last groups and fewer steps than slots included) give bit for bit what
    # one-call steps give, per-step losses and edge counts too
    dims, fan, n, m, batch = (100, 256, 47), (25, 10), 30_000, 400_000, 512
    _rp, _col, table, labels, ws, bs, g, targets = _pipeline_inputs(kind, dims, fan, n, m, batch)
    table = table.to(DEV)
    nrm = gnn.gcn_norm(g)
    print(f"[pipeline] kind={kind} precision={precision} slots={nslot} steps={steps}: one-call steps", flush=True)
    ref = gnn.Trainer(kind, dims, fan, precision, n, batch, ws, bs, device=DEV)
    edges_ref = torch.zeros(steps, dtype=torch.int64, device=DEV)
    loss_ref = []
    for s in range(steps):
        ref.step(g, table, labels, targets[s % len(targets)], seed=3, step=s, lr=0.05, gcn_norm_t=nrm,
                 edges_out=edges_ref[s:s + 1])
        loss_ref.append(ref.loss.clone())
    torch.cuda.synchronize()
    print("[pipeline] gnn_train_steps", flush=True)
    tr = gnn.Trainer(kind, dims, fan, precision, n, batch, ws, bs, device=DEV, prepare_slots=nslot, one_call=False)
    edges = torch.zeros(steps, dtype=torch.int64, device=DEV)
    losses = torch.zeros(steps, dtype=torch.float32, device=DEV)
    tr.run_pipelined(g, table, labels, lambda s: targets[s % len(targets)], seed=3, first_step=0, steps=steps,
                     lr=0.05, gcn_norm_t=nrm, edges_out=edges, loss_out=losses)
    torch.cuda.synchronize()
    assert torch.equal(edges, edges_ref)
    assert torch.equal(losses.view(torch.int32), torch.cat(loss_ref).view(torch.int32))
    assert torch.equal(tr.loss.view(torch.int32), loss_ref[-1].view(torch.int32))
    for a, b in zip(_state(tr), _state(ref)):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    for h in (1, 2):
        got, want = tr.block_view(h), ref.block_view(h)
        for key in want:
            assert np.array_equal(np.asarray(got[key]), np.asarray(want[key])), (h, key)


def test_step_error_word_collects_the_blocks_flags():
    # The step's tail ORs every block's counts[3] into the compute
    # workspace's error word: a flag planted in a prepared (valid) block
    # reaches it; the first step of the next call writes the word afresh.
    dims, fan, n, m, batch = (32, 16, 8), (5, 5), 5_000, 40_000, 128
    kind = gnn.GNN_AGG_SAGE_MEAN
    _rp, _col, table, labels, ws, bs, g, targets = _pipeline_inputs(kind, dims, fan, n, m, batch)
    table = table.to(DEV)
    tr = gnn.Trainer(kind, dims, fan, gnn.GNN_F32, n, batch, ws, bs, device=DEV, prepare_slots=2, one_call=False)
    tr.prepare(0, g, table, targets[0], seed=1, step=0)
    tr.compute(0, labels, lr=0.05)
    tr.check_device_errors()
    tr.prepare(1, g, table, targets[1], seed=1, step=1)
    off = tr.layout.blk_counts[1]
    tr.prep_ws[1][off:off + 32].view(torch.int64)[3] = gnn.GNN_DEVERR_RANGE
    tr.compute(1, labels, lr=0.05)
    with pytest.raises(gnn.GnnError) as e:
        tr.check_device_errors()
    assert e.value.code == gnn.GNN_EDEVICE and "GNN_DEVERR_RANGE" in str(e.value)
    tr.prepare(0, g, table, targets[2], seed=1, step=2)
    tr.compute(0, labels, lr=0.05)
    tr.check_device_errors()
    tr.run_pipelined(g, table, labels, lambda s: targets[s], seed=1, first_step=3, steps=5, lr=0.05)
    tr.check_device_errors()
    assert int(tr.error_word().item()) == 0


def test_prepare_then_compute_from_pinned_host_fp16_table_matches_oracle():
    # the host-table model shape (768 -> 1024 -> 153, fanouts 25/15) on a
    # small R-MAT graph: fp16 table in pinned host memory, read over the host
    # link by the gather, bf16 GEMMs; one step against the oracle, then a
    # pipelined run against one-call steps on an HBM copy of the table
    dims, fan, n, m, batch = (768, 1024, 153), (25, 15), 20_000, 200_000, 64
    kind = gnn.GNN_AGG_SAGE_MEAN
    rowptr, col, table, labels, ws, bs, g, targets = _pipeline_inputs(kind, dims, fan, n, m, batch,
                                                                      table_dtype=torch.float16)
    pinned = table.pin_memory()
    print("[host-table] prepare + compute, one step", flush=True)
    tr = gnn.Trainer(kind, dims, fan, gnn.GNN_BF16, n, batch, ws, bs, device=DEV, prepare_slots=2, one_call=False)
    tr.prepare(0, g, pinned, targets[0], seed=1, step=0, loc=gnn.GNN_LOC_HOST_PINNED)
    tr.compute(0, labels, lr=0.05)
    torch.cuda.synchronize()
    cfg = oracle.StepConfig(kind=oracle.SAGE, dims=dims, fanouts=fan, precision=oracle.BF16, seed=1, step=0, lr=0.05)
    ref = oracle.train_step(rowptr.numpy(), col.numpy(), None, table.numpy(), labels.cpu().numpy(),
                            targets[0].cpu().numpy(), [w.numpy() for w in ws], [b.numpy() for b in bs], cfg)
    _check_step(tr, ref, oracle.BF16, 2)
    x0 = tr.tensor("x0", 0, ref["x0"].shape[0], dims[0], torch.bfloat16).cpu().view(torch.int16).numpy()
    assert np.array_equal(x0.view(np.uint16), ref["x0"])

    steps = 4
    print("[host-table] pipelined from the pinned table vs one-call from HBM", flush=True)
    a = gnn.Trainer(kind, dims, fan, gnn.GNN_BF16, n, batch, ws, bs, device=DEV, prepare_slots=2, one_call=False)
    a.run_pipelined(g, pinned, labels, lambda s: targets[s], seed=1, first_step=0, steps=steps, lr=0.05,
                    loc=gnn.GNN_LOC_HOST_PINNED)
    b = gnn.Trainer(kind, dims, fan, gnn.GNN_BF16, n, batch, ws, bs, device=DEV)
    t_dev = table.to(DEV)
    for s in range(steps):
        b.step(g, t_dev, labels, targets[s], seed=1, step=s, lr=0.05)
    torch.cuda.synchronize()
    for x, y in zip(_state(a), _state(b)):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))

