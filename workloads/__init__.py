"""Seeded synthetic inputs for the sampled-GNN training step.

This module produces graphs, feature tables, labels, target batches and
initial weights.  It holds none of the training method's arithmetic: no
sampling, aggregation, update, loss or optimizer code lives here.  Both the
HIP path and the CPU oracle consume what it produces.

Every generator draws from a ``torch.Generator`` seeded from a master seed
and a per-purpose sub-seed, so a given (seed, device) pair always yields the
same bytes.  The streams of torch's CPU and GPU generators differ, so a graph
drawn on ``cuda`` differs from one drawn on ``cpu``; tests that compare the
two paths copy the same tensors to both sides instead of regenerating.

Workload shapes follow the paper's datasets (Table III) and model setup
(Section VI-A): two-layer models with hidden width 256, batch 1024, fanouts
25 and 10; the papers100M-sized three-layer case uses the (15, 10, 5) sample
size of the DistDGLv2 comparison (Table V).  The paper's datasets are not
available, so R-MAT and Erdos-Renyi graphs of the same vertex and edge counts
stand in for them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Tuple

import torch

# Sub-seeds per purpose; the master seed is added to each.
SUB_GRAPH = 11
SUB_FEATURES = 23
SUB_LABELS = 37
SUB_WEIGHTS = 41
SUB_TARGETS = 53
SUB_PERM = 67


def _gen(seed: int, sub: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((int(seed) * 1_000_003 + sub) & ((1 << 62) - 1))
    return g


# ---------------------------------------------------------------------------
# Graphs: int64 CSR, rows sorted ascending by column.
# ---------------------------------------------------------------------------

def csr_from_edges(src: torch.Tensor, dst: torch.Tensor, n: int) -> Tuple[torch.Tensor, torch.Tensor]:
    """Build an int64 CSR (rowptr[n+1], col[nnz]) whose row v lists, in
    ascending order, every stored edge (v, u).  Duplicates are kept."""
    src = src.to(torch.int64)
    dst = dst.to(torch.int64)
    key = src * n + dst
    key, _ = torch.sort(key)
    rows = torch.div(key, n, rounding_mode="floor")
    col = key - rows * n
    counts = torch.bincount(rows, minlength=n)
    rowptr = torch.zeros(n + 1, dtype=torch.int64, device=src.device)
    torch.cumsum(counts, 0, out=rowptr[1:])
    return rowptr, col


def er_graph(n: int, m_undirected: int, seed: int = 0, device="cpu"):
    """G(n, m): m distinct unordered non-loop pairs drawn uniformly, each
    stored in both directions (nnz = 2m)."""
    if m_undirected > n * (n - 1) // 2:
        raise ValueError("too many edges for G(n, m)")
    g = _gen(seed, SUB_GRAPH, device)
    chosen = torch.empty(0, dtype=torch.int64, device=device)
    while chosen.numel() < m_undirected:
        need = m_undirected - chosen.numel()
        draw = max(1024, int(need * 1.2) + 16)
        u = torch.randint(0, n, (draw,), generator=g, device=device)
        v = torch.randint(0, n, (draw,), generator=g, device=device)
        keep = u != v
        lo = torch.minimum(u, v)[keep]
        hi = torch.maximum(u, v)[keep]
        cand = torch.cat([chosen, lo * n + hi])
        # keep first occurrence of every pair so the choice is order-stable
        uniq, inv = torch.unique(cand, return_inverse=True)
        first = torch.full((uniq.numel(),), cand.numel(), dtype=torch.int64, device=device)
        first.scatter_reduce_(0, inv, torch.arange(cand.numel(), device=device), reduce="amin")
        order = torch.sort(first).values
        chosen = cand[order][:m_undirected]
    lo = torch.div(chosen, n, rounding_mode="floor")
    hi = chosen - lo * n
    return csr_from_edges(torch.cat([lo, hi]), torch.cat([hi, lo]), n)


def rmat_graph(n: int, m: int, a=0.57, b=0.19, c=0.19, seed: int = 0, directed: bool = False,
               device="cpu", chunk: int = 1 << 26):
    """R-MAT edge draws on a 2^s x 2^s grid, s = ceil(log2 n).  Draws whose
    endpoint falls outside [0, n) or that form a self loop are redrawn.
    Duplicate edges are kept.  Vertex ids are relabelled by a seeded random
    permutation so hubs are spread over the id range.  Undirected graphs store
    both directions (nnz = 2m); directed graphs store (src -> dst) in row src.
    """
    s = max(1, math.ceil(math.log2(max(n, 2))))
    g = _gen(seed, SUB_GRAPH, device)
    p_ab = a + b
    p_abc = a + b + c
    srcs, dsts = [], []
    remaining = m
    while remaining > 0:
        cm = min(remaining, chunk)
        r = torch.zeros(cm, dtype=torch.int64, device=device)
        q = torch.zeros(cm, dtype=torch.int64, device=device)
        todo = torch.arange(cm, device=device)
        while todo.numel() > 0:
            rr = torch.zeros(todo.numel(), dtype=torch.int64, device=device)
            qq = torch.zeros(todo.numel(), dtype=torch.int64, device=device)
            for _ in range(s):
                x = torch.rand(todo.numel(), generator=g, device=device)
                row_bit = (x >= p_ab).to(torch.int64)
                col_bit = ((x >= a) & (x < p_ab)) | (x >= p_abc)
                rr = rr * 2 + row_bit
                qq = qq * 2 + col_bit.to(torch.int64)
            r[todo] = rr
            q[todo] = qq
            bad = (rr >= n) | (qq >= n) | (rr == qq)
            todo = todo[bad]
        srcs.append(r)
        dsts.append(q)
        remaining -= cm
    src = torch.cat(srcs)
    dst = torch.cat(dsts)
    del srcs, dsts
    perm = torch.randperm(n, generator=_gen(seed, SUB_PERM, device), device=device)
    src = perm[src]
    dst = perm[dst]
    if directed:
        return csr_from_edges(src, dst, n)
    return csr_from_edges(torch.cat([src, dst]), torch.cat([dst, src]), n)


def graph_stats(rowptr: torch.Tensor, col: torch.Tensor) -> dict:
    n = rowptr.numel() - 1
    deg = rowptr[1:] - rowptr[:-1]
    nnz = int(col.numel())
    rows = torch.repeat_interleave(torch.arange(n, device=rowptr.device), deg)
    same = (rows[1:] == rows[:-1]) & (col[1:] == col[:-1]) if nnz > 1 else torch.zeros(0, dtype=torch.bool)
    return {
        "n": n,
        "nnz": nnz,
        "max_degree": int(deg.max()) if n else 0,
        "mean_degree": nnz / max(n, 1),
        "isolated_fraction": float((deg == 0).sum()) / max(n, 1),
        "duplicate_edge_fraction": float(same.sum()) / max(nnz, 1),
    }


# ---------------------------------------------------------------------------
# Features, labels, targets, weights.
# ---------------------------------------------------------------------------

def features(n: int, f: int, seed: int = 0, dtype=torch.float32, device="cpu",
             out: Optional[torch.Tensor] = None, rows_per_chunk: int = 1 << 22) -> torch.Tensor:
    """n x f table of N(0, 1) draws stored in ``dtype`` (float32 or float16).
    ``out`` may be a preallocated (e.g. pinned host) tensor to fill in place."""
    g = _gen(seed, SUB_FEATURES, device)
    if out is None:
        out = torch.empty((n, f), dtype=dtype, device=device)
    for r0 in range(0, n, rows_per_chunk):
        r1 = min(n, r0 + rows_per_chunk)
        blk = torch.randn((r1 - r0, f), generator=g, device=device, dtype=torch.float32)
        out[r0:r1].copy_(blk.to(out.dtype))
    return out


def labels(n: int, num_classes: int, seed: int = 0, device="cpu") -> torch.Tensor:
    return torch.randint(0, num_classes, (n,), generator=_gen(seed, SUB_LABELS, device),
                         device=device, dtype=torch.int64)


def target_batches(n: int, batch: int, seed: int = 0, device="cpu") -> torch.Tensor:
    """Seeded permutation of [0, n); step s trains on perm[s*B:(s+1)*B]."""
    return torch.randperm(n, generator=_gen(seed, SUB_TARGETS, device), device=device)


def targets_for_step(perm: torch.Tensor, batch: int, step: int) -> torch.Tensor:
    n = perm.numel()
    nb = n // batch
    s = step % max(nb, 1)
    return perm[s * batch:(s + 1) * batch]


def glorot(k: int, nout: int, seed: int, layer: int, device="cpu") -> torch.Tensor:
    """Glorot-uniform K x N float32 matrix."""
    g = _gen(seed + 7919 * (layer + 1), SUB_WEIGHTS, device)
    bound = math.sqrt(6.0 / (k + nout))
    return (torch.rand((k, nout), generator=g, device=device, dtype=torch.float64) * 2 - 1).mul_(bound).to(torch.float32)


# ---------------------------------------------------------------------------
# Workload presets.
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    graph: str                # "er" or "rmat"
    n: int
    m: int                    # undirected pairs (er / undirected rmat) or directed edges
    directed: bool
    kind: str                 # "gcn", "sage" (mean) or "sage-max"
    dims: Tuple[int, ...]     # f^0 .. f^L
    fanouts: Tuple[int, ...]  # hop order: fanouts[0] is sampled around the targets
    batch: int
    precision: str            # "f32" or "bf16"
    table_dtype: str = "f32"  # "f32" or "f16"
    table_loc: str = "device"  # "device" or "host"
    seed: int = 0

    @property
    def num_layers(self) -> int:
        return len(self.dims) - 1

    @property
    def num_classes(self) -> int:
        return self.dims[-1]

    def k_of_layer(self, layer: int) -> int:
        """Width of the update GEMM's reduction for layer ``layer`` (1-based)."""
        f = self.dims[layer - 1]
        return f if self.kind == "gcn" else 2 * f


TINY = Workload("tiny-er10k-gcn", "er", 10_000, 50_000, False, "gcn", (32, 16, 8), (5, 5), 256, "f32")
RMAT_SAGE = Workload("rmat2.4m-sage", "rmat", 2_449_029, 61_859_140, False, "sage", (100, 256, 47), (25, 10),
                     1024, "bf16")
RMAT_GCN = Workload("rmat2.4m-gcn", "rmat", 2_449_029, 61_859_140, False, "gcn", (100, 256, 47), (25, 10),
                    1024, "bf16")
# the headline model with GraphSAGE's max aggregator instead of the mean
RMAT_SAGE_MAX = Workload("rmat2.4m-sagemax", "rmat", 2_449_029, 61_859_140, False, "sage-max", (100, 256, 47),
                         (25, 10), 1024, "bf16")
RMAT_SAGE3 = Workload("rmat111m-sage3", "rmat", 111_059_956, 1_615_685_872, True, "sage", (128, 256, 256, 172),
                      (15, 10, 5), 1024, "bf16")
RMAT_HOST = Workload("rmat244m-sage-hosttable", "rmat", 244_000_000, 1_700_000_000, True, "sage", (768, 1024, 153),
                     (25, 15), 1024, "bf16", table_dtype="f16", table_loc="host")

PRESETS = {w.name: w for w in (TINY, RMAT_SAGE, RMAT_GCN, RMAT_SAGE_MAX, RMAT_SAGE3, RMAT_HOST)}


def scaled(w: Workload, n: int, m: int, name: Optional[str] = None) -> Workload:
    """Same model, fanouts, batch and precision on a smaller graph."""
    return dataclasses.replace(w, n=n, m=m, name=name or f"{w.name}-n{n}")


def make_graph(w: Workload, device="cpu"):
    if w.graph == "er":
        return er_graph(w.n, w.m, w.seed, device)
    return rmat_graph(w.n, w.m, seed=w.seed, directed=w.directed, device=device)
