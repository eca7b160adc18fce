"""Dense brute-force forms of the sampled-block operators, for pinning the
oracle.  Built with Python loops and numpy/torch library calls only; nothing
here is shared with the oracle or the GPU path."""
import numpy as np


def block_edges(blk):
    """[(i, j)] for every sampled edge, row-major."""
    out = []
    for i in range(blk.n_dst):
        for e in range(int(blk.rowptr[i]), int(blk.rowptr[i + 1])):
            out.append((i, int(blk.col[e])))
    return out


def sage_mean_matrix(blk):
    """n_dst x n_src matrix M with (M H)[i] = mean of H over row i's sampled
    neighbours (zero row when there are none)."""
    M = np.zeros((blk.n_dst, blk.n_src))
    for i in range(blk.n_dst):
        deg = int(blk.rowptr[i + 1] - blk.rowptr[i])
        for e in range(int(blk.rowptr[i]), int(blk.rowptr[i + 1])):
            M[i, int(blk.col[e])] += 1.0 / deg
    return M


def gcn_matrix(blk, src_norm):
    """n_dst x n_src matrix with the GCN weights nrm_i nrm_j (each product
    rounded to fp32, as the training step defines it) on every sampled edge
    plus nrm_i^2 on the self column."""
    sn = np.asarray(src_norm, dtype=np.float32)
    M = np.zeros((blk.n_dst, blk.n_src))
    for i in range(blk.n_dst):
        M[i, i] += float(np.float32(sn[i] * sn[i]))
        for e in range(int(blk.rowptr[i]), int(blk.rowptr[i + 1])):
            j = int(blk.col[e])
            M[i, j] += float(np.float32(sn[i] * sn[j]))
    return M


def self_select_matrix(blk):
    S = np.zeros((blk.n_dst, blk.n_src))
    for i in range(blk.n_dst):
        S[i, i] = 1.0
    return S


def small_multigraph(rng, n, avg_deg, hubs=1, isolated=2, multi=True):
    """Random directed multigraph CSR on n vertices with a few hubs, a few
    isolated vertices and (optionally) repeated edges; rows sorted."""
    rows = []
    iso = set(rng.choice(n, size=min(isolated, n), replace=False).tolist()) if isolated else set()
    hub_ids = [v for v in rng.choice(n, size=min(hubs, n), replace=False).tolist() if v not in iso]
    for v in range(n):
        if v in iso:
            rows.append([])
            continue
        d = int(rng.poisson(avg_deg))
        if v in hub_ids:
            d = n * 2
        nb = rng.integers(0, n, size=d).tolist() if multi else rng.choice(n, size=min(d, n), replace=False).tolist()
        nb = [u for u in nb if u != v and u not in iso]
        rows.append(sorted(nb))
    rowptr = np.zeros(n + 1, dtype=np.int64)
    for v in range(n):
        rowptr[v + 1] = rowptr[v] + len(rows[v])
    col = np.array([u for r in rows for u in r], dtype=np.int64)
    return rowptr, col
