"""gnn_update_bwd_noalloc against gnn_update_bwd, through the C ABI.

The allocation-free entry point runs the same kernels with the library's
static scratch in place of a caller workspace, so its outputs must equal the
workspace entry point's bit for bit.  Two calls in a row, the second on a
smaller input, show that nothing left in the shared scratch by one call
leaks into the next; the workspace call gets a workspace full of NaN bit
patterns, so neither side can depend on zeroed scratch.
"""

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

gnn = pytest.importorskip("paper_2303_00158_amd.gnn")

DEV = torch.device("cuda:0")


def _dev(a: np.ndarray, code) -> torch.Tensor:
    if code == oracle.BF16:
        return torch.from_numpy(oracle.f32_to_bf16_bits(a).view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def _case(rng, m, cap, ke, n, code):
    a_s = rng.standard_normal((cap, ke)).astype(np.float32)
    a_n = rng.standard_normal((cap, ke)).astype(np.float32)
    K = 2 * ke
    w = (rng.standard_normal((K, n)) / np.sqrt(K)).astype(np.float32)
    g = rng.standard_normal((cap, n)).astype(np.float32)
    return a_s, a_n, w, g


def _bits(t: torch.Tensor) -> torch.Tensor:
    return t.detach().cpu().view(torch.int32)


@pytest.mark.parametrize("code", [oracle.BF16, oracle.F32])
def test_noalloc_update_bwd_equals_workspace_entry_point(code):
    rng = np.random.default_rng(11)
    # (rows used, row capacity, k_each, n_out): the headline model's layer-1
    # and layer-2 update shapes, the second call smaller than the first
    cases = [(7585, 7700, 100, 256), (1000, 1024, 256, 47)]
    for m, cap, ke, n in cases:
        print(f"[noalloc] code={code} m={m} cap={cap} k_each={ke} n_out={n}", flush=True)
        a_s, a_n, w, g = _case(rng, m, cap, ke, n, code)
        K = 2 * ke
        m_dev = torch.tensor([m], dtype=torch.int64, device=DEV)
        args = (_dev(a_s, code), _dev(a_n, code), _dev(w, oracle.F32), _dev(g, oracle.F32))
        nb = gnn._sz()
        gnn._check(gnn.lib().gnn_update_bwd_workspace_size(K, n, cap, code, gnn.ctypes.byref(nb)))
        assert 0 < nb.value <= 32 << 20
        ws = torch.full((nb.value,), 0xFF, dtype=torch.uint8, device=DEV)
        outs = []
        for noalloc in (False, True):
            dw = torch.full((K, n), 5.0, device=DEV)
            db = torch.full((n,), 5.0, device=DEV)
            da = torch.full((cap, K), 5.0, device=DEV)
            if noalloc:
                gnn.update_bwd_noalloc(*args, dw, db, da, code, m_dev=m_dev, cap_m=cap)
            else:
                gnn.update_bwd(*args, dw, db, da, code, m_dev=m_dev, cap_m=cap, ws=ws)
            torch.cuda.synchronize()
            outs.append((dw, db, da))
        for x, y in zip(outs[0], outs[1]):
            assert torch.equal(_bits(x), _bits(y))
        # and both against the oracle on the counted rows
        dw_w, db_w, da_w = oracle.update_bwd(
            oracle.f32_to_bf16_bits(a_s[:m]) if code == oracle.BF16 else a_s[:m],
            oracle.f32_to_bf16_bits(a_n[:m]) if code == oracle.BF16 else a_n[:m], w, g[:m], code, want_da=True)
        dw, db, da = (t.cpu().numpy().astype(np.float64) for t in outs[1])
        tol = 8e-3 if code == oracle.BF16 else 1e-5
        assert np.abs(dw - dw_w).max() <= tol * np.abs(dw_w).max()
        assert np.abs(db - db_w).max() <= 1e-5 * np.abs(db_w).max()
        assert np.abs(da[:m] - da_w).max() <= tol * np.abs(da_w).max()
        assert np.all(da[m:] == 5.0)  # rows past the device count untouched


def test_noalloc_update_bwd_rejects_shapes_beyond_the_static_scratch():
    # the wide first layer of the host-table model (K = 1,536, n_out = 1,024)
    # at 26,624 rows needs more than 32 MiB of dW partials
    cap, ke, n = 26624, 768, 1024
    nb = gnn._sz()
    gnn._check(gnn.lib().gnn_update_bwd_workspace_size(2 * ke, n, cap, gnn.GNN_BF16, gnn.ctypes.byref(nb)))
    assert nb.value > 32 << 20
    a = torch.zeros((cap, ke), dtype=torch.bfloat16, device=DEV)
    w = torch.zeros((2 * ke, n), device=DEV)
    g = torch.zeros((cap, n), device=DEV)
    dw = torch.zeros((2 * ke, n), device=DEV)
    with pytest.raises(gnn.GnnError) as e:
        gnn.update_bwd_noalloc(a, a, w, g, dw, None, None, gnn.GNN_BF16)
    assert e.value.code == gnn.GNN_ESIZE
    assert "static scratch" in str(e.value)
