"""ctypes binding of libgnn.so (see include/gnn.h).

Argument marshalling only: torch tensors supply device memory and the current
HIP stream; every step runs in the library's kernels.  Importing this module
does not need a GPU; calling anything that launches work does.  If the
library has not been built the first call raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgnn.so")

GNN_OK, GNN_EINVAL, GNN_ESIZE, GNN_EHIP, GNN_EUNSUPPORTED, GNN_EDEVICE = 0, -1, -2, -3, -4, -5
GNN_DEVERR_WAIT, GNN_DEVERR_RANGE = 1, 2
GNN_F32, GNN_BF16, GNN_F16 = 0, 1, 2
GNN_AGG_SAGE_MEAN, GNN_AGG_GCN_SYM, GNN_AGG_SAGE_MAX = 0, 1, 2
GNN_LOC_DEVICE, GNN_LOC_HOST_PINNED = 0, 1
GNN_MAX_LAYERS = 4

_i64, _i32, _u64, _f32, _vp, _sz = (ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_float,
                                    ctypes.c_void_p, ctypes.c_size_t)


class GnnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class Graph(ctypes.Structure):
    _fields_ = [("n", _i64), ("nnz", _i64), ("rowptr", _vp), ("col", _vp)]


class Block(ctypes.Structure):
    _fields_ = [("cap_dst", _i64), ("cap_src", _i64), ("cap_nnz", _i64), ("counts", _vp), ("src_ids", _vp),
                ("rowptr", _vp), ("col", _vp), ("cscptr", _vp), ("cscrow", _vp), ("src_norm", _vp)]


class Model(ctypes.Structure):
    _fields_ = [("num_layers", _i32), ("kind", _i32), ("precision", _i32),
                ("dims", _i32 * (GNN_MAX_LAYERS + 1)), ("fanouts", _i32 * GNN_MAX_LAYERS),
                ("w", _vp * GNN_MAX_LAYERS), ("b", _vp * GNN_MAX_LAYERS),
                ("dw", _vp * GNN_MAX_LAYERS), ("db", _vp * GNN_MAX_LAYERS), ("wt", _vp * GNN_MAX_LAYERS)]


_ML = GNN_MAX_LAYERS


class StepLayout(ctypes.Structure):
    _fields_ = [("total_bytes", _sz), ("prep_bytes", _sz), ("compute_bytes", _sz),
                ("sampler_ws", _sz), ("sampler_ws_bytes", _sz),
                ("cap_dst", _i64 * _ML), ("cap_src", _i64 * _ML), ("cap_nnz", _i64 * _ML),
                ("blk_counts", _sz * _ML), ("blk_src_ids", _sz * _ML), ("blk_rowptr", _sz * _ML),
                ("blk_col", _sz * _ML), ("blk_cscptr", _sz * _ML), ("blk_cscrow", _sz * _ML),
                ("blk_src_norm", _sz * _ML), ("blk_csc_ws", _sz * _ML),
                ("x0", _sz), ("agg", _sz * (_ML + 1)), ("h", _sz * (_ML + 1)), ("grad", _sz * (_ML + 1)),
                ("d_a", _sz * (_ML + 1)), ("fwd_ws", _sz), ("fwd_ws_bytes", _sz), ("bwd_ws", _sz),
                ("bwd_ws_bytes", _sz), ("loss_ws", _sz),
                ("loss_ws_bytes", _sz), ("edges", _sz), ("error", _sz), ("loss", _sz),
                ("argmax", _sz * (_ML + 1))]


_P = ctypes.POINTER
_SIGNATURES = {
    "gnn_last_error": (ctypes.c_char_p, []),
    "gnn_abi_version": (_i32, []),
    "gnn_gcn_norm": (_i32, [_P(Graph), _vp, _vp]),
    "gnn_block_bounds": (_i32, [_i64, _i64, _i32, _P(_i64), _P(_i64)]),
    "gnn_sampler_workspace_size": (_i32, [_i64, _i64, _i32, _P(_sz)]),
    "gnn_sampler_workspace_init": (_i32, [_vp, _sz, _i64, _vp]),
    "gnn_build_block": (_i32, [_P(Graph), _vp, _vp, _vp, _i32, _u64, _u64, _i32, _i32, _P(Block), _vp, _sz, _vp]),
    "gnn_gather_features": (_i32, [_vp, _i32, _i32, _i64, _i64, _i64, _vp, _vp, _i64, _vp, _i32, _vp]),
    "gnn_aggregate_fwd": (_i32, [_P(Block), _i32, _vp, _i32, _i64, _vp, _i32, _vp]),
    "gnn_aggregate_fwd_dedup": (_i32, [_P(Block), _i32, _vp, _i32, _i64, _vp, _i32, _vp]),
    "gnn_aggregate_bwd": (_i32, [_P(Block), _i32, _vp, _i64, _vp, _i32, _vp, _vp]),
    "gnn_aggregate_fwd_max": (_i32, [_P(Block), _vp, _i32, _i64, _vp, _i32, _vp, _vp]),
    "gnn_aggregate_bwd_max": (_i32, [_P(Block), _vp, _vp, _i64, _vp, _i32, _vp, _vp]),
    "gnn_layer_fwd": (_i32, [_P(Block), _i32, _i32, _vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _i64, _vp, _vp, _vp]),
    "gnn_two_layer_fwd": (_i32, [_P(Block), _i32, _i32, _vp, _vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _i64, _vp,
                                 _vp, _vp, _i64, _vp, _vp, _vp, _vp]),
    "gnn_two_layer_fwd_max": (_i32, [_P(Block), _i32, _vp, _vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _i64, _vp,
                                     _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp]),
    "gnn_two_layer_bwd_workspace_size": (_i32, [_i32, _i64, _i64, _i64, _i64, _i64, _P(_sz)]),
    "gnn_two_layer_bwd": (_i32, [_P(Block), _i32, _vp, _vp, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _vp, _i64, _vp,
                                 _vp, _vp, _vp, _vp, _sz, _vp]),
    "gnn_two_layer_bwd_max": (_i32, [_P(Block), _vp, _vp, _i64, _vp, _i64, _vp, _i64, _vp, _vp, _vp, _vp, _i64,
                                     _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "gnn_update_fwd_workspace_size": (_i32, [_i64, _i64, _i64, _i32, _P(_sz)]),
    "gnn_update_fwd": (_i32, [_vp, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _vp, _i64, _i32, _i32, _vp, _i32, _vp, _sz,
                              _vp]),
    "gnn_update_bwd_workspace_size": (_i32, [_i64, _i64, _i64, _i32, _P(_sz)]),
    "gnn_update_bwd": (_i32, [_vp, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _i64, _i32, _vp, _vp, _vp, _vp, _sz,
                              _vp]),
    "gnn_update_bwd_noalloc": (_i32, [_vp, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _i64, _i32, _vp, _vp, _vp, _vp]),
    "gnn_softmax_ce_workspace_size": (_i32, [_i64, _P(_sz)]),
    "gnn_softmax_ce": (_i32, [_vp, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "gnn_sgd": (_i32, [_vp, _vp, _i64, _f32, _vp]),
    "gnn_model_sync_shadow": (_i32, [_P(Model), _vp]),
    "gnn_train_step_layout": (_i32, [_P(Model), _i64, _i64, _P(StepLayout)]),
    "gnn_train_step_workspace_size": (_i32, [_P(Model), _i64, _i64, _P(_sz)]),
    "gnn_train_step_workspace_init": (_i32, [_P(Model), _i64, _i64, _vp, _sz, _vp]),
    "gnn_train_step": (_i32, [_P(Model), _P(Graph), _vp, _vp, _i32, _i32, _i64, _vp, _vp, _i64, _u64, _u64, _f32,
                              _vp, _vp, _vp, _sz, _vp]),
    "gnn_step_prepare_workspace_init": (_i32, [_P(Model), _i64, _i64, _vp, _sz, _vp]),
    "gnn_step_prepare": (_i32, [_P(Model), _P(Graph), _vp, _vp, _i32, _i32, _i64, _vp, _i64, _u64, _u64, _vp, _sz,
                                _vp]),
    "gnn_step_compute": (_i32, [_P(Model), _i64, _vp, _i64, _f32, _vp, _vp, _vp, _sz, _vp, _sz, _vp]),
    "gnn_decode_device_errors": (_i32, [_i64]),
    "gnn_check_device_errors": (_i32, [_vp, _vp]),
    "gnn_debug_sampler_fault": (_i32, [_i64, ctypes.c_uint32]),
    "gnn_train_steps": (_i32, [_P(Model), _P(Graph), _vp, _vp, _i32, _i32, _i64, _vp, _vp, _i64, _u64, _u64, _i64,
                               _f32, _vp, _vp, _P(_vp), _i32, _sz, _vp, _sz, _vp, _vp]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """Load libgnn.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2303_00158_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def exported_symbols() -> List[str]:
    return list(_SIGNATURES)


def _check(code: int) -> None:
    if code != GNN_OK:
        raise GnnError(code, lib().gnn_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def dtype_code(dt: torch.dtype) -> int:
    return {torch.float32: GNN_F32, torch.bfloat16: GNN_BF16, torch.float16: GNN_F16}[dt]


def torch_dtype(code: int) -> torch.dtype:
    return {GNN_F32: torch.float32, GNN_BF16: torch.bfloat16, GNN_F16: torch.float16}[code]


def _aligned_empty(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# graph and blocks
# ---------------------------------------------------------------------------

class DeviceGraph:
    """An int64 CSR on the device plus its ctypes descriptor."""

    def __init__(self, rowptr: torch.Tensor, col: torch.Tensor):
        assert rowptr.dtype == torch.int64 and col.dtype == torch.int64
        self.rowptr = rowptr.contiguous()
        self.col = col.contiguous()
        self.n = self.rowptr.numel() - 1
        self.c = Graph(self.n, self.col.numel(), _ptr(self.rowptr), _ptr(self.col))


def gcn_norm(graph: DeviceGraph, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if out is None:
        out = torch.empty(graph.n, dtype=torch.float32, device=graph.rowptr.device)
    _check(lib().gnn_gcn_norm(ctypes.byref(graph.c), _ptr(out), _stream(stream)))
    return out


def block_bounds(graph_n: int, cap_dst: int, fanout: int):
    cs, cn = _i64(), _i64()
    _check(lib().gnn_block_bounds(graph_n, cap_dst, fanout, ctypes.byref(cs), ctypes.byref(cn)))
    return cs.value, cn.value


class DeviceBlock:
    """Device buffers of one block at its capacity bounds."""

    def __init__(self, graph_n: int, cap_dst: int, fanout: int, want_csc: bool, want_norm: bool, device):
        cap_src, cap_nnz = block_bounds(graph_n, cap_dst, fanout)
        z = lambda n, dt: torch.zeros(max(n, 1), dtype=dt, device=device)  # noqa: E731
        self.counts = z(4, torch.int64)
        self.src_ids = z(cap_src, torch.int64)
        self.rowptr = z(cap_dst + 1, torch.int64)
        self.col = z(cap_nnz, torch.int32)
        self.cscptr = z(cap_src + 1, torch.int64) if want_csc else None
        self.cscrow = z(cap_nnz, torch.int32) if want_csc else None
        self.src_norm = z(cap_src, torch.float32) if want_norm else None
        self.c = Block(cap_dst, cap_src, cap_nnz, _ptr(self.counts), _ptr(self.src_ids), _ptr(self.rowptr),
                       _ptr(self.col), _ptr(self.cscptr), _ptr(self.cscrow), _ptr(self.src_norm))

    def host(self) -> dict:
        """Copy the used part of the block to host numpy arrays (synchronises)."""
        c = self.counts.cpu().tolist()
        n_dst, n_src, nnz = int(c[0]), int(c[1]), int(c[2])
        out = {
            "n_dst": n_dst, "n_src": n_src, "nnz": nnz,
            "src_ids": self.src_ids[:n_src].cpu().numpy(),
            "rowptr": self.rowptr[:n_dst + 1].cpu().numpy(),
            "col": self.col[:nnz].cpu().numpy(),
        }
        if self.cscptr is not None:
            out["cscptr"] = self.cscptr[:n_src + 1].cpu().numpy()
            out["cscrow"] = self.cscrow[:nnz].cpu().numpy()
        if self.src_norm is not None:
            out["src_norm"] = self.src_norm[:n_src].cpu().numpy()
        return out


def sampler_workspace(graph_n: int, cap_dst: int, fanout: int, device, stream=None) -> torch.Tensor:
    nb = _sz()
    _check(lib().gnn_sampler_workspace_size(graph_n, cap_dst, fanout, ctypes.byref(nb)))
    ws = _aligned_empty(nb.value, device)
    _check(lib().gnn_sampler_workspace_init(_ptr(ws), ws.numel(), graph_n, _stream(stream)))
    return ws


def build_block(graph: DeviceGraph, dst_ids: torch.Tensor, fanout: int, seed: int, step: int, hop: int,
                out: DeviceBlock, ws: torch.Tensor, n_dst_dev: Optional[torch.Tensor] = None,
                gcn_norm_t: Optional[torch.Tensor] = None, want_csc: bool = True, stream=None) -> DeviceBlock:
    # the sampler reads up to cap_dst ids (the device count, if given, is
    # clamped to cap_dst)
    if dst_ids.numel() < out.c.cap_dst:
        raise ValueError(f"dst_ids holds {dst_ids.numel()} ids, the block's cap_dst is {out.c.cap_dst}")
    _check(lib().gnn_build_block(ctypes.byref(graph.c), _ptr(gcn_norm_t), _ptr(dst_ids), _ptr(n_dst_dev), fanout,
                                 seed, step, hop, int(want_csc), ctypes.byref(out.c), _ptr(ws), ws.numel(),
                                 _stream(stream)))
    return out


# ---------------------------------------------------------------------------
# kernels of one layer
# ---------------------------------------------------------------------------

def gather_features(table: torch.Tensor, ids: torch.Tensor, out: torch.Tensor, n_ids_dev: Optional[torch.Tensor] = None,
                    loc: int = GNN_LOC_DEVICE, row_stride: Optional[int] = None, stream=None) -> torch.Tensor:
    n_rows, dim = table.shape
    rs = table.stride(0) if row_stride is None else row_stride
    _check(lib().gnn_gather_features(_ptr(table), dtype_code(table.dtype), loc, n_rows, dim, rs, _ptr(ids),
                                     _ptr(n_ids_dev), out.shape[0], _ptr(out), dtype_code(out.dtype),
                                     _stream(stream)))
    return out


def aggregate_fwd(block: DeviceBlock, kind: int, h_src: torch.Tensor, out: torch.Tensor, stream=None) -> torch.Tensor:
    f = h_src.shape[1]
    _check(lib().gnn_aggregate_fwd(ctypes.byref(block.c), kind, _ptr(h_src), dtype_code(h_src.dtype), f, _ptr(out),
                                   dtype_code(out.dtype), _stream(stream)))
    return out


def aggregate_fwd_dedup(block: DeviceBlock, kind: int, h_src: torch.Tensor, out: torch.Tensor,
                        stream=None) -> torch.Tensor:
    f = h_src.shape[1]
    _check(lib().gnn_aggregate_fwd_dedup(ctypes.byref(block.c), kind, _ptr(h_src), dtype_code(h_src.dtype), f,
                                         _ptr(out), dtype_code(out.dtype), _stream(stream)))
    return out


def aggregate_bwd(block: DeviceBlock, kind: int, d_a: torch.Tensor, f: int, d_src: torch.Tensor,
                  h_below: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    hb_code = dtype_code(h_below.dtype) if h_below is not None else GNN_F32
    _check(lib().gnn_aggregate_bwd(ctypes.byref(block.c), kind, _ptr(d_a), f, _ptr(h_below), hb_code, _ptr(d_src),
                                   _stream(stream)))
    return d_src


def aggregate_fwd_max(block: DeviceBlock, h_src: torch.Tensor, out: torch.Tensor, argmax: Optional[torch.Tensor],
                      stream=None) -> torch.Tensor:
    """gnn_aggregate_fwd_max: GraphSAGE's max aggregator; argmax (int32, the
    shape of out, or None: not kept) receives the winning local source of
    every element."""
    assert argmax is None or argmax.dtype == torch.int32
    f = h_src.shape[1]
    _check(lib().gnn_aggregate_fwd_max(ctypes.byref(block.c), _ptr(h_src), dtype_code(h_src.dtype), f, _ptr(out),
                                       dtype_code(out.dtype), _ptr(argmax), _stream(stream)))
    return out


def aggregate_bwd_max(block: DeviceBlock, argmax: torch.Tensor, d_a: torch.Tensor, f: int, d_src: torch.Tensor,
                      h_below: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """gnn_aggregate_bwd_max: the max aggregator's backward from its argmax
    table (d_a rows hold 2f values: self part, then max part)."""
    assert argmax.dtype == torch.int32
    hb_code = dtype_code(h_below.dtype) if h_below is not None else GNN_F32
    _check(lib().gnn_aggregate_bwd_max(ctypes.byref(block.c), _ptr(argmax), _ptr(d_a), f, _ptr(h_below), hb_code,
                                       _ptr(d_src), _stream(stream)))
    return d_src


def layer_fwd(block: "DeviceBlock", kind: int, max_row_len: int, h_src: torch.Tensor, wt: torch.Tensor,
              bias: Optional[torch.Tensor], agg_out: torch.Tensor, out: torch.Tensor,
              labels: Optional[torch.Tensor] = None, batch: int = 0, g_out: Optional[torch.Tensor] = None,
              row_loss: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """gnn_layer_fwd: aggregation and update of one layer in one launch (bf16
    h_src, bf16 W^T wt).  With labels, out receives fp32 logits and g_out /
    row_loss the loss gradient and per-row losses of the first batch rows."""
    _check(lib().gnn_layer_fwd(ctypes.byref(block.c), kind, int(max_row_len), _ptr(h_src), h_src.shape[1], _ptr(wt),
                               _ptr(bias), wt.shape[0], _ptr(agg_out), _ptr(out), _ptr(labels), int(batch),
                               _ptr(g_out), _ptr(row_loss), _stream(stream)))
    return out


def two_layer_fwd(last: "DeviceBlock", kind: int, fanout: int, x_self: Optional[torch.Tensor], m1: torch.Tensor,
                  wt1: torch.Tensor, b1: Optional[torch.Tensor], h1: torch.Tensor, wt2: torch.Tensor,
                  b2: Optional[torch.Tensor], agg_out: torch.Tensor, logits: torch.Tensor, labels: torch.Tensor,
                  batch: int, g_out: torch.Tensor, row_loss: torch.Tensor, d_a: Optional[torch.Tensor] = None,
                  stream=None) -> torch.Tensor:
    """gnn_two_layer_fwd: both layers of a two-layer model in one launch (bf16
    rows x_self / m1 of layer 1, bf16 W^T shadows wt1 / wt2); h1, agg_out,
    logits, g_out, row_loss and (when given) d_a receive H^1, the last
    layer's aggregation, its logits, the loss gradient, the per-row losses and
    layer 2's input gradient."""
    _check(lib().gnn_two_layer_fwd(ctypes.byref(last.c), kind, int(fanout), _ptr(x_self), _ptr(m1), m1.shape[1],
                                   _ptr(wt1), _ptr(b1), wt1.shape[0], _ptr(h1), _ptr(wt2), _ptr(b2), wt2.shape[0],
                                   _ptr(agg_out), _ptr(logits), _ptr(labels), int(batch), _ptr(g_out),
                                   _ptr(row_loss), _ptr(d_a), _stream(stream)))
    return logits


def two_layer_fwd_max(last: "DeviceBlock", fanout: int, x_self: torch.Tensor, m1: torch.Tensor, wt1: torch.Tensor,
                      b1: Optional[torch.Tensor], h1: torch.Tensor, wt2: torch.Tensor, b2: Optional[torch.Tensor],
                      agg_out: torch.Tensor, argmax: torch.Tensor, logits: torch.Tensor, labels: torch.Tensor,
                      batch: int, g_out: torch.Tensor, row_loss: torch.Tensor, d_a: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """gnn_two_layer_fwd_max: two_layer_fwd with GraphSAGE's max aggregator
    in layer 2; argmax (int32, the shape of agg_out) receives its table."""
    assert argmax.dtype == torch.int32
    _check(lib().gnn_two_layer_fwd_max(ctypes.byref(last.c), int(fanout), _ptr(x_self), _ptr(m1), m1.shape[1],
                                       _ptr(wt1), _ptr(b1), wt1.shape[0], _ptr(h1), _ptr(wt2), _ptr(b2),
                                       wt2.shape[0], _ptr(agg_out), _ptr(argmax), _ptr(logits), _ptr(labels),
                                       int(batch), _ptr(g_out), _ptr(row_loss), _ptr(d_a), _stream(stream)))
    return logits


def two_layer_bwd_workspace(kind: int, f0: int, f1: int, n_out: int, cap_m1: int, cap_m2: int,
                            device) -> torch.Tensor:
    """A workspace for gnn_two_layer_bwd with these sizes."""
    nb = _sz()
    _check(lib().gnn_two_layer_bwd_workspace_size(kind, f0, f1, n_out, cap_m1, cap_m2, ctypes.byref(nb)))
    return torch.zeros(max(nb.value, 256), dtype=torch.uint8, device=device)


def two_layer_bwd(last: "DeviceBlock", kind: int, x_self: Optional[torch.Tensor], m1: torch.Tensor,
                  m1_rows: torch.Tensor, cap_m1: int, h1: torch.Tensor, agg2: torch.Tensor, d_a2: torch.Tensor,
                  g2: torch.Tensor, dw1: torch.Tensor, db1: Optional[torch.Tensor], dw2: torch.Tensor,
                  db2: Optional[torch.Tensor], ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """gnn_two_layer_bwd: both layers' weight gradients below the loss (layer
    2's aggregation backward folded into layer 1's dW).  m1_rows: device int64
    count of layer 1's rows (at most cap_m1); ws: workspace (allocated when
    None)."""
    f0, f1, n_out = m1.shape[1], h1.shape[1], g2.shape[1]
    if ws is None:
        ws = two_layer_bwd_workspace(kind, f0, f1, n_out, cap_m1, last.c.cap_dst, m1.device)
    _check(lib().gnn_two_layer_bwd(ctypes.byref(last.c), kind, _ptr(x_self), _ptr(m1), f0, _ptr(m1_rows), int(cap_m1),
                                   _ptr(h1), f1, _ptr(agg2), _ptr(d_a2), _ptr(g2), n_out, _ptr(dw1), _ptr(db1),
                                   _ptr(dw2), _ptr(db2), _ptr(ws), ws.numel(), _stream(stream)))


def two_layer_bwd_max(last: "DeviceBlock", x_self: torch.Tensor, m1: torch.Tensor, m1_rows: torch.Tensor,
                      cap_m1: int, h1: torch.Tensor, agg2: torch.Tensor, argmax2: torch.Tensor, d_a2: torch.Tensor,
                      g2: torch.Tensor, dw1: torch.Tensor, db1: Optional[torch.Tensor], dw2: torch.Tensor,
                      db2: Optional[torch.Tensor], ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """gnn_two_layer_bwd_max: two_layer_bwd for GraphSAGE with the max
    aggregator, from the argmax table gnn_two_layer_fwd_max wrote."""
    assert argmax2.dtype == torch.int32
    f0, f1, n_out = m1.shape[1], h1.shape[1], g2.shape[1]
    if ws is None:
        ws = two_layer_bwd_workspace(GNN_AGG_SAGE_MAX, f0, f1, n_out, cap_m1, last.c.cap_dst, m1.device)
    _check(lib().gnn_two_layer_bwd_max(ctypes.byref(last.c), _ptr(x_self), _ptr(m1), f0, _ptr(m1_rows), int(cap_m1),
                                       _ptr(h1), f1, _ptr(agg2), _ptr(argmax2), _ptr(d_a2), _ptr(g2), n_out,
                                       _ptr(dw1), _ptr(db1), _ptr(dw2), _ptr(db2), _ptr(ws), ws.numel(),
                                       _stream(stream)))


def update_fwd(a_self: torch.Tensor, a_nbr: Optional[torch.Tensor], w: torch.Tensor, bias: Optional[torch.Tensor],
               out: torch.Tensor, relu: bool, gemm_dtype: int, m_dev: Optional[torch.Tensor] = None,
               cap_m: Optional[int] = None, ws: Optional[torch.Tensor] = None, split: bool = True,
               wt: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """ws: workspace for split reductions (allocated when None and split is
    True); split=False runs without a workspace (no reduction split).  wt:
    optional bf16 W^T shadow (n_out x K) read instead of w in bf16 mode."""
    cap = a_self.shape[0] if cap_m is None else cap_m
    K = a_self.shape[1] * (2 if a_nbr is not None else 1)
    if ws is None and split:
        nb = _sz()
        _check(lib().gnn_update_fwd_workspace_size(K, w.shape[1], cap, gemm_dtype, ctypes.byref(nb)))
        ws = torch.zeros(max(nb.value, 256), dtype=torch.uint8, device=a_self.device)
    _check(lib().gnn_update_fwd(_ptr(a_self), _ptr(a_nbr), dtype_code(a_self.dtype), a_self.shape[1], _ptr(m_dev), cap,
                                _ptr(w), _ptr(wt), _ptr(bias), w.shape[1], int(relu), gemm_dtype, _ptr(out),
                                dtype_code(out.dtype), _ptr(ws), ws.numel() if ws is not None else 0,
                                _stream(stream)))
    return out


def update_bwd_workspace(k: int, n_out: int, cap_m: int, gemm_dtype: int, device) -> torch.Tensor:
    nb = _sz()
    _check(lib().gnn_update_bwd_workspace_size(k, n_out, cap_m, gemm_dtype, ctypes.byref(nb)))
    return torch.zeros(max(nb.value, 256), dtype=torch.uint8, device=device)


def update_bwd(a_self: torch.Tensor, a_nbr: Optional[torch.Tensor], w: torch.Tensor, g: torch.Tensor,
               dw: torch.Tensor, db: Optional[torch.Tensor], d_a: Optional[torch.Tensor], gemm_dtype: int,
               m_dev: Optional[torch.Tensor] = None, cap_m: Optional[int] = None, ws: Optional[torch.Tensor] = None,
               stream=None):
    cap = a_self.shape[0] if cap_m is None else cap_m
    K = a_self.shape[1] * (2 if a_nbr is not None else 1)
    if ws is None:
        ws = update_bwd_workspace(K, w.shape[1], cap, gemm_dtype, a_self.device)
    _check(lib().gnn_update_bwd(_ptr(a_self), _ptr(a_nbr), dtype_code(a_self.dtype), a_self.shape[1], _ptr(m_dev),
                                cap, _ptr(w), _ptr(g), w.shape[1], gemm_dtype, _ptr(dw), _ptr(db), _ptr(d_a),
                                _ptr(ws), ws.numel(), _stream(stream)))
    return dw, db, d_a


def update_bwd_noalloc(a_self: torch.Tensor, a_nbr: Optional[torch.Tensor], w: torch.Tensor, g: torch.Tensor,
                       dw: torch.Tensor, db: Optional[torch.Tensor], d_a: Optional[torch.Tensor], gemm_dtype: int,
                       m_dev: Optional[torch.Tensor] = None, cap_m: Optional[int] = None, stream=None):
    """gnn_update_bwd_noalloc: update_bwd with the library's static scratch."""
    cap = a_self.shape[0] if cap_m is None else cap_m
    _check(lib().gnn_update_bwd_noalloc(_ptr(a_self), _ptr(a_nbr), dtype_code(a_self.dtype), a_self.shape[1],
                                        _ptr(m_dev), cap, _ptr(w), _ptr(g), w.shape[1], gemm_dtype, _ptr(dw),
                                        _ptr(db), _ptr(d_a), _stream(stream)))
    return dw, db, d_a


def check_device_errors(word: torch.Tensor, stream=None) -> None:
    """gnn_check_device_errors on an int64 device word (a block's counts[3:4]
    or a step's error word); raises GnnError (GNN_EDEVICE) if a flag is set."""
    assert word.dtype == torch.int64 and word.is_cuda
    _check(lib().gnn_check_device_errors(_ptr(word), _stream(stream)))


def decode_device_errors(word: int) -> None:
    """gnn_decode_device_errors (host only)."""
    _check(lib().gnn_decode_device_errors(int(word)))


def debug_sampler_fault(silent_row_tile: int, spin_limit: int) -> None:
    """gnn_debug_sampler_fault: the test hook of the device error path."""
    _check(lib().gnn_debug_sampler_fault(int(silent_row_tile), int(spin_limit)))


def softmax_ce(logits: torch.Tensor, labels: torch.Tensor, targets: Optional[torch.Tensor], g_out: torch.Tensor,
               loss_out: torch.Tensor, stream=None):
    b, c = logits.shape
    nb = _sz()
    _check(lib().gnn_softmax_ce_workspace_size(b, ctypes.byref(nb)))
    ws = _aligned_empty(nb.value, logits.device)
    _check(lib().gnn_softmax_ce(_ptr(logits), b, c, _ptr(labels), _ptr(targets), _ptr(g_out), _ptr(loss_out),
                                _ptr(ws), ws.numel(), _stream(stream)))
    return g_out, loss_out


def sgd(w: torch.Tensor, dw: torch.Tensor, lr: float, stream=None) -> torch.Tensor:
    _check(lib().gnn_sgd(_ptr(w), _ptr(dw), w.numel(), float(lr), _stream(stream)))
    return w


# ---------------------------------------------------------------------------
# whole training step
# ---------------------------------------------------------------------------

_COMPUTE_BUFFERS = ("agg", "h", "grad", "d_a", "fwd_ws", "bwd_ws", "loss_ws", "edges", "error", "loss", "argmax")


class Trainer:
    """Owns the model buffers (fp32 master weights, gradients, and for bf16
    models the bf16 W^T shadows) and the step workspaces.

    step() calls gnn_train_step on one workspace.  With prepare_slots > 0
    the trainer also owns that many prepare workspaces and one compute
    workspace for the two-stage calls (prepare() / compute(), and
    run_pipelined(), which overlaps the prepare stage of step s+1 with the
    compute stage of step s on two streams)."""

    def __init__(self, kind: int, dims: Sequence[int], fanouts: Sequence[int], precision: int, graph_n: int,
                 batch: int, weights: Sequence[torch.Tensor], biases: Sequence[torch.Tensor], device="cuda",
                 shadows: bool = True, prepare_slots: int = 0, one_call: bool = True):
        L = len(dims) - 1
        assert len(fanouts) == L and len(weights) == L and len(biases) == L
        self.device = torch.device(device)
        self.kind, self.dims, self.fanouts, self.precision = kind, list(dims), list(fanouts), precision
        self.graph_n, self.batch = graph_n, batch
        self.w = [w.to(self.device, torch.float32).contiguous().clone() for w in weights]
        self.b = [b.to(self.device, torch.float32).contiguous().clone() for b in biases]
        self.dw = [torch.zeros_like(w) for w in self.w]
        self.db = [torch.zeros_like(b) for b in self.b]
        m = Model()
        m.num_layers, m.kind, m.precision = L, kind, precision
        for i, d in enumerate(dims):
            m.dims[i] = d
        for i, k in enumerate(fanouts):
            m.fanouts[i] = k
        for l in range(L):
            m.w[l], m.b[l], m.dw[l], m.db[l] = _ptr(self.w[l]), _ptr(self.b[l]), _ptr(self.dw[l]), _ptr(self.db[l])
        self.wt = []
        if shadows and precision == GNN_BF16:
            self.wt = [torch.empty((w.shape[1], w.shape[0]), dtype=torch.bfloat16, device=self.device) for w in self.w]
            for l in range(L):
                m.wt[l] = _ptr(self.wt[l])
        self.model = m
        if self.wt:
            _check(lib().gnn_model_sync_shadow(ctypes.byref(m), _stream(None)))
        self.layout = StepLayout()
        _check(lib().gnn_train_step_layout(ctypes.byref(m), graph_n, batch, ctypes.byref(self.layout)))
        self.ws = None
        if one_call:
            self.ws = _aligned_empty(self.layout.total_bytes, self.device)
            _check(lib().gnn_train_step_workspace_init(ctypes.byref(m), graph_n, batch, _ptr(self.ws),
                                                       self.ws.numel(), _stream(None)))
        self.prep_ws: List[torch.Tensor] = []
        for _ in range(prepare_slots):
            ws = _aligned_empty(self.layout.prep_bytes, self.device)
            _check(lib().gnn_step_prepare_workspace_init(ctypes.byref(m), graph_n, batch, _ptr(ws), ws.numel(),
                                                         _stream(None)))
            self.prep_ws.append(ws)
        self.comp_ws = _aligned_empty(self.layout.compute_bytes, self.device) if prepare_slots else None
        self.loss = torch.zeros(1, dtype=torch.float32, device=self.device)
        self.edges = torch.zeros(1, dtype=torch.int64, device=self.device)
        self._viewing = None  # (prepare ws, compute ws) that the views read

    def step(self, graph: DeviceGraph, table: torch.Tensor, labels: torch.Tensor, targets: torch.Tensor, seed: int,
             step: int, lr: float, gcn_norm_t: Optional[torch.Tensor] = None, loc: int = GNN_LOC_DEVICE,
             edges_out: Optional[torch.Tensor] = None, stream=None) -> None:
        """Enqueue one training step.  The loss lands in self.loss and the
        sampled-edge count in edges_out (an int64 device scalar view) or
        self.edges."""
        e = self.edges if edges_out is None else edges_out
        _check(lib().gnn_train_step(ctypes.byref(self.model), ctypes.byref(graph.c), _ptr(gcn_norm_t), _ptr(table),
                                    dtype_code(table.dtype), loc, table.stride(0), _ptr(labels), _ptr(targets),
                                    self.batch, seed, step, float(lr), _ptr(self.loss), _ptr(e),
                                    _ptr(self.ws), self.ws.numel(), _stream(stream)))
        self._viewing = None

    def prepare(self, slot: int, graph: DeviceGraph, table: torch.Tensor, targets: torch.Tensor, seed: int, step: int,
                gcn_norm_t: Optional[torch.Tensor] = None, loc: int = GNN_LOC_DEVICE, stream=None) -> None:
        """Enqueue the prepare stage of one step into prepare slot ``slot``."""
        ws = self.prep_ws[slot]
        _check(lib().gnn_step_prepare(ctypes.byref(self.model), ctypes.byref(graph.c), _ptr(gcn_norm_t), _ptr(table),
                                      dtype_code(table.dtype), loc, table.stride(0), _ptr(targets), self.batch, seed,
                                      step, _ptr(ws), ws.numel(), _stream(stream)))

    def compute(self, slot: int, labels: torch.Tensor, lr: float, edges_out: Optional[torch.Tensor] = None,
                stream=None) -> None:
        """Enqueue the compute stage of the step prepared in slot ``slot``."""
        e = self.edges if edges_out is None else edges_out
        ws = self.prep_ws[slot]
        _check(lib().gnn_step_compute(ctypes.byref(self.model), self.graph_n, _ptr(labels), self.batch, float(lr),
                                      _ptr(self.loss), _ptr(e), _ptr(ws), ws.numel(), _ptr(self.comp_ws),
                                      self.comp_ws.numel(), _stream(stream)))
        self._viewing = (ws, self.comp_ws)

    def run_pipelined(self, graph: DeviceGraph, table: torch.Tensor, labels: torch.Tensor, targets, seed: int,
                      first_step: int, steps: int, lr: float, gcn_norm_t: Optional[torch.Tensor] = None,
                      loc: int = GNN_LOC_DEVICE, edges_out: Optional[torch.Tensor] = None,
                      loss_out: Optional[torch.Tensor] = None, prep_stream=None, stream=None) -> None:
        """Enqueue ``steps`` steps through gnn_train_steps: the prepare stage
        (sampling and the gather of X') of a later step runs on prep_stream
        while the compute stage of the current one runs on ``stream``.
        targets: int64 device tensor (steps x batch), or a callable giving
        the target tensor of step number s (stacked here).  edges_out /
        loss_out, if given, are int64 / fp32 device tensors of ``steps``
        per-step values; self.loss holds the last step's loss."""
        nslot = len(self.prep_ws)
        assert nslot >= 2, "run_pipelined needs prepare_slots >= 2"
        if steps == 0:
            return
        if callable(targets):
            targets = torch.stack([targets(first_step + i) for i in range(steps)])
        assert targets.dtype == torch.int64 and targets.is_contiguous() and targets.numel() == steps * self.batch
        ps = prep_stream if prep_stream is not None else torch.cuda.Stream(self.device)
        ws = (_vp * nslot)(*[_ptr(w) for w in self.prep_ws])
        lo = loss_out if loss_out is not None else self._loss_steps(steps)
        _check(lib().gnn_train_steps(ctypes.byref(self.model), ctypes.byref(graph.c), _ptr(gcn_norm_t), _ptr(table),
                                     dtype_code(table.dtype), loc, table.stride(0), _ptr(labels), _ptr(targets),
                                     self.batch, seed, first_step, steps, float(lr), _ptr(lo), _ptr(edges_out), ws,
                                     nslot, self.prep_ws[0].numel(), _ptr(self.comp_ws), self.comp_ws.numel(),
                                     _stream(stream), _stream(ps)))
        with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream(self.device)):
            self.loss.copy_(lo[steps - 1:steps])
        self._keep = (targets, lo)  # alive until the next call; the stream orders their reuse
        # the slot of the last step, as gnn_train_steps assigns them: groups of
        # G = min(4, max(1, nslot // 2)) steps alternate between two halves
        G = min(4, max(1, nslot // 2))
        last = steps - 1
        self._viewing = (self.prep_ws[((last // G) % 2) * G + last % G], self.comp_ws)

    def _loss_steps(self, steps: int) -> torch.Tensor:
        if getattr(self, "_loss_buf", None) is None or self._loss_buf.numel() < steps:
            self._loss_buf = torch.zeros(steps, dtype=torch.float32, device=self.device)
        return self._loss_buf[:steps]

    # --- views into the workspaces (for inspection and tests) --------------
    def _view(self, off: int, numel: int, dtype: torch.dtype, compute: bool = False) -> torch.Tensor:
        esz = torch.empty(0, dtype=dtype).element_size()
        if self._viewing is not None:
            base = self._viewing[1] if compute else self._viewing[0]
        else:
            base = self.ws[self.layout.prep_bytes:] if compute else self.ws
        return base[off:off + numel * esz].view(dtype)

    def block_view(self, h: int) -> dict:
        """Host copy of the block built at hop h (1-based) by the last step."""
        lay = self.layout
        i = h - 1
        counts = self._view(lay.blk_counts[i], 4, torch.int64).cpu().tolist()
        n_dst, n_src, nnz = counts[0], counts[1], counts[2]
        out = {
            "n_dst": n_dst, "n_src": n_src, "nnz": nnz,
            "src_ids": self._view(lay.blk_src_ids[i], n_src, torch.int64).cpu().numpy(),
            "rowptr": self._view(lay.blk_rowptr[i], n_dst + 1, torch.int64).cpu().numpy(),
            "col": self._view(lay.blk_col[i], nnz, torch.int32).cpu().numpy(),
        }
        if lay.blk_cscptr[i]:
            out["cscptr"] = self._view(lay.blk_cscptr[i], n_src + 1, torch.int64).cpu().numpy()
            out["cscrow"] = self._view(lay.blk_cscrow[i], nnz, torch.int32).cpu().numpy()
        return out

    def error_word(self) -> torch.Tensor:
        """The device error word of the last call (view of one int64)."""
        return self._view(self.layout.error, 1, torch.int64, compute=True)

    def check_device_errors(self, stream=None) -> None:
        """Raise GnnError (GNN_EDEVICE) if the last call's blocks flagged a
        device-side error."""
        check_device_errors(self.error_word(), stream)

    def act_dtype(self) -> torch.dtype:
        return torch_dtype(self.precision)

    def tensor(self, name: str, layer: int, rows: int, cols: int, dtype: torch.dtype) -> torch.Tensor:
        """View of a step buffer of the last step (agg/h/grad/d_a/argmax per
        layer; x0 and the rest by name)."""
        per_layer = ("agg", "h", "grad", "d_a", "argmax")
        off = getattr(self.layout, name)[layer] if name in per_layer else getattr(self.layout, name)
        compute = name in _COMPUTE_BUFFERS and not (name == "agg" and layer == 1)  # layer 1's: prepare stage
        return self._view(off, rows * cols, dtype, compute=compute).view(rows, cols)
