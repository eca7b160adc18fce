"""CPU oracle for sampled mini-batch GNN training (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU product path never imports it, and it imports
nothing from that path.

The arithmetic lives in ``oracle.c`` (plain loops, double-precision sums);
this module marshals numpy arrays into it and composes one training step in
the order the paper gives (Section II-B: sample, load features, L forward
layers, loss, backward in reverse, weight update; Section V, equation
T_Trainer: the first layer's backward is the update alone).

Array conventions: float32 -> fp32, float64 -> fp64, float16 -> fp16, and
uint16 arrays hold raw bfloat16 bits.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
import threading
from typing import List, Optional, Sequence

import numpy as np

F32, BF16, F16, F64 = 0, 1, 2, 3
SAGE, GCN = 0, 1
SAGE_MAX = 2  # GraphSAGE with the max aggregator (its update reads [h_self || max] like SAGE)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_SO = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with gcc (plain C11 + OpenMP)."""
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        tmp = _SO + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _SO)
    return _SO


def lib():
    global _lib
    with _lock:
        if _lib is None:
            build()
            L = ctypes.CDLL(_SO)
            u64, i64, i32, vp, dbl = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_double
            L.orc_mix64.restype = u64
            L.orc_mix64.argtypes = [u64]
            L.orc_sample_key.restype = u64
            L.orc_sample_key.argtypes = [u64, u64, u64, u64, u64]
            L.orc_bounded.restype = u64
            L.orc_bounded.argtypes = [u64, u64]
            L.orc_sample_positions.restype = i64
            L.orc_sample_positions.argtypes = [i64, i32, u64, u64, i32, i64, vp]
            L.orc_gcn_norm.restype = None
            L.orc_gcn_norm.argtypes = [i64, vp, vp]
            L.orc_build_block.restype = ctypes.c_int
            L.orc_build_block.argtypes = [i64, vp, vp, vp, i64, i32, u64, u64, i32, i64, i64,
                                          vp, vp, vp, vp, vp, vp, vp]
            L.orc_gather.restype = None
            L.orc_gather.argtypes = [vp, ctypes.c_int, i64, i64, vp, i64, vp, ctypes.c_int]
            L.orc_aggregate_fwd.restype = None
            L.orc_aggregate_fwd.argtypes = [ctypes.c_int, i64, vp, vp, vp, vp, ctypes.c_int, i64, vp, ctypes.c_int]
            L.orc_aggregate_fwd_max.restype = None
            L.orc_aggregate_fwd_max.argtypes = [i64, vp, vp, vp, ctypes.c_int, i64, vp, ctypes.c_int, vp]
            L.orc_aggregate_bwd_max.restype = None
            L.orc_aggregate_bwd_max.argtypes = [i64, i64, vp, vp, ctypes.c_int, i64, vp, ctypes.c_int, vp,
                                                ctypes.c_int]
            L.orc_aggregate_bwd.restype = None
            L.orc_aggregate_bwd.argtypes = [ctypes.c_int, i64, i64, vp, vp, vp, vp, ctypes.c_int, i64,
                                            vp, ctypes.c_int, vp, ctypes.c_int]
            L.orc_update_fwd.restype = None
            L.orc_update_fwd.argtypes = [i64, vp, vp, ctypes.c_int, i64, vp, ctypes.c_int, vp, ctypes.c_int,
                                         i64, ctypes.c_int, ctypes.c_int, vp, ctypes.c_int]
            L.orc_update_bwd.restype = None
            L.orc_update_bwd.argtypes = [i64, vp, vp, ctypes.c_int, i64, vp, ctypes.c_int, vp, ctypes.c_int,
                                         i64, ctypes.c_int, vp, vp, vp, ctypes.c_int]
            L.orc_softmax_ce.restype = dbl
            L.orc_softmax_ce.argtypes = [i64, i64, vp, ctypes.c_int, vp, vp, ctypes.c_int]
            L.orc_sgd.restype = None
            L.orc_sgd.argtypes = [i64, vp, ctypes.c_int, vp, ctypes.c_int, dbl]
            L.orc_f32_to_bf16.restype = ctypes.c_uint16
            L.orc_f32_to_bf16.argtypes = [ctypes.c_float]
            L.orc_bf16_to_f32.restype = ctypes.c_float
            L.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
            L.orc_f16_to_f32.restype = ctypes.c_float
            L.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
            L.orc_set_threads.restype = None
            L.orc_set_threads.argtypes = [ctypes.c_int]
            L.orc_get_threads.restype = ctypes.c_int
            L.orc_get_threads.argtypes = []
            _lib = L
    return _lib


# ---------------------------------------------------------------------------
# helpers
# ---------------------------------------------------------------------------

def _code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.float64:
        return F64
    if a.dtype == np.float16:
        return F16
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"unsupported dtype {a.dtype}")


def _np_dtype(code: int):
    return {F32: np.float32, F64: np.float64, F16: np.float16, BF16: np.uint16}[code]


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "arrays passed to the oracle must be C-contiguous"
    return a.ctypes.data


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def set_threads(n: int) -> None:
    lib().orc_set_threads(int(n))


def get_threads() -> int:
    return int(lib().orc_get_threads())


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16, vectorised over the C routine's rule
    (used only to prepare expected values, never on the product path)."""
    x = _c(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def bf16_bits_to_f32(b) -> np.ndarray:
    return (_c(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_float64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


# ---------------------------------------------------------------------------
# sampler
# ---------------------------------------------------------------------------

def mix64(z: int) -> int:
    return int(lib().orc_mix64(z & 0xFFFFFFFFFFFFFFFF))


def sample_key(seed, step, hop, v, t) -> int:
    return int(lib().orc_sample_key(seed, step, hop, v, t))


def bounded(key: int, bound: int) -> int:
    return int(lib().orc_bounded(key, bound))


def sample_positions(d: int, k: int, seed: int, step: int, hop: int, v: int) -> np.ndarray:
    out = np.zeros(max(1, min(d, k)), dtype=np.int64)
    cnt = lib().orc_sample_positions(d, k, seed, step, hop, v, _p(out))
    return out[:cnt].copy()


def gcn_norm(rowptr: np.ndarray) -> np.ndarray:
    rowptr = _c(rowptr, np.int64)
    n = rowptr.size - 1
    out = np.zeros(n, dtype=np.float32)
    lib().orc_gcn_norm(n, _p(rowptr), _p(out))
    return out


@dataclasses.dataclass
class Block:
    src_ids: np.ndarray   # int64 [n_src], dst first
    rowptr: np.ndarray    # int64 [n_dst+1]
    col: np.ndarray       # int32 [nnz] local source index
    cscptr: np.ndarray    # int64 [n_src+1]
    cscrow: np.ndarray    # int32 [nnz]
    n_dst: int

    @property
    def n_src(self) -> int:
        return int(self.src_ids.size)

    @property
    def nnz(self) -> int:
        return int(self.col.size)


def build_block(rowptr, col, dst, fanout: int, seed: int, step: int, hop: int) -> Block:
    rowptr = _c(rowptr, np.int64)
    col = _c(col, np.int64)
    dst = _c(dst, np.int64)
    n = rowptr.size - 1
    n_dst = dst.size
    cap_nnz = max(1, n_dst * fanout)
    cap_src = n_dst + cap_nnz
    src_ids = np.zeros(cap_src, dtype=np.int64)
    brow = np.zeros(n_dst + 1, dtype=np.int64)
    bcol = np.zeros(cap_nnz, dtype=np.int32)
    cscptr = np.zeros(cap_src + 1, dtype=np.int64)
    cscrow = np.zeros(cap_nnz, dtype=np.int32)
    n_src = np.zeros(1, dtype=np.int64)
    nnz = np.zeros(1, dtype=np.int64)
    rc = lib().orc_build_block(n, _p(rowptr), _p(col), _p(dst), n_dst, fanout, seed, step, hop, cap_src, cap_nnz,
                               _p(src_ids), _p(n_src), _p(brow), _p(bcol), _p(nnz), _p(cscptr), _p(cscrow))
    if rc != 0:
        raise ValueError(f"orc_build_block failed with {rc}")
    ns, ne = int(n_src[0]), int(nnz[0])
    return Block(src_ids[:ns].copy(), brow, bcol[:ne].copy(), cscptr[:ns + 1].copy(), cscrow[:ne].copy(), n_dst)


# ---------------------------------------------------------------------------
# gather, aggregation, update, loss, optimizer
# ---------------------------------------------------------------------------

def gather(table: np.ndarray, ids, out_code: int) -> np.ndarray:
    table = np.ascontiguousarray(table)
    ids = _c(ids, np.int64)
    dim = table.shape[1]
    out = np.zeros((ids.size, dim), dtype=_np_dtype(out_code))
    lib().orc_gather(_p(table), _code(table), dim, dim, _p(ids), ids.size, _p(out), out_code)
    return out


def aggregate_fwd(kind: int, blk: Block, src_norm: Optional[np.ndarray], h: np.ndarray, out_code: int) -> np.ndarray:
    h = np.ascontiguousarray(h)
    f = h.shape[1]
    assert h.shape[0] >= blk.n_src
    out = np.zeros((blk.n_dst, f), dtype=_np_dtype(out_code))
    sn = _c(src_norm, np.float32) if src_norm is not None else None
    if kind not in (SAGE, GCN):
        raise ValueError(f"aggregate_fwd: kind {kind} (the max aggregator is aggregate_fwd_max)")
    if kind == GCN and sn is None:
        raise ValueError("GCN aggregation needs per-source norms")
    lib().orc_aggregate_fwd(kind, blk.n_dst, _p(blk.rowptr), _p(blk.col), _p(sn), _p(h), _code(h), f,
                            _p(out), out_code)
    return out


def aggregate_bwd(kind: int, blk: Block, src_norm, d_a: np.ndarray, f: int, h_below: Optional[np.ndarray],
                  out_code: int) -> np.ndarray:
    if kind not in (SAGE, GCN):
        raise ValueError(f"aggregate_bwd: kind {kind} (the max aggregator is aggregate_bwd_max)")
    d_a = np.ascontiguousarray(d_a)
    sn = _c(src_norm, np.float32) if src_norm is not None else None
    out = np.zeros((blk.n_src, f), dtype=_np_dtype(out_code))
    hb = np.ascontiguousarray(h_below) if h_below is not None else None
    lib().orc_aggregate_bwd(kind, blk.n_dst, blk.n_src, _p(blk.rowptr), _p(blk.col), _p(sn), _p(d_a), _code(d_a), f,
                            _p(hb), _code(hb) if hb is not None else F32, _p(out), out_code)
    return out


def aggregate_fwd_max(blk: Block, h: np.ndarray, out_code: int):
    """GraphSAGE's max aggregator: (out, argmax) with argmax the winning
    source of each output element (-1 for rows without neighbours)."""
    h = np.ascontiguousarray(h)
    f = h.shape[1]
    assert h.shape[0] >= blk.n_src
    out = np.zeros((blk.n_dst, f), dtype=_np_dtype(out_code))
    arg = np.zeros((blk.n_dst, f), dtype=np.int32)
    lib().orc_aggregate_fwd_max(blk.n_dst, _p(blk.rowptr), _p(blk.col), _p(h), _code(h), f, _p(out), out_code,
                                _p(arg))
    return out, arg


def aggregate_bwd_max(blk: Block, argmax: np.ndarray, d_a: np.ndarray, f: int, h_below: Optional[np.ndarray],
                      out_code: int) -> np.ndarray:
    """Backward of the max aggregator from its argmax table; d_a has 2f
    columns (self part, then max part)."""
    d_a = np.ascontiguousarray(d_a)
    argmax = _c(argmax, np.int32)
    out = np.zeros((blk.n_src, f), dtype=_np_dtype(out_code))
    hb = np.ascontiguousarray(h_below) if h_below is not None else None
    lib().orc_aggregate_bwd_max(blk.n_dst, blk.n_src, _p(argmax), _p(d_a), _code(d_a), f, _p(hb),
                                _code(hb) if hb is not None else F32, _p(out), out_code)
    return out


def update_fwd(a_self: np.ndarray, a_nbr: Optional[np.ndarray], w: np.ndarray, b: Optional[np.ndarray], relu: bool,
               gemm_code: int, out_code: int) -> np.ndarray:
    a_self = np.ascontiguousarray(a_self)
    m, k_each = a_self.shape
    if a_nbr is not None:
        a_nbr = np.ascontiguousarray(a_nbr)
        assert a_nbr.shape == a_self.shape and a_nbr.dtype == a_self.dtype
    w = np.ascontiguousarray(w)
    nout = w.shape[1]
    out = np.zeros((m, nout), dtype=_np_dtype(out_code))
    bb = np.ascontiguousarray(b) if b is not None else None
    lib().orc_update_fwd(m, _p(a_self), _p(a_nbr), _code(a_self), k_each, _p(w), _code(w), _p(bb),
                         _code(bb) if bb is not None else F32, nout, int(relu), gemm_code, _p(out), out_code)
    return out


def update_bwd(a_self: np.ndarray, a_nbr: Optional[np.ndarray], w: np.ndarray, g: np.ndarray, gemm_code: int,
               want_da: bool, out_code: int = F32):
    a_self = np.ascontiguousarray(a_self)
    m, k_each = a_self.shape
    if a_nbr is not None:
        a_nbr = np.ascontiguousarray(a_nbr)
    K = 2 * k_each if a_nbr is not None else k_each
    w = np.ascontiguousarray(w)
    g = np.ascontiguousarray(g)
    nout = w.shape[1]
    dt = _np_dtype(out_code)
    dw = np.zeros((K, nout), dtype=dt)
    db = np.zeros(nout, dtype=dt)
    da = np.zeros((m, K), dtype=dt) if want_da else None
    lib().orc_update_bwd(m, _p(a_self), _p(a_nbr), _code(a_self), k_each, _p(w), _code(w), _p(g), _code(g), nout,
                         gemm_code, _p(dw), _p(db), _p(da), out_code)
    return dw, db, da


def softmax_ce(logits: np.ndarray, y, out_code: int = F32):
    logits = np.ascontiguousarray(logits)
    y = _c(y, np.int64)
    b, c = logits.shape
    g = np.zeros((b, c), dtype=_np_dtype(out_code))
    loss = lib().orc_softmax_ce(b, c, _p(logits), _code(logits), _p(y), _p(g), out_code)
    return float(loss), g


def sgd(w: np.ndarray, dw: np.ndarray, lr: float) -> np.ndarray:
    w = np.array(w, copy=True, order="C")
    dw = np.ascontiguousarray(dw)
    lib().orc_sgd(w.size, _p(w), _code(w), _p(dw), _code(dw), float(lr))
    return w


# ---------------------------------------------------------------------------
# one training step
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class StepConfig:
    kind: int                  # SAGE, GCN or SAGE_MAX
    dims: Sequence[int]        # f^0..f^L
    fanouts: Sequence[int]     # hop order: fanouts[0] sampled around the targets
    precision: int             # F32, BF16 or F64 (storage of X', M, H; GEMM operand rounding)
    seed: int = 0
    step: int = 0
    lr: float = 0.01


def sample_blocks(rowptr, col, targets, cfg: StepConfig) -> List[Block]:
    """blocks[h-1] is built at hop h; it is the block of layer L-h+1."""
    blocks: List[Block] = []
    dst = np.asarray(targets, dtype=np.int64)
    for h in range(1, len(cfg.fanouts) + 1):
        blk = build_block(rowptr, col, dst, cfg.fanouts[h - 1], cfg.seed, cfg.step, h)
        blocks.append(blk)
        dst = blk.src_ids
    return blocks


def _flip_decisions(h: np.ndarray, flip: np.ndarray) -> np.ndarray:
    """Copy of stored activations h whose test h > 0 is inverted where flip
    is True (values elsewhere unchanged).  Only the backward ReLU mask reads
    the copy."""
    hv = to_float64(h)
    f = np.asarray(flip, dtype=bool)
    assert f.shape == hv.shape
    out = np.array(h, copy=True)
    off = f & (hv > 0)
    on = f & ~(hv > 0)
    if out.dtype == np.uint16:          # bf16 bits
        out[off] = 0
        out[on] = 0x3F80                # 1.0
    else:
        out[off] = 0
        out[on] = 1
    return out


def train_step(rowptr, col, nrm, table, labels, targets, weights, biases, cfg: StepConfig,
               blocks: Optional[List[Block]] = None, relu_flip: Optional[dict] = None) -> dict:
    """One iteration of sampled mini-batch training; returns every
    intermediate plus the updated weights.

    Storage precision: X', M^l (or A^l) and H^l (l < L) are stored in the
    precision mode (bf16 in bf16 mode); logits, gradients and weights are
    fp32 (fp64 in fp64 mode).  GEMM operands are rounded to bf16 in bf16 mode.

    relu_flip (optional): {l: bool array shaped like H^l} inverting the
    backward's ReLU decision (H^l > 0) at the marked positions, for parity
    checks where an implementation that sums in another order takes the other
    side of a decision whose pre-activation is within rounding of zero.  The
    forward pass is not changed.
    """
    L = len(cfg.dims) - 1
    assert len(cfg.fanouts) == L and len(weights) == L
    act = cfg.precision                                   # storage of activations
    wide = F64 if cfg.precision == F64 else F32           # logits / gradients
    gemm = BF16 if cfg.precision == BF16 else cfg.precision
    if blocks is None:
        blocks = sample_blocks(rowptr, col, targets, cfg)
    layer_block = {l: blocks[L - l] for l in range(1, L + 1)}
    x0 = gather(table, blocks[-1].src_ids, act)
    src_norms = {}
    if cfg.kind == GCN:
        for l in range(1, L + 1):
            src_norms[l] = np.ascontiguousarray(nrm[layer_block[l].src_ids], dtype=np.float32)

    cat = cfg.kind in (SAGE, SAGE_MAX)                    # A = [h_self || aggregation]
    H = {0: x0}
    AGG, ARG = {}, {}
    for l in range(1, L + 1):
        blk = layer_block[l]
        if cfg.kind == SAGE_MAX:
            AGG[l], ARG[l] = aggregate_fwd_max(blk, H[l - 1], act)
        else:
            AGG[l] = aggregate_fwd(cfg.kind, blk, src_norms.get(l), H[l - 1], act)
        last = l == L
        a_self = np.ascontiguousarray(H[l - 1][:blk.n_dst]) if cat else AGG[l]
        a_nbr = AGG[l] if cat else None
        H[l] = update_fwd(a_self, a_nbr, weights[l - 1], biases[l - 1], relu=not last, gemm_code=gemm,
                          out_code=wide if last else act)
    y = np.asarray(labels, dtype=np.int64)[np.asarray(targets, dtype=np.int64)]
    loss, G = softmax_ce(H[L], y, wide)

    dW, dB, GR = {}, {}, {L: G}
    for l in range(L, 0, -1):
        blk = layer_block[l]
        a_self = np.ascontiguousarray(H[l - 1][:blk.n_dst]) if cat else AGG[l]
        a_nbr = AGG[l] if cat else None
        dw, db, da = update_bwd(a_self, a_nbr, weights[l - 1], GR[l], gemm, want_da=l > 1, out_code=wide)
        dW[l], dB[l] = dw, db
        if l > 1:
            f = cfg.dims[l - 1]
            h_mask = H[l - 1]
            if relu_flip and (l - 1) in relu_flip:
                h_mask = _flip_decisions(H[l - 1], relu_flip[l - 1])
            if cfg.kind == SAGE_MAX:
                GR[l - 1] = aggregate_bwd_max(blk, ARG[l], da, f, h_mask, wide)
            else:
                GR[l - 1] = aggregate_bwd(cfg.kind, blk, src_norms.get(l), da, f, h_mask, wide)
    new_w = [sgd(weights[l - 1], dW[l], cfg.lr) for l in range(1, L + 1)]
    new_b = [sgd(biases[l - 1], dB[l], cfg.lr) for l in range(1, L + 1)]
    return {
        "blocks": blocks, "x0": x0, "H": H, "AGG": AGG, "ARG": ARG, "loss": loss, "G": GR, "dW": dW, "dB": dB,
        "new_w": new_w, "new_b": new_b, "edges": int(sum(b.nnz for b in blocks)),
    }
