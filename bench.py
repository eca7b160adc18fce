"""Throughput of sampled mini-batch GNN training steps on one MI355X.

Default workload: R-MAT graph with 2,449,029 vertices and 61,859,140
undirected edges (products-sized), 100-dim fp32 features resident in HBM,
47 classes, 2-layer GraphSAGE-mean (hidden 256), batch 1024, fanouts (25, 10),
bf16 GEMM operands with fp32 accumulation.  Inputs are synthetic and seeded.

One step = sample both hops, gather X', forward, loss, backward, SGD, all in
one gnn_train_step call.  Prints one JSON line:
  value          sampled edges per second over the timed steps (sum of the
                 device edge counters / elapsed time)
  steps_per_s    training steps per second
  roofline       the dominant single-kernel stage, timed with HIP events in a
                 staged run of the same step, against its algorithmic bytes
  cpu_baseline   the CPU oracle on a bounded sample of the same workload
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402

HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
# Source files of each single-kernel stage's kernel (their hash ties a
# counter measurement to the code it was taken on).
KERNEL_SOURCES = {
    "fwd_l1l2": ["paper_2303_00158_amd/csrc/fused_two.hip", "paper_2303_00158_amd/csrc/fused_dev.h",
                 "paper_2303_00158_amd/csrc/internal.h"],
    "layer_fwd": ["paper_2303_00158_amd/csrc/fused_layer.hip", "paper_2303_00158_amd/csrc/fused_dev.h",
                  "paper_2303_00158_amd/csrc/internal.h"],
    "update_fwd": ["paper_2303_00158_amd/csrc/gemm_fwd.hip", "paper_2303_00158_amd/csrc/fused_layer.hip",
                   "paper_2303_00158_amd/csrc/gemm_engine.h", "paper_2303_00158_amd/csrc/internal.h"],
    "agg_fwd": ["paper_2303_00158_amd/csrc/aggregate.hip", "paper_2303_00158_amd/csrc/aggregate_dev.h",
                "paper_2303_00158_amd/csrc/jobs.h", "paper_2303_00158_amd/csrc/internal.h"],
    "gather": ["paper_2303_00158_amd/csrc/gather.hip", "paper_2303_00158_amd/csrc/gather_dev.h",
               "paper_2303_00158_amd/csrc/jobs.h", "paper_2303_00158_amd/csrc/internal.h"],
    "agg_bwd": ["paper_2303_00158_amd/csrc/aggregate.hip", "paper_2303_00158_amd/csrc/aggregate_dev.h",
                "paper_2303_00158_amd/csrc/jobs.h", "paper_2303_00158_amd/csrc/internal.h"],
    "bwd_l1l2": ["paper_2303_00158_amd/csrc/bwd_two.hip", "paper_2303_00158_amd/csrc/bwd_pull_dev.h",
                 "paper_2303_00158_amd/csrc/gemm_bwd_dev.h", "paper_2303_00158_amd/csrc/gemm_engine.h",
                 "paper_2303_00158_amd/csrc/aggregate_dev.h", "paper_2303_00158_amd/csrc/jobs.h",
                 "paper_2303_00158_amd/csrc/internal.h"],
    "update_bwd": ["paper_2303_00158_amd/csrc/gemm_bwd.hip", "paper_2303_00158_amd/csrc/gemm_bwd_dev.h",
                   "paper_2303_00158_amd/csrc/gemm_engine.h", "paper_2303_00158_amd/csrc/jobs.h",
                   "paper_2303_00158_amd/csrc/internal.h"],
}
HOST_LINK_PEAK_GBS = 64.0  # PCIe Gen5 x16, one direction
BF16_PEAK_TFLOPS = 2500.0
FP32_PEAK_TFLOPS = 157.3


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default=workloads.RMAT_SAGE.name, choices=sorted(workloads.PRESETS))
    p.add_argument("--stage-steps", type=int, default=5, help="steps of the event-instrumented staged run")
    p.add_argument("--no-stages", action="store_true")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="CPU oracle baseline: run whole oracle steps until this much time has passed")
    p.add_argument("--replays", type=int, default=20, help="back-to-back launches timing the roofline kernel")
    p.add_argument("--lr", type=float, default=0.01)
    p.add_argument("--scale-batches", default="8192,32768",
                   help="comma-separated mini-batch sizes at which the single-kernel stages are also timed "
                        "(same graph and model; empty: skip)")
    p.add_argument("--scale-n", type=int, default=0, help="run the workload's model on an R-MAT graph of this many "
                   "vertices (the edge count scales with it unless --scale-m is given)")
    p.add_argument("--scale-m", type=int, default=0)
    p.add_argument("--prepare-slots", type=int, default=8,
                   help="prepare workspaces of the pipelined steps; steps go in groups of half as many")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="first run a plain device copy (fp32 -> int32 elementwise) of this many MiB three times, the "
                        "known-size kernel that scales HBM traffic counters")
    p.add_argument("--other-workloads", default="rmat2.4m-gcn,rmat2.4m-sagemax,tiny-er10k-gcn,fp32,rmat111m-sage3,"
                                                 "rmat244m-sage-hosttable",
                   help="comma-separated workloads also timed (pipelined) after the headline, each with its own "
                        "roofline; 'fp32' is the headline workload in fp32; empty: none")
    p.add_argument("--other-steps", type=int, default=20)
    p.add_argument("--other-warmup", type=int, default=5)
    p.add_argument("--host-table-n", type=int, default=30_000_000,
                   help="vertices of the graph the host-table workload is scaled to (its full table needs 375 GB "
                        "of pinned host memory)")
    p.add_argument("--cpu-seconds-one-thread", type=float, default=6.0,
                   help="CPU oracle baseline: also run it on one thread for about this long")
    p.add_argument("--pipeline", action=argparse.BooleanOptionalAction, default=None,
                   help="two-stage steps (gnn_train_steps) with the prepare stage (sampling, gather) of step s+1 "
                        "overlapping the compute stage of step s (default: on; --no-pipeline times one "
                        "gnn_train_step call per step)")
    return p.parse_args()


def source_hash(stage: str) -> str:
    import hashlib
    key = next((k for k in KERNEL_SOURCES if stage.startswith(k)), None)
    if key is None:
        return ""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[key]:
        with open(os.path.join(ROOT, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(stage: str, workload: str):
    """HBM bytes per launch of `stage` on `workload` from the committed
    counter summaries (profiles/*_hbm_counters.md: rows of
    | stage | workload | source hash | FETCH_SIZE KiB | WRITE_SIZE KiB | fetch scale | write scale | bytes |),
    or None when there is none for the current source of the kernel."""
    if not os.path.isdir(PROFILES):
        return None
    want = source_hash(stage)
    for fn in sorted(os.listdir(PROFILES)):
        if not fn.endswith("_hbm_counters.md"):
            continue
        for line in open(os.path.join(PROFILES, fn)):
            cells = [c.strip().strip("`") for c in line.strip().strip("|").split("|")]
            if len(cells) == 8 and cells[0] == stage and cells[1] == workload and cells[2] == want and want:
                try:
                    return int(cells[7])
                except ValueError:
                    return None
    return None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kind_code(gnn, kind: str) -> int:
    return {"sage": gnn.GNN_AGG_SAGE_MEAN, "gcn": gnn.GNN_AGG_GCN_SYM, "sage-max": gnn.GNN_AGG_SAGE_MAX}[kind]


# ---------------------------------------------------------------------------
# staged step: the same iteration through the individual ABI calls, with HIP
# events between them (on torch's current stream, which the calls use)
# ---------------------------------------------------------------------------

class StagedStep:
    def __init__(self, gnn, w: workloads.Workload, graph, batch_size, act, loc):
        self.gnn, self.w, self.graph, self.act, self.loc = gnn, w, graph, act, loc
        dev = graph.rowptr.device
        L = w.num_layers
        self.L = L
        self.kind = kind_code(gnn, w.kind)
        self.maxagg = self.kind == gnn.GNN_AGG_SAGE_MAX
        self.blocks = []
        cap = batch_size
        ws_bytes = 0
        for h in range(L):
            blk = gnn.DeviceBlock(graph.n, cap, w.fanouts[h], h < L - 1, w.kind == "gcn", dev)
            self.blocks.append(blk)
            nb = ctypes.c_size_t()
            gnn._check(gnn.lib().gnn_sampler_workspace_size(graph.n, cap, w.fanouts[h], ctypes.byref(nb)))
            ws_bytes = max(ws_bytes, nb.value)
            cap = blk.c.cap_src
        self.samp_ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        gnn._check(gnn.lib().gnn_sampler_workspace_init(self.samp_ws.data_ptr(), ws_bytes, graph.n,
                                                        gnn._stream(None)))
        dims = w.dims
        self.x0 = torch.empty((self.blocks[-1].c.cap_src, dims[0]), dtype=act, device=dev)
        self.agg, self.h, self.grad, self.da, self.argmax = {}, {}, {}, {}, {}
        for l in range(1, L + 1):
            rows = self.blocks[L - l].c.cap_dst
            self.agg[l] = torch.empty((rows, dims[l - 1]), dtype=act, device=dev)
            # the max aggregator's argmax tables, kept for the layers whose
            # aggregation has a backward (as in the training step)
            self.argmax[l] = (torch.empty((rows, dims[l - 1]), dtype=torch.int32, device=dev)
                              if self.maxagg and l > 1 else None)
            self.h[l] = torch.empty((rows, dims[l]), dtype=act if l < L else torch.float32, device=dev)
            self.grad[l] = torch.empty((rows, dims[l]), dtype=torch.float32, device=dev)
            if l > 1:
                self.da[l] = torch.empty((rows, w.k_of_layer(l)), dtype=torch.float32, device=dev)
        self.loss = torch.zeros(1, device=dev)
        self.row_loss = torch.empty(batch_size, device=dev)
        self.fused = {}  # layer -> whether gnn_layer_fwd serves it (as inside the training step)
        self.two = None  # whether gnn_two_layer_fwd serves both layers (as inside the training step)
        self.two_bwd = None  # whether gnn_two_layer_bwd serves their backward (as inside the training step)
        self.two_ws = None
        gemm = gnn.GNN_BF16 if act == torch.bfloat16 else gnn.GNN_F32
        self.fwd_ws, self.bwd_ws = {}, {}
        for l in range(1, L + 1):
            rows = self.blocks[L - l].c.cap_dst
            nb = ctypes.c_size_t()
            gnn._check(gnn.lib().gnn_update_fwd_workspace_size(w.k_of_layer(l), dims[l], rows, gemm, ctypes.byref(nb)))
            self.fwd_ws[l] = torch.zeros(max(nb.value, 256), dtype=torch.uint8, device=dev)
            self.bwd_ws[l] = gnn.update_bwd_workspace(w.k_of_layer(l), dims[l], rows, gemm, dev)

    def layer_fwd(self, l, trainer, labels):
        """gnn_layer_fwd for layer l on the blocks of the last run."""
        gnn, L = self.gnn, self.L
        blk, hin = self.blocks[L - l], (self.x0 if l == 1 else self.h[l - 1])
        kw = {}
        if l == L:
            kw = dict(labels=labels, batch=self.blocks[0].c.cap_dst, g_out=self.grad[L], row_loss=self.row_loss)
        gnn.layer_fwd(blk, self.kind, self.w.fanouts[L - l], hin, trainer.wt[l - 1], trainer.b[l - 1], self.agg[l],
                      self.h[l], **kw)

    def two_layer_fwd(self, trainer, labels):
        """gnn_two_layer_fwd on the blocks of the last run (layer 1's
        aggregation already in agg[1])."""
        gnn = self.gnn
        if self.maxagg:
            gnn.two_layer_fwd_max(self.blocks[0], self.w.fanouts[0], self.x0, self.agg[1], trainer.wt[0],
                                  trainer.b[0], self.h[1], trainer.wt[1], trainer.b[1], self.agg[2], self.argmax[2],
                                  self.h[2], labels, self.blocks[0].c.cap_dst, self.grad[2], self.row_loss,
                                  self.da[2])
            return
        sage = self.kind == gnn.GNN_AGG_SAGE_MEAN
        gnn.two_layer_fwd(self.blocks[0], self.kind, self.w.fanouts[0], self.x0 if sage else None, self.agg[1],
                          trainer.wt[0], trainer.b[0], self.h[1], trainer.wt[1], trainer.b[1], self.agg[2], self.h[2],
                          labels, self.blocks[0].c.cap_dst, self.grad[2], self.row_loss, self.da[2])

    def two_layer_bwd(self, trainer):
        """gnn_two_layer_bwd on the blocks and forward values of the last run."""
        gnn = self.gnn
        sage = self.kind == gnn.GNN_AGG_SAGE_MEAN
        b0, b1 = self.blocks
        if self.two_ws is None:
            self.two_ws = gnn.two_layer_bwd_workspace(self.kind, self.w.dims[0], self.w.dims[1], self.w.dims[2],
                                                      b1.c.cap_dst, b0.c.cap_dst, self.x0.device)
        if self.maxagg:
            gnn.two_layer_bwd_max(b0, self.x0, self.agg[1], b1.counts[0:1], b1.c.cap_dst, self.h[1], self.agg[2],
                                  self.argmax[2], self.da[2], self.grad[2], trainer.dw[0], trainer.db[0],
                                  trainer.dw[1], trainer.db[1], ws=self.two_ws)
            return
        gnn.two_layer_bwd(b0, self.kind, self.x0 if sage else None, self.agg[1], b1.counts[0:1], b1.c.cap_dst,
                          self.h[1], self.agg[2], self.da[2], self.grad[2], trainer.dw[0], trainer.db[0],
                          trainer.dw[1], trainer.db[1], ws=self.two_ws)

    def aggregate_fwd(self, blk, l, hin):
        if self.maxagg:
            self.gnn.aggregate_fwd_max(blk, hin, self.agg[l], self.argmax[l])
        else:
            self.gnn.aggregate_fwd(blk, self.kind, hin, self.agg[l])

    def aggregate_bwd(self, blk, l, hin):
        f = self.w.dims[l - 1]
        if self.maxagg:
            self.gnn.aggregate_bwd_max(blk, self.argmax[l], self.da[l], f, self.grad[l - 1], h_below=hin)
        else:
            self.gnn.aggregate_bwd(blk, self.kind, self.da[l], f, self.grad[l - 1], h_below=hin)

    def replay(self, name: str, trainer, table, reps: int, labels=None) -> float:
        """Launch the single ABI call of stage `name` `reps` times back to back
        on the blocks of the last run; returns the mean ms per launch (HIP
        events on the stream the call uses)."""
        gnn, L, w = self.gnn, self.L, self.w
        sage = self.kind != gnn.GNN_AGG_GCN_SYM  # A = [h_self || aggregation]
        gemm = gnn.GNN_BF16 if self.act == torch.bfloat16 else gnn.GNN_F32
        if name == "gather":
            b0 = self.blocks[-1]
            call = lambda: gnn.gather_features(table, b0.src_ids, self.x0, n_ids_dev=b0.counts[1:2],  # noqa
                                               loc=self.loc)
        elif name.startswith("agg_fwd_l"):
            l = int(name[-1])
            blk, hin = self.blocks[L - l], (self.x0 if l == 1 else self.h[l - 1])
            call = lambda: self.aggregate_fwd(blk, l, hin)  # noqa
        elif name.startswith("agg_dedup_l"):
            l = int(name[-1])
            blk, hin = self.blocks[L - l], (self.x0 if l == 1 else self.h[l - 1])
            call = lambda: gnn.aggregate_fwd_dedup(blk, self.kind, hin, self.agg[l])  # noqa
        elif name.startswith("update_fwd_l"):
            l = int(name[-1])
            blk, hin = self.blocks[L - l], (self.x0 if l == 1 else self.h[l - 1])
            call = lambda: gnn.update_fwd(hin if sage else self.agg[l], self.agg[l] if sage else None,  # noqa
                                          trainer.w[l - 1], trainer.b[l - 1], self.h[l], l < L, gemm,
                                          m_dev=blk.counts[0:1], cap_m=blk.c.cap_dst, ws=self.fwd_ws[l],
                                          wt=trainer.wt[l - 1] if trainer.wt else None)
        elif name.startswith("layer_fwd_l"):
            l = int(name[-1])
            call = lambda: self.layer_fwd(l, trainer, labels)  # noqa
        elif name == "fwd_l1l2":
            call = lambda: self.two_layer_fwd(trainer, labels)  # noqa
        elif name == "bwd_l1l2":
            call = lambda: self.two_layer_bwd(trainer)  # noqa
        elif name.startswith("agg_bwd_l"):
            l = int(name[-1])
            blk, hin = self.blocks[L - l], (self.x0 if l == 1 else self.h[l - 1])
            call = lambda: self.aggregate_bwd(blk, l, hin)  # noqa
        elif name.startswith("update_bwd_l"):
            l = int(name[-1])
            blk, hin = self.blocks[L - l], (self.x0 if l == 1 else self.h[l - 1])
            da = None if self.two else self.da.get(l)
            call = lambda: gnn.update_bwd(hin if sage else self.agg[l], self.agg[l] if sage else None,  # noqa
                                          trainer.w[l - 1], self.grad[l], trainer.dw[l - 1], trainer.db[l - 1],
                                          da, gemm, m_dev=blk.counts[0:1], cap_m=blk.c.cap_dst,
                                          ws=self.bwd_ws[l])
        elif name == "sgd":
            def call():
                for l in range(L):
                    gnn.sgd(trainer.w[l], trainer.dw[l], 0.0)
                    gnn.sgd(trainer.b[l], trainer.db[l], 0.0)
        else:
            raise ValueError(name)
        call()
        torch.cuda.synchronize()
        if hasattr(torch.cuda, "_sleep"):
            torch.cuda._sleep(20_000_000)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            call()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def launches(self, name: str) -> int:
        """Kernel launches of a multi-launch stage's ABI calls."""
        if name.startswith("update_bwd") or name == "bwd_l1l2":
            return 2  # the dA/dW GEMMs, then the split-order reduction
        if name == "sgd":
            return 2 * self.L  # one gnn_sgd for W and one for b per layer
        return 1

    def block_sizes(self):
        return [{k: int(v) for k, v in blk.host().items() if k in ("n_dst", "n_src", "nnz")} for blk in self.blocks]

    def run(self, trainer, table, labels, targets, nrm, seed, step, lr, events=None):
        """Enqueue one step; when `events` is a list, record (name, event) pairs."""
        gnn, L, w = self.gnn, self.L, self.w

        def mark(name):
            if events is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                events.append((name, e))

        mark("begin")
        dst, n_dst = targets, None
        for h in range(L):
            blk = self.blocks[h]
            gnn.build_block(self.graph, dst, w.fanouts[h], seed, step, h + 1, blk, self.samp_ws, n_dst_dev=n_dst,
                            gcn_norm_t=nrm if w.kind == "gcn" else None, want_csc=h < L - 1)
            mark(f"sample_hop{h + 1}")
            dst, n_dst = blk.src_ids, blk.counts[1:2]
        b0 = self.blocks[-1]
        gnn.gather_features(table, b0.src_ids, self.x0, n_ids_dev=b0.counts[1:2], loc=self.loc)
        mark("gather")
        sage = self.kind != gnn.GNN_AGG_GCN_SYM  # A = [h_self || aggregation]
        gemm = gnn.GNN_BF16 if self.act == torch.bfloat16 else gnn.GNN_F32
        loss_fused = False
        if L == 2 and self.two is not False and trainer.wt:
            # as in the training step: layer 1's aggregation (the prepare
            # stage's), then both layers, the loss and dA^2 in one launch
            self.aggregate_fwd(self.blocks[1], 1, self.x0)
            mark("agg_fwd_l1")
            try:
                self.two_layer_fwd(trainer, labels)
                self.two = loss_fused = True
                mark("fwd_l1l2")
            except gnn.GnnError as e:
                if e.code != gnn.GNN_EUNSUPPORTED:
                    raise
                self.two = False
        for l in range(1, L + 1 if not self.two else 1):
            blk = self.blocks[L - l]
            hin = self.x0 if l == 1 else self.h[l - 1]
            # as in the training step: layer 1's aggregation belongs to the
            # prepare stage, its update reads it (fused kernel in A-load mode
            # inside gnn_update_fwd); later layers in one gnn_layer_fwd
            if (l > 1 or L == 1) and self.fused.get(l, bool(trainer.wt) and not self.maxagg):  # (sums only)
                try:
                    self.layer_fwd(l, trainer, labels)
                    self.fused[l] = True
                    loss_fused = l == L
                    mark(f"layer_fwd_l{l}")
                    continue
                except gnn.GnnError as e:
                    if e.code != gnn.GNN_EUNSUPPORTED:
                        raise
            self.fused[l] = False
            self.aggregate_fwd(blk, l, hin)
            mark(f"agg_fwd_l{l}")
            gnn.update_fwd(hin if sage else self.agg[l], self.agg[l] if sage else None, trainer.w[l - 1],
                           trainer.b[l - 1], self.h[l], l < L, gemm, m_dev=blk.counts[0:1], cap_m=blk.c.cap_dst,
                           ws=self.fwd_ws[l], wt=trainer.wt[l - 1] if trainer.wt else None)
            mark(f"update_fwd_l{l}")
        if not loss_fused:
            gnn.softmax_ce(self.h[L], labels, targets, self.grad[L], self.loss)
            mark("loss")
        if self.two and self.two_bwd is not False:
            # as in the training step: both layers' dW (layer 2's aggregation
            # backward folded into layer 1's) and their reductions
            try:
                self.two_layer_bwd(trainer)
                self.two_bwd = True
                mark("bwd_l1l2")
            except gnn.GnnError as e:
                if e.code != gnn.GNN_EUNSUPPORTED:
                    raise
                self.two_bwd = False
        for l in range(L, 0, -1) if not self.two_bwd else ():
            blk = self.blocks[L - l]
            hin = self.x0 if l == 1 else self.h[l - 1]
            gnn.update_bwd(hin if sage else self.agg[l], self.agg[l] if sage else None, trainer.w[l - 1],
                           self.grad[l], trainer.dw[l - 1], trainer.db[l - 1],
                           None if self.two else self.da.get(l), gemm, m_dev=blk.counts[0:1], cap_m=blk.c.cap_dst,
                           ws=self.bwd_ws[l])
            mark(f"update_bwd_l{l}")
            if l > 1:
                self.aggregate_bwd(blk, l, hin)
                mark(f"agg_bwd_l{l}")
        for l in range(L):
            gnn.sgd(trainer.w[l], trainer.dw[l], lr)
            gnn.sgd(trainer.b[l], trainer.db[l], lr)
        mark("sgd")

    def stage_bytes(self, name: str):
        """Algorithmic HBM bytes (and flops) of a single-kernel stage, from the
        block sizes of the last run (host copies; call after synchronising)."""
        L, w = self.L, self.w
        S_H = 2 if self.act == torch.bfloat16 else 4
        S_X = 2 if w.table_dtype == "f16" else 4
        if name == "gather":
            b = self.blocks[-1].host()
            n0 = b["n_src"]
            if self.loc == self.gnn.GNN_LOC_HOST_PINNED:
                return n0 * w.dims[0] * S_X, 0  # bytes over the host link
            return n0 * w.dims[0] * (S_X + S_H) + 8 * n0, 0
        if name.startswith("agg_fwd_l"):
            l = int(name[-1])
            b = self.blocks[L - l].host()
            f = w.dims[l - 1]
            R = np.unique(b["col"]).size
            extra = (b["n_dst"] * f * S_H + 4 * b["n_src"]) if w.kind == "gcn" else 0
            if self.argmax.get(l) is not None:
                extra = 4 * b["n_dst"] * f  # the int32 argmax table
            return R * f * S_H + 4 * b["nnz"] + 8 * (b["n_dst"] + 1) + b["n_dst"] * f * S_H + extra, 0
        if name.startswith("update_fwd_l"):
            l = int(name[-1])
            b = self.blocks[L - l].host()
            M, K, N = b["n_dst"], w.k_of_layer(l), w.dims[l]
            out = S_H if l < L else 4
            S_W = 2 if S_H == 2 else 4  # the bf16 shadow of W in bf16 mode
            return M * K * S_H + K * N * S_W + N * 4 + M * N * out, 2 * M * K * N
        if name.startswith("layer_fwd_l"):
            l = int(name[-1])
            b = self.blocks[L - l].host()
            f, N, K = w.dims[l - 1], w.dims[l], w.k_of_layer(l)
            M = b["n_dst"]
            # distinct source rows read: the sampled columns and the rows' own (self) rows
            R = np.union1d(np.unique(b["col"]), np.arange(M)).size
            byts = R * f * S_H + 4 * b["nnz"] + 8 * (M + 1) + K * N * 2 + 4 * N + M * f * S_H
            if w.kind == "gcn":
                byts += 4 * R
            if l == L:
                B = self.blocks[0].c.cap_dst
                byts += M * N * 4 + B * (16 + N * 4 + 4)  # logits; labels, targets, gradient, row loss
            else:
                byts += M * N * S_H
            return byts, 2 * M * K * N
        if name == "fwd_l1l2":
            # reads: the last block, its targets and labels, the A^1 rows of
            # its distinct sources, both layers' weights; writes: H^1 of
            # those rows, M^2, logits, the loss gradient and row losses, dA^2
            b = self.blocks[0].host()
            M, B = b["n_dst"], self.blocks[0].c.cap_dst
            f0, f1, C = w.dims
            K1, K2 = w.k_of_layer(1), w.k_of_layer(2)
            R = np.union1d(np.unique(b["col"]), np.arange(M)).size
            byts = (8 * (M + 1) + 4 * b["nnz"] + 16 * M + R * K1 * S_H + K1 * f1 * 2 + 4 * f1 + K2 * C * 2 + 4 * C
                    + R * f1 * S_H + M * f1 * S_H + M * C * 4 + B * (C * 4 + 4) + M * K2 * 4)
            if w.kind == "gcn":
                byts += 4 * R
            if self.maxagg:
                byts += 4 * M * f1  # the argmax table of M^2
            return byts, 2 * R * K1 * f1 + 4 * M * K2 * C
        if name == "bwd_l1l2":
            # reads: layer 1's A rows, H^1 (the mask), dA^2 (the neighbour
            # part of every destination row, the self part of the
            # destinations), the transpose and row pointers, layer 2's A rows
            # and G^2; writes: both layers' dW and db (the partials of the
            # split reductions are not counted)
            b, b1 = self.blocks[0].host(), self.blocks[1].host()
            M1, M2 = b1["n_dst"], b["n_dst"]
            f0, f1, C = w.dims
            K1, K2 = w.k_of_layer(1), w.k_of_layer(2)
            byts = (M1 * K1 * S_H + M1 * f1 * S_H + M2 * K2 * 4 + 4 * b["nnz"] + 8 * (b["n_src"] + 1)
                    + 8 * (M2 + 1) + M2 * K2 * S_H + M2 * C * 4 + (K1 * f1 + f1 + K2 * C + C) * 4)
            if w.kind == "gcn":
                byts += 4 * b["n_src"]
            return byts, 2 * M1 * K1 * f1 + 2 * M2 * K2 * C
        if name.startswith("agg_bwd_l"):
            l = int(name[-1])
            b = self.blocks[L - l].host()
            f = w.dims[l - 1]
            rows_used = np.unique(b["cscrow"]).size
            if self.maxagg:
                # the argmax rows and the max part of dA of the rows that
                # sampled anything (each element read where it was won), the
                # self part, the transpose, the mask and the output
                return (2 * rows_used * f * 4 + b["n_dst"] * f * 4 + 4 * b["nnz"] + 8 * (b["n_src"] + 1)
                        + b["n_src"] * f * S_H + b["n_src"] * f * 4), 0
            return (rows_used * f * 4 + b["n_dst"] * f * 4 + 4 * b["nnz"] + 8 * (b["n_src"] + 1)
                    + 8 * (b["n_dst"] + 1) + b["n_src"] * f * S_H + b["n_src"] * f * 4), 0
        if name.startswith("update_bwd_l"):
            # dW = A^T G and db (reads A and G, writes dW and db); above the
            # first layer also dA = G W^T (reads W, writes dA)
            l = int(name[-1])
            b = self.blocks[L - l].host()
            M, K, N = b["n_dst"], w.k_of_layer(l), w.dims[l]
            byts = M * K * S_H + M * N * 4 + K * N * 4 + N * 4
            flops = 2 * M * K * N
            if l > 1 and not self.two:
                byts += K * N * 4 + M * K * 4
                flops *= 2
            return byts, flops
        if name == "sgd":
            P = sum(w.k_of_layer(l) * w.dims[l] + w.dims[l] for l in range(1, L + 1))
            return 3 * 4 * P, 2 * P  # read W and dW, write W; one multiply-add per parameter
        return None, None


def roofline_of(staged, name: str, ms: float, host_link: bool) -> dict:
    """Roofline entry of single-kernel stage `name` of `staged` at `ms` per
    launch: the bound (HBM, matrix cores or host link) its algorithmic bytes
    and flops put it under, and the achieved fraction of that peak."""
    byts, flops = staged.stage_bytes(name)
    t = ms / 1e3
    ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    if name == "gather" and host_link:
        ach = byts / t / 1e9
        r = {"bound": "host_link", "achieved": ach, "peak": HOST_LINK_PEAK_GBS, "unit": "GB/s",
             "frac": ach / HOST_LINK_PEAK_GBS}
    elif flops and flops / max(byts, 1) > ridge:
        ach = flops / t / 1e12
        r = {"bound": "mfma", "achieved": ach, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
             "frac": ach / BF16_PEAK_TFLOPS}
    else:
        ach = byts / t / 1e9
        r = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS}
    r.update({"algorithmic_bytes": int(byts), "flops": int(flops or 0), "avg_ms": ms})
    return r


def scale_report(gnn, w, graph, tr, table, labels, nrm, perm, act, loc, batches, reps, lr):
    """The single-kernel stages of the same model and graph at larger
    mini-batches: one staged step builds the blocks, then each stage's ABI
    call is replayed back to back.  At the workload's own batch the kernels
    are launch- and latency-bound; these sizes show where they stand once a
    launch has enough work to fill the chip."""
    out = []
    host_link = loc == gnn.GNN_LOC_HOST_PINNED
    for B in batches:
        st = StagedStep(gnn, w, graph, B, act, loc)
        tg = workloads.targets_for_step(perm, B, 0).contiguous()
        for s in range(2):
            st.run(tr, table, labels, tg, nrm, w.seed, 20_000 + s, lr)
        torch.cuda.synchronize()
        L = w.num_layers
        names = ["gather", "agg_fwd_l1", "update_fwd_l1"]
        names += [f"layer_fwd_l{l}" if st.fused.get(l) else f"agg_fwd_l{l}" for l in range(2, L + 1)]
        names += [f"agg_bwd_l{l}" for l in range(2, L + 1)]
        kern = {}
        for k in names:
            ms = st.replay(k, tr, table, reps, labels=labels)
            kern[k] = {kk: (round(vv, 6) if isinstance(vv, float) else vv)
                       for kk, vv in roofline_of(st, k, ms, host_link).items()}
        out.append({"batch": B, "block_sizes": st.block_sizes(), "kernels": kern})
        log(f"batch {B}: " + ", ".join(f"{k} {v['frac']:.2f} of {v['bound']}" for k, v in kern.items()))
        del st
        torch.cuda.empty_cache()
    return out


def wide_gemm_report(gnn, dev, reps, m=26_624, ke=768, n=1024):
    """The update GEMMs of a wide GraphSAGE layer (the 768 -> 1024 first
    layer of the host-table model: K = 1,536, at its hop-2 row bound of
    26,624), where they are bound by the matrix cores rather than HBM: the
    forward (with the bf16 W^T shadow), dA + dW, and dW alone, in TFLOP/s
    against the dense bf16 peak; torch.matmul on the same bf16 operands is
    timed beside them for context.  Random bf16 operands."""
    g = torch.Generator(device=dev).manual_seed(0)
    K = 2 * ke
    a_s = torch.randn(m, ke, device=dev, generator=g).to(torch.bfloat16)
    a_n = torch.randn(m, ke, device=dev, generator=g).to(torch.bfloat16)
    w = torch.randn(K, n, device=dev, generator=g) / K ** 0.5
    bias = torch.zeros(n, device=dev)
    wt = w.t().contiguous().to(torch.bfloat16)
    out = torch.empty(m, n, dtype=torch.bfloat16, device=dev)
    grad = torch.randn(m, n, device=dev, generator=g)
    dw, db = torch.empty(K, n, device=dev), torch.empty(n, device=dev)
    da = torch.empty(m, K, device=dev)
    ws = gnn.update_bwd_workspace(K, n, m, gnn.GNN_BF16, dev)
    a_cat, w_b = torch.cat([a_s, a_n], 1), w.to(torch.bfloat16)
    flops = 2.0 * m * K * n

    def rate(ms, times=1):
        t = times * flops / (ms / 1e3) / 1e12
        return {"ms": round(ms, 5), "tflops": round(t, 1), "frac": round(t / BF16_PEAK_TFLOPS, 4)}
    r = {"shape": {"m": m, "k": K, "n": n}, "peak_tflops": BF16_PEAK_TFLOPS}
    r["update_fwd"] = rate(time_calls(lambda: gnn.update_fwd(a_s, a_n, w, bias, out, True, gnn.GNN_BF16, wt=wt), reps))
    r["update_bwd_dA_dW"] = rate(time_calls(lambda: gnn.update_bwd(a_s, a_n, w, grad, dw, db, da, gnn.GNN_BF16,
                                                                   ws=ws), reps), 2)
    r["update_bwd_dW"] = rate(time_calls(lambda: gnn.update_bwd(a_s, a_n, w, grad, dw, db, None, gnn.GNN_BF16,
                                                                ws=ws), reps))
    r["torch_matmul_fwd"] = rate(time_calls(lambda: torch.matmul(a_cat, w_b), reps))
    return r


def tile_bytes(rowptr, col, f, elem, rows=16):
    """Source bytes an aggregation fetches: per edge (every edge reads its
    source row) and per tile-distinct source (each distinct source of a tile
    of `rows` destination rows read once)."""
    per_edge = int(col.size) * f * elem
    distinct = 0
    for r0 in range(0, rowptr.size - 1, rows):
        seg = col[rowptr[r0]:rowptr[min(r0 + rows, rowptr.size - 1)]]
        distinct += np.unique(seg).size
    return per_edge, distinct * f * elem


def time_calls(call, reps):
    call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def hub_block_case(gnn, dev, reps, n=50_000, hubs=128, n_dst=8192, fanout=25, f=256):
    """A sampled hub-heavy block: every non-hub vertex links to all `hubs`
    hubs and to two random vertices, so the rows of a tile share most of
    their sources.  Pull against tile-deduplicated aggregation (bf16 in and
    out): time per launch and source bytes."""
    rng = np.random.default_rng(5)
    deg = np.full(n, hubs + 2, np.int64)
    deg[:hubs] = 0
    rowptr = np.zeros(n + 1, np.int64)
    rowptr[1:] = np.cumsum(deg)
    col = np.empty(int(rowptr[-1]), np.int64)
    body = np.concatenate([np.tile(np.arange(hubs), (n - hubs, 1)), rng.integers(0, n, (n - hubs, 2))], axis=1)
    col[rowptr[hubs]:] = body.reshape(-1)
    graph = gnn.DeviceGraph(torch.from_numpy(rowptr).to(dev), torch.from_numpy(col).to(dev))
    blk = gnn.DeviceBlock(n, n_dst, fanout, False, False, dev)
    nb = ctypes.c_size_t()
    gnn._check(gnn.lib().gnn_sampler_workspace_size(n, n_dst, fanout, ctypes.byref(nb)))
    ws = torch.empty(nb.value, dtype=torch.uint8, device=dev)
    gnn._check(gnn.lib().gnn_sampler_workspace_init(ws.data_ptr(), nb.value, n, gnn._stream(None)))
    dst = torch.from_numpy(rng.choice(np.arange(hubs, n), n_dst, replace=False).astype(np.int64)).to(dev)
    gnn.build_block(graph, dst, fanout, 5, 0, 1, blk, ws, want_csc=False)
    hb = blk.host()
    h = torch.randn((blk.c.cap_src, f), device=dev).to(torch.bfloat16)
    out = torch.empty((n_dst, f), dtype=torch.bfloat16, device=dev)
    out2 = torch.empty_like(out)
    kind = gnn.GNN_AGG_SAGE_MEAN
    t_pull = time_calls(lambda: gnn.aggregate_fwd(blk, kind, h, out), reps)
    t_dedup = time_calls(lambda: gnn.aggregate_fwd_dedup(blk, kind, h, out2), reps)
    same = bool(torch.equal(out.view(torch.int16), out2.view(torch.int16)))
    per_edge, distinct = tile_bytes(hb["rowptr"], hb["col"], f, 2)
    return {"block": {"n_dst": hb["n_dst"], "n_src": hb["n_src"], "nnz": hb["nnz"], "f": f},
            "pull_ms": t_pull, "dedup_ms": t_dedup, "bitwise_equal": same,
            "source_bytes_per_edge": per_edge, "source_bytes_tile_distinct": distinct}


def dedup_report(gnn, staged, w, reps, dev):
    """Section IV-C's feature duplicator as tile-deduplicated aggregation
    (gnn_aggregate_fwd_dedup) against the pull kernel: on the staged step's
    blocks and on a hub-heavy block."""
    out = {"tile_rows": 16}
    elem = 2 if staged.act == torch.bfloat16 else 4
    for l in range(1, staged.L + 1):
        hb = staged.blocks[staged.L - l].host()
        per_edge, distinct = tile_bytes(hb["rowptr"], hb["col"], w.dims[l - 1], elem)
        out[f"layer{l}"] = {"pull_ms": staged.replay(f"agg_fwd_l{l}", None, None, reps),
                            "dedup_ms": staged.replay(f"agg_dedup_l{l}", None, None, reps),
                            "source_bytes_per_edge": per_edge, "source_bytes_tile_distinct": distinct}
    out["hub_block"] = hub_block_case(gnn, dev, reps)
    return out


def effective_rates(dev, host_table):
    """Effective device-memory bandwidth (a plain 256 MiB device copy, read +
    write bytes over its time) and, for a host table, the pinned host ->
    device copy bandwidth: the burst bandwidths the performance model
    divides by."""
    n = 64 << 20  # fp32 elements: 256 MiB
    src = torch.empty(n, device=dev)
    dst = torch.empty(n, device=dev)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    bw_mem = 5 * 2 * n * 4 / (e0.elapsed_time(e1) / 1e3)
    del src, dst
    bw_link = HOST_LINK_PEAK_GBS * 1e9
    if host_table:
        h = torch.empty(n // 4, pin_memory=True)
        d = torch.empty(n // 4, device=dev)
        d.copy_(h, non_blocking=True)
        e0.record()
        for _ in range(3):
            d.copy_(h, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        bw_link = 3 * n * 4 / 4 / (e0.elapsed_time(e1) / 1e3)
        del h, d
    return bw_mem, bw_link


def perf_model_report(w, staged, stage_ms, ms_per_step, host_table, table, dev):
    """Section V's model for the staged step's blocks, with the published
    MI355X peaks and with effective rates measured here, beside the measured
    step and stage times.  T_samp is the staged run's sampling time (the
    paper measures it too)."""
    from paper_2303_00158_amd import perf_model as pm
    layers = pm.layers_from_blocks(staged.block_sizes(), w.dims)
    n_input = staged.block_sizes()[-1]["n_src"]
    t_samp = sum(v for k, v in stage_ms.items() if k.startswith("sample_hop")) / 1e3
    s_table = table.element_size()
    s_act = 2 if w.precision == "bf16" else 4
    bw_mem, bw_link = effective_rates(dev, host_table)
    eff = pm.Hardware(bw_mem=bw_mem, bw_link=bw_link, mac_rate=pm.MI355X_PEAK.mac_rate, name="MI355X effective")
    prop_stages = [k for k in stage_ms if not k.startswith("sample_hop") and k != "gather"]
    measured = {"samp": t_samp, "load" if not host_table else "load+trans": stage_ms.get("gather", 0.0) / 1e3,
                "prop (staged, one launch per stage)": sum(stage_ms[k] for k in prop_stages) / 1e3}
    out = {"readings": "one trainer, no T_sync; (+) = max (fused aggregate -> update); t_agg over f^{l-1}-wide "
                       "inputs of the layer's own block; t_upd with K = 2 f^{l-1} (SAGE) or f^{l-1} (GCN)",
           "rates": {"peak": {"bw_mem_GBs": pm.MI355X_PEAK.bw_mem / 1e9, "bw_link_GBs": pm.MI355X_PEAK.bw_link / 1e9,
                              "mac_per_s": pm.MI355X_PEAK.mac_rate},
                     "effective": {"bw_mem_GBs": bw_mem / 1e9, "bw_link_GBs": bw_link / 1e9,
                                   "mac_per_s": eff.mac_rate}}}
    for name, hw in (("peak", pm.MI355X_PEAK), ("effective", eff)):
        p = pm.predict(layers, n_input, w.kind, hw, t_samp, s_table, s_act, host_table=host_table)
        out[name] = pm.report(p, ms_per_step / 1e3, measured)
    return out


class Inputs:
    """Seeded synthetic inputs of one workload on the GPU (the graph and
    feature table may be shared with another workload of the same graph)."""

    def __init__(self, gnn, w, dev, share=None, precision=None):
        self.w = w
        self.host_table = w.table_loc == "host"
        self.loc = gnn.GNN_LOC_HOST_PINNED if self.host_table else gnn.GNN_LOC_DEVICE
        prec = precision or w.precision
        self.act = torch.bfloat16 if prec == "bf16" else torch.float32
        self.precision = gnn.GNN_BF16 if prec == "bf16" else gnn.GNN_F32
        self.kind = kind_code(gnn, w.kind)
        t0 = time.time()
        if share is not None:
            self.rowptr, self.col, self.graph, self.table = share.rowptr, share.col, share.graph, share.table
            self.labels, self.perm, self.nrm = share.labels, share.perm, share.nrm
        else:
            log(f"generating {w.name}: {w.graph} n={w.n} m={w.m}")
            self.rowptr, self.col = workloads.make_graph(w, device=dev)
            self.graph = gnn.DeviceGraph(self.rowptr, self.col)
            tdt = torch.float16 if w.table_dtype == "f16" else torch.float32
            if self.host_table:
                # drawn on the GPU in chunks and copied into pinned host memory
                self.table = torch.empty((w.n, w.dims[0]), dtype=tdt, pin_memory=True)
                workloads.features(w.n, w.dims[0], seed=w.seed, device=dev, out=self.table)
            else:
                self.table = workloads.features(w.n, w.dims[0], seed=w.seed, device=dev, dtype=tdt)
            self.labels = workloads.labels(w.n, w.num_classes, seed=w.seed, device=dev)
            self.perm = workloads.target_batches(w.n, w.batch, seed=w.seed, device=dev)
            self.nrm = gnn.gcn_norm(self.graph)
        L = w.num_layers
        self.weights = [workloads.glorot(w.k_of_layer(l + 1), w.dims[l + 1], w.seed, l) for l in range(L)]
        self.biases = [torch.zeros(w.dims[l + 1]) for l in range(L)]
        torch.cuda.synchronize()
        if share is None:
            log(f"inputs ready in {time.time() - t0:.1f}s")


def timed_training(gnn, inp, dev, steps, warmup, lr, pipeline, prepare_slots, one_call_compare=False):
    """Warm up, then time `steps` training steps (pipelined through
    gnn_train_steps, or one gnn_train_step call per step) between two HIP
    events; the sampled edges come from the device counters."""
    w = inp.w
    tr = gnn.Trainer(inp.kind, w.dims, w.fanouts, inp.precision, w.n, w.batch, inp.weights, inp.biases, device=dev,
                     prepare_slots=prepare_slots if pipeline else 0, one_call=one_call_compare or not pipeline)
    nb = w.n // w.batch
    n_t = min(nb, warmup + steps + (warmup + steps if one_call_compare else 0))
    tgt = [workloads.targets_for_step(inp.perm, w.batch, s).contiguous() for s in range(max(n_t, 1))]
    edges = torch.zeros(steps, dtype=torch.int64, device=dev)
    prep_stream = torch.cuda.Stream(dev) if pipeline else None

    def step_targets(first, count):
        return torch.stack([tgt[(first + i) % len(tgt)] for i in range(count)])

    def run_steps(first, count, edges_out=None, pipelined=pipeline, targets=None):
        if pipelined:
            tr.run_pipelined(inp.graph, inp.table, inp.labels,
                             step_targets(first, count) if targets is None else targets, w.seed, first, count, lr,
                             gcn_norm_t=inp.nrm, loc=inp.loc, edges_out=edges_out, prep_stream=prep_stream)
            return
        for i in range(count):
            tr.step(inp.graph, inp.table, inp.labels, tgt[(first + i) % len(tgt)], w.seed, first + i, lr,
                    gcn_norm_t=inp.nrm, loc=inp.loc, edges_out=None if edges_out is None else edges_out[i:i + 1])

    def timed(first, count, edges_out, pipelined=pipeline):
        targets = step_targets(first, count) if pipelined else None
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        ev0.record()
        run_steps(first, count, edges_out, pipelined, targets)
        t_enq = time.perf_counter() - t
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1), time.perf_counter() - t, t_enq

    run_steps(0, warmup)
    torch.cuda.synchronize()
    log(f"{w.name}: warmup done ({warmup} steps, {'pipelined two-stage' if pipeline else 'one-call'} steps), "
        f"loss {tr.loss.item():.4f}")
    ms_total, t_wall, t_enqueue = timed(warmup, steps, edges)
    if pipeline:
        tr.check_device_errors()  # the blocks of the timed steps were built without a device-side failure
    total_edges = int(edges.sum().item())
    out = {"ms_per_step": ms_total / steps, "value": total_edges / (ms_total / 1e3),
           "edges_per_step": total_edges / steps, "host_enqueue_ms_per_step": 1e3 * t_enqueue / steps,
           "loss": tr.loss.item()}
    log(f"{w.name}: timed {steps} steps: {out['ms_per_step']:.3f} ms/step (wall {1e3 * t_wall / steps:.3f}, host "
        f"enqueue {out['host_enqueue_ms_per_step']:.3f}), {out['edges_per_step']:.0f} edges/step, "
        f"loss {out['loss']:.4f}")
    if pipeline and one_call_compare:
        # the same steps without the overlap (one-call steps on one stream)
        e2 = torch.zeros(steps, dtype=torch.int64, device=dev)
        run_steps(0, warmup, pipelined=False)  # warms up the one-call path
        ms2, _, _ = timed(warmup + steps, steps, e2, pipelined=False)
        out["sequential_ms_per_step"] = ms2 / steps
        log(f"{w.name}: without the overlap: {out['sequential_ms_per_step']:.3f} ms/step")
    return out, tr, tgt


# single-kernel stages (one launch per ABI call) and multi-launch ones
MULTI_LAUNCH = ("update_bwd", "sgd", "bwd_l1l2")


def staged_report(gnn, inp, tr, tgt, stage_steps, replays, lr):
    """Event-timed staged steps (one ABI call per stage), then back-to-back
    replays of each stage's call: per-stage times, the roofline of every
    stage and of the dominant single-kernel stage."""
    w = inp.w
    staged = StagedStep(gnn, w, inp.graph, w.batch, inp.act, inp.loc)
    sums, counts = {}, {}
    for s in range(stage_steps + 1):
        evs = []
        torch.cuda.synchronize()
        if hasattr(torch.cuda, "_sleep"):
            torch.cuda._sleep(20_000_000)  # let the host enqueue the whole step before the GPU starts it
        staged.run(tr, inp.table, inp.labels, tgt[s % len(tgt)], inp.nrm, w.seed, 10_000 + s, lr, events=evs)
        torch.cuda.synchronize()
        if s == 0:
            continue  # first staged step warms up the allocations
        for (n0, e0), (n1, e1) in zip(evs[:-1], evs[1:]):
            sums[n1] = sums.get(n1, 0.0) + e0.elapsed_time(e1)
            counts[n1] = counts.get(n1, 0) + 1
    stage_ms = {k: sums[k] / counts[k] for k in sums}
    host_link = inp.loc == gnn.GNN_LOC_HOST_PINNED
    replayable = [k for k in stage_ms
                  if k in ("gather", "fwd_l1l2", "bwd_l1l2")
                  or k.startswith(("agg_fwd", "update_fwd", "layer_fwd", "agg_bwd", "update_bwd"))
                  or k == "sgd"]
    launch_ms = {k: staged.replay(k, tr, inp.table, replays, labels=inp.labels) for k in replayable}
    single = [k for k in replayable if not k.startswith(MULTI_LAUNCH)]
    dom = max(single, key=lambda k: launch_ms[k])
    roof = roofline_of(staged, dom, launch_ms[dom], host_link)
    roof.update({"kernel": dom, "traffic": measured_traffic(dom, w.name), "source_hash": source_hash(dom)})
    kernels = {}
    for k in replayable:
        e = {kk: (round(vv, 6) if isinstance(vv, float) else vv)
             for kk, vv in roofline_of(staged, k, launch_ms[k], host_link).items()}
        e["traffic"] = measured_traffic(k, w.name)
        if k.startswith(MULTI_LAUNCH):
            e["launches"] = staged.launches(k)
        kernels[k] = e
    log(f"{w.name}: stages (ms): {json.dumps({k: round(v, 5) for k, v in stage_ms.items()})}")
    log(f"{w.name}: per-call (ms): {json.dumps({k: round(v, 5) for k, v in launch_ms.items()})}")
    return staged, stage_ms, roof, kernels


def other_workload(gnn, w, dev, args, share=None, precision=None, label=None):
    """Measured figures of a workload besides the headline: pipelined
    steps (edges/s, steps/s) and the roofline of its dominant kernel."""
    inp = Inputs(gnn, w, dev, share=share, precision=precision)
    steps, warmup = args.other_steps, args.other_warmup
    t, tr, tgt = timed_training(gnn, inp, dev, steps, warmup, args.lr, True, args.prepare_slots)
    staged, stage_ms, roof, kernels = staged_report(gnn, inp, tr, tgt, 2, max(5, args.replays // 2), args.lr)
    out = {"workload": label or w.name,
           "config": {"graph": f"{w.graph} n={w.n} m={w.m} {'directed' if w.directed else 'undirected'}",
                      "aggregation": w.kind, "dims": list(w.dims), "fanouts": list(w.fanouts), "batch": w.batch,
                      "features": f"{w.table_dtype} in {'pinned host memory' if inp.host_table else 'HBM'}",
                      "precision": precision or w.precision},
           "value": t["value"], "unit": "edges/s", "ms_per_step": t["ms_per_step"],
           "steps_per_s": 1e3 / t["ms_per_step"], "edges_per_step": t["edges_per_step"], "steps": steps,
           "warmup": warmup, "roofline": roof, "block_sizes": staged.block_sizes(),
           "stages_ms": {k: round(v, 5) for k, v in stage_ms.items()}}
    if inp.host_table:
        link_bytes = staged.stage_bytes("gather")[0]
        ach = link_bytes / (t["ms_per_step"] / 1e3) / 1e9
        out["host_link"] = {"bytes_per_step": int(link_bytes), "achieved": ach, "peak": HOST_LINK_PEAK_GBS,
                            "unit": "GB/s", "frac": ach / HOST_LINK_PEAK_GBS}
    log(f"{out['workload']}: {t['value']:.3g} edges/s, {out['steps_per_s']:.0f} steps/s, dominant {roof['kernel']} "
        f"{roof['frac']:.3f} of {roof['bound']}")
    del staged, tr, inp
    torch.cuda.empty_cache()
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1 (multi-GPU sharding is "
                                   "described in the design notes, not built)", "n_gpus": args.gpus}))
        sys.exit(1)
    from paper_2303_00158_amd import gnn
    if not os.path.exists(gnn.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.randn(n, device=dev)
        dst = torch.empty(n, dtype=torch.int32, device=dev)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {args.copy_calibration} MiB read + {args.copy_calibration} MiB written per launch")
        del src, dst
    w = workloads.PRESETS[args.workload]
    if args.scale_n:
        m = args.scale_m or int(round(w.m * args.scale_n / w.n))
        w = workloads.scaled(w, args.scale_n, m)
    pipeline = True if args.pipeline is None else args.pipeline

    inp = Inputs(gnn, w, dev)
    log(f"graph: {workloads.graph_stats(inp.rowptr, inp.col)}")
    t, tr, tgt = timed_training(gnn, inp, dev, args.steps, args.warmup, args.lr, pipeline, args.prepare_slots,
                                one_call_compare=pipeline)
    ms_per_step = t["ms_per_step"]
    host_table, loc, act, precision = inp.host_table, inp.loc, inp.act, inp.precision

    result = {
        "metric": "sampled edges/sec (fwd+bwd) and train steps/sec, 2-layer GraphSAGE, 1 GPU",
        "value": t["value"],
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "steps_per_s": 1e3 / ms_per_step,
        "edges_per_step": t["edges_per_step"],
        "host_enqueue_ms_per_step": t["host_enqueue_ms_per_step"],
        "step_mode": "two-stage pipelined (prepare of step s+1 overlaps compute of step s)" if pipeline
                     else "one call per step",
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if act == torch.bfloat16 else "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name, "graph": f"{w.graph} n={w.n} m={w.m} {'directed' if w.directed else 'undirected'}",
            "aggregation": w.kind, "dims": list(w.dims), "fanouts": list(w.fanouts), "batch": w.batch,
            "features": f"{w.table_dtype} in {'pinned host memory' if w.table_loc == 'host' else 'HBM'}",
            "scope": "sample + gather + forward + loss + backward + SGD",
            "scaled_from": None if not args.scale_n else workloads.PRESETS[args.workload].name,
            "parallelism": "single GPU",
        },
    }
    if "sequential_ms_per_step" in t:
        result["sequential_ms_per_step"] = t["sequential_ms_per_step"]

    # ---- staged run with events per stage --------------------------------
    if not args.no_stages:
        staged, stage_ms, roof, kernels = staged_report(gnn, inp, tr, tgt, args.stage_steps, args.replays, args.lr)
        result["stages_ms"] = {k: round(v, 5) for k, v in stage_ms.items()}
        result["roofline"] = roof
        result["kernels"] = kernels
        result["block_sizes"] = staged.block_sizes()
        if host_table:
            # X' rows moved over the host link per step, against the step time
            link_bytes = staged.stage_bytes("gather")[0]
            ach = link_bytes / (ms_per_step / 1e3) / 1e9
            result["host_link"] = {"bytes_per_step": int(link_bytes), "achieved": ach, "peak": HOST_LINK_PEAK_GBS,
                                   "unit": "GB/s", "frac": ach / HOST_LINK_PEAK_GBS}
        result["perf_model"] = perf_model_report(w, staged, stage_ms, ms_per_step, host_table, inp.table, dev)
        result["dedup_aggregation"] = dedup_report(gnn, staged, w, args.replays, dev)
        log(f"dedup aggregation: {json.dumps(result['dedup_aggregation'])}")
        if precision == gnn.GNN_BF16:
            result["wide_gemm"] = wide_gemm_report(gnn, dev, args.replays)
            log(f"wide-layer GEMMs: {json.dumps(result['wide_gemm'])}")
        batches = [int(x) for x in args.scale_batches.split(",") if x.strip()]
        if batches:
            result["kernels_at_batch"] = scale_report(gnn, w, inp.graph, tr, inp.table, inp.labels, inp.nrm,
                                                      inp.perm, act, loc, batches, args.replays, args.lr)
        pmr = result["perf_model"]["effective"]
        log(f"performance model (effective rates): T_execution {pmr['predicted_us']['T_execution (max, eq. 6)']:.1f} us "
            f"(max of stages), serial {pmr['predicted_us']['serial sum']:.1f} us; measured {pmr['measured_step_us']:.1f} us")
        del staged

    # ---- the other workloads, pipelined -----------------------------------
    others = [x.strip() for x in args.other_workloads.split(",") if x.strip()] if not args.scale_n else []
    if others:
        result["other_workloads"] = []
        for name in others:
            if name == "fp32":
                # the headline workload computed in fp32 throughout (the
                # paper models features as 4-byte values)
                e = other_workload(gnn, w, dev, args, share=inp, precision="f32", label=f"{w.name} (fp32)")
            else:
                ow = workloads.PRESETS[name]
                lbl = None
                if ow.table_loc == "host" and ow.n > args.host_table_n:
                    # the 375 GB host table does not fit the host memory of one
                    # run: same model, batch and fanouts on a smaller graph
                    m = int(round(ow.m * args.host_table_n / ow.n))
                    ow = workloads.scaled(ow, args.host_table_n, m)
                    lbl = f"{name} scaled to n={ow.n}"
                share = inp if (ow.graph == w.graph and ow.n == w.n and ow.m == w.m and ow.directed == w.directed
                                and ow.dims[0] == w.dims[0] and ow.table_loc == w.table_loc
                                and ow.table_dtype == w.table_dtype and ow.num_classes == w.num_classes) else None
                e = other_workload(gnn, ow, dev, args, share=share, label=lbl)
            result["other_workloads"].append(e)

    # ---- CPU oracle baseline ---------------------------------------------
    if not args.no_cpu_baseline:
        import oracle
        threads = len(os.sched_getaffinity(0))
        rp_h, col_h = inp.rowptr.cpu().numpy(), inp.col.cpu().numpy()
        nrm_h = inp.nrm.cpu().numpy()
        table_h = inp.table.cpu().numpy()
        labels_h = inp.labels.cpu().numpy()
        okind = oracle.SAGE if w.kind == "sage" else oracle.GCN
        oprec = oracle.BF16 if w.precision == "bf16" else oracle.F32

        def oracle_rate(nthreads, seconds):
            oracle.set_threads(nthreads)
            w_h = [x.numpy() for x in inp.weights]
            b_h = [x.numpy() for x in inp.biases]
            tot_e, tot_t, n_steps = 0, 0.0, 0
            while n_steps < 1 or tot_t < seconds:
                s = n_steps
                cfg = oracle.StepConfig(kind=okind, dims=w.dims, fanouts=w.fanouts, precision=oprec, seed=w.seed,
                                        step=s, lr=args.lr)
                tt = time.perf_counter()
                ref = oracle.train_step(rp_h, col_h, nrm_h, table_h, labels_h, tgt[s % len(tgt)].cpu().numpy(), w_h,
                                        b_h, cfg)
                tot_t += time.perf_counter() - tt
                tot_e += ref["edges"]
                w_h, b_h = ref["new_w"], ref["new_b"]
                n_steps += 1
            return tot_e, tot_t, n_steps, oracle.get_threads()

        tot_e, tot_t, n_steps, used = oracle_rate(threads, args.cpu_seconds)
        e1, t1, n1, _ = oracle_rate(1, args.cpu_seconds_one_thread)
        result["cpu_baseline"] = {
            "value": tot_e / tot_t, "unit": "edges/s", "cores": used, "kind": "oracle",
            "sample": f"{n_steps} full training steps (sample, gather, forward, loss, backward, SGD) of the "
                      f"same workload, fp64 sums, {tot_t:.1f} s",
            "steps_per_s": n_steps / tot_t,
            "one_thread": {"value": e1 / t1, "unit": "edges/s", "steps": n1, "seconds": round(t1, 2),
                           "steps_per_s": n1 / t1},
            "cpu_model": cpu_model(),
        }
        log(f"cpu oracle: {tot_e / tot_t:.0f} edges/s with {used} threads, {e1 / t1:.0f} with 1 thread")

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
