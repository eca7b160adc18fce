"""The paper's performance model (Section V), instantiated for one MI355X.

Host-side arithmetic only: it predicts the time of one training iteration
from the sizes of its sampled blocks and from bandwidth and compute rates,
so that the prediction can be set beside measured stage times.

The model (Section V):
  throughput   = sum over trainers and layers of |E^l| / T_execution   (eq. 5)
  T_execution  = max(T_samp, T_load, T_trans, T_prop)                  (eq. 6)
  T_samp       measured, not modelled (the paper measures it too)
  T_load       = |V^0| f^0 S_feat / BW_mem                             (eq. 7)
  T_trans      = |V^0| f^0 S_feat / BW_link                            (eq. 8)
  T_prop       = max over trainers of T_trainer + T_sync               (eq. 9)
  T_trainer    = sum_{l=1..L} (+)(t_agg^l, t_upd^l)                    (forward)
                 + t_upd^1 + sum_{l=2..L} (+)(t_agg^l, t_upd^l)         (backward)  (eq. 10)
  t_agg^l      = edges x feature width x S_feat / BW_mem               (eq. 11)
  t_upd^l      = MACs of the layer's update / (N x freq)               (eq. 12)
  T_sync       = 2 x model bytes / BW_link                             (eq. 13)
(+) is max when aggregation and update are pipelined (the fused kernel
here, like the paper's FPGA datapath) and sum when they are not.

Readings (the paper's layer indices are not consistent between its
equations): layer l aggregates the |E^l| edges of its own block over
features of width f^{l-1} (its input), and its update multiplies
|V^l| x K_l by K_l x f^l, with K_l = 2 f^{l-1} for GraphSAGE (self and
mean concatenated) and f^{l-1} for GCN.  With one GPU there is one
trainer and no T_sync.  T_trans applies only when the feature table
lives in host memory.  Every stage runs on the same device here, so
besides the paper's pipeline bound (the max of eq. 6) the serial bound
T_samp + T_load + T_trans + T_prop is reported: a pipelined step on one
GPU lies between the two.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence


@dataclass
class Hardware:
    """Rates the model divides by (bytes/s and MAC/s)."""
    bw_mem: float            # device memory bandwidth the gather and aggregation see
    bw_link: float           # host link bandwidth (T_trans, T_sync)
    mac_rate: float          # N x freq: multiply-accumulates per second of the update
    name: str = "MI355X"


# Published MI355X figures: 8 TB/s HBM3E, PCIe Gen5 x16 (64 GB/s one way),
# 2.5 PFLOP/s dense bf16 on the matrix cores (1.25e15 MAC/s).
MI355X_PEAK = Hardware(bw_mem=8.0e12, bw_link=64e9, mac_rate=2.5e15 / 2)


@dataclass
class Layer:
    edges: int       # |E^l|: sampled edges of the layer's block
    n_dst: int       # |V^l|: destination rows of the block
    f_in: int        # f^{l-1}
    f_out: int       # f^l


@dataclass
class Prediction:
    t_samp: float
    t_load: float
    t_trans: float
    t_sync: float
    t_agg: List[float]
    t_upd: List[float]
    t_forward: float
    t_backward: float
    t_prop: float
    t_pipeline: float        # eq. 6: max of the stages
    t_serial: float          # the stages one after another
    edges: int
    throughput_pipeline: float   # eq. 5 with t_pipeline
    throughput_serial: float
    stages: Dict[str, float] = field(default_factory=dict)


def layers_from_blocks(blocks: Sequence[dict], dims: Sequence[int]) -> List[Layer]:
    """Layers 1..L from hop-ordered block sizes (blocks[0] is hop 1, the last
    layer's block) and the layer widths dims[0..L]."""
    L = len(dims) - 1
    if len(blocks) != L:
        raise ValueError(f"{len(blocks)} blocks for {L} layers")
    out = []
    for l in range(1, L + 1):
        b = blocks[L - l]
        out.append(Layer(edges=int(b["nnz"]), n_dst=int(b["n_dst"]), f_in=int(dims[l - 1]), f_out=int(dims[l])))
    return out


def predict(layers: Sequence[Layer], n_input: int, kind: str, hw: Hardware, t_samp: float,
            s_table: int, s_act: int, host_table: bool = False, fused: bool = True,
            n_trainers: int = 1, s_model: int = 4) -> Prediction:
    """Predicted iteration time (seconds) for one trainer's blocks.

    layers: layers 1..L; n_input: |V^0| (rows of X'); kind: "sage", "gcn" or
    "sage-max" (the max aggregator moves the mean's bytes);
    t_samp: measured sampling time; s_table: bytes per feature of the table
    (S_feat of eqs. 7-8); s_act: bytes per activation the aggregation reads
    (S_feat of eq. 11); fused: (+) is max, else sum."""
    if kind not in ("sage", "gcn", "sage-max"):
        raise ValueError(kind)
    f0 = layers[0].f_in
    t_load = n_trainers * n_input * f0 * s_table / hw.bw_mem
    t_trans = n_input * f0 * s_table / hw.bw_link if host_table else 0.0
    t_agg, t_upd = [], []
    for ly in layers:
        t_agg.append(ly.edges * ly.f_in * s_act / hw.bw_mem)
        k = (1 if kind == "gcn" else 2) * ly.f_in
        t_upd.append(ly.n_dst * k * ly.f_out / hw.mac_rate)
    comb = max if fused else (lambda a, b: a + b)
    L = len(layers)
    t_fwd = sum(comb(t_agg[i], t_upd[i]) for i in range(L))
    t_bwd = t_upd[0] + sum(comb(t_agg[i], t_upd[i]) for i in range(1, L))
    model_bytes = sum((1 if kind == "gcn" else 2) * ly.f_in * ly.f_out for ly in layers) * s_model
    t_sync = 2 * model_bytes / hw.bw_link if n_trainers > 1 else 0.0
    t_prop = t_fwd + t_bwd + t_sync
    t_pipe = max(t_samp, t_load, t_trans, t_prop)
    t_ser = t_samp + t_load + t_trans + t_prop
    edges = n_trainers * sum(ly.edges for ly in layers)
    return Prediction(t_samp=t_samp, t_load=t_load, t_trans=t_trans, t_sync=t_sync, t_agg=t_agg, t_upd=t_upd,
                      t_forward=t_fwd, t_backward=t_bwd, t_prop=t_prop, t_pipeline=t_pipe, t_serial=t_ser,
                      edges=edges, throughput_pipeline=edges / t_pipe if t_pipe > 0 else float("inf"),
                      throughput_serial=edges / t_ser if t_ser > 0 else float("inf"),
                      stages={"samp": t_samp, "load": t_load, "trans": t_trans, "prop": t_prop})


def report(p: Prediction, measured_step_s: float, measured: Optional[Dict[str, float]] = None) -> dict:
    """JSON-ready comparison of a prediction with measured times (seconds in,
    microseconds out)."""
    us = lambda x: round(x * 1e6, 3)
    out = {
        "predicted_us": {"T_samp (measured)": us(p.t_samp), "T_load": us(p.t_load), "T_trans": us(p.t_trans),
                         "T_prop": us(p.t_prop), "t_forward": us(p.t_forward), "t_backward": us(p.t_backward),
                         "t_agg": [us(x) for x in p.t_agg], "t_upd": [us(x) for x in p.t_upd],
                         "T_execution (max, eq. 6)": us(p.t_pipeline), "serial sum": us(p.t_serial)},
        "measured_step_us": us(measured_step_s),
        "ratio_measured_to_max": measured_step_s / p.t_pipeline if p.t_pipeline > 0 else None,
        "ratio_measured_to_serial": measured_step_s / p.t_serial if p.t_serial > 0 else None,
    }
    if measured:
        out["measured_stage_us"] = {k: us(v) for k, v in measured.items()}
    return out
