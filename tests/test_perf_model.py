"""The performance model of Section V against hand-worked values.

Sizes and rates are chosen so that every term comes out as a round number
computed here by hand (the comments show the arithmetic), not by restating
the module's expressions."""
import math

import pytest

from paper_2303_00158_amd import perf_model as pm

# rates: 1 GB/s memory, 0.5 GB/s host link, 1e9 MAC/s
HW = pm.Hardware(bw_mem=1e9, bw_link=0.5e9, mac_rate=1e9, name="toy")

# two layers, dims 10 -> 20 -> 5; hop 1 (layer 2's block): 4 targets, 12
# edges; hop 2 (layer 1's block): 16 rows, 40 edges
BLOCKS = [{"n_dst": 4, "n_src": 16, "nnz": 12}, {"n_dst": 16, "n_src": 50, "nnz": 40}]
DIMS = [10, 20, 5]


def test_layers_follow_hop_order():
    ls = pm.layers_from_blocks(BLOCKS, DIMS)
    assert [(l.edges, l.n_dst, l.f_in, l.f_out) for l in ls] == [(40, 16, 10, 20), (12, 4, 20, 5)]
    with pytest.raises(ValueError):
        pm.layers_from_blocks(BLOCKS[:1], DIMS)


def test_sage_fused_terms():
    ls = pm.layers_from_blocks(BLOCKS, DIMS)
    p = pm.predict(ls, n_input=50, kind="sage", hw=HW, t_samp=1e-6, s_table=4, s_act=2)
    # eq. 7: 50 rows x 10 features x 4 B / 1e9 = 2 us
    assert p.t_load == pytest.approx(2e-6)
    assert p.t_trans == 0.0 and p.t_sync == 0.0
    # eq. 11: layer 1 40 x 10 x 2 B = 800 B -> 0.8 us; layer 2 12 x 20 x 2 = 480 B -> 0.48 us
    assert p.t_agg == pytest.approx([0.8e-6, 0.48e-6])
    # eq. 12 (SAGE, K = 2 f_in): layer 1 16 x 20 x 20 = 6400 MAC -> 6.4 us;
    # layer 2 4 x 40 x 5 = 800 MAC -> 0.8 us
    assert p.t_upd == pytest.approx([6.4e-6, 0.8e-6])
    # eq. 10 with max: forward 6.4 + 0.8; backward t_upd^1 + max(0.48, 0.8)
    assert p.t_forward == pytest.approx(7.2e-6)
    assert p.t_backward == pytest.approx(7.2e-6)
    assert p.t_prop == pytest.approx(14.4e-6)
    # eq. 6: max(1, 2, 0, 14.4) us; serial sum 17.4 us; eq. 5: 52 edges
    assert p.t_pipeline == pytest.approx(14.4e-6)
    assert p.t_serial == pytest.approx(17.4e-6)
    assert p.edges == 52
    assert p.throughput_pipeline == pytest.approx(52 / 14.4e-6)


def test_unfused_sum_and_gcn_width():
    ls = pm.layers_from_blocks(BLOCKS, DIMS)
    p = pm.predict(ls, n_input=50, kind="gcn", hw=HW, t_samp=0.0, s_table=4, s_act=4, fused=False)
    # GCN: K = f_in; updates 16 x 10 x 20 = 3200 MAC, 4 x 20 x 5 = 400 MAC
    assert p.t_upd == pytest.approx([3.2e-6, 0.4e-6])
    # 4-byte activations: aggregations 1.6 us and 0.96 us
    assert p.t_agg == pytest.approx([1.6e-6, 0.96e-6])
    # sum operator: forward (1.6 + 3.2) + (0.96 + 0.4); backward 3.2 + (0.96 + 0.4)
    assert p.t_forward == pytest.approx(6.16e-6)
    assert p.t_backward == pytest.approx(4.56e-6)


def test_host_link_and_sync():
    ls = pm.layers_from_blocks(BLOCKS, DIMS)
    p = pm.predict(ls, n_input=50, kind="sage", hw=HW, t_samp=0.0, s_table=2, s_act=2, host_table=True,
                   n_trainers=2)
    # eq. 8: 50 x 10 x 2 B = 1000 B over 0.5 GB/s = 2 us; eq. 7 counts both trainers: 2000 B / 1 GB/s
    assert p.t_trans == pytest.approx(2e-6)
    assert p.t_load == pytest.approx(2e-6)
    # eq. 13: model (20 x 20 + 40 x 5) fp32 = 2400 B, twice over the link = 9.6 us
    assert p.t_sync == pytest.approx(9.6e-6)
    # eq. 9: the trainer plus the synchronisation
    assert p.t_prop == pytest.approx(p.t_forward + p.t_backward + 9.6e-6)
    # eq. 5 counts every trainer's edges
    assert p.edges == 104


def test_report_units():
    ls = pm.layers_from_blocks(BLOCKS, DIMS)
    p = pm.predict(ls, n_input=50, kind="sage", hw=HW, t_samp=1e-6, s_table=4, s_act=2)
    r = pm.report(p, measured_step_s=28.8e-6, measured={"prop": 20e-6})
    assert r["predicted_us"]["T_execution (max, eq. 6)"] == pytest.approx(14.4)
    assert r["measured_step_us"] == pytest.approx(28.8)
    assert r["ratio_measured_to_max"] == pytest.approx(2.0)
    assert r["measured_stage_us"]["prop"] == pytest.approx(20.0)
    assert math.isfinite(r["ratio_measured_to_serial"])
