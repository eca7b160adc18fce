"""The C ABI library loads, exports every entry point its header declares,
and rejects bad arguments on the host before touching the GPU.  CPU only:
nothing here launches a kernel."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gnn.h")


@pytest.fixture(scope="module")
def gnn():
    from paper_2303_00158_amd import gnn as g
    if not os.path.exists(g.LIB_PATH):
        from paper_2303_00158_amd import build
        build.build()
    return g


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gnn_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_paper_calls():
    names = header_functions()
    for f in ("gnn_build_block", "gnn_gather_features", "gnn_aggregate_fwd", "gnn_aggregate_bwd",
              "gnn_update_fwd", "gnn_update_bwd", "gnn_train_step"):
        assert f in names


def test_library_exports_every_declared_symbol(gnn):
    out = subprocess.run(["nm", "-D", "--defined-only", gnn.LIB_PATH], capture_output=True, text=True, check=True)
    exported = set(line.split()[-1] for line in out.stdout.splitlines() if line.strip())
    missing = [f for f in header_functions() if f not in exported]
    assert not missing, missing
    lib = gnn.lib()
    for f in header_functions():
        assert hasattr(lib, f)
    # the binding declares a signature for every header function
    assert sorted(gnn.exported_symbols()) == header_functions()


def test_host_validation_errors(gnn):
    lib = gnn.lib()
    cs, cn = ctypes.c_int64(), ctypes.c_int64()
    assert lib.gnn_block_bounds(100, 10, 0, ctypes.byref(cs), ctypes.byref(cn)) == gnn.GNN_EINVAL
    assert b"fanout" in lib.gnn_last_error()
    assert lib.gnn_block_bounds(100, 10, 25, ctypes.byref(cs), ctypes.byref(cn)) == gnn.GNN_OK
    assert (cs.value, cn.value) == (100, 250)
    assert lib.gnn_block_bounds(10**9, 1024, 25, ctypes.byref(cs), ctypes.byref(cn)) == gnn.GNN_OK
    assert (cs.value, cn.value) == (1024 * 26, 1024 * 25)
    assert lib.gnn_last_error() == b""
    # NULL weights, unsupported dtypes, bad sizes: rejected before any launch
    assert lib.gnn_update_fwd(None, None, gnn.GNN_F32, 8, None, 4, None, None, None, 8, 0, gnn.GNN_F32, None,
                              gnn.GNN_F32, None, 0, None) == gnn.GNN_EINVAL
    assert lib.gnn_update_fwd(None, None, gnn.GNN_F16, 8, None, 4, None, None, None, 8, 0, gnn.GNN_F32, None,
                              gnn.GNN_F32, None, 0, None) == gnn.GNN_EUNSUPPORTED
    assert lib.gnn_update_fwd(None, None, gnn.GNN_F32, 0, None, 4, None, None, None, 8, 0, gnn.GNN_F32, None,
                              gnn.GNN_F32, None, 0, None) == gnn.GNN_EINVAL
    # a bf16 shadow must be 8-byte aligned
    fake = 1 << 24
    assert lib.gnn_update_fwd(fake, fake, gnn.GNN_BF16, 8, None, 4, fake, fake + 2, None, 8, 1, gnn.GNN_BF16, fake,
                              gnn.GNN_BF16, None, 0, None) == gnn.GNN_EINVAL
    assert lib.gnn_gather_features(None, gnn.GNN_F32, gnn.GNN_LOC_DEVICE, 10, 4, 4, None, None, 3, None,
                                   gnn.GNN_F16, None) == gnn.GNN_EUNSUPPORTED
    assert lib.gnn_gather_features(None, gnn.GNN_F32, 7, 10, 4, 4, None, None, 3, None,
                                   gnn.GNN_F32, None) == gnn.GNN_EINVAL
    assert lib.gnn_gather_features(None, gnn.GNN_F32, gnn.GNN_LOC_DEVICE, 10, 4, 2, None, None, 3, None,
                                   gnn.GNN_F32, None) == gnn.GNN_EINVAL
    assert lib.gnn_sgd(None, None, -1, 0.1, None) == gnn.GNN_EINVAL
    assert lib.gnn_aggregate_fwd(None, 0, None, 0, 4, None, 0, None) == gnn.GNN_EINVAL
    assert lib.gnn_softmax_ce(None, 4, 0, None, None, None, None, None, 0, None) == gnn.GNN_EINVAL
    blk = gnn.Block(4, 8, 8, None, None, None, None, None, None, None)
    assert lib.gnn_aggregate_bwd(ctypes.byref(blk), 0, None, 4, None, 0, None, None) == gnn.GNN_EINVAL
    g = gnn.Graph(10, 20, None, None)
    assert lib.gnn_build_block(ctypes.byref(g), None, None, None, 5, 0, 0, 1, 1, ctypes.byref(blk), None, 0,
                               None) == gnn.GNN_EINVAL
    nb = ctypes.c_size_t()
    assert lib.gnn_update_bwd_workspace_size(0, 4, 4, gnn.GNN_BF16, ctypes.byref(nb)) == gnn.GNN_EINVAL
    assert lib.gnn_update_fwd_workspace_size(8, 4, 4, gnn.GNN_F16, ctypes.byref(nb)) == gnn.GNN_EUNSUPPORTED
    assert lib.gnn_update_fwd_workspace_size(8, 4, 1000, gnn.GNN_BF16, ctypes.byref(nb)) == gnn.GNN_OK


def _model(gnn, kind, dims, fanouts, precision):
    m = gnn.Model()
    m.num_layers, m.kind, m.precision = len(dims) - 1, kind, precision
    for i, d in enumerate(dims):
        m.dims[i] = d
    for i, k in enumerate(fanouts):
        m.fanouts[i] = k
    return m


def test_step_layout_capacities_and_disjoint_buffers(gnn):
    lib = gnn.lib()
    m = _model(gnn, gnn.GNN_AGG_SAGE_MEAN, (100, 256, 47), (25, 10), gnn.GNN_BF16)
    lay = gnn.StepLayout()
    assert lib.gnn_train_step_layout(ctypes.byref(m), 2_449_029, 1024, ctypes.byref(lay)) == gnn.GNN_OK
    # no-duplicate upper bounds of the two hops
    assert list(lay.cap_dst[:2]) == [1024, 26_624]
    assert list(lay.cap_nnz[:2]) == [25_600, 266_240]
    assert list(lay.cap_src[:2]) == [26_624, 292_864]
    # hop 1 (the last layer's block) has a transpose, hop 2 (first layer) has none
    assert lay.blk_cscptr[0] and not lay.blk_cscptr[1]
    # the prepare buffers tile the prepare workspace without overlap, the
    # compute buffers the compute workspace
    cd, cs, cn = lay.cap_dst, lay.cap_src, lay.cap_nnz
    prep = [(lay.sampler_ws, lay.sampler_ws_bytes), (lay.x0, cs[1] * 100 * 2)]
    for h in range(2):
        prep += [(lay.blk_counts[h], 32), (lay.blk_src_ids[h], cs[h] * 8), (lay.blk_rowptr[h], (cd[h] + 1) * 8),
                 (lay.blk_col[h], cn[h] * 4)]
    prep += [(lay.blk_cscptr[0], (cs[0] + 1) * 8), (lay.blk_cscrow[0], cn[0] * 4), (lay.blk_csc_ws[0], 1)]
    prep += [(lay.agg[1], cd[1] * 100 * 2)]  # layer 1's aggregation is made by the prepare stage
    comp = [(lay.fwd_ws, lay.fwd_ws_bytes), (lay.bwd_ws, lay.bwd_ws_bytes), (lay.loss_ws, lay.loss_ws_bytes),
            (lay.edges, 8), (lay.error, 8), (lay.loss, 4)]
    comp += [(lay.agg[2], cd[0] * 256 * 2)]
    for l, rows in ((1, cd[1]), (2, cd[0])):
        f_out = (100, 256, 47)[l]
        comp += [(lay.h[l], rows * f_out * (2 if l < 2 else 4)), (lay.grad[l], rows * f_out * 4)]
    comp += [(lay.d_a[2], cd[0] * 512 * 4)]
    for spans, size in ((prep, lay.prep_bytes), (comp, lay.compute_bytes)):
        spans = sorted(spans)
        assert all(a + n <= b for (a, n), (b, _) in zip(spans, spans[1:])), spans
        assert spans[-1][0] + spans[-1][1] <= size and size % 256 == 0
    assert lay.total_bytes == lay.prep_bytes + lay.compute_bytes
    nb = ctypes.c_size_t()
    assert lib.gnn_train_step_workspace_size(ctypes.byref(m), 2_449_029, 1024, ctypes.byref(nb)) == gnn.GNN_OK
    assert nb.value == lay.total_bytes
    bad = _model(gnn, gnn.GNN_AGG_SAGE_MEAN, (100, 256, 47), (25, 0), gnn.GNN_BF16)
    assert lib.gnn_train_step_workspace_size(ctypes.byref(bad), 1000, 10, ctypes.byref(nb)) == gnn.GNN_EINVAL
    bad = _model(gnn, gnn.GNN_AGG_SAGE_MEAN, (100, 256, 47), (25, 10), gnn.GNN_F16)
    assert lib.gnn_train_step_workspace_size(ctypes.byref(bad), 1000, 10, ctypes.byref(nb)) == gnn.GNN_EUNSUPPORTED
    assert lib.gnn_train_step_workspace_size(ctypes.byref(m), 1000, 2000, ctypes.byref(nb)) == gnn.GNN_EINVAL


def test_max_aggregator_host_validation(gnn):
    # GraphSAGE's max aggregator: every error path is taken on the host
    lib = gnn.lib()
    fake = 1 << 24  # aligned stand-in addresses, never dereferenced
    blk = gnn.Block(4, 8, 8, fake, fake, fake, fake, None, None, None)  # no transpose
    B = ctypes.byref(blk)
    assert lib.gnn_aggregate_fwd_max(None, fake, gnn.GNN_F32, 4, fake, gnn.GNN_F32, fake, None) == gnn.GNN_EINVAL
    assert lib.gnn_aggregate_fwd_max(B, fake, gnn.GNN_F16, 4, fake, gnn.GNN_F32, fake, None) == gnn.GNN_EUNSUPPORTED
    assert lib.gnn_aggregate_fwd_max(B, fake, gnn.GNN_F32, 0, fake, gnn.GNN_F32, fake, None) == gnn.GNN_EINVAL
    assert lib.gnn_aggregate_fwd_max(B, fake, gnn.GNN_F32, 4, None, gnn.GNN_F32, fake, None) == gnn.GNN_EINVAL
    assert lib.gnn_aggregate_fwd_max(B, fake, gnn.GNN_F32, 4, fake, gnn.GNN_F32, fake + 2, None) == gnn.GNN_EINVAL
    assert b"misaligned" in lib.gnn_last_error()
    # the backward needs the transpose and the argmax table
    assert lib.gnn_aggregate_bwd_max(B, fake, fake, 4, None, gnn.GNN_F32, fake, None) == gnn.GNN_EINVAL
    assert b"transpose" in lib.gnn_last_error()
    blk_t = gnn.Block(4, 8, 8, fake, fake, fake, fake, fake, fake, None)
    assert lib.gnn_aggregate_bwd_max(ctypes.byref(blk_t), None, fake, 4, None, gnn.GNN_F32, fake,
                                     None) == gnn.GNN_EINVAL
    assert lib.gnn_aggregate_bwd_max(ctypes.byref(blk_t), fake, fake, 4, fake, gnn.GNN_F16, fake,
                                     None) == gnn.GNN_EUNSUPPORTED
    # the sum aggregations do not take the max kind
    assert lib.gnn_aggregate_fwd(B, gnn.GNN_AGG_SAGE_MAX, fake, gnn.GNN_F32, 4, fake, gnn.GNN_F32,
                                 None) == gnn.GNN_EINVAL
    assert b"unknown aggregation" in lib.gnn_last_error()
    # the two-layer launches: x_self and the table are required
    lab = fake
    assert lib.gnn_two_layer_fwd_max(B, 4, None, fake, 32, fake, None, 64, fake, fake, None, 8, fake, fake, fake, lab,
                                     4, fake, fake, None, None) == gnn.GNN_EINVAL
    assert lib.gnn_two_layer_fwd_max(B, 4, fake, fake, 32, fake, None, 64, fake, fake, None, 8, fake, None, fake, lab,
                                     4, fake, fake, None, None) == gnn.GNN_EINVAL
    assert lib.gnn_two_layer_bwd_max(ctypes.byref(blk_t), fake, fake, 32, fake, 8, fake, 64, fake, None, fake, fake,
                                     8, fake, fake, fake, fake, fake, 1 << 20, None) == gnn.GNN_EINVAL
    nb = ctypes.c_size_t()
    assert lib.gnn_two_layer_bwd_workspace_size(gnn.GNN_AGG_SAGE_MAX, 100, 256, 47, 100, 10,
                                                ctypes.byref(nb)) == gnn.GNN_OK
    n_max = nb.value
    assert lib.gnn_two_layer_bwd_workspace_size(gnn.GNN_AGG_SAGE_MEAN, 100, 256, 47, 100, 10,
                                                ctypes.byref(nb)) == gnn.GNN_OK
    assert nb.value == n_max  # the same dW partials as the mean model's


def test_max_model_step_layout(gnn):
    # the max model keeps an argmax table per layer from 2 on, disjoint
    # from every other compute buffer; layer 1 keeps none
    lib = gnn.lib()
    m = _model(gnn, gnn.GNN_AGG_SAGE_MAX, (100, 256, 256, 47), (15, 10, 5), gnn.GNN_BF16)
    lay = gnn.StepLayout()
    assert lib.gnn_train_step_layout(ctypes.byref(m), 2_449_029, 1024, ctypes.byref(lay)) == gnn.GNN_OK
    cd = lay.cap_dst
    assert lay.argmax[1] == 0 and lay.argmax[2] and lay.argmax[3]
    dims = (100, 256, 256, 47)
    spans = [(lay.fwd_ws, lay.fwd_ws_bytes), (lay.bwd_ws, lay.bwd_ws_bytes), (lay.loss_ws, lay.loss_ws_bytes),
             (lay.edges, 8), (lay.error, 8), (lay.loss, 4)]
    for l in (1, 2, 3):
        rows = cd[3 - l]
        spans += [(lay.h[l], rows * dims[l] * (2 if l < 3 else 4)), (lay.grad[l], rows * dims[l] * 4)]
        if l >= 2:
            spans += [(lay.agg[l], rows * dims[l - 1] * 2), (lay.d_a[l], rows * 2 * dims[l - 1] * 4),
                      (lay.argmax[l], rows * dims[l - 1] * 4)]
    spans = sorted(spans)
    assert all(a + n <= b for (a, n), (b, _) in zip(spans, spans[1:])), spans
    assert spans[-1][0] + spans[-1][1] <= lay.compute_bytes
    mean = _model(gnn, gnn.GNN_AGG_SAGE_MEAN, (100, 256, 256, 47), (15, 10, 5), gnn.GNN_BF16)
    lay_m = gnn.StepLayout()
    assert lib.gnn_train_step_layout(ctypes.byref(mean), 2_449_029, 1024, ctypes.byref(lay_m)) == gnn.GNN_OK
    assert all(lay_m.argmax[l] == 0 for l in range(5))


def test_two_stage_step_validation(gnn):
    # argument checks of the prepare / compute entry points run on the host
    # before anything is enqueued (the pointers below are never dereferenced)
    lib = gnn.lib()
    m = _model(gnn, gnn.GNN_AGG_SAGE_MEAN, (32, 16, 8), (5, 5), gnn.GNN_F32)
    for l in range(2):
        m.w[l] = m.b[l] = m.dw[l] = m.db[l] = 1 << 20
    lay = gnn.StepLayout()
    assert lib.gnn_train_step_layout(ctypes.byref(m), 1000, 64, ctypes.byref(lay)) == gnn.GNN_OK
    fake = 1 << 24
    assert lib.gnn_step_prepare_workspace_init(ctypes.byref(m), 1000, 64, fake, lay.prep_bytes - 256,
                                               None) == gnn.GNN_ESIZE
    assert lib.gnn_step_prepare_workspace_init(ctypes.byref(m), 1000, 64, fake + 8, lay.prep_bytes,
                                               None) == gnn.GNN_EINVAL
    assert lib.gnn_step_compute(ctypes.byref(m), 1000, fake, 64, 0.1, None, None, fake, lay.prep_bytes, fake,
                                lay.compute_bytes - 256, None) == gnn.GNN_ESIZE
    assert lib.gnn_step_compute(ctypes.byref(m), 1000, fake, 64, 0.1, None, None, fake, lay.prep_bytes - 256, fake,
                                lay.compute_bytes, None) == gnn.GNN_ESIZE
    assert lib.gnn_step_compute(ctypes.byref(m), 1000, None, 64, 0.1, None, None, fake, lay.prep_bytes, fake,
                                lay.compute_bytes, None) == gnn.GNN_EINVAL
    assert lib.gnn_step_compute(ctypes.byref(m), 1000, fake, 2000, 0.1, None, None, fake, lay.prep_bytes, fake,
                                lay.compute_bytes, None) == gnn.GNN_EINVAL
    g = gnn.Graph(1000, 5000, fake, fake)
    assert lib.gnn_step_prepare(ctypes.byref(m), None, None, fake, gnn.GNN_F32, gnn.GNN_LOC_DEVICE, 32, fake, 64, 0,
                                0, fake, lay.prep_bytes, None) == gnn.GNN_EINVAL
    assert lib.gnn_step_prepare(ctypes.byref(m), ctypes.byref(g), None, fake, gnn.GNN_F32, gnn.GNN_LOC_DEVICE, 32,
                                fake, 64, 0, 0, fake, lay.prep_bytes - 256, None) == gnn.GNN_ESIZE
    assert lib.gnn_step_prepare(ctypes.byref(m), ctypes.byref(g), None, fake, gnn.GNN_F32, gnn.GNN_LOC_DEVICE, 16,
                                fake, 64, 0, 0, fake, lay.prep_bytes, None) == gnn.GNN_EINVAL


def test_pipelined_steps_validation(gnn):
    # gnn_train_steps checks its slot array, workspaces and counts on the
    # host before creating events or enqueueing anything
    lib = gnn.lib()
    m = _model(gnn, gnn.GNN_AGG_SAGE_MEAN, (32, 16, 8), (5, 5), gnn.GNN_F32)
    for l in range(2):
        m.w[l] = m.b[l] = m.dw[l] = m.db[l] = 1 << 20
    lay = gnn.StepLayout()
    assert lib.gnn_train_step_layout(ctypes.byref(m), 1000, 64, ctypes.byref(lay)) == gnn.GNN_OK
    fake = 1 << 24
    g = gnn.Graph(1000, 5000, fake, fake)

    def call(slots, n_prep=None, steps=3, prep_bytes=lay.prep_bytes, comp=fake, comp_bytes=lay.compute_bytes):
        arr = (ctypes.c_void_p * max(len(slots), 1))(*slots)
        return lib.gnn_train_steps(ctypes.byref(m), ctypes.byref(g), None, fake, gnn.GNN_F32, gnn.GNN_LOC_DEVICE, 32,
                                   fake, fake, 64, 0, 0, steps, 0.1, None, None, arr,
                                   len(slots) if n_prep is None else n_prep, prep_bytes, comp, comp_bytes, None, None)

    a, b, c = fake, fake + (1 << 22), fake + (2 << 22)
    assert call([a]) == gnn.GNN_EINVAL                      # one slot cannot overlap anything
    assert b"n_prep" in lib.gnn_last_error()
    assert call([a, b], n_prep=9) == gnn.GNN_EINVAL         # above GNN_MAX_PREPARE_SLOTS
    assert call([a, a]) == gnn.GNN_EINVAL                   # the same workspace twice
    assert call([a, b + 8]) == gnn.GNN_EINVAL               # misaligned
    assert call([a, 0]) == gnn.GNN_EINVAL                   # NULL slot
    assert call([a, b], steps=-1) == gnn.GNN_EINVAL
    assert call([a, b, c], prep_bytes=lay.prep_bytes - 256) == gnn.GNN_ESIZE
    assert call([a, b], comp_bytes=lay.compute_bytes - 256) == gnn.GNN_ESIZE
    assert call([a, b], comp=None) == gnn.GNN_EINVAL


def test_device_error_decode(gnn):
    # the device error flags of a block (counts[3]) and of a step's error
    # word decode on the host into a status and a message naming each flag
    lib = gnn.lib()
    assert lib.gnn_decode_device_errors(0) == gnn.GNN_OK
    assert lib.gnn_last_error() == b""
    assert lib.gnn_decode_device_errors(gnn.GNN_DEVERR_WAIT) == gnn.GNN_EDEVICE
    msg = lib.gnn_last_error()
    assert b"GNN_DEVERR_WAIT" in msg and b"GNN_DEVERR_RANGE" not in msg
    assert lib.gnn_decode_device_errors(gnn.GNN_DEVERR_RANGE) == gnn.GNN_EDEVICE
    msg = lib.gnn_last_error()
    assert b"GNN_DEVERR_RANGE" in msg and b"GNN_DEVERR_WAIT" not in msg
    assert lib.gnn_decode_device_errors(3) == gnn.GNN_EDEVICE
    msg = lib.gnn_last_error()
    assert b"GNN_DEVERR_WAIT" in msg and b"GNN_DEVERR_RANGE" in msg and b"0x3" in msg
    assert lib.gnn_decode_device_errors(0x10 | 1) == gnn.GNN_EDEVICE
    assert b"unknown flags 0x10" in lib.gnn_last_error()
    with pytest.raises(gnn.GnnError) as e:
        gnn.decode_device_errors(2)
    assert e.value.code == gnn.GNN_EDEVICE
    # a NULL or misaligned device word is rejected before any HIP call
    assert lib.gnn_check_device_errors(None, None) == gnn.GNN_EINVAL
    assert lib.gnn_check_device_errors((1 << 24) + 4, None) == gnn.GNN_EINVAL


def test_sampler_fault_hook_validation(gnn):
    lib = gnn.lib()
    assert lib.gnn_debug_sampler_fault(-2, 10) == gnn.GNN_EINVAL
    assert lib.gnn_debug_sampler_fault(1, 0) == gnn.GNN_EINVAL
    assert lib.gnn_debug_sampler_fault(1, 64) == gnn.GNN_OK
    assert lib.gnn_debug_sampler_fault(-1, 0) == gnn.GNN_OK  # back to normal
