"""MI355X (gfx950) hot path of sampled mini-batch GNN training.

``gnn`` is the ctypes binding of ``libgnn.so`` (C ABI in include/gnn.h);
``build`` compiles the library with hipcc.
"""
from . import gnn  # noqa: F401
from .gnn import (GNN_AGG_GCN_SYM, GNN_AGG_SAGE_MEAN, GNN_BF16, GNN_F16, GNN_F32, GNN_LOC_DEVICE,  # noqa: F401
                  GNN_LOC_HOST_PINNED, DeviceBlock, DeviceGraph, GnnError, Trainer)
