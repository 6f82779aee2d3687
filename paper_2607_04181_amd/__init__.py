"""MI355X-native hot path of layer-wise replication (one decoder-layer replica
serving its row subset of a decode or prefill batch).

The compute runs in hand-written gfx950 HIP kernels behind the C ABI in
include/coco.h (libcoco.so, built in-tree by build.py); this package is the
thin ctypes binding over it plus the build step.
"""
from ._lib import (  # noqa: F401
    COCO_BF16, COCO_F32, COCO_WS_H, COCO_WS_H2, COCO_WS_O, COCO_WS_Q, COCO_WS_U, COCO_WS_X,
    COCO_WS_X1, CocoError, Handle, LIB_PATH, coco_kv_append, coco_last_error, coco_layer_destroy,
    coco_layer_forward, coco_layer_forward_noalloc, coco_layer_init, coco_layer_set_validate, coco_layer_span_forward,
    coco_layer_workspace, coco_version, make_config, coco_layer_set_timing,
    coco_layer_read_timing, KERNEL_KINDS, coco_probe_read, coco_probe_mfma_bf16,
    make_scale_model, coco_split_batch, coco_comm_time, coco_speedup, coco_cost_mem,
    coco_cost_comp, coco_speedup_vec, coco_scale_candidates,
)
