"""fp64 CPU oracle of the layer-replica hot path. TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product path (the HIP library and its
Python binding) never imports, calls or links anything here, and this package
imports nothing from the product path.

What it computes. A layer replica runs the unchanged decoder layer on a subset
of the in-flight requests (Sec. 3.1, replication mechanism) and its outputs are
bit-wise consistent with the unreplicated model (Sec. 5.2, interference
isolation). So the oracle is the plain definition of a pre-norm decoder layer
(RMSNorm, QKV projection, rotary embedding, grouped-query attention over the
request's cached keys/values, output projection with residual, RMSNorm, SwiGLU
MLP with residual -- the SwiGLU block is the one the cost model of Sec. 4.2
assumes) applied per selected row, in float64, with the row gather before and
the scatter after (the segment-boundary scatter/gather of Sec. 3.1). A span of
consecutive layers (Sec. 3.1) applies it layer after layer.

``oracle/scaling.py`` holds the paper's speedup and cost model (Sec. 4.2) and
the candidate ranking of its scaling step (Sec. 4.4) in plain float64 Python.

Parity status of each function is in its docstring; every function is pinned
by the CPU tests (brute force on tiny shapes, closed forms, invariants, and
library routines of torch in float64).
"""
from .layer import (  # noqa: F401
    rms_norm, rope, silu, attend, layer_forward, span_forward, KVCache,
)
