"""EDiT layer-wise outer synchronization step on AMD Instinct MI355X (gfx950).

The HIP library (libedit_outer.so, C ABI in include/edit_outer.h) does all
of the work; `outer` is its Python binding and `synth` makes seeded
synthetic workloads shaped like Llama decoder layers.
"""
from .outer import (  # noqa: F401
    AE, GC, ONE_PASS, WA, EditOuter, EditOuterError, LayerState, OuterConfig, SyncGroupWorker,
    copy_probe, load_library, min_warmup,
)
