"""MI355X (gfx950) MoE expert stage with tile-level signaling (producer/consumer overlap).

The compute path lives in the HIP library ``_lib/libmoe_stage.so`` behind the
C ABI of ``include/moe_stage.h``; ``binding`` is its ctypes binding and
``workload`` makes seeded synthetic inputs.  Importing the package loads
nothing: the library is loaded on first use.
"""
__all__ = ["binding", "workload", "build"]
