"""ZeRO P_os+g shard optimizer step for AMD Instinct MI355X (gfx950).

The step itself lives in the HIP/C-ABI library ``libzeroshard.so`` built from
``csrc/``; ``paper_1910_02054_amd.binding`` marshals arguments to it.  Nothing
is imported eagerly so that the workload generators can be used without the
library.
"""
__all__ = ["binding", "workloads"]
