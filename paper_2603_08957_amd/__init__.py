"""Tensor-relational (upper-case-lower-case) EinSum on AMD Instinct MI355X.

One binary EinSum over two tensor relations (keys + dense tiles) runs as a
GPU join on the shared promoted labels, an MFMA tile contraction of every
matched pair accumulated per output key, and an atomic-free segmented sum
(Tang et al., PVLDB 19(6), 2026, Sec. 5).  The work is done by the HIP
library ``libtre.so`` through the C ABI in ``include/tre.h``; this package is
its ctypes binding.
"""
from .tre import (  # noqa: F401
    EXPORTS, Einsum3, JoinResult, Output, Plan, TreError, Timing, alloc_workspace, cast_f32_bf16, contract, einsum,
    execute, execute3, execute_async, execute_noalloc, join, join_keys, lib, noalloc_scratch_bytes, output_bounds,
    repartition, scale_f32, stack_rows, tiles_from_entries,
)
