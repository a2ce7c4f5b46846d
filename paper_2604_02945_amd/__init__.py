"""MI355X (gfx950) implementation of MSAO's fine-grained sparsity analysis.

The HIP kernels and the C ABI live in libmsao.so (sources in csrc/, ABI in
include/msao.h at the repository root); `binding` is a thin ctypes layer over
it with the same entry-point names.
"""
from .binding import (  # noqa: F401
    AUDIO, BF16, F32, FLAG_TEMPORAL_LITERAL, IMAGE, TEXT, VIDEO,
    Context, DeviceSegment, MsaoError, Outputs, Plan, compact_layout, compacted_rows, default_params, lib,
    msao_compact, msao_mas_score, msao_run, msao_select_tokens, msao_temporal_redundancy, prepare, sizes,
)
