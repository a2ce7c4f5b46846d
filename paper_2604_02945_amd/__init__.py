"""MI355X (gfx950) implementation of MSAO's fine-grained sparsity analysis
(Sec. 4.1, with the MAS-guided selection and compaction it drives) and of the
decoding-side pieces of its speculative offloading (Sec. 4.2): the draft
model's confidence on the GPU and Algorithm 1's threshold logic on the host.

The HIP kernels and the C ABI live in libmsao.so (sources in csrc/, ABI in
include/msao.h at the repository root); `binding` is a thin ctypes layer over
it with the same entry-point names.
"""
from .binding import (  # noqa: F401
    AUDIO, BF16, F32, FLAG_TEMPORAL_LITERAL, IMAGE, TEXT, VIDEO,
    Context, DeviceSegment, MsaoError, Outputs, Plan, compact_layout, compacted_rows, default_params, lib,
    msao_compact, msao_mas_score, msao_run, msao_select_tokens, msao_temporal_redundancy, prepare, sizes,
    DECIDE_HOLD, DECIDE_OFFLOAD, DECIDE_SEND, Scheduler, comm_latency, expected_e2e_latency,
    expected_spec_tokens, msao_draft_entropy, p_conf, retention_floor, sched_default_params,
    msao_mas_score_learned, msao_temporal_simhash, msao_run_simhash, FLAG_SELECT_PER_FRAME,
    msao_run_noalloc, msao_stream_read, msao_run_learned,
)
