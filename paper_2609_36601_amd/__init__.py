"""SAKI coupling-and-routing path on AMD MI355X (gfx950).

The compute lives in libsaki.so (HIP kernels behind the C ABI of
include/saki.h); this package is its thin Python binding.
"""
from .binding import (  # noqa: F401
    COUPLE_FIELDS, EXPORTED, SAKI_BF16, SAKI_CHUNK, SAKI_F32, SAKI_MAX_VOCAB, SAKI_OP_COUPLE,
    SAKI_OP_ROUTE, SAKI_OP_SELECT, SAKI_OP_VERIFY, SAKI_SELECT_RANDOM, SAKI_SELECT_TV_WEIGHTED, SAKI_STATIC_MAX_ROWS,
    SAKI_TARGET_MODE, SAKI_TARGET_SAMPLE, SEQ_FINISHED, SEQ_RUNNING, SEQ_STOPPED, SakiError,
    alloc_couple_out, alloc_rows, alloc_traj, couple, load,
    probe_metrics, route_loss, sample, saki_commit, saki_couple, saki_couple_static, saki_probe_metrics, saki_route_loss,
    saki_sample, saki_select_positions, saki_spec_verify, select_positions, spec_verify,
    workspace_bytes)
from .speculative import rollout  # noqa: F401
