"""DAVET hot path on MI355X (gfx950): Python binding of libdavet.so.

Every step of the path runs in the HIP library; this package only marshals
arguments (see ``_lib``).  Import fails loudly if the library is not built.
"""

from ._lib import (  # noqa: F401
    DAVET_BF16, DAVET_F16, DAVET_F32, DAVET_HEAD_ROWS, DAVET_HEAD_TILED,
    DAVET_REALIZER_MERGE, DAVET_REALIZER_POOL, DAVET_REALIZER_PRUNE,
    MAX_REALIZER_GRID, MAX_SEQS, STATIC_SCRATCH_BYTES, EXPORTED, LIB_PATH, DavetError,
    LayerWeights, Mailbox, ModelCfg, Policy, ViewGeom, Weights, WeightsT,
    davet_set_wait_limit, default_mailbox,
    davet_build_views, davet_build_views_static, davet_convert, davet_demand_prior, davet_denoise_step,
    davet_fp16_overflow_count, davet_set_attention_split,
    davet_head_tiled_elems, davet_pack_head, davet_parse_operation,
    davet_policy_envelope, davet_policy_step, davet_policy_step_device,
    davet_realizer_key_count,
    davet_realizer_keys, davet_realizer_maps, davet_run_schedule,
    davet_step_stats, davet_unmask, davet_version, davet_view_map_sizes,
    davet_view_sizes, davet_views_scratch_bytes,
    davet_workspace_bytes, prof_enable, prof_only, prof_read, prof_reset, raw,
)
