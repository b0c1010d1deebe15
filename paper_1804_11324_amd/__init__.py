"""MI355X-native batched NMT beam decoding with LMBR n-gram posteriors.

The compute path is the HIP library liblmbr.so (include/lmbr.h); this package
is its ctypes binding (``_abi``) and its in-tree build (``build``).
"""
from ._abi import (LMBR_DEV_NONFINITE, LMBR_DEV_TABLE, LMBR_E_CAPACITY, LMBR_E_DEVICE, LMBR_E_INVALID,
                   LMBR_FINISH_AT_T,
                   LMBR_FINISH_EOS_BACKUP, LMBR_STATE_FN, LMBR_STEP_FUSED, LMBR_STEP_TWO_PASS,
                   BeamState, Context, LmbrError, lmbr_device_status, lmbr_workspace_bytes,
                   lmbr_static_scratch_bytes, lmbr_beam_step_logits_static, lmbr_projected_rows,
                   lmbr_set_lmbr_layout, LMBR_L_SPARSE, LMBR_L_DENSE, lmbr_plan_batches,
                   lmbr_beam_step, lmbr_beam_step_logits, lmbr_config, lmbr_create, lmbr_decode,
                   lmbr_destroy, lmbr_device_bytes, lmbr_gather_rows, lmbr_load_posteriors,
                   lmbr_load_posteriors_into, lmbr_table_bytes,
                   lmbr_project, lmbr_score, lmbr_score_logits, lmbr_select, lmbr_set_constraints,
                   lmbr_set_decode_options, lmbr_set_projection, lmbr_set_sentence_steps, lmbr_set_step_path,
                   lmbr_state_init, lmbr_state_probe, lmbr_synth_hidden, lmbr_table_build,
                   lmbr_traceback, make_config, lib)

__all__ = [n for n in dir() if n.startswith("lmbr_")] + [
    "BeamState", "Context", "LmbrError", "make_config", "lib", "LMBR_FINISH_AT_T",
    "LMBR_FINISH_EOS_BACKUP", "LMBR_STEP_TWO_PASS", "LMBR_STEP_FUSED", "LMBR_E_DEVICE",
    "LMBR_E_CAPACITY", "LMBR_E_INVALID",
    "LMBR_DEV_NONFINITE", "LMBR_DEV_TABLE", "LMBR_STATE_FN", "LMBR_L_SPARSE", "LMBR_L_DENSE"]
