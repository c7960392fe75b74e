"""CPU oracle for the SBD decode step (test infrastructure only; see sbd_oracle)."""
from .sbd_oracle import (Model, SeqCache, BlockResult, attention, apply_rope, decode_weight,
                         eb_select, eb_select_from_entropy, inference_mask, rms_norm,
                         rope_cos_sin, round_to_bf16, row_entropy, silu)
