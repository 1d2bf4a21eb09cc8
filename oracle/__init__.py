"""Float64 CPU oracle of the functional-reconstruction step (test infrastructure only)."""
from .mla_recon_oracle import (  # noqa: F401
    rope_tables, rope_apply, rope_apply_transpose, causal_softmax, causal_attention,
    teacher_forward, teacher_logits, student_logits, student_forward, recon_loss,
    student_backward, reconstruction_step,
)
from .adamw_oracle import adamw_step  # noqa: F401
from .stack_oracle import rms_norm, capture  # noqa: F401
from .decode_oracle import absorbed_decode  # noqa: F401
