"""CPU oracle for the unified attention path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct implementations of what the GPU path
computes, written from the paper's definitions (Sections 3.1, 3.2 and 4.1)
and checked against closed forms, brute force and library routines by the
``-m "not gpu"`` tests.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it.  It shares no code with
the HIP kernels or the binding, and neither imports the other.
"""
from .attention import (  # noqa: F401
    CHUNK_KEYS,
    LSE_ABS,
    MAX_ABS,
    MAX_SLACK,
    MEAN_ABS,
    REL_BF16,
    TILE_KEYS,
    attention_row_fp64,
    attention_rows_fp64,
    bf16_to_f64,
    causal_attention_fp64,
    default_scale,
    gather_paged,
    paged_decode_fp64,
    parity_report,
    round_to_bf16,
    tile_emulate_fp32,
    tile_emulate_rows_fp32,
    to_bf16_bits,
)
from .kv_cache import kv_write  # noqa: F401
from .lm_head import abs_dot, lm_head_logprob_fp64, logits_bf16, logits_fp64  # noqa: F401
from .logprob import logprob_fp64  # noqa: F401
from .norm_rope import qk_norm_rope, rms_norm_bf16, rope_neox, rope_table  # noqa: F401
from .attention_backward import attention_backward_fp64, backward_error_scales, dq_rows_fp64  # noqa: F401
