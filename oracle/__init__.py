"""CPU oracle for the anchor-branched greedy rollout -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct NumPy implementation of what
the rollout computes, written from the paper (Eq. 3 of Sec. 3.2, "Labels from
the target's rollout", and the "Rollout implementation" paragraph of App. A,
"Training Configuration").  It exists to check the HIP path.  Only the test
suite, the smoke entry point and the benchmark's CPU-baseline leg may import
it; the product path never routes through it.  It shares no code with the HIP
library: inputs come from the seeded generator module, which holds none of the
method's arithmetic.

Every function computes in float64 by default.  Parity pins: see the
``tests/test_oracle_*.py`` files; every function below is pinned (no
"parity unpinned" function exists in this package).
"""
from .reference import (  # noqa: F401
    Params,
    bf16_round,
    rmsnorm,
    rope,
    silu,
    causal_gqa_attention,
    log_softmax,
    greedy_argmax,
    embed_rows,
    decoder_forward,
    decoder_layer_at,
    head_logits,
    prefill_outputs,
    rollout_naive,
    rollout_teacher_forced,
    rollout_kv_shared,
)
