"""fp64 CPU oracle of the ReCycle stage hot path — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never does and has no CPU fallback.

Parity of every function here is pinned by ``tests/test_oracle_pins.py``.
"""
from .stage import (  # noqa: F401
    AdamHP, LayerShape, OracleStage, StageError, adamw_update, attention, attention_grad,
    gelu, gelu_prime, layer_backward_fused, layer_backward_input, layer_backward_weight,
    layer_forward, layer_norm, layer_norm_grad_input, merge_heads, softmax_rows, split_heads,
    stage_backward_fused, stage_backward_input, stage_backward_weight, stage_forward, to_heads,
    OP_F, OP_B, OP_W, OP_STEP, OP_SKIP, OP_ROLLBACK, adamw_rollback, stash_bytes,
)
from .run import run_oplist, OracleRun  # noqa: F401
