"""Stage shapes of the synthetic GPT workloads.

The paper evaluates Megatron GPT-3 stages (Evaluation, Workloads paragraph:
GPT-3 Medium/3.35B/6.7B with TP = 1, micro-batch 1 for the large models).  It
states no sequence length; these workloads use GPT-3's 2048.  The five named
configurations are the measured workloads; the ``TEST_CONFIGS`` are small,
deliberately ragged shapes (not multiples of the GEMM tiles) that the fp64
oracle finishes in seconds, used for element-by-element parity.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple


@dataclass(frozen=True)
class StageConfig:
    name: str
    layers: int
    hidden: int
    heads: int
    ffn: int
    seq: int
    micro_batch: int
    causal: bool
    dtype: str                      # "f32" or "bf16" (storage type of activations/weights)
    n_mb: int                       # micro-batches this stage executes per iteration
    rerouted: Tuple[int, ...] = ()  # micro-batch ids j that were re-routed from a failed peer
    reroute_origin: int = 1         # their original pipeline k
    schedule: str = "1f1b"          # op-list family, see synth.schedules
    warmup: int = 4                 # 1F1B warm-up depth
    ln_eps: float = 1e-5
    seed: int = 0
    w_std: float = 0.02
    x_std: float = 1.0
    dy_std: float = 0.01
    perturbed: bool = False         # non-trivial biases / LN affine (tests only)
    max_stashed_mb: int = 0         # 0 -> n_mb
    max_inflight_mb: int = 0        # 0 -> n_mb

    @property
    def head_dim(self) -> int:
        return self.hidden // self.heads

    @property
    def tokens(self) -> int:
        return self.micro_batch * self.seq

    @property
    def stash_slots(self) -> int:
        return self.max_stashed_mb or self.n_mb

    @property
    def inflight_slots(self) -> int:
        return self.max_inflight_mb or self.n_mb

    def with_(self, **kw) -> "StageConfig":
        return replace(self, **kw)

    # Algorithmic work per layer per micro-batch (causal attention counted at
    # half: the masked half is work the method need not do).
    def flops_per_layer(self) -> Tuple[float, float, float]:
        T, h, f, s, b = self.tokens, self.hidden, self.ffn, self.seq, self.micro_batch
        lin = 2.0 * T * (4 * h * h + 2 * h * f)
        att = (b * s * s * h) if self.causal else (2.0 * b * s * s * h)
        return lin + 2 * att, lin + 4 * att, lin

    def linear_flops_per_layer(self) -> float:
        T, h, f = self.tokens, self.hidden, self.ffn
        return 2.0 * T * (4 * h * h + 2 * h * f)

    def n_params(self) -> int:
        h, f = self.hidden, self.ffn
        return self.layers * (4 * h * h + 2 * h * f + 9 * h + f)


CONFIGS = {
    "tiny": StageConfig(
        name="tiny", layers=1, hidden=256, heads=4, ffn=1024, seq=128, micro_batch=1,
        causal=True, dtype="f32", n_mb=4, rerouted=(3,), schedule="tiny", warmup=2),
    "gpt1.3b": StageConfig(
        name="gpt1.3b", layers=6, hidden=2048, heads=16, ffn=8192, seq=2048, micro_batch=2,
        causal=True, dtype="bf16", n_mb=8, rerouted=(6, 7), schedule="1f1b_cooldown_w"),
    "gpt6.7b": StageConfig(
        name="gpt6.7b", layers=4, hidden=4096, heads=32, ffn=16384, seq=2048, micro_batch=1,
        causal=True, dtype="bf16", n_mb=16, schedule="1f1b_deferred_shuffled_w"),
    "gpt13b": StageConfig(
        name="gpt13b", layers=2, hidden=5120, heads=40, ffn=20480, seq=2048, micro_batch=1,
        causal=True, dtype="bf16", n_mb=12, rerouted=(8, 9, 10, 11), schedule="1f1b_deferred_w"),
    "gpt175b": StageConfig(
        name="gpt175b", layers=1, hidden=12288, heads=96, ffn=49152, seq=2048, micro_batch=1,
        causal=True, dtype="bf16", n_mb=8, schedule="coupled", max_stashed_mb=1,
        max_inflight_mb=1),
}

# Small shapes for element-by-element parity: several GEMM tiles plus a ragged
# tail in every dimension (hidden 384 = 1.5 tiles of 256, seq 320 = 1.25 tiles),
# head dim 128 and 64 as in the real workloads.
TEST_CONFIGS = {
    "small_bf16": StageConfig(
        name="small_bf16", layers=2, hidden=384, heads=3, ffn=1536, seq=320, micro_batch=2,
        causal=True, dtype="bf16", n_mb=4, rerouted=(3,), schedule="1f1b_deferred_shuffled_w",
        warmup=2, perturbed=True),
    "small_f32": StageConfig(
        name="small_f32", layers=2, hidden=192, heads=3, ffn=768, seq=136, micro_batch=2,
        causal=True, dtype="f32", n_mb=3, rerouted=(2,), schedule="1f1b_deferred_shuffled_w",
        warmup=2, perturbed=True),
    # A wide FFN makes the FC1 forward, FC2 input-gradient and FC1/FC2 weight
    # products large enough to take 256 x 256 GEMM tiles, with ragged edges
    # (640 tokens = 2.5 tiles, hidden 1152 = 4.5 tiles).
    "wide_bf16": StageConfig(
        name="wide_bf16", layers=1, hidden=1152, heads=9, ffn=12288, seq=320, micro_batch=2,
        causal=True, dtype="bf16", n_mb=2, rerouted=(1,), schedule="1f1b_deferred_shuffled_w",
        warmup=2, perturbed=True),
    # Causal attention whose grid of query-block pairs (4 sequences x 10 heads
    # x 4 pairs = 160) would fill the last round of 256 compute units poorly,
    # so F and B_input run the per-query-block kernels, over 8 query blocks of
    # 128 (key ranges of 2 .. 16 key blocks), as the 40-head 13B stage does.
    "block_bf16": StageConfig(
        name="block_bf16", layers=1, hidden=1280, heads=10, ffn=2048, seq=1024, micro_batch=4,
        causal=True, dtype="bf16", n_mb=2, rerouted=(1,), schedule="1f1b_deferred_shuffled_w",
        warmup=2, perturbed=True),
    # Weight-gradient products of more than one round of 256 x 256 tiles with
    # ragged edges (FC1: [1152, 16200] = 5 x 64 tiles, FC2: 64 x 5), which the
    # launcher gives to the persistent kernel on a 256-CU device.
    "persist_bf16": StageConfig(
        name="persist_bf16", layers=1, hidden=1152, heads=9, ffn=16200, seq=128, micro_batch=2,
        causal=True, dtype="bf16", n_mb=3, rerouted=(2,), schedule="1f1b_deferred_shuffled_w",
        warmup=2, perturbed=True),
    "tiny_noncausal": CONFIGS["tiny"].with_(name="tiny_noncausal", causal=False),
    "tiny_perturbed": CONFIGS["tiny"].with_(name="tiny_perturbed", perturbed=True),
}


def get_config(name: str) -> StageConfig:
    if name in CONFIGS:
        return CONFIGS[name]
    return TEST_CONFIGS[name]
