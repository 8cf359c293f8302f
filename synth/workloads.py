"""Workload recipes: the five synthetic configurations of the batched RPS step.

Each recipe fixes the model shape, arithmetic type, sequence layout, pivot
and candidate parameters and the seeds.  Prompts are uniform on the vocabulary
without [MASK]; the response is all [MASK] at the start of a step.  These
stand in for the paper's benchmark prompts (generation length 256, block 32).
"""
from __future__ import annotations

from dataclasses import dataclass, field

from .inputs import ModelShape, TINY, B8

SEED_WEIGHTS = 0
SEED_PROMPT = 1
SEED_SCALE = 2


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    dtype: str                 # "f32" or "bf16"
    prompt_len: int            # random prompt tokens (or cached prefix length)
    gen_len: int               # masked response length
    block: int                 # semi-autoregressive block size
    pivot_mode: str            # "band" (percentile band, multi-pivot) or "paper" (mass filter)
    n_pivots: int
    n_cand: int
    k_max: int = 10
    r: float = 0.0
    tau_pivot: float = 0.9
    pct_lo: float = 25.0
    pct_hi: float = 75.0
    lam: float = 0.0
    tau_conf: float = -1.0     # < 0: no confidence commit inside the step
    logit_scale: float = 1.0
    scale_range: tuple = field(default=())   # (s_lo, s_hi): per-position scales
    topk: int = 16
    cached: bool = False
    capacity: int = 16         # lookahead batch capacity

    @property
    def seq(self) -> int:
        return self.prompt_len + (self.block if self.cached else self.gen_len)


WORKLOADS = {
    # 2-layer fp32 model, 32 prompt + 32 masked, 2 band pivots x top-4 = 8 branches
    "tiny_rps_step_f32": Workload(
        name="tiny_rps_step_f32", model=TINY, dtype="f32", prompt_len=32, gen_len=32, block=32,
        pivot_mode="band", n_pivots=2, n_cand=4, logit_scale=4.0, capacity=8),
    # 8B-class single denoising forward, batch 1 x 512
    "b8_forward_bf16": Workload(
        name="b8_forward_bf16", model=B8, dtype="bf16", prompt_len=256, gen_len=256, block=256,
        pivot_mode="band", n_pivots=4, n_cand=4, capacity=1),
    # 8B-class RPS lookahead step: 4 pivots x 4 candidates = 16 sequences of 512
    "b8_rps_step_bf16": Workload(
        name="b8_rps_step_bf16", model=B8, dtype="bf16", prompt_len=256, gen_len=256, block=256,
        pivot_mode="band", n_pivots=4, n_cand=4, capacity=16),
    # 8B-class full blockwise decode (Algorithm 1): confidence commit + one pivot lookahead
    "b8_decode_bf16": Workload(
        name="b8_decode_bf16", model=B8, dtype="bf16", prompt_len=256, gen_len=256, block=32,
        pivot_mode="paper", n_pivots=1, n_cand=10, k_max=10, r=0.1, tau_pivot=0.9, lam=0.1,
        tau_conf=0.9, scale_range=(2.6, 16.0), capacity=16),
    # 8B-class KV-cached step: 1024 cached prefix + one 32-position block, 16 branches
    "b8_cached_step_bf16": Workload(
        name="b8_cached_step_bf16", model=B8, dtype="bf16", prompt_len=1024, gen_len=32, block=32,
        pivot_mode="band", n_pivots=4, n_cand=4, cached=True, capacity=16),
}
