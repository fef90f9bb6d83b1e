"""The five workloads the library is checked and measured on.

Shapes follow the paper's model table (SmolLM2-135M, Qwen2.5-1.5B and
Gemma 3-4B rows, Section 4, Table "tab:models" and Appendix A).  Weights and
residuals are synthetic (seeded, random-init); no trained checkpoint is used.
Unstated parameters take the readings documented in the design doc: gamma =
1 + N(0, 0.1) and eps = 1e-6 for every config.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    dtype: str            # "f32" or "bf16"
    d_model: int
    n_q: int
    n_kv: int
    head_dim: int
    layers: int
    batch: int
    ctx: int              # checkpointed context tokens per sequence (recomputed)
    rope_theta: float = 1.0e4
    rms_eps: float = 1.0e-6
    w_std: float = 0.02
    gamma_std: float = 0.1
    layer_scale: tuple = (1.0, 1.0)    # per-layer residual scale ~ U(lo, hi)
    pos_offset_max: int = 0            # pos0[b] ~ U{0 .. pos_offset_max-1} (0: all zero)
    batches: tuple = field(default=())  # batch sweep (crossover workload)
    turns: int = 0                     # multi-turn workload: turns of turn_tokens
    turn_tokens: int = 0

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv


SMOLLM_FP32 = Workload(
    name="smollm2-135m-layer-fp32", cfg_id=0, dtype="f32", d_model=576, n_q=9, n_kv=3,
    head_dim=64, layers=1, batch=1, ctx=256)

GEMMA3_4B = Workload(
    name="gemma3-4b-34L-b1-ctx4096-bf16", cfg_id=1, dtype="bf16", d_model=2560, n_q=8, n_kv=4,
    head_dim=256, layers=34, batch=1, ctx=4096, layer_scale=(0.5, 4.0))

GEMMA3_SWEEP = Workload(
    name="gemma3-4b-layer-ctx2048-batch-sweep-bf16", cfg_id=2, dtype="bf16", d_model=2560, n_q=8,
    n_kv=4, head_dim=256, layers=1, batch=1, ctx=2048, batches=(1, 2, 4, 8, 16, 32, 64))

QWEN_1_5B = Workload(
    name="qwen-1.5b-28L-b8-ctx16384-bf16", cfg_id=3, dtype="bf16", d_model=1536, n_q=12, n_kv=2,
    head_dim=128, layers=28, batch=8, ctx=16384, rope_theta=1.0e6, pos_offset_max=1024)

GEMMA3_MULTITURN = Workload(
    name="gemma3-4b-34L-b16-20x256-multiturn-bf16", cfg_id=4, dtype="bf16", d_model=2560, n_q=8,
    n_kv=4, head_dim=256, layers=34, batch=16, ctx=5120, turns=20, turn_tokens=256)

ALL = (SMOLLM_FP32, GEMMA3_4B, GEMMA3_SWEEP, QWEN_1_5B, GEMMA3_MULTITURN)
