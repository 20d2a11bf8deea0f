"""Model and workload shapes of the five benchmark configurations.

Shapes only (no arithmetic).  ``ctx_layers`` are 1-based indices of the base
layers whose residual outputs form the micro-decoder context: by default
C = min(4, L) layers, l_i = ceil(i * L / C), or an explicit ``ctx_layer_set``
(in the paper the micro decoder is conditioned on outputs of intermediate base
layers plus the final one, Sec. 3.3 and Fig. 2a; which layers is a reading).
"""
from __future__ import annotations

import dataclasses
import math

STOP_HEAD, STOP_TOKEN, STOP_FORCED, STOP_FORCED_TOKEN = 0, 1, 2, 3
F32, BF16 = 0, 1


@dataclasses.dataclass(frozen=True)
class HamShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    micro_layers: int
    max_group: int = 4
    stop_mode: int = STOP_FORCED
    stop_id: int = 0
    stop_conf: float = 0.5
    rope_theta: float = 500000.0
    norm_eps: float = 1e-5
    dtype: int = BF16
    ctx_layer_set: tuple = ()   # explicit 1-based context layers; empty = the default reading

    @property
    def ctx_layers(self) -> tuple:
        if self.ctx_layer_set:
            return tuple(int(x) for x in self.ctx_layer_set)
        c = min(4, self.n_layers)
        return tuple(int(math.ceil(i * self.n_layers / c)) for i in range(1, c + 1))

    @property
    def qkv_dim(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: HamShape
    batch: int
    prompt_len: int
    max_new: int          # output-token budget per sequence (0 = unlimited)
    macro_steps: int      # ham_macro_step calls to make (for budgeted runs: until done)
    seed_weights: int
    seed_prompt: int
    seed_sched: int


TINY = HamShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=704,
                vocab=1024, micro_layers=1, max_group=4, stop_mode=STOP_TOKEN, stop_id=1023,
                dtype=F32)
SHAPE_1B = HamShape(n_layers=16, d_model=2048, n_heads=32, n_kv_heads=8, head_dim=64,
                    ffn_dim=8192, vocab=128256, micro_layers=2)
SHAPE_8B = HamShape(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                    ffn_dim=14336, vocab=128256, micro_layers=2)

WORKLOADS = {
    # tiny fp32 model, TOKEN stop (reserved id 1023), 128 macro-steps, no budget
    "c1_tiny_f32": Workload("c1_tiny_f32", TINY, 1, 64, 0, 128, 1001, 2001, 3001),
    # 1B-shaped bf16, forced geometric group lengths, 512 output tokens
    "c2_1b_bf16": Workload("c2_1b_bf16", SHAPE_1B, 1, 512, 512, 0, 1002, 2002, 3002),
    # 8B-shaped bf16, batch 1
    "c3_8b_bf16": Workload("c3_8b_bf16", SHAPE_8B, 1, 1024, 1024, 0, 1003, 2003, 3003),
    # 8B-shaped bf16, batch 32 with ragged smashed-KV lengths
    "c4_8b_b32": Workload("c4_8b_b32", SHAPE_8B, 32, 2048, 512, 0, 1004, 2004, 3004),
    # 8B-shaped bf16, long context
    "c5_8b_long": Workload("c5_8b_long", SHAPE_8B, 4, 32768, 1024, 0, 1005, 2005, 3005),
}


def with_shape(w: Workload, **kw) -> Workload:
    return dataclasses.replace(w, shape=dataclasses.replace(w.shape, **kw))
