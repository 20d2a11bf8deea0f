"""Long-context and batched launch paths of the decode loop, teacher-forced
against the oracle at the 8B attention shape (32 q-heads, 8 kv-heads, head dim
128) with a narrow model (d 512, ffn 1024, vocab 4096, 2 base + 2 micro layers)
so the float64 oracle can run a multi-thousand-token prefill in seconds.

* batch 8, prompt 5200: the prefill runs three chunks (2048 + 2048 + 1104
  rows; the later chunks attend over the earlier chunks' cache entries), and
  every macro-step's fused attention step runs 4 slot splits of about 41 key
  blocks, so each wave loops over two more key chunks after its first (the
  long-context workload's launch, where each wave takes about 16 blocks);
* batch 32, prompt 1300: one attention workgroup per (sequence, kv head), each
  wave about 5 of its sequence's own key blocks (the batched workload's launch).

The oracle follows some rows of each batch; the others are fed seeded groups of
the forced lengths (they only fill the launch).
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleHam
from synth.configs import SHAPE_8B
from tests.gpu_util import teacher_forced

pytestmark = pytest.mark.gpu

NARROW_8B_ATTN = dataclasses.replace(SHAPE_8B, n_layers=2, micro_layers=2, d_model=512, ffn_dim=1024, vocab=4096)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


def _splits(B, P, steps):
    from paper_2505_20438_amd import ham
    return ham.ham_op_attention_step_splits(1, B, 8, 128, P + steps - 1)


def test_three_chunk_prefill_and_split_attention_loop(torch_cuda):
    shp = NARROW_8B_ATTN
    B, P, steps = 8, 5200, 4
    nsplit = _splits(B, P, steps)
    blocks = (P + steps - 1 + 31) // 32
    per_wave = -(-blocks // nsplit) / 8
    print("splits", nsplit, "key blocks per wave", per_wave, flush=True)
    assert nsplit == 4 and per_wave > 4   # the first chunk (2 blocks) and at least two more
    prompts = synth.prompt_ids(4101, B, P, shp.vocab)
    sched = synth.group_schedule(5101, B, steps + 1, 4)
    om = OracleHam(shp, 6101)
    exact, ties = teacher_forced(om, shp, prompts, [0] * B, steps, sched, 6101, debug_steps=steps + 1,
                                 check_rows=[0, 5])
    assert ties <= 1 and exact >= 10


def test_batch32_per_row_attention_loop(torch_cuda):
    shp = NARROW_8B_ATTN
    B, P, steps = 32, 1300, 4
    nsplit = _splits(B, P, steps)
    per_wave = (P + 31) // 32 / 8
    print("splits", nsplit, "key blocks per wave", per_wave, flush=True)
    assert nsplit == 1 and per_wave > 4
    prompts = synth.prompt_ids(4102, B, P, shp.vocab)
    sched = synth.group_schedule(5102, B, steps + 1, 4)
    om = OracleHam(shp, 6102)
    exact, ties = teacher_forced(om, shp, prompts, [0] * B, steps, sched, 6102, debug_steps=steps + 1,
                                 check_rows=[0, 7, 19, 31])
    assert ties <= 1 and exact >= 20
