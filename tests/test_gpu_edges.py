"""Edge cases of the decode loop on the GPU, free-running fp32 against the oracle
(group boundaries, tokens and KV counters exact):

* the largest batch (64 sequences) with a one-token prompt, a group cap of 3 and
  ragged budgets, including budgets that end inside the prefill's group and
  sequences that finish long before the others (they write no further slot);
* HEAD mode at confidence 0 (never stops: every group fills to its cap) and at
  cap 2 with a budget, the degenerate settings of the stop test (Sec. 3.3).

Marked ``gpu``: needs an MI355X and ``libham.so`` built in-tree.
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleHam
from synth.configs import STOP_FORCED, STOP_HEAD, TINY
from tests.gpu_util import config_for, oracle_groups_for, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


def _check(res, orcs, budgets, P):
    for b, o in enumerate(orcs):
        assert res.groups[b] == o.groups, b
        st = res.stats[b]
        assert st["kv_len"] == o.kv_len == P + st["gen_slots"], b
        assert st["gen_slots"] == len(o.groups) - 1 and st["groups"] == len(o.groups), b
        assert st["tokens"] == o.tokens and st["device_error"] == 0, b
        if budgets[b] and o.tokens == budgets[b]:  # the budget was spent within the steps run
            assert st["done"] == 1, b


def test_max_batch_one_token_prompt_cap3_ragged_budgets(torch_cuda):
    from paper_2505_20438_amd import ham
    shp = dataclasses.replace(TINY, stop_mode=STOP_FORCED, max_group=3)
    B, P, steps, seed = 64, 1, 12, 71
    prompts = synth.prompt_ids(72, B, P, shp.vocab)
    sched = np.minimum(synth.group_schedule(73, B, steps + 1, 4), 3)
    budgets = [[0, 1, 2, 3, 5, 9, 17, 30][b % 8] for b in range(B)]
    om = OracleHam(shp, seed)
    orcs = oracle_groups_for(om, prompts, budgets, steps, sched)
    rt = ham.HamRuntime(config_for(shp, B, P, steps), seed)
    res = run_gpu(rt, prompts, budgets, steps, sched)
    _check(res, orcs, budgets, P)
    assert sum(1 for b in range(B) if budgets[b] and orcs[b].tokens == budgets[b]) >= 40
    assert max(len(g) for gs in res.groups for g in gs) == 3
    assert any(len(res.groups[b]) == 1 for b in range(B))   # budgets ending inside the first group


@pytest.mark.parametrize("cap,conf,budget", [(4, 0.0, 0), (2, 0.0, 37), (4, 0.5, 29)])
def test_head_mode_extremes(torch_cuda, cap, conf, budget):
    from paper_2505_20438_amd import ham
    shp = dataclasses.replace(TINY, stop_mode=STOP_HEAD, stop_conf=conf, max_group=cap)
    B, P, steps, seed = 3, 20, 24, 81
    prompts = synth.prompt_ids(82, B, P, shp.vocab)
    budgets = [budget] * B
    om = OracleHam(shp, seed)
    orcs = oracle_groups_for(om, prompts, budgets, steps)
    rt = ham.HamRuntime(config_for(shp, B, P, steps), seed)
    res = run_gpu(rt, prompts, budgets, steps)
    _check(res, orcs, budgets, P)
    if conf == 0.0:  # never stops: every group is full except one cut by the budget
        for gs in res.groups:
            assert all(len(g) == cap for g in gs[:-1])
