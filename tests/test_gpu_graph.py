"""Graph replay of the macro-step equals launching every kernel on the stream.

ham_macro_step captures its launches (after the step's first kernel) as a HIP
graph once and replays it.  Each replay here is preceded by the step's own
eager kernel and followed by host synchronisation and reads, and every step's
outputs must equal the stream launches bit for bit (the kernels are
deterministic): emitted groups, the model's own tokens, debug logits, counters
and the KV cache.

Marked ``gpu``: needs an MI355X and ``libham.so`` built in-tree.
"""
import dataclasses

import numpy as np
import pytest

import synth
from synth.configs import STOP_FORCED, STOP_HEAD
from tests.gpu_util import SMALL16, config_for, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


def _run(shp, seed, prompts, budgets, steps, sched, graph: bool):
    from paper_2505_20438_amd import ham
    B, P = prompts.shape
    rt = ham.HamRuntime(config_for(shp, B, P, steps), seed)
    rt.set_graph(graph)
    res = run_gpu(rt, prompts, budgets, steps, sched, debug_steps=steps + 1)
    kv = [tuple(t.cpu().numpy() for t in rt.kv_cache(l, P + steps)) for l in (0, shp.n_layers - 1)]
    return res, kv


@pytest.mark.parametrize("mode", [STOP_FORCED, STOP_HEAD])
def test_graph_replay_equals_stream_launches(torch_cuda, mode):
    shp = dataclasses.replace(SMALL16, stop_mode=mode, stop_conf=0.5)
    B, P, steps, seed = 3, 48, 30, 61
    prompts = synth.prompt_ids(62, B, P, shp.vocab)
    sched = synth.group_schedule(63, B, steps + 1, 4) if mode == STOP_FORCED else None
    budgets = [0, 23, 57]
    g, kv_g = _run(shp, seed, prompts, budgets, steps, sched, graph=True)
    s, kv_s = _run(shp, seed, prompts, budgets, steps, sched, graph=False)
    assert g.groups == s.groups and g.own == s.own
    assert g.stats == s.stats
    assert sum(len(x) for x in g.groups) > B * 10
    assert g.logits.keys() == s.logits.keys()
    for key in g.logits:
        assert np.array_equal(g.logits[key], s.logits[key]), key
        assert np.array_equal(g.hidden[key], s.hidden[key]), key
        assert g.stop[key] == s.stop[key], key
    for (kg, vg), (ks, vs) in zip(kv_g, kv_s):
        assert np.array_equal(kg, ks) and np.array_equal(vg, vs)
