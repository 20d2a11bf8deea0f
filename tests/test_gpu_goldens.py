"""The full-depth workload models against the oracle's stored decisions.

``tests/golden/golden_<workload>.json`` holds what the float64 oracle computed
(``tests/golden/make_goldens.py``, which calls only the oracle and the seeded
generators) for sequence 0 of a workload: the emitted groups of the prefill and
the first macro-steps, and per token decision the token, the stop logit, the
16 largest logits, and seeded samples of the logits and of the normed hidden
state.  Here the GPU runs the same model at full depth (the 8B shape at 32
layers, the 1B shape at 16), built with the workload's own capacity so every
launch has the benchmark's shape, teacher-forced with the oracle's groups:

* logits at the sampled ids and at the oracle's top 16, the normed hidden
  state at the sampled coordinates and the stop logit within 2e-2;
* every token equal to the oracle's, or a near tie that the measured error
  explains (the oracle's logit of the GPU's token is among its top 16 and
  within twice the largest measured error of the winner);
* group boundaries and KV counts exact (one KV entry per consumed group).
"""
import json
import os

import numpy as np
import pytest

import synth
from synth.configs import WORKLOADS
from tests.gpu_util import TOL, config_for, run_gpu

pytestmark = pytest.mark.gpu

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


@pytest.mark.parametrize("name", ["c3_8b_bf16", "c2_1b_bf16"])
def test_full_depth_against_oracle_goldens(torch_cuda, name):
    from paper_2505_20438_amd import ham
    g = json.load(open(os.path.join(HERE, f"golden_{name}.json")))
    w = WORKLOADS[name]
    s = w.shape
    assert (g["seed_weights"], g["seed_prompt"], g["seed_sched"], g["prompt_len"]) == \
        (w.seed_weights, w.seed_prompt, w.seed_sched, w.prompt_len)
    steps = g["macro_steps"]
    prompts = synth.prompt_ids(w.seed_prompt, 1, w.prompt_len, s.vocab)
    sched = synth.group_schedule(w.seed_sched, 1, steps + 1, s.max_group)
    rt = ham.HamRuntime(config_for(s, 1, w.prompt_len, w.max_new), w.seed_weights)
    res = run_gpu(rt, prompts, [w.max_new], steps, sched, teacher=[g["groups"]], debug_steps=steps + 1)
    tol = TOL[s.dtype]
    li = np.array(g["logit_idx"])
    hi = np.array(g["hidden_idx"])
    worst = {"logits": 0.0, "hidden": 0.0, "stop": 0.0}
    ties = exact = 0
    decs = {(d["step"], d["k"]): d for d in g["decisions"]}
    assert len(res.own[0]) == len(g["groups"])
    for step, toks in enumerate(res.own[0]):
        assert len(toks) == len(g["groups"][step]), step          # group boundaries exact
        for k, t in enumerate(toks):
            d = decs[(step, k)]
            lg = res.logits[(0, step, k)]
            top_id = np.array([p[0] for p in d["top"]])
            top_v = np.array([p[1] for p in d["top"]])
            e_l = max(float(np.max(np.abs(lg[li] - np.array(d["logits"])))),
                      float(np.max(np.abs(lg[top_id] - top_v))))
            e_h = float(np.max(np.abs(res.hidden[(0, step, k)][hi] - np.array(d["hidden"]))))
            e_s = abs(res.stop[(0, step, k)] - d["stop_logit"])
            worst = {"logits": max(worst["logits"], e_l), "hidden": max(worst["hidden"], e_h),
                     "stop": max(worst["stop"], e_s)}
            assert e_l <= tol and e_h <= tol and e_s <= tol, (step, k, e_l, e_h, e_s)
            if t == d["token"]:
                exact += 1
                continue
            assert t in top_id, (step, k, t, d["token"])
            gap = top_v[0] - top_v[list(top_id).index(t)]
            assert gap <= 2 * e_l, (step, k, t, d["token"], gap, e_l)
            ties += 1
    st = res.stats[0]
    assert st["kv_len"] == g["kv_len"] and st["gen_slots"] == g["gen_slots"] == steps
    assert st["tokens"] == g["tokens"] and st["groups"] == len(g["groups"]) and st["device_error"] == 0
    print(name, "decisions", exact + ties, "near ties", ties, "max errors", worst, flush=True)
    assert ties <= 1
