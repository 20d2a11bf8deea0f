"""GPU parity of the decode loop against the oracle, through the C ABI.

Marked ``gpu``: needs an MI355X and ``libham.so`` built in-tree.
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleHam
from synth.configs import BF16, SHAPE_1B, STOP_FORCED, STOP_FORCED_TOKEN, STOP_HEAD, STOP_TOKEN, TINY, WORKLOADS
from tests.gpu_util import SMALL16, TOL, check_decision, config_for, oracle_groups_for, run_gpu, teacher_forced

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


def _runtime(shape, seed, batch, prompt, steps):
    from paper_2505_20438_amd import ham
    return ham.HamRuntime(config_for(shape, batch, prompt, steps), seed)


def test_weights_match_seeded_generator(torch_cuda):
    # the device initialiser and the shared input generator implement one definition
    shp = TINY
    rt = _runtime(shp, 1001, 1, 64, 8)
    ids = [synth.T_EMBED, synth.T_RELPOS, synth.T_AQ, synth.T_AV, synth.T_ALIN, synth.T_LMHEAD, synth.T_STOP,
           synth.layer_tensor_id(0, synth.L_WQ), synth.layer_tensor_id(1, synth.L_WG),
           synth.layer_tensor_id(1, synth.L_WU), synth.layer_tensor_id(2, synth.L_WD)]
    for tid in ids:
        got = rt.tensor(tid).cpu().numpy()
        want = synth.normal_tensor(1001, tid, got.size, bf16=False).reshape(got.shape)
        # float64 libm differences can move a value by one fp32 ulp at a rounding boundary
        mism = np.mean(got != want)
        assert mism < 1e-5 and np.max(np.abs(got - want)) <= 1e-8, (tid, mism)


def test_weights_match_generator_bf16_1b_sample(torch_cuda):
    import torch
    shp = SHAPE_1B
    rt = _runtime(shp, 1002, 1, 64, 4)
    rng = np.random.default_rng(0)
    for tid in (synth.T_EMBED, synth.T_LMHEAD, synth.layer_tensor_id(7, synth.L_WU),
                synth.layer_tensor_id(17, synth.L_WD)):
        t = rt.tensor(tid)
        rows, cols = t.shape
        idx = rng.integers(0, rows * cols, 20000)
        got = t.reshape(-1)[torch.from_numpy(idx).to(t.device)].cpu().numpy().view(np.uint16)
        want = synth.normal_elements(1002, tid, idx, bf16=True)
        assert np.mean(got != want) < 1e-4, tid


@pytest.mark.parametrize("mode", ["c1", "head", "forced", "forced_token"])
def test_tiny_fp32_free_running_exact(torch_cuda, mode):
    # configuration 1: fp32, TOKEN stop id 1023, 64-token prompt, 128 macro-steps, no budget;
    # plus HEAD (c = 0.5) and FORCED variants on the same weights
    w = WORKLOADS["c1_tiny_f32"]
    shp = w.shape
    sched = None
    if mode == "head":
        shp = dataclasses.replace(shp, stop_mode=STOP_HEAD, stop_conf=0.5)
    elif mode in ("forced", "forced_token"):
        shp = dataclasses.replace(shp, stop_mode=STOP_FORCED if mode == "forced" else STOP_FORCED_TOKEN)
        sched = synth.group_schedule(w.seed_sched, 1, w.macro_steps + 1, 4)
    prompts = synth.prompt_ids(w.seed_prompt, 1, w.prompt_len, shp.vocab)
    om = OracleHam(shp, w.seed_weights)
    orc = oracle_groups_for(om, prompts, [0], w.macro_steps, sched, record=True)[0]
    rt = _runtime(shp, w.seed_weights, 1, w.prompt_len, w.macro_steps)
    res = run_gpu(rt, prompts, [0], w.macro_steps, sched, debug_steps=6)
    # logits and normed hidden states of the first steps within the fp32 tolerance
    decs = {(d.step, d.k): d for d in orc.decisions}
    for (b, step, k), lg in res.logits.items():
        d = decs[(step, k)]
        assert np.max(np.abs(lg - d.logits)) <= TOL[0], (step, k)
        assert np.max(np.abs(res.hidden[(b, step, k)] - d.h)) <= TOL[0], (step, k)
        assert abs(res.stop[(b, step, k)] - d.stop_logit) <= TOL[0], (step, k)
    assert res.groups[0] == orc.groups
    st = res.stats[0]
    assert st["kv_len"] == orc.kv_len and st["gen_slots"] == w.macro_steps
    assert st["tokens"] == orc.tokens and st["groups"] == len(orc.groups)
    assert st["device_error"] == 0
    assert sum(st["len_hist"]) == len(orc.groups)




def _teacher_forced(om, shp, prompts, budgets, steps, sched, seed, debug_steps):
    return teacher_forced(om, shp, prompts, budgets, steps, sched, seed, debug_steps)


def test_small_bf16_teacher_forced_ragged_batch(torch_cuda):
    shp = SMALL16
    B, P, steps = 3, 100, 24
    prompts = synth.prompt_ids(77, B, P, shp.vocab)
    sched = synth.group_schedule(78, B, steps + 1, 4)
    budgets = [0, 17, 40]
    om = OracleHam(shp, 76)
    exact, ties = _teacher_forced(om, shp, prompts, budgets, steps, sched, 76, debug_steps=steps + 1)
    assert ties <= max(1, exact // 50)


def test_small_fp32_teacher_forced_ragged_batch(torch_cuda):
    # the same shape in fp32: any error beyond rounding would show up here
    shp = dataclasses.replace(SMALL16, dtype=0)
    B, P, steps = 3, 100, 24
    prompts = synth.prompt_ids(77, B, P, shp.vocab)
    sched = synth.group_schedule(78, B, steps + 1, 4)
    om = OracleHam(shp, 76)
    exact, ties = _teacher_forced(om, shp, prompts, [0, 17, 40], steps, sched, 76, debug_steps=steps + 1)
    assert ties == 0


def test_small_fp32_long_prompt_teacher_forced(torch_cuda):
    # prompt chunks above 256 rows: the prefill runs the 128x128-tile GEMM and
    # several 64-row attention chunks, in fp32 (no rounding to hide behind)
    shp = dataclasses.replace(SMALL16, dtype=0)
    B, P, steps = 2, 300, 6
    prompts = synth.prompt_ids(79, B, P, shp.vocab)
    sched = synth.group_schedule(80, B, steps + 1, 4)
    om = OracleHam(shp, 81)
    exact, ties = _teacher_forced(om, shp, prompts, [0, 9], steps, sched, 81, debug_steps=steps + 1)
    assert ties == 0


def test_1b_bf16_teacher_forced_prefix(torch_cuda):
    # configuration 2 shape and prompt length; the first macro-steps against the oracle
    w = WORKLOADS["c2_1b_bf16"]
    shp = w.shape
    steps = 4
    prompts = synth.prompt_ids(w.seed_prompt, 1, w.prompt_len, shp.vocab)
    sched = synth.group_schedule(w.seed_sched, 1, steps + 1, 4)
    om = OracleHam(shp, w.seed_weights)
    exact, ties = _teacher_forced(om, shp, prompts, [w.max_new], steps, sched, w.seed_weights,
                                  debug_steps=steps + 1)
    assert ties <= 1


def _free_running_compare(orc, res, tol, tau):
    """Walk the free-running GPU groups against the oracle's until the first
    divergence, which must be a near tie the measured error explains (of the
    token argmax, or of the stop logit against tau).  Returns exact decisions."""
    decs = {(d.step, d.k): d for d in orc.decisions}
    exact = 0
    for step, (g_gpu, g_orc) in enumerate(zip(res.groups[0], orc.groups)):
        for k in range(min(len(g_gpu), len(g_orc))):
            d = decs[(step, k)]
            lg = res.logits[(0, step, k)]
            assert np.max(np.abs(lg - d.logits)) <= tol, (step, k)
            assert np.max(np.abs(res.hidden[(0, step, k)] - d.h)) <= tol, (step, k)
            if g_gpu[k] != g_orc[k]:
                check_decision(d, g_gpu[k], lg, tol)
                return exact
            exact += 1
        if len(g_gpu) != len(g_orc):  # the stop test at the shorter group's last token differed
            k = min(len(g_gpu), len(g_orc)) - 1
            d = decs[(step, k)]
            err = abs(res.stop[(0, step, k)] - d.stop_logit)
            assert err <= tol and abs(d.stop_logit - tau) <= 2 * err, (step, k, d.stop_logit, err)
            return exact
    assert len(res.groups[0]) == len(orc.groups)
    return exact


def test_1b_dims_head_mode_free_running(torch_cuda):
    # model-driven stopping (HEAD mode, c = 0.5) at the 1B layer shape and full vocabulary,
    # two base layers and one micro layer; free-running against the free-running oracle
    shp = dataclasses.replace(SHAPE_1B, n_layers=2, micro_layers=1, stop_mode=STOP_HEAD, stop_conf=0.5)
    P, steps = 64, 10
    prompts = synth.prompt_ids(4010, 1, P, shp.vocab)
    om = OracleHam(shp, 6010)
    orc = oracle_groups_for(om, prompts, [0], steps, None, record=True)[0]
    rt = _runtime(shp, 6010, 1, P, steps)
    res = run_gpu(rt, prompts, [0], steps, debug_steps=steps + 1)
    exact = _free_running_compare(orc, res, TOL[BF16], 0.0)
    lens = [len(g) for g in orc.groups]
    print("oracle group lengths", lens, "exact decisions", exact)
    assert exact >= 10
    assert len(set(lens)) > 1  # the stop head actually varies the group length here


def test_head_c1_equals_one_token_decoding(torch_cuda):
    # c = 1 stops after every token: the loop reduces to plain decoding, and must give the
    # same tokens as the same weights configured with max group 1 (the base comparator)
    import torch
    w = WORKLOADS["c2_1b_bf16"]
    shp_h = dataclasses.replace(w.shape, n_layers=4, stop_mode=STOP_HEAD, stop_conf=1.0)
    shp_1 = dataclasses.replace(w.shape, n_layers=4, max_group=1)
    P, steps = 128, 24
    prompts = synth.prompt_ids(4011, 2, P, shp_h.vocab)
    res_h = run_gpu(_runtime(shp_h, 6011, 2, P, steps), prompts, [0, 0], steps)
    sched = np.ones((2, steps + 1), dtype=np.int64)
    res_1 = run_gpu(_runtime(shp_1, 6011, 2, P, steps), prompts, [0, 0], steps, sched)
    for b in range(2):
        assert all(len(g) == 1 for g in res_h.groups[b])
        assert res_h.groups[b] == res_1.groups[b]
        assert res_h.stats[b]["kv_len"] == res_1.stats[b]["kv_len"] == P + steps


@pytest.mark.parametrize("layers,dtype,B", [((1, 3), 0, 1), ((1, 2, 3, 5, 7, 8), BF16, 3)])
def test_configured_context_layers_teacher_forced(torch_cuda, layers, dtype, B):
    # a non-default set of base layers conditions the micro decoder (Sec. 3.3, Fig. 2a):
    # C context rows at local positions 0..C-1, here C = 2 (fp32, one sequence) and C = 6
    shp = dataclasses.replace(SMALL16, n_layers=4 if max(layers) <= 4 else 8, ctx_layer_set=layers, dtype=dtype)
    P, steps = 40, 8
    prompts = synth.prompt_ids(4020 + B, B, P, shp.vocab)
    sched = synth.group_schedule(5020 + B, B, steps + 1, 4)
    om = OracleHam(shp, 6020 + B)
    exact, ties = teacher_forced(om, shp, prompts, [0] * B, steps, sched, 6020 + B, debug_steps=steps + 1)
    assert ties == 0 if dtype == 0 else ties <= 1


def test_max_group_one_against_oracle_plain_decoding(torch_cuda):
    # the base comparator (max group 1): no embedder fusion, no micro steps, one KV entry
    # per token, i.e. the base model's own computation (Sec. 3.4; Sec. 3.7 "Minimal
    # Overhead"), at the 1B layer shape and full vocabulary against the oracle's group-size-1
    # run: teacher-forced on two sequences, then free-running on one
    w = WORKLOADS["c2_1b_bf16"]
    shp = dataclasses.replace(w.shape, n_layers=4, max_group=1)
    B, P, steps = 2, 128, 24
    prompts = synth.prompt_ids(4012, B, P, shp.vocab)
    sched = np.ones((B, steps + 1), dtype=np.int32)
    om = OracleHam(shp, 6012)
    exact, ties = teacher_forced(om, shp, prompts, [0] * B, steps, sched, 6012, debug_steps=steps + 1)
    assert ties <= 1 and exact >= 48
    orc = om.generate(prompts[0], 0, steps, forced=lambda st: 1, record=True)
    rt = _runtime(shp, 6012, 1, P, steps)
    res = run_gpu(rt, prompts[:1], [0], steps, sched[:1], debug_steps=steps + 1)
    free_exact = _free_running_compare(orc, res, TOL[BF16], 0.0)
    st = res.stats[0]
    print("free-running exact decisions", free_exact, flush=True)
    assert all(len(g) == 1 for g in res.groups[0])
    assert st["gen_slots"] == st["tokens"] - 1 == steps and st["kv_len"] == P + steps
    assert free_exact >= 10
