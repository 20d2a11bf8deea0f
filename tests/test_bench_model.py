"""The benchmark's byte model (algorithmic HBM bytes of the decode loop) on the CPU.

Degenerate schedules reduce the model to closed forms written out here term by
term: groups of one token never fuse inputs or run micro steps (plain decoding,
one KV entry per token); groups of the cap fuse every input after the first and
run every micro step.  The seeded workload schedules are checked against the
expected bytes per macro-step and per token that follow from the group-length
distribution (p = 1/2 before the cap of 4): weights and LM head once, the
embedder when a consumed group has more than one token, E[micro steps] times
(micro weights + LM head), and the K and V of every visible slot plus the new one.
"""
import dataclasses

import numpy as np
import pytest

import bench
import synth
from synth.configs import BF16, SHAPE_1B, WORKLOADS, Workload


def _sizes(s):
    es = 2 if s.dtype == BF16 else 4
    layer = (2 * s.d_model * s.n_heads * s.head_dim + 2 * s.d_model * s.n_kv_heads * s.head_dim
             + 3 * s.d_model * s.ffn_dim) * es
    return dict(base=s.n_layers * layer, micro=s.micro_layers * layer, lm=(s.vocab + 1) * s.d_model * es,
                emb=5 * s.d_model ** 2 * es, slot=s.n_layers * 2 * s.n_kv_heads * s.head_dim * es)


def _workload(batch, prompt_len, max_new):
    return Workload("t", SHAPE_1B, batch, prompt_len, max_new, 0, 1, 2, 3)


def test_one_token_groups_are_plain_decoding():
    w = _workload(2, 10, 7)
    z = _sizes(w.shape)
    lens = [[1] * 7, [1] * 7]
    # macro-step st reads the prompt plus st generated slots and writes one
    expect = sum(z["base"] + z["lm"] + 2 * ((10 + st) * z["slot"] + z["slot"]) for st in range(1, 7))
    assert bench.algorithmic_bytes(w, lens) == pytest.approx(expect, rel=1e-12)


def test_full_groups_fuse_and_run_every_micro_step():
    w = _workload(1, 33, 16)
    z = _sizes(w.shape)
    lens = [[4, 4, 4, 4]]
    per = z["base"] + z["lm"] + z["emb"] + 3 * (z["micro"] + z["lm"])
    expect = sum(per + (33 + st) * z["slot"] + z["slot"] for st in range(1, 4))
    assert bench.algorithmic_bytes(w, lens) == pytest.approx(expect, rel=1e-12)


def test_ragged_batch_runs_the_longest_micro_loop_and_stops_finished_rows():
    w = _workload(2, 5, 6)
    z = _sizes(w.shape)
    lens = [[1, 1, 4], [2, 4]]          # sequence 1 is done after macro-step 1
    step1 = z["base"] + z["lm"] + z["emb"] + 3 * (z["micro"] + z["lm"]) + 2 * (6 * z["slot"] + z["slot"])
    step2 = z["base"] + z["lm"] + 3 * (z["micro"] + z["lm"]) + (7 * z["slot"] + z["slot"])
    assert bench.algorithmic_bytes(w, lens) == pytest.approx(step1 + step2, rel=1e-12)


def test_reserved_token_variant_adds_one_micro_step_per_short_group():
    w = _workload(1, 8, 20)
    z = _sizes(w.shape)
    lens = [[2] * 10]
    plain = bench.algorithmic_bytes(w, lens)
    variant = bench.algorithmic_bytes(w, lens, token_variant=True)
    # every consumed-and-emitted group of two takes one more micro step, except the
    # last one, which the budget cuts
    assert variant - plain == pytest.approx(8 * (z["micro"] + z["lm"]), rel=1e-12)


def test_group_lengths_cut_by_budget():
    assert bench.group_lengths(np.array([4, 3, 1, 4, 2]), 10) == [4, 3, 1, 2]
    assert bench.group_lengths(np.array([1, 1, 1]), 0) == []


@pytest.mark.parametrize("name", ["c2_1b_bf16", "c3_8b_bf16", "c4_8b_b32", "c5_8b_long"])
def test_seeded_schedules_match_the_expected_bytes(name):
    w = WORKLOADS[name]
    s = w.shape
    z = _sizes(s)
    B = w.batch
    sched = synth.group_schedule(w.seed_sched, B, w.max_new + 1, s.max_group)
    lens = [bench.group_lengths(sched[b], w.max_new) for b in range(B)]
    steps = max(len(l) for l in lens) - 1
    total = bench.algorithmic_bytes(w, lens)
    # expected value per macro-step under P(L = 1, 2, 3, 4) = 1/2, 1/4, 1/8, 1/8
    p_le = [0.5, 0.75, 0.875]
    e_micro = sum(1 - q ** B for q in p_le)
    p_fuse = 1 - 0.5 ** B
    mean_len = 1 * 0.5 + 2 * 0.25 + 3 * 0.125 + 4 * 0.125
    mean_kv = w.prompt_len + w.max_new / mean_len / 2
    expect_step = (z["base"] + z["lm"] + p_fuse * z["emb"] + e_micro * (z["micro"] + z["lm"])
                   + B * (mean_kv + 1) * z["slot"])
    assert total / steps == pytest.approx(expect_step, rel=0.05)
    expect_token = expect_step / (B * mean_len)
    assert total / (B * w.max_new) == pytest.approx(expect_token, rel=0.06)
    # one KV entry per group after the prefill's: about 1 / 1.875 per output token
    gen_slots = sum(len(l) - 1 for l in lens)
    assert gen_slots / (B * w.max_new) == pytest.approx(1 / mean_len, rel=0.06)


def test_micro_steps_needed_counts_the_longest_group_of_the_running_rows():
    w = _workload(2, 10, 6)
    lens = [[4, 1, 3, 2], [2, 4]]            # row 1 finishes after macro-step 1
    # step 1: groups 1 and 4 -> 3 micro steps; consumed 4 and 2 -> fused
    # step 2: row 0 only, group 3 -> 2; consumed 1 -> not fused
    # step 3: group 2 -> 1; consumed 3 -> fused
    assert bench.micro_steps_needed(w, lens, 3) == (6, 2)
    assert bench.micro_steps_needed(w, lens, 1) == (3, 1)


def test_cost_model_of_sec_3_7_closed_forms():
    # r = sum n C(S) / sum (C(S) + (n - 1) c): groups of one give r = 1 (the base model's
    # own computation, Sec. 3.7 "Minimal Overhead"); full groups give 4 C / (C + 3 c) per step
    w = _workload(1, 100, 12)
    z = _sizes(w.shape)
    assert bench.cost_model_speedup(w, [[1] * 13], 12) == pytest.approx(1.0, rel=1e-12)
    lens = [[4, 4, 4]]
    C = [z["base"] + z["lm"] + (100 + 1 + i) * z["slot"] for i in range(2)]
    c = z["micro"] + z["lm"]
    expect = sum(4 * x for x in C) / sum(x + 3 * c for x in C)
    assert bench.cost_model_speedup(w, lens, 2) == pytest.approx(expect, rel=1e-12)
    assert 1.0 < expect < 4.0
