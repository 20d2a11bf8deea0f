"""Pins of the oracle's whole decode loop.

* against an independent full-recompute reading written with torch primitives;
* group size forced to 1 reduces to textbook greedy decoding (one KV per token);
* one full causal forward over the recorded inputs equals the incremental run;
* KV slots count the groups, not the tokens; budgets and the group cap hold.
"""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import OracleHam
from synth.configs import BF16, STOP_FORCED, STOP_FORCED_TOKEN, STOP_HEAD, STOP_TOKEN, TINY
from tests.ref_torch import RefHam, plain_greedy

SMALL = dataclasses.replace(TINY, vocab=96, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96,
                            n_layers=3, micro_layers=2)


def _prompt(seed, P, V):
    return synth.prompt_ids(seed, 1, P, V)[0]


def _check_counts(res, P, budget=0):
    assert res.kv_len == P + res.gen_slots
    assert res.gen_slots == len(res.groups) - 1          # one KV entry per consumed group
    assert res.tokens == sum(len(g) for g in res.groups)
    assert all(1 <= len(g) <= 4 for g in res.groups)
    if budget:
        assert res.tokens == budget


@pytest.mark.parametrize("mode,conf,dtype", [
    (STOP_HEAD, 0.5, 0), (STOP_HEAD, 0.6, 0), (STOP_TOKEN, 0.5, 0), (STOP_FORCED, 0.5, 0),
    (STOP_HEAD, 0.5, BF16), (STOP_FORCED, 0.5, BF16)])
def test_oracle_matches_full_recompute_reference(mode, conf, dtype):
    shp = dataclasses.replace(SMALL, stop_mode=mode, stop_conf=conf, dtype=dtype, stop_id=7)
    om, ref = OracleHam(shp, 31), RefHam(shp, 31)
    prompt = _prompt(41, 12, shp.vocab)
    sched = synth.group_schedule(51, 1, 64, 4)[0]
    forced = (lambda st: int(sched[st])) if mode == STOP_FORCED else None
    res = om.generate(prompt, 0, 10, forced=forced, record=True)
    rec = []
    assert res.groups == ref.generate(prompt, 0, 10, forced=forced, record=rec)
    assert len(rec) == len(res.decisions)
    for d, (t, st, lg) in zip(res.decisions, rec):
        assert d.token == t
        assert abs(d.stop_logit - st) <= 1e-9 * max(1.0, abs(st))
        assert np.allclose(d.logits, lg, rtol=1e-5, atol=1e-6)  # oracle keeps a float32 copy
    _check_counts(res, 12)
    if mode == STOP_FORCED:
        assert [len(g) for g in res.groups] == [int(x) for x in sched[:11]]


def test_token_mode_never_emits_stop_id_after_first():
    shp = dataclasses.replace(SMALL, stop_mode=STOP_TOKEN)
    om = OracleHam(shp, 32)
    prompt = _prompt(42, 10, shp.vocab)
    first = om.generate(prompt, 0, 12)
    later = [t for g in first.groups for t in g[1:]]
    common = int(np.bincount(later).argmax())        # make the reserved id a frequent one
    shp2 = dataclasses.replace(shp, stop_id=common)
    om2, ref2 = OracleHam(shp2, 32), RefHam(shp2, 32)
    res = om2.generate(prompt, 0, 12)
    assert res.groups == ref2.generate(prompt, 0, 12)
    assert any(len(g) < 4 for g in res.groups)         # the stop path was exercised
    assert all(common not in g[1:] for g in res.groups)


@pytest.mark.parametrize("budget", [1, 7, 23])
def test_budget_is_exact_and_truncates_last_group(budget):
    shp = dataclasses.replace(SMALL, stop_mode=STOP_FORCED)
    om = OracleHam(shp, 33)
    sched = synth.group_schedule(52, 1, 64, 4)[0]
    res = om.generate(_prompt(43, 9, shp.vocab), budget, 0, forced=lambda st: int(sched[st]))
    _check_counts(res, 9, budget)
    lens = [len(g) for g in res.groups]
    assert lens[:-1] == [int(x) for x in sched[:len(lens) - 1]]
    assert lens[-1] == min(int(sched[len(lens) - 1]), budget - sum(lens[:-1]))


@pytest.mark.parametrize("how", ["forced1", "head_c1"])
def test_group_size_one_reduces_to_plain_greedy(how):
    # north star check: with groups of one token the macro-step is ordinary decoding
    mode = STOP_FORCED if how == "forced1" else STOP_HEAD
    shp = dataclasses.replace(SMALL, stop_mode=mode, stop_conf=1.0)
    om = OracleHam(shp, 34)
    prompt = _prompt(44, 11, shp.vocab)
    res = om.generate(prompt, 0, 15, forced=lambda st: 1)
    toks = [g[0] for g in res.groups]
    assert all(len(g) == 1 for g in res.groups)
    assert res.gen_slots == res.tokens - 1 and res.kv_len == 11 + 15
    assert toks == plain_greedy(RefHam(shp, 34), prompt, 16)


def test_plain_greedy_on_config1_shape():
    shp = dataclasses.replace(TINY, stop_mode=STOP_FORCED)
    om = OracleHam(shp, 1001)
    prompt = _prompt(2001, 64, shp.vocab)[:24]
    res = om.generate(prompt, 0, 6, forced=lambda st: 1)
    assert [g[0] for g in res.groups] == plain_greedy(RefHam(shp, 1001), prompt, 7)


@pytest.mark.parametrize("dtype", [0, BF16])
def test_full_prefill_equals_incremental_macro_steps(dtype):
    # north star check: one causal forward over [prompt, z_1..z_S] at the recorded positions
    # reproduces every KV slot and the last hidden state of the incremental run
    shp = dataclasses.replace(SMALL, stop_mode=STOP_HEAD, dtype=dtype)
    om = OracleHam(shp, 35)
    inputs = []
    res = om.generate(_prompt(45, 13, shp.vocab), 0, 9, inputs=inputs)
    inc_caches = om.last_caches
    X = np.concatenate([x for x, _ in inputs])
    pos = np.concatenate([p for _, p in inputs])
    assert X.shape[0] == res.kv_len
    assert np.all(np.diff(pos) >= 1)
    caches = om.new_caches(shp.n_layers)
    Xo, _ = om.forward_rows(om.layers[:shp.n_layers], X, pos, caches)
    tol = 1e-10 if dtype == 0 else 0.0
    for (k1, v1), (k2, v2) in zip(caches, inc_caches):
        if dtype == 0:
            assert np.allclose(k1, k2, rtol=tol, atol=1e-13) and np.allclose(v1, v2, rtol=tol, atol=1e-13)
        else:  # bf16-stored slots: equal up to a rare one-ulp flip at a rounding boundary
            assert np.mean(k1 != k2) < 1e-3 and np.abs(k1 - k2).max() <= 2 ** -7 * np.abs(k2).max()
    t_full, _, _, _ = om.decide(Xo[-1], om.g_final, False)
    assert t_full == res.groups[-1][0]


def test_positions_advance_by_group_size():
    shp = dataclasses.replace(SMALL, stop_mode=STOP_FORCED)
    om = OracleHam(shp, 36)
    inputs = []
    sched = synth.group_schedule(53, 1, 64, 4)[0]
    res = om.generate(_prompt(46, 8, shp.vocab), 0, 12, forced=lambda st: int(sched[st]), inputs=inputs)
    pos = np.concatenate([p for _, p in inputs])
    assert list(pos[:8]) == list(range(8))
    assert list(np.diff(pos[7:])) == [len(g) for g in res.groups[:-1]]


def test_forced_token_costs_one_extra_micro_step_per_short_group():
    # the reserved-token variant (Sec. 4.4) on forced lengths: the same groups as the
    # stop-head control flow, plus one discarded decision for every group shorter than
    # the cap (a group of one needs a micro step it would otherwise skip)
    sched = synth.group_schedule(57, 1, 40, 4)[0]
    prompt = _prompt(58, 12, SMALL.vocab)
    res = {}
    for mode in (STOP_FORCED, STOP_FORCED_TOKEN):
        om = OracleHam(dataclasses.replace(SMALL, stop_mode=mode), 37)
        res[mode] = om.generate(prompt, 0, 30, forced=lambda st: int(sched[st]))
    head, tok = res[STOP_FORCED], res[STOP_FORCED_TOKEN]
    assert tok.groups == head.groups and tok.kv_len == head.kv_len
    assert [len(g) for g in head.groups] == [int(x) for x in sched[:31]]
    extra = sum(1 for g in head.groups if len(g) < 4)
    assert extra > 5
    assert len(tok.decisions) == len(head.decisions) + extra
    for g, n_dec in zip(head.groups, np.bincount([d.step for d in tok.decisions])):
        assert n_dec == len(g) + (1 if len(g) < 4 else 0)


@pytest.mark.parametrize("layers", [(1,), (2, 3), (1, 3)])
def test_explicit_context_layers_match_reference_and_matter(layers):
    # the micro decoder's context rows come from the configured base layers (Sec. 3.3,
    # Fig. 2a): both readings follow the set, and a different set changes the decisions
    shp = dataclasses.replace(SMALL, stop_mode=STOP_FORCED, ctx_layer_set=layers)
    om, ref = OracleHam(shp, 33), RefHam(shp, 33)
    prompt = _prompt(43, 10, shp.vocab)
    sched = synth.group_schedule(53, 1, 64, 4)[0]
    forced = lambda st: int(sched[st])  # noqa: E731
    res = om.generate(prompt, 0, 6, forced=forced, record=True)
    rec = []
    assert res.groups == ref.generate(prompt, 0, 6, forced=forced, record=rec)
    for d, (t, st, lg) in zip(res.decisions, rec):
        assert np.allclose(d.logits, lg, rtol=1e-5, atol=1e-6)
    default = OracleHam(dataclasses.replace(shp, ctx_layer_set=()), 33).generate(prompt, 0, 6, forced=forced,
                                                                                 record=True)
    micro = [(a.logits, b.logits) for a, b in zip(res.decisions, default.decisions) if a.k >= 1]
    assert micro and all(not np.allclose(a, b) for a, b in micro)
    # decisions from the base model (k = 0) do not depend on the context set
    base = [(a.logits, b.logits) for a, b in zip(res.decisions, default.decisions) if a.k == 0]
    assert all(np.array_equal(a, b) for a, b in base[:1])
