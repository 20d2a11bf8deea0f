#!/usr/bin/env python3
"""Write the oracle's expected decisions for the full-depth workload models.

Calls only the oracle (``oracle/``) and the seeded input generators
(``synth/``).  For each named workload it runs the float64 oracle on sequence 0
of the workload's seeded prompt, with the workload's seeded forced group
lengths (reading 11 of the decode loop: a geometric law, p = 1/2, capped at 4),
for a few macro-steps after the prefill, and stores per token decision (Sec. 3.3
micro index k, Sec. 3.4 for k = 0):

* the emitted token (greedy argmax, Sec. 4.1) and the stop-head logit;
* the oracle's 16 largest logits with their ids (the near-tie rule needs the
  oracle's logit of any token the GPU might pick instead);
* the logits at a fixed seeded sample of ids and the normed hidden state at a
  fixed seeded sample of coordinates (element-by-element comparison);
* the emitted groups (fed back to the GPU as teacher tokens) and the KV counts
  (one entry per consumed group, Sec. 3.1).

The full model at 32 layers is too slow for the oracle inside a GPU test, so
its values are computed once here and committed as ``golden_<workload>.json``.

    python tests/golden/make_goldens.py c3_8b_bf16 c2_1b_bf16
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import OracleHam  # noqa: E402
from synth.configs import WORKLOADS  # noqa: E402

MACRO_STEPS = {"c2_1b_bf16": 24, "c3_8b_bf16": 7}
N_LOGITS, N_HIDDEN, TOP = 192, 96, 16


def _f(x) -> float:
    """The float32 value, written with the fewest digits that read back to it."""
    return float(str(np.float32(x)))


def make(name: str) -> dict:
    w = WORKLOADS[name]
    s = w.shape
    steps = MACRO_STEPS[name]
    t0 = time.time()
    om = OracleHam(s, w.seed_weights, cache_f64=False)
    t1 = time.time()
    prompt = synth.prompt_ids(w.seed_prompt, 1, w.prompt_len, s.vocab)[0]
    sched = synth.group_schedule(w.seed_sched, 1, steps + 2, s.max_group)[0]
    res = om.generate(prompt, w.max_new, steps, forced=lambda st: int(sched[st]), record=True)
    t2 = time.time()
    rng = np.random.default_rng(12345)
    logit_idx = np.unique(np.concatenate([[0, s.vocab - 1], rng.integers(0, s.vocab, N_LOGITS)]))
    hidden_idx = np.unique(np.concatenate([[0, s.d_model - 1], rng.integers(0, s.d_model, N_HIDDEN)]))
    decisions = []
    for d in res.decisions:
        lg = d.logits.astype(np.float64)
        top = np.argsort(-lg, kind="stable")[:TOP]
        decisions.append({
            "step": d.step, "k": d.k, "token": d.token, "stop_logit": _f(d.stop_logit),
            "top": [[int(i), _f(lg[i])] for i in top],
            "logits": [_f(lg[i]) for i in logit_idx],
            "hidden": [_f(d.h[i]) for i in hidden_idx],
        })
    return {
        "workload": name,
        "what": "float64 oracle, sequence 0, forced group lengths, first macro-steps after prefill",
        "generator": "tests/golden/make_goldens.py",
        "paper": "Sec. 3.1-3.4 (macro-step, embedder, micro-step decoder, stop head), Sec. 4.1 (greedy)",
        "seed_weights": w.seed_weights, "seed_prompt": w.seed_prompt, "seed_sched": w.seed_sched,
        "prompt_len": w.prompt_len, "max_new": w.max_new, "macro_steps": steps,
        "groups": res.groups, "kv_len": res.kv_len, "gen_slots": res.gen_slots, "tokens": res.tokens,
        "logit_idx": [int(i) for i in logit_idx], "hidden_idx": [int(i) for i in hidden_idx],
        "decisions": decisions,
        "oracle_seconds": {"weights": round(t1 - t0, 1), "generate": round(t2 - t1, 1)},
    }


def main() -> int:
    names = sys.argv[1:] or sorted(MACRO_STEPS)
    for name in names:
        g = make(name)
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"golden_{name}.json")
        with open(path, "w") as f:
            json.dump(g, f, separators=(",", ":"))
            f.write("\n")
        print(name, "->", path, g["oracle_seconds"], flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
