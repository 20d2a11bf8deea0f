"""Helpers of the GPU parity tests: run the library through its C ABI (ctypes
binding) and compare with the oracle under the token-parity rule.

Token rule: a GPU decision must equal the oracle's, except at a near tie that
the measured logit error explains: with err = max |logits_gpu - logits_oracle|
on that decision (and err within the dtype's tolerance), a different token t' is
accepted iff logit_oracle[t_oracle] - logit_oracle[t'] <= 2 * err.  Group
boundaries and KV counts must match exactly.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

import synth
from synth.configs import BF16, STOP_FORCED, HamShape

TOL = {0: 1e-4, BF16: 2e-2}

# a small bf16 model of several tiles per GEMM dimension, FORCED stops
SMALL16 = HamShape(n_layers=4, d_model=512, n_heads=8, n_kv_heads=2, head_dim=64, ffn_dim=1024, vocab=4096,
                   micro_layers=2, max_group=4, stop_mode=STOP_FORCED, stop_id=1023, dtype=BF16)


def config_for(shape: HamShape, batch: int, prompt: int, steps: int):
    from paper_2505_20438_amd import ham
    return ham.make_config(
        n_layers=shape.n_layers, d_model=shape.d_model, n_heads=shape.n_heads, n_kv_heads=shape.n_kv_heads,
        head_dim=shape.head_dim, ffn_dim=shape.ffn_dim, vocab=shape.vocab, micro_layers=shape.micro_layers,
        max_group=shape.max_group, stop_mode=shape.stop_mode, stop_id=shape.stop_id, stop_conf=shape.stop_conf,
        rope_theta=shape.rope_theta, norm_eps=shape.norm_eps, dtype=shape.dtype, max_batch=batch,
        max_prompt=prompt, max_steps=steps)


@dataclasses.dataclass
class GpuRun:
    groups: List[List[List[int]]]          # [b][step] -> emitted group
    own: List[List[List[int]]]             # [b][step] -> the model's own argmax per position
    stats: List[dict]
    logits: Dict[tuple, np.ndarray]        # (b, step, k) -> float32 logits (debug capture)
    hidden: Dict[tuple, np.ndarray]
    stop: Dict[tuple, float]


def run_gpu(rt, prompts: np.ndarray, budgets, steps: int, sched: Optional[np.ndarray] = None,
            teacher: Optional[List[List[List[int]]]] = None, debug_steps: int = 0) -> GpuRun:
    """Prefill + ``steps`` macro-steps (stops early once every budget is spent).

    ``sched`` [B][steps+1] forced lengths; ``teacher[b][step]`` the group to feed back.
    """
    import torch
    from paper_2505_20438_amd import ham
    dev = rt.device
    B, P = prompts.shape
    cfg = rt.cfg
    V, d = cfg.vocab, cfg.d_model
    dbg = None
    if debug_steps:
        dbg = torch.zeros(4 * cfg.max_batch * (V + d + 1), dtype=torch.float32, device=dev)
        ham.ham_set_debug(rt.handle, dbg)
    prompt_t = torch.from_numpy(prompts.astype(np.int32)).to(dev)
    groups = [[] for _ in range(B)]
    own = [[] for _ in range(B)]
    logits, hidden, stop = {}, {}, {}

    def forced(step):
        if sched is None:
            return None
        return torch.from_numpy(np.ascontiguousarray(sched[:, step]).astype(np.int32)).to(dev)

    def teach(step):
        if teacher is None:
            return None
        t = np.zeros((B, 4), dtype=np.int32)
        for b in range(B):
            g = teacher[b][step] if step < len(teacher[b]) else []
            t[b, :len(g)] = g
        return torch.from_numpy(t).to(dev)

    for step in range(steps + 1):
        if step == 0:
            rt.prefill(prompt_t, budgets, forced(0), teach(0))
        else:
            rt.macro_step(forced(step), teach(step))
        toks = rt.out_tokens[:B].cpu().numpy()
        lens = rt.out_lens[:B].cpu().numpy()
        if dbg is not None and step < debug_steps:
            D = dbg.cpu().numpy()
            Bm = cfg.max_batch
            lg = D[:4 * Bm * V].reshape(4, Bm, V)
            hd_ = D[4 * Bm * V: 4 * Bm * (V + d)].reshape(4, Bm, d)
            st = D[4 * Bm * (V + d):].reshape(4, Bm)
        for b in range(B):
            n = int(lens[b])
            if n == 0:
                continue
            tb = teacher[b][step] if teacher is not None else None
            groups[b].append(list(tb) if tb is not None else [int(t) for t in toks[b, :n]])
            own[b].append([int(t) for t in toks[b, :4] if t >= 0])
            if dbg is not None and step < debug_steps:
                for k in range(len(own[b][-1])):
                    logits[(b, step, k)] = lg[k, b].copy()
                    hidden[(b, step, k)] = hd_[k, b].copy()
                    stop[(b, step, k)] = float(st[k, b])
        if step > 0 and all(int(l) == 0 for l in lens):
            break
    if dbg is not None:
        ham.ham_set_debug(rt.handle, None)
    return GpuRun(groups, own, rt.kv_stats(), logits, hidden, stop)


def check_decision(orc_dec, gpu_tok: int, gpu_logits: Optional[np.ndarray], tol: float) -> str:
    """'exact', 'near_tie' (accepted) or raises AssertionError."""
    if gpu_tok == orc_dec.token:
        return "exact"
    assert gpu_logits is not None and orc_dec.logits is not None, "token mismatch without logits to explain it"
    err = float(np.max(np.abs(gpu_logits.astype(np.float64) - orc_dec.logits.astype(np.float64))))
    gap = float(orc_dec.logits[orc_dec.token]) - float(orc_dec.logits[gpu_tok])
    assert err <= tol, f"logit error {err} above tolerance {tol}"
    assert gap <= 2 * err, f"token {gpu_tok} vs oracle {orc_dec.token}: gap {gap} not explained by error {err}"
    return "near_tie"


def oracle_groups_for(om, prompts, budgets, steps, sched=None, record=False):
    out = []
    for b in range(prompts.shape[0]):
        forced = (lambda st, b=b: int(sched[b, st])) if sched is not None else None
        out.append(om.generate(prompts[b], int(budgets[b]), steps, forced=forced, record=record))
    return out
