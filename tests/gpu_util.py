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
        max_prompt=prompt, max_steps=steps, ctx_layers=shape.ctx_layer_set)


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


def act_rows(torch, x, dtype):
    """fp32 rows -> the library's activation layout (bf16 hi/lo planes for bf16)."""
    if dtype == 0:
        return x.contiguous()
    hi = x.to(torch.bfloat16)
    lo = (x - hi.float()).to(torch.bfloat16)
    return torch.cat([hi, lo], dim=1).contiguous()


def from_act(torch, buf, width, dtype):
    """The library's activation layout -> fp32 rows."""
    if dtype == 0:
        return buf.float()
    return buf[:, :width].float() + buf[:, width:].float()


def tiled_v(torch, V):
    """V [R][Hkv][S][hd] -> the cache's 32-slot tiles, d-major inside a tile: [R][Hkv][S/32][hd][32]."""
    R, Hk, S, hd = V.shape
    return V.reshape(R, Hk, S // 32, 32, hd).transpose(3, 4).contiguous()


def untiled_v(torch, VT):
    R, Hk, nt, hd, _ = VT.shape
    return VT.transpose(3, 4).reshape(R, Hk, nt * 32, hd)


def synthetic_groups(seed: int, sched_row, steps: int, vocab: int) -> List[List[int]]:
    """Teacher groups for a row the oracle does not follow: the forced lengths,
    seeded uniform token ids (any valid input will do for such a row)."""
    ids = synth.prompt_ids(seed, 1, 4 * (steps + 1), vocab)[0]
    return [[int(t) for t in ids[4 * st: 4 * st + int(sched_row[st])]] for st in range(steps + 1)]


def teacher_forced(om, shp, prompts, budgets, steps, sched, seed, debug_steps, check_rows=None, cap_steps=None):
    """Teacher-forced parity: the oracle runs free on ``check_rows`` (all rows by
    default); the GPU is fed the oracle's groups on those rows (and seeded
    synthetic groups of the forced lengths, unbudgeted, on the others), and every
    captured decision of a checked row is compared: logits and normed hidden
    within the tolerance, tokens exact or an explained near tie, group boundaries
    and KV counts exact.  ``cap_steps`` sets the model's macro-step capacity
    (default ``steps``), which fixes the decode-attention launch shape.
    Returns (exact decisions, accepted near ties)."""
    from paper_2505_20438_amd import ham
    B = prompts.shape[0]
    rows = list(range(B)) if check_rows is None else list(check_rows)
    orc_of = {}
    for b in rows:
        forced = (lambda st, b=b: int(sched[b, st]))
        orc_of[b] = om.generate(prompts[b], int(budgets[b]), steps, forced=forced, record=True)
    teacher = []
    for b in range(B):
        if b in orc_of:
            teacher.append(orc_of[b].groups)
        else:
            assert budgets[b] == 0, "rows the oracle does not follow run unbudgeted"
            teacher.append(synthetic_groups(9000 + b, sched[b], steps, shp.vocab))
    cfg = config_for(shp, B, prompts.shape[1], steps if cap_steps is None else cap_steps)
    rt = ham.HamRuntime(cfg, seed)
    res = run_gpu(rt, prompts, budgets, steps, sched, teacher=teacher, debug_steps=debug_steps)
    tol = TOL[shp.dtype]
    ties = exact = 0
    errs = []
    for b, o in orc_of.items():
        decs = {(d.step, d.k): d for d in o.decisions}
        for (bb, step, k), lg in res.logits.items():
            if bb == b:
                d = decs[(step, k)]
                errs.append((float(np.max(np.abs(lg - d.logits))),
                             float(np.max(np.abs(res.hidden[(b, step, k)] - d.h))),
                             float(np.sqrt(np.mean((res.hidden[(b, step, k)] - d.h) ** 2))), b, step, k))
    e = np.array([x[:3] for x in errs])
    print("decisions", len(errs), "logit err max/mean", e[:, 0].max(), e[:, 0].mean(),
          "hidden max/mean", e[:, 1].max(), e[:, 1].mean(), "hidden rms mean", e[:, 2].mean(), flush=True)
    for x in sorted(errs, key=lambda x: -x[1])[:8]:
        print("  worst", x)
    for b, o in orc_of.items():
        decs = {(d.step, d.k): d for d in o.decisions}
        assert len(res.own[b]) == len(o.groups)
        for step, toks in enumerate(res.own[b]):
            assert len(toks) == len(o.groups[step])          # group boundaries exact
            for k, t in enumerate(toks):
                lg = res.logits.get((b, step, k))
                if lg is not None:
                    d = decs[(step, k)]
                    assert np.max(np.abs(lg - d.logits)) <= tol, (b, step, k)
                    assert np.max(np.abs(res.hidden[(b, step, k)] - d.h)) <= tol, (b, step, k)
                    assert abs(res.stop[(b, step, k)] - d.stop_logit) <= tol, (b, step, k)
                r = check_decision(decs[(step, k)], t, lg, tol)
                ties += r == "near_tie"
                exact += r == "exact"
        st = res.stats[b]
        assert st["kv_len"] == o.kv_len and st["gen_slots"] == o.gen_slots and st["tokens"] == o.tokens
        assert st["groups"] == len(o.groups) and st["device_error"] == 0
    for b in range(B):
        assert res.stats[b]["device_error"] == 0, b
        if b not in orc_of:   # unfollowed rows: one KV entry per consumed group all the same
            assert res.stats[b]["gen_slots"] == steps and res.stats[b]["kv_len"] == prompts.shape[1] + steps, b
    return exact, ties
