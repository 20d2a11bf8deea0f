"""Full-sequence prefill over fused inputs equals the incremental macro-steps,
on the GPU through the C ABI (the smashed KV cache holds one entry per base
input, Sec. 3.1; a fused input sits at its group's last position, Sec. 3.2).

The oracle records the base inputs of a generation: the prompt tokens'
embeddings at 0..P-1, then each macro-step's fused vector at its position.
``ham_prefill_embeds`` runs one causal forward over all of them.  Its KV cache,
its decision at the last position and the macro-step after it must match the
incremental GPU run (teacher-forced with the oracle's groups) and the oracle.

Marked ``gpu``: needs an MI355X and ``libham.so`` built in-tree.
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleHam
from synth.configs import BF16
from tests.gpu_util import SMALL16, TOL, check_decision, config_for, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(1e-30, float(np.max(np.abs(b)))))


@pytest.mark.parametrize("dtype", [0, BF16])
def test_prefill_embeds_equals_incremental(torch_cuda, dtype):
    import torch
    from paper_2505_20438_amd import ham
    shp = dataclasses.replace(SMALL16, dtype=dtype)
    tol = TOL[dtype]
    B, P, S, seed = 2, 40, 20, 91          # S macro-steps recorded, then one more
    prompts = synth.prompt_ids(92, B, P, shp.vocab)
    sched = synth.group_schedule(93, B, S + 2, 4)
    om = OracleHam(shp, seed)
    orcs, recs, orc_caches = [], [], []
    for b in range(B):
        rec = []
        orcs.append(om.generate(prompts[b], 0, S + 1, forced=lambda st, b=b: int(sched[b, st]), record=True,
                                inputs=rec))
        recs.append(rec)
        orc_caches.append(om.last_caches)
    T = P + S
    X = np.stack([np.concatenate([x for x, _ in r])[:T] for r in recs]).astype(np.float32)
    pos = np.stack([np.concatenate([p for _, p in r])[:T] for r in recs]).astype(np.int32)
    assert X.shape == (B, T, shp.d_model)
    assert np.all(np.diff(pos, axis=1) >= 1) and np.any(np.diff(pos, axis=1) > 1)   # fused inputs skip positions
    assert not np.array_equal(pos[0], pos[1])                                       # ragged across the batch
    teacher = [o.groups for o in orcs]
    dev = torch.device("cuda:0")

    # incremental: prefill + S + 1 macro-steps
    rt = ham.HamRuntime(config_for(shp, B, P, S + 1), seed)
    inc = run_gpu(rt, prompts, [0] * B, S + 1, sched, teacher=teacher, debug_steps=S + 2)
    inc_kv = [rt.kv_cache(l, T + 1) for l in range(shp.n_layers)]

    # full-sequence prefill over the first T inputs, then the last macro-step
    V, d = shp.vocab, shp.d_model
    dbg = torch.zeros(4 * B * (V + d + 1), dtype=torch.float32, device=dev)
    ham.ham_set_debug(rt.handle, dbg)
    tch = np.zeros((B, 4), dtype=np.int32)
    for b in range(B):
        tch[b, :len(teacher[b][S])] = teacher[b][S]
    rt.prefill_embeds(torch.from_numpy(X).to(dev), torch.from_numpy(pos).to(dev), [0] * B,
                      torch.from_numpy(np.ascontiguousarray(sched[:, S]).astype(np.int32)).to(dev),
                      torch.from_numpy(tch).to(dev))
    torch.cuda.synchronize()
    lg_full = dbg[:4 * B * V].view(4, B, V).cpu().numpy().copy()
    own_full = rt.out_tokens[:B].cpu().numpy().copy()
    lens_full = rt.out_lens[:B].cpu().numpy().copy()
    full_kv = [rt.kv_cache(l, T) for l in range(shp.n_layers)]
    st = rt.kv_stats()
    for b in range(B):
        assert st[b]["kv_len"] == T and st[b]["device_error"] == 0
        assert lens_full[b] == len(teacher[b][S])

    for l in range(shp.n_layers):
        for which in range(2):   # K, V
            g_full = full_kv[l][which].cpu().numpy().astype(np.float64)
            g_inc = inc_kv[l][which][:, :, :T].cpu().numpy().astype(np.float64)
            assert _rel(g_full, g_inc) <= tol, (l, which, _rel(g_full, g_inc))
            for b in range(B):
                o = np.transpose(orc_caches[b][l][which][:T], (1, 0, 2))   # [Hkv][T][hd]
                assert _rel(g_full[b], o) <= tol, (l, which, b)

    # the decision at the last input equals the last recorded macro-step's (step S)
    for b in range(B):
        decs = {(dd.step, dd.k): dd for dd in orcs[b].decisions}
        for k in range(lens_full[b]):
            assert np.max(np.abs(lg_full[k, b] - inc.logits[(b, S, k)])) <= tol, (b, k)
            check_decision(decs[(S, k)], int(own_full[b, k]), lg_full[k, b], tol)

    # one macro-step after the full prefill continues exactly like the incremental run
    for b in range(B):
        tch[b] = 0
        tch[b, :len(teacher[b][S + 1])] = teacher[b][S + 1]
    rt.macro_step(torch.from_numpy(np.ascontiguousarray(sched[:, S + 1]).astype(np.int32)).to(dev),
                  torch.from_numpy(tch).to(dev))
    torch.cuda.synchronize()
    lg_next = dbg[:4 * B * V].view(4, B, V).cpu().numpy().copy()
    lens_next = rt.out_lens[:B].cpu().numpy()
    ham.ham_set_debug(rt.handle, None)
    st = rt.kv_stats()
    for b in range(B):
        assert st[b]["kv_len"] == T + 1 and st[b]["device_error"] == 0
        assert lens_next[b] == len(teacher[b][S + 1])
        for k in range(lens_next[b]):
            assert np.max(np.abs(lg_next[k, b] - inc.logits[(b, S + 1, k)])) <= tol, (b, k)
    for l in range(shp.n_layers):
        for which in range(2):
            g = rt.kv_cache(l, T + 1)[which][:, :, T].cpu().numpy().astype(np.float64)
            ref = inc_kv[l][which][:, :, T].cpu().numpy().astype(np.float64)
            assert _rel(g, ref) <= tol, (l, which)
