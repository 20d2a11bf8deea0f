"""GPU checks at the 8B shapes and at the full sizes of the five workloads.

* 8B layer shapes (d 4096, head dim 128, ffn 14336, vocab 128256) at reduced
  depth, teacher-forced against the oracle: same kernels, same launch shapes as
  the full models, at a depth the oracle finishes in about a minute;
* batch 20 with ragged budgets: the batched tile paths (two row tiles, the
  LDS-tiled GEMM for the micro decoder's context rows) against the oracle;
* the decode attention kernel through its C-ABI entry point at the 32K-slot
  context of the long-context workload, against the oracle's attention;
* every workload at full size: exact token budgets, group lengths equal to the
  forced schedule, KV entries equal to the macro-steps run, no device error,
  bitwise-identical reruns.
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import OracleHam
from oracle.ham import attend
from synth.configs import BF16, SHAPE_8B, STOP_FORCED, WORKLOADS
from tests.gpu_util import TOL, check_decision, config_for, oracle_groups_for, run_gpu
from tests.test_gpu_parity import _teacher_forced

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


def _act_rows(torch, x, dtype):
    """fp32 rows -> the library's activation layout (bf16 hi/lo planes for bf16)."""
    if dtype == 0:
        return x.contiguous()
    hi = x.to(torch.bfloat16)
    lo = (x - hi.float()).to(torch.bfloat16)
    return torch.cat([hi, lo], dim=1).contiguous()


def _from_act(torch, buf, width, dtype):
    if dtype == 0:
        return buf.float()
    return buf[:, :width].float() + buf[:, width:].float()


@pytest.mark.parametrize("case", ["long_bf16", "short_bf16", "fp32"])
def test_decode_attention_op(torch_cuda, case):
    torch = torch_cuda
    from paper_2505_20438_amd import ham
    rng = np.random.default_rng(7)
    if case == "long_bf16":   # the long-context workload: 4 sequences near 33K slots, one finished
        dtype, H, Hk, hd, S = BF16, 32, 8, 128, 33792
        lens = [33314, 32769, 33792, 1000]
        enable = [1, 1, 1, 0]
    elif case == "short_bf16":
        dtype, H, Hk, hd, S = BF16, 32, 8, 64, 1088
        lens = [1, 31, 33, 785, 1088]
        enable = [1] * 5
    else:
        dtype, H, Hk, hd, S = 0, 4, 2, 64, 192
        lens = [1, 17, 130, 192]
        enable = [1] * 4
    R = len(lens)
    q = rng.standard_normal((R, H * hd)).astype(np.float32)
    K = rng.standard_normal((R, Hk, S, hd)).astype(np.float32)
    V = rng.standard_normal((R, Hk, S, hd)).astype(np.float32)
    tdt = torch.bfloat16 if dtype == BF16 else torch.float32
    dev = "cuda:0"
    Kt = torch.from_numpy(K).to(dev).to(tdt)
    Vt = torch.from_numpy(V).to(dev).to(tdt)
    # V in 32-slot tiles, d-major inside a tile: [R][Hk][S/32][hd][32]
    VTt = Vt.reshape(R, Hk, S // 32, 32, hd).transpose(3, 4).contiguous()
    Kf = Kt.float().cpu().numpy()       # the stored (rounded) values both sides use
    Vf = Vt.float().cpu().numpy()
    qt = _act_rows(torch, torch.from_numpy(q).to(dev), dtype)
    out = torch.zeros_like(qt)
    ws = torch.empty(ham.ham_op_attention_workspace_bytes(R, H, Hk, hd), dtype=torch.uint8, device=dev)
    lt = torch.tensor(lens, dtype=torch.int32, device=dev)
    et = torch.tensor(enable, dtype=torch.int32, device=dev)
    ham.ham_op_decode_attention(dtype, qt, Kt, VTt, lt, et, max(lens), out, ws,
                                torch.cuda.current_stream().cuda_stream, H, Hk, hd, S)
    torch.cuda.synchronize()
    got = _from_act(torch, out, H * hd, dtype).cpu().numpy().reshape(R, H, hd)
    for r in range(R):
        if not enable[r]:
            assert np.all(got[r] == 0)
            continue
        ref = attend(q[r].reshape(1, H, hd).astype(np.float64), Kf[r].transpose(1, 0, 2),
                     Vf[r].transpose(1, 0, 2), [lens[r]], Hk)[0]
        tol = 2e-3 if dtype == BF16 else 1e-5
        assert np.max(np.abs(got[r] - ref)) <= tol, (case, r, np.max(np.abs(got[r] - ref)))


def test_8b_shapes_reduced_depth_teacher_forced(torch_cuda):
    # every kernel at the 8B-shaped launch configuration (head dim 128, d 4096, ffn 14336,
    # vocab 128256), two base layers and one micro layer so the oracle stays fast
    shp = dataclasses.replace(SHAPE_8B, n_layers=2, micro_layers=1)
    B, P, steps = 1, 48, 3
    prompts = synth.prompt_ids(4003, B, P, shp.vocab)
    sched = synth.group_schedule(5003, B, steps + 1, 4)
    om = OracleHam(shp, 6003)
    exact, ties = _teacher_forced(om, shp, prompts, [0], steps, sched, 6003, debug_steps=steps + 1)
    assert ties <= 1


def test_8b_dims_long_prompt_split_attention_teacher_forced(torch_cuda):
    # head dim 128 with a prompt long enough for several decode-attention splits,
    # merged in the o-projection's prologue
    shp = dataclasses.replace(SHAPE_8B, n_layers=2, micro_layers=1, vocab=8192)
    B, P, steps = 1, 560, 4
    prompts = synth.prompt_ids(4006, B, P, shp.vocab)
    sched = synth.group_schedule(5006, B, steps + 1, 4)
    om = OracleHam(shp, 6006)
    exact, ties = _teacher_forced(om, shp, prompts, [0], steps, sched, 6006, debug_steps=steps + 1)
    assert ties <= 1


def test_batch20_ragged_8b_dims_teacher_forced(torch_cuda):
    # batch above 16 rows (two row tiles) and micro context rows above 64 (LDS-tiled GEMM)
    shp = dataclasses.replace(SHAPE_8B, n_layers=2, micro_layers=1, vocab=8192)
    B, P, steps = 20, 40, 4
    prompts = synth.prompt_ids(4004, B, P, shp.vocab)
    sched = synth.group_schedule(5004, B, steps + 1, 4)
    budgets = [0, 3, 7, 12] * 5
    om = OracleHam(shp, 6004, cache_f64=True)
    exact, ties = _teacher_forced(om, shp, prompts, budgets, steps, sched, 6004, debug_steps=steps + 1)
    assert ties <= max(1, exact // 50)


def test_batch32_one_workgroup_per_row_attention(torch_cuda):
    # 32 rows x 8 KV heads fill the GPU with one attention workgroup per (row, head):
    # the waves split each row's own cached blocks (rows of different lengths)
    shp = dataclasses.replace(SHAPE_8B, n_layers=2, micro_layers=1, vocab=8192)
    B, P, steps = 32, 100, 4
    prompts = synth.prompt_ids(4005, B, P, shp.vocab)
    sched = synth.group_schedule(5005, B, steps + 1, 4)
    budgets = [0, 2, 5, 9] * 8
    om = OracleHam(shp, 6005, cache_f64=True)
    exact, ties = _teacher_forced(om, shp, prompts, budgets, steps, sched, 6005, debug_steps=steps + 1)
    assert ties <= max(1, exact // 50)


def _expected_lengths(sched_row, budget):
    out, emitted, s = [], 0, 0
    while emitted < budget:
        n = min(int(sched_row[s]), budget - emitted)
        out.append(n)
        emitted += n
        s += 1
    return out


def _full_run(torch, name, repeat=1):
    from paper_2505_20438_amd import ham
    w = WORKLOADS[name]
    s = w.shape
    cfg = config_for(s, w.batch, w.prompt_len, w.max_new)
    rt = ham.HamRuntime(cfg, w.seed_weights)
    dev = rt.device
    prompts = torch.from_numpy(synth.prompt_ids(w.seed_prompt, w.batch, w.prompt_len, s.vocab)).to(dev)
    sched = synth.group_schedule(w.seed_sched, w.batch, w.max_new + 1, s.max_group)
    sched_t = torch.from_numpy(np.ascontiguousarray(sched.T)).to(dev)
    expect = [_expected_lengths(sched[b], w.max_new) for b in range(w.batch)]
    n_steps = max(len(e) for e in expect) - 1
    runs = []
    for _ in range(repeat):
        toks_steps, lens_steps = [], []
        rt.prefill(prompts, [w.max_new] * w.batch, sched_t[0])
        toks_steps.append(rt.out_tokens[:w.batch].clone())
        lens_steps.append(rt.out_lens[:w.batch].clone())
        for st in range(1, n_steps + 1):
            rt.macro_step(sched_t[st])
            toks_steps.append(rt.out_tokens[:w.batch].clone())
            lens_steps.append(rt.out_lens[:w.batch].clone())
        torch.cuda.synchronize()
        toks = torch.stack(toks_steps).cpu().numpy()    # [step][B][4]
        lens = torch.stack(lens_steps).cpu().numpy()    # [step][B]
        runs.append((toks, lens, rt.kv_stats()))
    return w, expect, runs


@pytest.mark.parametrize("name", ["c2_1b_bf16", "c3_8b_bf16", "c4_8b_b32", "c5_8b_long"])
def test_full_workload_counts_and_determinism(torch_cuda, name):
    torch = torch_cuda
    w, expect, runs = _full_run(torch, name, repeat=2 if name in ("c2_1b_bf16", "c4_8b_b32") else 1)
    toks, lens, stats = runs[0]
    for b in range(w.batch):
        got = [int(n) for n in lens[:, b] if n > 0]
        assert got == expect[b], (b, got[:10], expect[b][:10])          # group boundaries exact
        st = stats[b]
        assert st["tokens"] == w.max_new and st["done"] == 1
        assert st["gen_slots"] == len(expect[b]) - 1 == st["groups"] - 1   # one KV entry per consumed group
        assert st["kv_len"] == w.prompt_len + st["gen_slots"]
        assert st["device_error"] == 0
        assert sum(st["len_hist"]) == st["groups"]
        emitted = np.concatenate([toks[s, b, :lens[s, b]] for s in range(len(lens)) if lens[s, b] > 0])
        assert emitted.min() >= 0 and emitted.max() < w.shape.vocab
    total_tokens = sum(st["tokens"] for st in stats)
    total_slots = sum(st["gen_slots"] for st in stats)
    assert 0.45 < total_slots / total_tokens < 0.62     # about 1/1.875 under the capped geometric law
    if len(runs) > 1:
        assert np.array_equal(runs[0][0], runs[1][0]) and np.array_equal(runs[0][1], runs[1][1])


@pytest.mark.parametrize("name,steps", [("c5_8b_long", 6), ("c4_8b_b32", 6)])
def test_full_size_batch_rows_equal_the_sequence_alone(torch_cuda, name, steps):
    # A property that holds at any size: a sequence decoded inside the workload's batch
    # gives the decisions it gives alone (rows never mix; only the launch shapes, and so
    # the rounding, differ).  Sequence 0 of the long-context and batched workloads at full
    # size, the first macro-steps, teacher-forced with its own batch-1 groups: logits,
    # normed hidden states and stop logits within the bf16 tolerance, group boundaries
    # and KV counts exact; row 1 of the batch is checked the same way.
    from paper_2505_20438_amd import ham
    w = WORKLOADS[name]
    s = w.shape
    prompts = synth.prompt_ids(w.seed_prompt, w.batch, w.prompt_len, s.vocab)
    sched = synth.group_schedule(w.seed_sched, w.batch, steps + 1, s.max_group)
    tol = TOL[BF16]
    alone = {}
    for b in (0, 1):
        rt1 = ham.HamRuntime(config_for(s, 1, w.prompt_len, w.max_new), w.seed_weights)
        alone[b] = run_gpu(rt1, prompts[b:b + 1], [w.max_new], steps, sched[b:b + 1], debug_steps=steps + 1)
        del rt1
        torch_cuda.cuda.empty_cache()
    teacher = [alone[b].groups[0] if b in alone else alone[0].groups[0] for b in range(w.batch)]
    sched_t = sched.copy()
    for b in range(2, w.batch):   # other rows: row 0's groups, so every row has consistent lengths
        sched_t[b] = sched[0]
    rt = ham.HamRuntime(config_for(s, w.batch, w.prompt_len, w.max_new), w.seed_weights)
    res = run_gpu(rt, prompts, [w.max_new] * w.batch, steps, sched_t, teacher=teacher, debug_steps=steps + 1)
    worst = 0.0
    for b in (0, 1):
        one = alone[b]
        assert [len(g) for g in res.own[b]] == [len(g) for g in one.groups[0]], b
        for key, lg in one.logits.items():
            _, step, k = key
            bk = (b, step, k)
            e = max(float(np.max(np.abs(res.logits[bk] - lg))),
                    float(np.max(np.abs(res.hidden[bk] - one.hidden[key]))),
                    abs(res.stop[bk] - one.stop[key]))
            worst = max(worst, e)
            assert e <= tol, (name, b, step, k, e)
        assert res.stats[b]["kv_len"] == one.stats[0]["kv_len"] == w.prompt_len + steps
        assert res.stats[b]["device_error"] == 0
    print(name, "batch row vs alone: max difference", worst, flush=True)
