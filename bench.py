#!/usr/bin/env python3
"""Benchmark of the HAMburger macro-step decode loop on one MI355X.

One step = one whole generation of the workload: prefill (timed separately and
excluded from the decode rate) then macro-steps until every sequence has spent
its output-token budget.  Inputs (weights, prompts, group-length schedule) are
seeded and resident in HBM before timing starts.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2_1b_bf16]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from synth.configs import BF16, STOP_FORCED, STOP_FORCED_TOKEN, WORKLOADS, Workload  # noqa: E402

METRIC = "output tokens/s at 1 GPU; KV entries per output token; decode HBM GB/s"
HBM_PEAK_GBS = 8000.0
PROF_NAMES = ["qkv", "o_proj", "gate_up", "down", "micro_gemm", "embed_gemm", "lm_head_k0", "lm_head_micro",
              "attn_decode"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_gate_up_c2_1b_bf16.txt")
GEMM_SOURCE = os.path.join(ROOT, "paper_2505_20438_amd", "csrc", "kernels_gemm.hip")


def gate_up_kernel(w: Workload) -> str:
    """Profiler name of the base-layer gate/up kernel at this workload.

    Batches whose normalised rows fit the staged prologue (rows * d_model <= 4096)
    run the staged GEMM (X built in LDS; template: element type, 16-column tiles
    per workgroup, epilogue 3 = SwiGLU, tag 0 = base layer, X source 1 = RMSNorm);
    larger batches the plain skinny GEMM after a separate RMSNorm kernel.
    """
    s = w.shape
    elem = "unsigned short" if s.dtype == BF16 else "float"
    tn = 2 if (2 * s.ffn_dim) // 32 >= 512 else 1
    if w.batch <= 8 and w.batch * s.d_model <= 4096:
        return f"k_gemm_staged<{elem}, {tn}, 3, 0, 1>"
    mt = 1 if w.batch <= 16 else (2 if w.batch <= 32 else 4)
    return f"k_gemm_skinny<{elem}, {mt}, {tn}, 3, 0>"


def measured_traffic(w: Workload, kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter summary, or None
    when the summary is for another kernel or workload, or the GEMM source changed."""
    import hashlib
    try:
        fields = dict(l.split("=", 1) for l in open(TRAFFIC_FILE).read().split("\n") if "=" in l and not l.startswith("#"))
        src = hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    if fields.get("kernel") != kernel or fields.get("workload") != w.name or fields.get("source_sha256") != src:
        return None
    return float(fields["fetch_bytes_per_launch"]) + float(fields["write_bytes_per_launch"])


def group_lengths(sched: np.ndarray, budget: int) -> list:
    """Realised group sizes of one sequence: the forced length, cut by the budget."""
    out, emitted, s = [], 0, 0
    while emitted < budget:
        n = min(int(sched[s]), budget - emitted)
        out.append(n)
        emitted += n
        s += 1
    return out


def algorithmic_bytes(w: Workload, lens: list, max_steps: int = 0, token_variant: bool = False) -> float:
    """Bytes the decode loop must move (closed form over the realised schedule).

    Per macro-step s (consuming group s-1, emitting group s), while any sequence
    runs: all base-layer weights and the LM head once; the embedder weights if a
    consumed group has more than one token; for every micro step some sequence
    still needs, the micro-decoder weights and the LM head again; per running
    sequence the K and V of every visible slot, plus the new slot written.
    With ``token_variant`` a group of n < max_group tokens (not cut by the
    budget) takes one more micro step: the decision taken as the reserved id.
    """
    s = w.shape
    es = 2 if s.dtype == BF16 else 4
    d, H, Hk, hd, F, V = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim, s.vocab
    layer = (2 * d * H * hd + 2 * d * Hk * hd + 3 * d * F) * es
    W_base, W_micro = s.n_layers * layer, s.micro_layers * layer
    W_lm = (V + 1) * d * es
    W_emb = 5 * d * d * es
    kv_slot = s.n_layers * 2 * Hk * hd * es
    steps = max(len(l) for l in lens) - 1
    if max_steps > 0:
        steps = min(steps, max_steps)
    total = 0.0
    for st in range(1, steps + 1):
        run = [b for b in range(len(lens)) if st < len(lens[b])]
        if not run:
            break
        total += W_base + W_lm
        if any(lens[b][st - 1] > 1 for b in run):
            total += W_emb
        def steps_of(b):
            n = lens[b][st]
            cut = st == len(lens[b]) - 1 and sum(lens[b]) == w.max_new  # the budget ends this group
            return n if (token_variant and n < s.max_group and not cut) else n - 1
        micro = max(steps_of(b) for b in run)
        total += micro * (W_micro + W_lm)
        for b in run:
            kv_len = w.prompt_len + st
            total += kv_len * kv_slot + kv_slot
    return total


def cpu_baseline(w: Workload, sample_steps: int) -> dict:
    """The float64 oracle on this host's cores over the first macro-steps of one sequence."""
    from oracle import OracleHam
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    om = OracleHam(w.shape, w.seed_weights)
    prompt = synth.prompt_ids(w.seed_prompt, 1, w.prompt_len, w.shape.vocab)[0]
    sched = synth.group_schedule(w.seed_sched, 1, sample_steps + 2, w.shape.max_group)[0]
    timing = {}
    res = om.generate(prompt, w.max_new, sample_steps, forced=lambda st: int(sched[st]), timing=timing)
    tokens = res.tokens - len(res.groups[0])   # tokens emitted by the timed macro-steps
    return {"value": tokens / timing["decode_s"], "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{w.name}: sequence 0, prompt {w.prompt_len}, first {sample_steps} macro-steps "
                      f"({tokens} tokens, {timing['decode_s']:.1f} s of decode; prefill {timing['prefill_s']:.1f} s "
                      f"excluded), float64 numpy, {platform.processor() or platform.machine()}"}


def _config(w: Workload, **over):
    from paper_2505_20438_amd import ham
    s = w.shape
    kw = dict(n_layers=s.n_layers, d_model=s.d_model, n_heads=s.n_heads, n_kv_heads=s.n_kv_heads,
              head_dim=s.head_dim, ffn_dim=s.ffn_dim, vocab=s.vocab, micro_layers=s.micro_layers,
              max_group=s.max_group, stop_mode=s.stop_mode, stop_id=s.stop_id, dtype=s.dtype,
              max_batch=w.batch, max_prompt=w.prompt_len, max_steps=w.max_new)
    kw.update(over)
    return ham.make_config(**kw)


def base_comparator(w: Workload, prompts, warmup: int, steps: int) -> dict:
    """The same weights decoding one token per forward (max group 1: no embedder
    fusion, no micro steps, one KV entry per token) on the same kernels."""
    import torch
    from paper_2505_20438_amd import ham
    rt = ham.HamRuntime(_config(w, max_group=1), w.seed_weights, "cuda:0")
    B = w.batch
    ones = torch.ones((w.max_new + 1, B), dtype=torch.int32, device=prompts.device)
    times = []
    for i in range(warmup + steps):
        rt.prefill(prompts, [w.max_new] * B, ones[0])
        e1, e2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e1.record(rt.stream)
        for st in range(1, w.max_new):
            rt.macro_step(ones[st])
        e2.record(rt.stream)
        torch.cuda.synchronize()
        if i >= warmup:
            times.append(e1.elapsed_time(e2))
    stats = rt.kv_stats()
    assert all(st["tokens"] == w.max_new and st["gen_slots"] == w.max_new - 1 for st in stats), stats
    ms = float(np.median(times))
    del rt
    torch.cuda.empty_cache()
    return {"value": B * w.max_new / (ms / 1000.0), "unit": "tokens/s", "ms_per_run": ms,
            "kv_entries_per_output_token": (w.max_new - 1) / float(w.max_new),
            "what": "same weights and kernels, max group 1: plain one-token-per-forward decoding"}


def token_cost_run(w: Workload, prompts, sched, lens, n_steps: int, warmup: int, steps: int) -> dict:
    """The same forced schedule with the reserved-token variant's control flow
    (Sec. 4.4): a group shorter than the cap ends on one more micro step, whose
    decision is discarded.  Emits the same tokens; measures that step's cost."""
    import torch
    from paper_2505_20438_amd import ham
    rt = ham.HamRuntime(_config(w, stop_mode=ham.HAM_STOP_FORCED_TOKEN), w.seed_weights, "cuda:0")
    B = w.batch
    times = []
    for i in range(warmup + steps):
        rt.prefill(prompts, [w.max_new] * B, sched[0])
        e1, e2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e1.record(rt.stream)
        for st in range(1, n_steps + 1):
            rt.macro_step(sched[st])
        e2.record(rt.stream)
        torch.cuda.synchronize()
        if i >= warmup:
            times.append(e1.elapsed_time(e2))
    stats = rt.kv_stats()
    assert all(st["tokens"] == w.max_new and st["device_error"] == 0 for st in stats), stats
    ms = float(np.median(times))
    nbytes = algorithmic_bytes(w, lens, n_steps, token_variant=True)
    del rt
    torch.cuda.empty_cache()
    return {"value": B * w.max_new / (ms / 1000.0), "unit": "tokens/s", "ms_per_run": ms,
            "algorithmic_bytes_per_run": nbytes, "decode_hbm_gbs": (nbytes / 1e9) / (ms / 1000.0),
            "what": "same schedule and kernels, reserved-token control flow: one more micro step per short group"}


def head_mode_run(w: Workload, prompts, conf: float) -> dict:
    """Model-driven groups: the stop head's logit against ln((1-c)/c).  The
    number of macro-steps is found by an untimed run, then one run is timed."""
    import torch
    from paper_2505_20438_amd import ham
    rt = ham.HamRuntime(_config(w, stop_mode=ham.HAM_STOP_HEAD, stop_conf=conf), w.seed_weights, "cuda:0")
    B = w.batch
    rt.prefill(prompts, [w.max_new] * B)
    n = 0
    while not all(st["done"] for st in rt.kv_stats()):
        if n >= w.max_new:  # every macro-step emits at least one token of an unfinished sequence
            raise RuntimeError("HEAD-mode decode did not spend its budget")
        rt.macro_step()
        n += 1
    rt.prefill(prompts, [w.max_new] * B)
    e1, e2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e1.record(rt.stream)
    for _ in range(n):
        rt.macro_step()
    e2.record(rt.stream)
    torch.cuda.synchronize()
    stats = rt.kv_stats()
    tokens = sum(st["tokens"] for st in stats)
    groups = sum(st["groups"] for st in stats)
    ms = e1.elapsed_time(e2)
    del rt
    torch.cuda.empty_cache()
    return {"confidence": conf, "value": tokens / (ms / 1000.0), "unit": "tokens/s", "macro_steps": n,
            "mean_group": tokens / float(groups),
            "kv_entries_per_output_token": sum(st["gen_slots"] for st in stats) / float(tokens)}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="c2_1b_bf16", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-steps", type=int, default=3, help="macro-steps of the oracle sample (0 = skip)")
    ap.add_argument("--max-macro-steps", type=int, default=0,
                    help="stop each run after this many macro-steps (profiler passes only; 0 = whole workload)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="first run one plain device-to-device copy of this size (HBM counter calibration)")
    ap.add_argument("--base", choices=("auto", "on", "off"), default="auto",
                    help="also time the same model decoding one token per forward (groups of one; auto: prompts <= 4096)")
    ap.add_argument("--token-cost", action="store_true",
                    help="also time the same schedule with the reserved-token stop variant (one more micro step per short group)")
    ap.add_argument("--graph", choices=("on", "off"), default="on",
                    help="replay each macro-step's launches from a HIP graph (on) or launch them on the stream")
    ap.add_argument("--head-sweep", default="",
                    help="comma-separated confidences: also time the model-driven stop head (HEAD mode) at each")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for {args.gpus}); the batch would shard "
              "data-parallel over sequences with no exchange, which is not built.", file=sys.stderr)
        return 2

    import torch
    from paper_2505_20438_amd import ham

    w = WORKLOADS[args.workload]
    s = w.shape
    # unbudgeted workloads (the tiny fp32 model: TOKEN stop, 128 macro-steps) run
    # a fixed number of macro-steps; their tokens are counted on the device
    unbudgeted = w.max_new <= 0
    forced_mode = s.stop_mode in (STOP_FORCED, STOP_FORCED_TOKEN)
    B, P = w.batch, w.prompt_len
    dev = torch.device("cuda:0")
    cfg = ham.make_config(n_layers=s.n_layers, d_model=s.d_model, n_heads=s.n_heads, n_kv_heads=s.n_kv_heads,
                          head_dim=s.head_dim, ffn_dim=s.ffn_dim, vocab=s.vocab, micro_layers=s.micro_layers,
                          max_group=s.max_group, stop_mode=s.stop_mode, stop_id=s.stop_id, dtype=s.dtype,
                          max_batch=B, max_prompt=P, max_steps=w.macro_steps if unbudgeted else w.max_new)
    rt = ham.HamRuntime(cfg, w.seed_weights, "cuda:0")
    rt.set_graph(args.graph == "on")
    stream = rt.stream
    prompts = torch.from_numpy(synth.prompt_ids(w.seed_prompt, B, P, s.vocab)).to(dev)
    n_sched = (w.macro_steps if unbudgeted else w.max_new) + 1
    sched_np = synth.group_schedule(w.seed_sched, B, n_sched, s.max_group)
    sched_dev = torch.from_numpy(np.ascontiguousarray(sched_np.T)).to(dev)   # [step][B], resident
    sched = [sched_dev[st] if forced_mode else None for st in range(n_sched)]
    budgets = [max(w.max_new, 0)] * B
    if unbudgeted:
        lens = None
        n_steps = w.macro_steps
        rt.prefill(prompts, budgets, sched[0])   # the prefill's group, excluded from the decode tokens
        first = int(rt.out_lens[:B].sum())
        for st in range(1, n_steps + 1):
            rt.macro_step(sched[st])
        tokens_per_run = sum(x["tokens"] for x in rt.kv_stats()) - first
    else:
        lens = [group_lengths(sched_np[b], w.max_new) for b in range(B)]
        n_steps = max(len(l) for l in lens) - 1
        tokens_per_run = sum(budgets)
    if not unbudgeted and args.max_macro_steps > 0 and args.max_macro_steps < n_steps:
        n_steps = args.max_macro_steps   # profiler passes: the JSON line is then not a benchmark result
        tokens_per_run = sum(sum(l[:n_steps + 1]) for l in lens)
    if args.copy_calibration_mb > 0:
        src = torch.ones(args.copy_calibration_mb << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def one_run(profile: bool = False):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record(stream)
        rt.prefill(prompts, budgets, sched[0])
        e1.record(stream)
        if profile:
            ham.load_library().ham_profile(rt.handle, 1)
        # the host's enqueue time is taken from an idle GPU: otherwise the loop
        # would also wait for the prefill through the full launch queue
        torch.cuda.synchronize()
        h0 = time.perf_counter()
        for st in range(1, n_steps + 1):
            rt.macro_step(sched[st])
        host_enqueue.append(time.perf_counter() - h0)
        e2.record(stream)
        if profile:
            ham.load_library().ham_profile(rt.handle, 0)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1), e1.elapsed_time(e2)

    host_enqueue = []
    for _ in range(args.warmup):
        one_run()
    torch.cuda.synchronize()
    decode_ms, prefill_ms = [], []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        pf, dc = one_run()
        prefill_ms.append(pf)
        decode_ms.append(dc)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dec_med = float(np.median(decode_ms))
    stats = rt.kv_stats()
    truncated = (not unbudgeted) and n_steps < max(len(l) for l in lens) - 1
    assert all((unbudgeted or truncated or st["tokens"] == w.max_new) and st["device_error"] == 0
               for st in stats), stats
    if unbudgeted:
        assert sum(st["tokens"] for st in stats) - first == tokens_per_run   # deterministic across runs
    gen_slots = sum(st["gen_slots"] for st in stats)
    dec_ms = dec_med
    value = tokens_per_run / (dec_ms / 1000.0)
    # the tiny model's 20 MB stay in the caches: no HBM bytes model for it
    alg_bytes = None if unbudgeted else algorithmic_bytes(w, lens, n_steps)

    # per-kernel-class timing: one more run with HIP events attached to the
    # dispatch of every launch of the classes (same launch configuration, outside
    # the timed runs above; the events mark each kernel's own start and end)
    one_run(profile=True)
    prof = (ham.HamProfT * ham.HAM_PROF_KINDS)()
    ham.check(ham.load_library().ham_profile_read(rt.handle, prof, ham.HAM_PROF_KINDS))
    kernels = {}
    for i, name in enumerate(PROF_NAMES):
        p = prof[i]
        if p.launches:
            kernels[name] = {"launches": p.launches, "avg_us": 1000.0 * p.ms / p.launches,
                             "bytes_per_launch": p.bytes / p.launches,
                             "gbs": (p.bytes / 1e9) / (p.ms / 1000.0) if p.ms > 0 else None}
    dom = max(("qkv", "o_proj", "gate_up", "down", "lm_head_k0", "attn_decode"),
              key=lambda k: kernels.get(k, {}).get("avg_us", 0) * kernels.get(k, {}).get("launches", 0))
    kd = kernels[dom]
    roofline = {"bound": "hbm", "achieved": kd["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": kd["gbs"] / HBM_PEAK_GBS, "traffic": None, "kernel": dom,
                "bytes_per_launch": kd["bytes_per_launch"], "avg_us": kd["avg_us"]}
    if unbudgeted:
        roofline["note"] = "the tiny model stays in the on-chip caches: launch-latency bound, HBM fraction not meaningful"
    if dom == "gate_up":
        roofline["kernel_name"] = gate_up_kernel(w)
        roofline["traffic"] = measured_traffic(w, roofline["kernel_name"])

    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": dec_ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if s.dtype == BF16 else "f32", "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "prompt_len": P, "output_tokens_per_seq": w.max_new,
                   "layers": s.n_layers, "d_model": s.d_model, "micro_layers": s.micro_layers,
                   "schedule": ("forced geometric group lengths p=1/2, cap 4" if forced_mode
                                else f"model-driven stops (mode {s.stop_mode}, stop id {s.stop_id})"),
                   "macro_steps": n_steps},
        "kv_entries_per_output_token": gen_slots / float(sum(st["tokens"] for st in stats)),
        "kv_entries_per_token_incl_prompt": (B * P + gen_slots) / float(B * P + sum(st["tokens"] for st in stats)),
        "decode_hbm_gbs": None if alg_bytes is None else (alg_bytes / 1e9) / (dec_ms / 1000.0),
        "decode_hbm_frac": None if alg_bytes is None else (alg_bytes / 1e9) / (dec_ms / 1000.0) / HBM_PEAK_GBS,
        "algorithmic_bytes_per_run": alg_bytes,
        "prefill_ms": float(np.mean(prefill_ms)),
        "us_per_macro_step": 1000.0 * dec_ms / n_steps,
        "host_enqueue_us_per_macro_step": 1e6 * float(np.median(host_enqueue[args.warmup:args.warmup + args.steps])) / n_steps,
        "graph": args.graph == "on",
        "wall_s_timed": wall,
        "roofline": roofline,
        "kernels": kernels,
    }
    out["decode_ms_runs"] = [float(x) for x in decode_ms]
    del rt
    torch.cuda.empty_cache()
    if not unbudgeted and (args.base == "on" or (args.base == "auto" and P <= 4096 and not truncated)):
        out["base_comparator"] = base_comparator(w, prompts, args.warmup, args.steps)
        out["speedup_vs_base"] = value / out["base_comparator"]["value"]
    if args.token_cost and not truncated and not unbudgeted:
        out["token_variant"] = token_cost_run(w, prompts, sched, lens, n_steps, args.warmup, args.steps)
        out["token_variant"]["slowdown_vs_stop_head"] = value / out["token_variant"]["value"]
        out["token_variant"]["bytes_ratio_vs_stop_head"] = out["token_variant"]["algorithmic_bytes_per_run"] / alg_bytes
    if args.head_sweep:
        out["head_sweep"] = [head_mode_run(w, prompts, float(c)) for c in args.head_sweep.split(",")]
    if args.cpu_steps > 0:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_steps)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
