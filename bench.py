#!/usr/bin/env python3
"""Benchmark of the HAMburger macro-step decode loop on one MI355X.

One step = one whole generation of the workload's decode: every macro-step
until each sequence has spent its output-token budget.  The prompt is
prefilled once (timed on its own and excluded from the decode rate); the
decode state it leaves (smashed KV cache and per-sequence counters) is saved
and restored before every run, so each run decodes from the same prefilled
cache.  Inputs (weights, prompts, group-length schedule) are seeded and
resident in HBM before timing starts.  Prints one JSON line on stdout and one
progress line per run on stderr.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c5_8b_long]

The default workload is the largest that fits one GPU: the 8B-shaped model,
4 sequences of 32768 prompt tokens, 1024 output tokens each.
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
              "attn_decode", "norm"]
CSRC = os.path.join(ROOT, "paper_2505_20438_amd", "csrc")
# the sources each measured kernel class is compiled from (a committed counter
# summary applies only while these are unchanged)
CLASS_SOURCES = {
    "gate_up": ["kernels_gemm.hip", "device_common.h", "ham_internal.h", "decide.h"],
    "attn_decode": ["kernels_attn.hip", "device_common.h", "ham_internal.h", "rows.h"],
}


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


def attention_kernel(w: Workload) -> str:
    """Profiler name of the base layers' fused decode-attention step."""
    elem = "unsigned short" if w.shape.dtype == BF16 else "float"
    return f"k_attn_step<{elem}, {w.shape.head_dim}>"


def sources_sha(cls: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in CLASS_SOURCES[cls]:
        h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()


def measured_traffic(w: Workload, cls: str, kernel: str):
    """HBM bytes per launch of ``kernel`` from the committed counter summary
    ``profiles/traffic_<class>_<workload>.txt``, or None when there is none for
    this kernel and workload or its sources have changed since."""
    path = os.path.join(ROOT, "profiles", f"traffic_{cls}_{w.name}.txt")
    try:
        fields = dict(l.split("=", 1) for l in open(path).read().split("\n") if "=" in l and not l.startswith("#"))
        src = sources_sha(cls)
    except (OSError, KeyError):
        return None
    if fields.get("kernel") != kernel or fields.get("workload") != w.name or fields.get("sources_sha256") != src:
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


def micro_steps_needed(w: Workload, lens: list, n_steps: int) -> tuple:
    """(micro steps some sequence needs, macro-steps that fuse a group) over the
    first ``n_steps`` macro-steps: every macro-step launches the micro-step and
    embedder kernels, which return at once on device when nothing needs them."""
    micro = fused = 0
    for st in range(1, n_steps + 1):
        run = [b for b in range(len(lens)) if st < len(lens[b])]
        if not run:
            break
        micro += max(lens[b][st] - 1 for b in run)
        fused += any(lens[b][st - 1] > 1 for b in run)
    return micro, fused


def cost_model_speedup(w: Workload, lens: list, n_steps: int) -> float:
    """The speedup the cost model of Sec. 3.7 predicts over one-token-per-forward
    decoding, r = sum n C(S) / sum (C(S) + (n - 1) c), with C(S) the bytes of one
    base forward at context S (weights, LM head, cached K and V) and c the bytes
    of one micro step (micro layers, LM head), summed over the realised groups of
    every sequence (the embedder, which the formula leaves out, is ignored)."""
    s = w.shape
    es = 2 if s.dtype == BF16 else 4
    d, H, Hk, hd, F, V = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim, s.vocab
    layer = (2 * d * H * hd + 2 * d * Hk * hd + 3 * d * F) * es
    W_lm = (V + 1) * d * es
    kv_slot = s.n_layers * 2 * Hk * hd * es
    c = s.micro_layers * layer + W_lm
    num = den = 0.0
    for b in range(len(lens)):
        S = w.prompt_len
        for st in range(1, min(n_steps, len(lens[b]) - 1) + 1):
            C = s.n_layers * layer + W_lm + (S + 1) * kv_slot
            n = lens[b][st]
            num += n * C
            den += C + (n - 1) * c
            S += 1
    return num / den


def cpu_baseline(w: Workload, sample_steps: int, prompt_len: int) -> dict:
    """The float64 oracle on this host's cores: sequence 0 of the workload's model,
    its seeded prompt cut to ``prompt_len`` tokens, timed over the first macro-steps."""
    from oracle import OracleHam
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    t0 = time.perf_counter()
    om = OracleHam(w.shape, w.seed_weights)
    t_init = time.perf_counter() - t0
    prompt = synth.prompt_ids(w.seed_prompt, 1, w.prompt_len, w.shape.vocab)[0][:prompt_len]
    sched = synth.group_schedule(w.seed_sched, 1, sample_steps + 2, w.shape.max_group)[0]
    timing = {}
    res = om.generate(prompt, w.max_new, sample_steps, forced=lambda st: int(sched[st]), timing=timing)
    tokens = res.tokens - len(res.groups[0])   # tokens emitted by the timed macro-steps
    cut = "" if prompt_len == w.prompt_len else (
        f" (of {w.prompt_len}: the oracle's macro-step cost is its weight streaming; attention over the full "
        f"prompt's slots is about {100.0 * kv_share(w):.0f}% of the bytes)")
    return {"value": tokens / timing["decode_s"], "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{w.name}: sequence 0, prompt {prompt_len}{cut}, first {sample_steps} macro-steps "
                      f"({tokens} tokens, {timing['decode_s']:.1f} s of decode; prefill {timing['prefill_s']:.1f} s "
                      f"and weight generation {t_init:.0f} s excluded), float64 numpy, "
                      f"{platform.processor() or platform.machine()}"}


def kv_share(w: Workload) -> float:
    """Share of the cached K and V in one base forward's bytes at the full prompt length."""
    s = w.shape
    es = 2 if s.dtype == BF16 else 4
    d, H, Hk, hd, F, V = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim, s.vocab
    kv = w.prompt_len * s.n_layers * 2 * Hk * hd * es
    base = s.n_layers * (2 * d * H * hd + 2 * d * Hk * hd + 3 * d * F) * es + (V + 1) * d * es
    return kv / (kv + base)


def _config(w: Workload, **over):
    from paper_2505_20438_amd import ham
    s = w.shape
    kw = dict(n_layers=s.n_layers, d_model=s.d_model, n_heads=s.n_heads, n_kv_heads=s.n_kv_heads,
              head_dim=s.head_dim, ffn_dim=s.ffn_dim, vocab=s.vocab, micro_layers=s.micro_layers,
              max_group=s.max_group, stop_mode=s.stop_mode, stop_id=s.stop_id, dtype=s.dtype,
              max_batch=w.batch, max_prompt=w.prompt_len,
              max_steps=w.macro_steps if w.max_new <= 0 else w.max_new)
    kw.update(over)
    return ham.make_config(**kw)


class Snapshot:
    """One prefill, then every run decodes from the state it left."""

    def __init__(self, rt, prompts, budgets, forced0):
        import torch
        self.rt = rt
        # a short untimed prefill first loads every prefill kernel (the first launch
        # of a kernel pays for loading its code object)
        rt.prefill(prompts[:, :min(512, prompts.shape[1])].contiguous(), budgets, forced0)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(rt.stream)
        rt.prefill(prompts, budgets, forced0)
        e1.record(rt.stream)
        self.buf = torch.empty(rt.state.numel(), dtype=torch.uint8, device=rt.state.device)
        rt.save_state(self.buf)
        torch.cuda.synchronize()
        self.prefill_ms = e0.elapsed_time(e1)
        self.first_tokens = int(rt.out_lens[:prompts.shape[0]].sum())

    def restore(self):
        self.rt.restore_state(self.buf)


def timed_decodes(rt, snap: Snapshot, sched, n_steps: int, warmup: int, steps: int, label: str) -> list:
    """Decode times (ms, HIP events on the model's stream) of ``steps`` runs after ``warmup``."""
    import torch
    times = []
    for i in range(warmup + steps):
        snap.restore()
        e1, e2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e1.record(rt.stream)
        for st in range(1, n_steps + 1):
            rt.macro_step(sched[st])
        e2.record(rt.stream)
        torch.cuda.synchronize()
        ms = e1.elapsed_time(e2)
        if i >= warmup:
            times.append(ms)
        print(f"bench: {label} {'warmup' if i < warmup else 'run'} {i + 1 - (warmup if i >= warmup else 0)}: "
              f"{ms:.1f} ms", file=sys.stderr, flush=True)
    return times


def base_comparator(w: Workload, prompts, warmup: int, steps: int) -> dict:
    """The same weights decoding one token per forward (max group 1: no embedder
    fusion, no micro steps, one KV entry per token) on the same kernels."""
    import torch
    from paper_2505_20438_amd import ham
    rt = ham.HamRuntime(_config(w, max_group=1), w.seed_weights, "cuda:0")
    B = w.batch
    ones = torch.ones((w.max_new + 1, B), dtype=torch.int32, device=prompts.device)
    snap = Snapshot(rt, prompts, [w.max_new] * B, ones[0])
    times = timed_decodes(rt, snap, ones, w.max_new - 1, warmup, steps, "base comparator")
    stats = rt.kv_stats()
    assert all(st["tokens"] == w.max_new and st["gen_slots"] == w.max_new - 1 for st in stats), stats
    ms = float(np.median(times))
    del snap, rt
    torch.cuda.empty_cache()
    # the prefill emits one token per sequence; the timed macro-steps the rest
    return {"value": B * (w.max_new - 1) / (ms / 1000.0), "unit": "tokens/s", "ms_per_run": ms, "runs": len(times),
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
    snap = Snapshot(rt, prompts, [w.max_new] * B, sched[0])
    times = timed_decodes(rt, snap, sched, n_steps, warmup, steps, "reserved-token variant")
    stats = rt.kv_stats()
    assert all(st["tokens"] == w.max_new and st["device_error"] == 0 for st in stats), stats
    ms = float(np.median(times))
    nbytes = algorithmic_bytes(w, lens, n_steps, token_variant=True)
    first = snap.first_tokens
    del snap, rt
    torch.cuda.empty_cache()
    return {"value": (B * w.max_new - first) / (ms / 1000.0), "unit": "tokens/s", "ms_per_run": ms,
            "algorithmic_bytes_per_run": nbytes, "decode_hbm_gbs": (nbytes / 1e9) / (ms / 1000.0),
            "what": "same schedule and kernels, reserved-token control flow: one more micro step per short group"}


def head_mode_run(w: Workload, prompts, conf: float) -> dict:
    """Model-driven groups: the stop head's logit against ln((1-c)/c).  The
    number of macro-steps is found by an untimed run, then one run is timed."""
    import torch
    from paper_2505_20438_amd import ham
    rt = ham.HamRuntime(_config(w, stop_mode=ham.HAM_STOP_HEAD, stop_conf=conf), w.seed_weights, "cuda:0")
    B = w.batch
    snap = Snapshot(rt, prompts, [w.max_new] * B, None)
    n = 0
    while not all(st["done"] for st in rt.kv_stats()):
        if n >= w.max_new:  # every macro-step emits at least one token of an unfinished sequence
            raise RuntimeError("HEAD-mode decode did not spend its budget")
        rt.macro_step()
        n += 1
    snap.restore()
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
    first = snap.first_tokens
    del snap, rt
    torch.cuda.empty_cache()
    return {"confidence": conf, "value": (tokens - first) / (ms / 1000.0), "unit": "tokens/s",
            "macro_steps": n, "mean_group": tokens / float(groups),
            "kv_entries_per_output_token": sum(st["gen_slots"] for st in stats) / float(tokens)}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="c5_8b_long", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-steps", type=int, default=2, help="macro-steps of the oracle sample (0 = skip)")
    ap.add_argument("--cpu-prompt", type=int, default=512,
                    help="prompt tokens of the oracle sample (at most the workload's)")
    ap.add_argument("--max-macro-steps", type=int, default=0,
                    help="stop each run after this many macro-steps (profiler passes only; 0 = whole workload)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="first run one plain device-to-device copy of this size (HBM counter calibration)")
    ap.add_argument("--base", choices=("auto", "on", "off"), default="auto",
                    help="also time the same model decoding one token per forward (groups of one)")
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
    rt = ham.HamRuntime(_config(w), w.seed_weights, "cuda:0")
    rt.set_graph(args.graph == "on")
    stream = rt.stream
    prompts = torch.from_numpy(synth.prompt_ids(w.seed_prompt, B, P, s.vocab)).to(dev)
    n_sched = (w.macro_steps if unbudgeted else w.max_new) + 1
    sched_np = synth.group_schedule(w.seed_sched, B, n_sched, s.max_group)
    sched_dev = torch.from_numpy(np.ascontiguousarray(sched_np.T)).to(dev)   # [step][B], resident
    sched = [sched_dev[st] if forced_mode else None for st in range(n_sched)]
    budgets = [max(w.max_new, 0)] * B
    snap = Snapshot(rt, prompts, budgets, sched[0])
    print(f"bench: {w.name} prefill {snap.prefill_ms:.1f} ms", file=sys.stderr, flush=True)
    if unbudgeted:
        lens = None
        n_steps = w.macro_steps
        for st in range(1, n_steps + 1):
            rt.macro_step(sched[st])
        tokens_per_run = sum(x["tokens"] for x in rt.kv_stats()) - snap.first_tokens
    else:
        lens = [group_lengths(sched_np[b], w.max_new) for b in range(B)]
        n_steps = max(len(l) for l in lens) - 1
        tokens_per_run = sum(budgets) - snap.first_tokens
    truncated = False
    if not unbudgeted and 0 < args.max_macro_steps < n_steps:
        n_steps = args.max_macro_steps   # profiler passes: the JSON line is then not a benchmark result
        tokens_per_run = sum(sum(l[1:n_steps + 1]) for l in lens)
        truncated = True
    if args.copy_calibration_mb > 0:
        src = torch.ones(args.copy_calibration_mb << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    host_enqueue = []

    def one_run(profile: bool = False):
        snap.restore()
        e1, e2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        # the host's enqueue time is taken from an idle GPU
        torch.cuda.synchronize()
        e1.record(stream)
        if profile:
            ham.load_library().ham_profile(rt.handle, 1)
        h0 = time.perf_counter()
        for st in range(1, n_steps + 1):
            rt.macro_step(sched[st])
        host_enqueue.append(time.perf_counter() - h0)
        if profile:
            ham.load_library().ham_profile(rt.handle, 0)
        e2.record(stream)
        torch.cuda.synchronize()
        return e1.elapsed_time(e2)

    for i in range(args.warmup):
        ms = one_run()
        print(f"bench: warmup {i + 1}/{args.warmup}: {ms:.1f} ms", file=sys.stderr, flush=True)
    host_enqueue.clear()
    decode_ms = []
    t0 = time.perf_counter()
    for i in range(args.steps):
        decode_ms.append(one_run())
        print(f"bench: run {i + 1}/{args.steps}: {decode_ms[-1]:.1f} ms", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dec_med = float(np.median(decode_ms))
    stats = rt.kv_stats()
    assert all((unbudgeted or truncated or st["tokens"] == w.max_new) and st["device_error"] == 0
               for st in stats), stats
    if unbudgeted:
        assert sum(st["tokens"] for st in stats) - snap.first_tokens == tokens_per_run   # deterministic runs
    gen_slots = sum(st["gen_slots"] for st in stats)
    value = tokens_per_run / (dec_med / 1000.0)
    # the tiny model's 20 MB stay in the caches: no HBM bytes model for it
    alg_bytes = None if unbudgeted else algorithmic_bytes(w, lens, n_steps)

    # per-kernel-class timing: one more run with HIP events attached to the
    # dispatch of every launch of the classes (same launch configuration, outside
    # the timed runs above; the events mark each kernel's own start and end)
    one_run(profile=True)
    prof = (ham.HamProfT * ham.HAM_PROF_KINDS)()
    ham.check(ham.load_library().ham_profile_read(rt.handle, prof, ham.HAM_PROF_KINDS))
    # micro-step and embedder launches return at once when nothing needs them:
    # their bytes count only for the launches that did work
    if lens is not None:
        micro_needed, fused_steps = micro_steps_needed(w, lens, n_steps)
        active = {"micro_gemm": micro_needed / float(3 * n_steps), "lm_head_micro": micro_needed / float(3 * n_steps),
                  "embed_gemm": fused_steps / float(n_steps)}
    else:
        active = {}
    kernels = {}
    for i, name in enumerate(PROF_NAMES):
        p = prof[i]
        if p.launches:
            frac = active.get(name, 1.0)
            kernels[name] = {"launches": p.launches, "avg_us": 1000.0 * p.ms / p.launches,
                             "bytes_per_launch": p.bytes / p.launches,
                             "launches_with_work": int(round(p.launches * frac)),
                             "gbs": (frac * p.bytes / 1e9) / (p.ms / 1000.0) if p.ms > 0 else None}
            if name in active:
                kernels[name]["note"] = ("bytes of the launches that did work over the time of all launches "
                                         "(launches that no sequence needs return at once)")
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
    elif dom == "attn_decode":
        roofline["kernel_name"] = attention_kernel(w)
    if "kernel_name" in roofline:
        roofline["traffic"] = measured_traffic(w, dom, roofline["kernel_name"])

    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": dec_med, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if s.dtype == BF16 else "f32", "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "prompt_len": P, "output_tokens_per_seq": w.max_new,
                   "layers": s.n_layers, "d_model": s.d_model, "micro_layers": s.micro_layers,
                   "schedule": ("forced geometric group lengths p=1/2, cap 4" if forced_mode
                                else f"model-driven stops (mode {s.stop_mode}, stop id {s.stop_id})"),
                   "macro_steps": n_steps},
        "kv_entries_per_output_token": gen_slots / float(sum(st["tokens"] for st in stats)),
        "kv_entries_per_token_incl_prompt": (B * P + gen_slots) / float(B * P + sum(st["tokens"] for st in stats)),
        "decode_hbm_gbs": None if alg_bytes is None else (alg_bytes / 1e9) / (dec_med / 1000.0),
        "decode_hbm_frac": None if alg_bytes is None else (alg_bytes / 1e9) / (dec_med / 1000.0) / HBM_PEAK_GBS,
        "algorithmic_bytes_per_run": alg_bytes,
        "tokens_per_run": tokens_per_run,
        "prefill_ms": snap.prefill_ms,
        "us_per_macro_step": 1000.0 * dec_med / n_steps,
        "host_enqueue_us_per_macro_step": 1e6 * float(np.median(host_enqueue[:args.steps])) / n_steps,
        "graph": args.graph == "on",
        "wall_s_timed": wall,
        "roofline": roofline,
        "kernels": kernels,
        "timing": "each run restores the state saved after one prefill and decodes the whole budget; value = "
                  "tokens emitted by the macro-steps / median decode time (prefill excluded, reported apart)",
    }
    out["decode_ms_runs"] = [float(x) for x in decode_ms]
    if not unbudgeted and not truncated:
        out["cost_model_speedup_vs_base"] = cost_model_speedup(w, lens, n_steps)
    del snap, rt
    torch.cuda.empty_cache()
    if not unbudgeted and not truncated and args.base != "off":
        out["base_comparator"] = base_comparator(w, prompts, 1 if args.base == "auto" else args.warmup,
                                                 min(args.steps, 3) if args.base == "auto" else args.steps)
        out["speedup_vs_base"] = value / out["base_comparator"]["value"]
    if args.token_cost and not truncated and not unbudgeted:
        out["token_variant"] = token_cost_run(w, prompts, sched, lens, n_steps, args.warmup, args.steps)
        out["token_variant"]["slowdown_vs_stop_head"] = value / out["token_variant"]["value"]
        out["token_variant"]["bytes_ratio_vs_stop_head"] = out["token_variant"]["algorithmic_bytes_per_run"] / alg_bytes
    if args.head_sweep:
        out["head_sweep"] = [head_mode_run(w, prompts, float(c)) for c in args.head_sweep.split(",")]
    if args.cpu_steps > 0:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_steps, min(args.cpu_prompt, P))
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
