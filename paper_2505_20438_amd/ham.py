"""Thin ctypes binding of libham (include/ham.h): argument marshalling only.

Every step of the decode loop runs in the library's HIP kernels; this module
passes device pointers (from torch tensors) and the caller's HIP stream.
It fails loudly when the compiled library is missing: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libham.so")

HAM_OK, HAM_EINVAL, HAM_ENOMEM, HAM_EHIP, HAM_ESTATE, HAM_ECAP = 0, -1, -2, -3, -4, -5
HAM_F32, HAM_BF16 = 0, 1
HAM_STOP_HEAD, HAM_STOP_TOKEN, HAM_STOP_FORCED, HAM_STOP_FORCED_TOKEN = 0, 1, 2, 3

(HAM_PROF_QKV, HAM_PROF_O, HAM_PROF_GU, HAM_PROF_DOWN, HAM_PROF_MICRO, HAM_PROF_EMBED, HAM_PROF_HEAD0, HAM_PROF_HEADK,
 HAM_PROF_ATTN, HAM_PROF_NORM) = range(10)
HAM_PROF_KINDS = 10

EXPORTED = ("ham_weights_bytes", "ham_state_bytes", "ham_workspace_bytes", "ham_init_weights",
            "ham_prefill", "ham_prefill_embeds", "ham_state_info", "ham_macro_step", "ham_kv_stats", "ham_set_debug", "ham_steps_done",
            "ham_tensor_info", "ham_set_graph", "ham_profile", "ham_profile_read", "ham_last_error", "ham_destroy",
            "ham_op_attention_workspace_bytes", "ham_op_decode_attention", "ham_op_attention_step",
            "ham_op_attention_step_splits", "ham_state_save", "ham_state_restore", "ham_op_attention_step_noalloc",
            "ham_op_attention_step_noalloc_max_bytes")


class HamConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab",
        "embed_layers", "micro_layers", "max_group", "n_ctx_layers")] + [
        ("ctx_layers", ctypes.c_int32 * 8)] + [(n, ctypes.c_int32) for n in ("stop_mode", "stop_id")] + [
        ("stop_conf", ctypes.c_float), ("rope_theta", ctypes.c_float), ("norm_eps", ctypes.c_float),
        ("dtype", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("max_prompt", ctypes.c_int32),
        ("max_steps", ctypes.c_int32)]


class HamKvStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "kv_len", "prompt_slots", "gen_slots", "tokens", "groups", "done")] + [
        ("len_hist", ctypes.c_int32 * 5), ("device_error", ctypes.c_int32)]

    def as_dict(self) -> dict:
        d = {n: getattr(self, n) for n, _ in self._fields_ if n != "len_hist"}
        d["len_hist"] = list(self.len_hist)
        return d


class HamProfT(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int32), ("ms", ctypes.c_double), ("bytes", ctypes.c_double)]


class HamError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libham error {code}: {msg}")
        self.code = code


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libham.so; raises if it has not been built (no fallback path exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is missing: build it with `python -m paper_2505_20438_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, SZ, U64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t, ctypes.c_uint64
    cfgp = ctypes.POINTER(HamConfig)
    for n in ("ham_weights_bytes", "ham_state_bytes", "ham_workspace_bytes"):
        getattr(lib, n).argtypes = [cfgp]
        getattr(lib, n).restype = SZ
    lib.ham_init_weights.argtypes = [cfgp, U64, P, SZ, P, SZ, P, SZ, P, ctypes.POINTER(P)]
    lib.ham_prefill.argtypes = [P, I32, P, I32, P, P, P, P, P]
    lib.ham_prefill_embeds.argtypes = [P, I32, P, P, I32, P, P, P, P, P]
    lib.ham_state_info.argtypes = [cfgp, I32, ctypes.POINTER(SZ), ctypes.POINTER(SZ), ctypes.POINTER(I32)]
    lib.ham_macro_step.argtypes = [P, P, P, P, P]
    lib.ham_kv_stats.argtypes = [P, ctypes.POINTER(HamKvStats)]
    lib.ham_set_debug.argtypes = [P, P, SZ]
    lib.ham_steps_done.argtypes = [P]
    lib.ham_tensor_info.argtypes = [cfgp, I32, ctypes.POINTER(SZ)] + [ctypes.POINTER(I32)] * 6
    lib.ham_profile.argtypes = [P, I32]
    lib.ham_set_graph.argtypes = [P, I32]
    lib.ham_profile_read.argtypes = [P, ctypes.POINTER(HamProfT), I32]
    lib.ham_op_attention_workspace_bytes.argtypes = [I32, I32, I32, I32]
    lib.ham_op_attention_workspace_bytes.restype = SZ
    lib.ham_op_decode_attention.argtypes = [I32, I32, I32, I32, I32, I32, P, P, P, P, P, I32, P, P, SZ, P]
    lib.ham_op_decode_attention.restype = I32
    lib.ham_op_attention_step.argtypes = [I32, I32, I32, I32, I32, I32, P, P, P, P, P, P, P, P, I32, P, P, P, SZ, P]
    lib.ham_op_attention_step.restype = I32
    lib.ham_op_attention_step_noalloc.argtypes = [I32, I32, I32, I32, I32, I32, P, P, P, P, P, P, P, P, I32, P, P, P]
    lib.ham_op_attention_step_noalloc.restype = I32
    lib.ham_op_attention_step_noalloc_max_bytes.argtypes = []
    lib.ham_op_attention_step_noalloc_max_bytes.restype = SZ
    lib.ham_op_attention_step_splits.argtypes = [I32, I32, I32, I32, I32]
    lib.ham_op_attention_step_splits.restype = I32
    lib.ham_state_save.argtypes = [P, P, SZ]
    lib.ham_state_restore.argtypes = [P, P, SZ]
    lib.ham_last_error.restype = ctypes.c_char_p
    lib.ham_destroy.argtypes = [P]
    lib.ham_destroy.restype = None
    for n in ("ham_init_weights", "ham_prefill", "ham_prefill_embeds", "ham_state_info", "ham_macro_step", "ham_kv_stats", "ham_set_debug",
              "ham_steps_done", "ham_tensor_info", "ham_set_graph", "ham_profile", "ham_profile_read",
              "ham_state_save", "ham_state_restore"):
        getattr(lib, n).restype = I32
    _lib = lib
    return lib


def check(rc: int) -> None:
    if rc != HAM_OK:
        raise HamError(rc, load_library().ham_last_error().decode())


_check = check


def make_config(**kw) -> HamConfig:
    c = HamConfig()
    defaults = dict(embed_layers=1, max_group=4, stop_mode=HAM_STOP_FORCED, stop_id=0, stop_conf=0.5,
                    rope_theta=500000.0, norm_eps=1e-5, dtype=HAM_BF16, max_batch=1, max_prompt=1, max_steps=0,
                    ctx_layers=())
    defaults.update(kw)
    layers = [int(x) for x in defaults.pop("ctx_layers")]
    if len(layers) > 8:
        raise ValueError("at most 8 context layers")
    c.n_ctx_layers = len(layers)
    for i, l in enumerate(layers):
        c.ctx_layers[i] = l
    for k, v in defaults.items():
        setattr(c, k, v)
    return c


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def ham_weights_bytes(cfg: HamConfig) -> int:
    return load_library().ham_weights_bytes(ctypes.byref(cfg))


def ham_state_bytes(cfg: HamConfig) -> int:
    return load_library().ham_state_bytes(ctypes.byref(cfg))


def ham_workspace_bytes(cfg: HamConfig) -> int:
    return load_library().ham_workspace_bytes(ctypes.byref(cfg))


def ham_tensor_info(cfg: HamConfig, tensor_id: int) -> dict:
    off = ctypes.c_size_t()
    v = [ctypes.c_int32() for _ in range(6)]
    _check(load_library().ham_tensor_info(ctypes.byref(cfg), tensor_id, ctypes.byref(off),
                                          *[ctypes.byref(x) for x in v]))
    keys = ("rows", "cols", "row_off", "mat_rows", "interleave", "tiled")
    d = {k: x.value for k, x in zip(keys, v)}
    d["offset"] = off.value
    return d


def ham_init_weights(cfg: HamConfig, seed: int, weights, state, workspace, stream: int) -> int:
    h = ctypes.c_void_p()
    _check(load_library().ham_init_weights(
        ctypes.byref(cfg), seed, weights.data_ptr(), weights.numel() * weights.element_size(), state.data_ptr(),
        state.numel() * state.element_size(), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
        stream, ctypes.byref(h)))
    return h.value


def ham_prefill(model: int, batch: int, prompt, prompt_len: int, max_new: Sequence[int], forced=None,
                teacher=None, out_tokens=None, out_lens=None) -> None:
    arr = (ctypes.c_int32 * batch)(*[int(x) for x in max_new])
    _check(load_library().ham_prefill(model, batch, _ptr(prompt), prompt_len, arr, _ptr(forced), _ptr(teacher),
                                      _ptr(out_tokens), _ptr(out_lens)))


def ham_prefill_embeds(model: int, embeds, positions, max_new: Sequence[int], forced=None, teacher=None,
                       out_tokens=None, out_lens=None) -> None:
    """embeds: fp32 [batch][n][d_model], positions: int32 [batch][n] (device tensors)."""
    batch, n = int(embeds.shape[0]), int(embeds.shape[1])
    arr = (ctypes.c_int32 * batch)(*[int(x) for x in max_new])
    _check(load_library().ham_prefill_embeds(model, batch, _ptr(embeds), _ptr(positions), n, arr, _ptr(forced),
                                             _ptr(teacher), _ptr(out_tokens), _ptr(out_lens)))


def ham_state_info(cfg: HamConfig, layer: int) -> dict:
    k, v, s = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_int32()
    _check(load_library().ham_state_info(ctypes.byref(cfg), layer, ctypes.byref(k), ctypes.byref(v),
                                         ctypes.byref(s)))
    return {"k_offset": k.value, "v_offset": v.value, "slots": s.value}


def ham_macro_step(model: int, forced=None, teacher=None, out_tokens=None, out_lens=None) -> None:
    _check(load_library().ham_macro_step(model, _ptr(forced), _ptr(teacher), _ptr(out_tokens), _ptr(out_lens)))


def ham_kv_stats(model: int, batch: int) -> List[dict]:
    out = (HamKvStats * batch)()
    _check(load_library().ham_kv_stats(model, out))
    return [o.as_dict() for o in out]


def ham_set_debug(model: int, buf) -> None:
    _check(load_library().ham_set_debug(model, _ptr(buf), 0 if buf is None else buf.numel() * buf.element_size()))


def ham_op_decode_attention(dtype: int, q, k, vt, kv_len, enable, kv_max: int, out, workspace, stream: int,
                            n_heads: int, n_kv_heads: int, head_dim: int, slots_cap: int) -> None:
    """Decode attention of one act row per sequence (include/ham_ops.h)."""
    rows = kv_len.numel()
    check(load_library().ham_op_decode_attention(
        dtype, rows, n_heads, n_kv_heads, head_dim, slots_cap, q.data_ptr(), k.data_ptr(), vt.data_ptr(),
        kv_len.data_ptr(), enable.data_ptr(), kv_max, out.data_ptr(), workspace.data_ptr(),
        workspace.numel() * workspace.element_size(), stream))


def ham_op_attention_step(dtype: int, qkv, cos, sin, k, vt, kv_len, new_slot, enable, kv_cap: int, err, out,
                          workspace, stream: int, n_heads: int, n_kv_heads: int, head_dim: int,
                          slots_cap: int) -> None:
    """Fused decode-attention step of one base layer, one row per sequence (include/ham_ops.h)."""
    rows = kv_len.numel()
    check(load_library().ham_op_attention_step(
        dtype, rows, n_heads, n_kv_heads, head_dim, slots_cap, qkv.data_ptr(), cos.data_ptr(), sin.data_ptr(),
        k.data_ptr(), vt.data_ptr(), kv_len.data_ptr(), new_slot.data_ptr(), enable.data_ptr(), kv_cap,
        err.data_ptr(), out.data_ptr(), workspace.data_ptr(), workspace.numel() * workspace.element_size(), stream))


def ham_op_attention_step_noalloc(dtype: int, qkv, cos, sin, k, vt, kv_len, new_slot, enable, kv_cap: int, err,
                                  out, stream: int, n_heads: int, n_kv_heads: int, head_dim: int,
                                  slots_cap: int) -> None:
    """ham_op_attention_step with its split records in the library's own device array."""
    rows = kv_len.numel()
    check(load_library().ham_op_attention_step_noalloc(
        dtype, rows, n_heads, n_kv_heads, head_dim, slots_cap, qkv.data_ptr(), cos.data_ptr(), sin.data_ptr(),
        k.data_ptr(), vt.data_ptr(), kv_len.data_ptr(), new_slot.data_ptr(), enable.data_ptr(), kv_cap,
        err.data_ptr(), out.data_ptr(), stream))


def ham_op_attention_step_splits(dtype: int, rows: int, n_kv_heads: int, head_dim: int, kv_cap: int) -> int:
    return load_library().ham_op_attention_step_splits(dtype, rows, n_kv_heads, head_dim, kv_cap)


def ham_op_attention_workspace_bytes(rows: int, n_heads: int, n_kv_heads: int, head_dim: int) -> int:
    return load_library().ham_op_attention_workspace_bytes(rows, n_heads, n_kv_heads, head_dim)


def ham_steps_done(model: int) -> int:
    return load_library().ham_steps_done(model)


def ham_destroy(model: int) -> None:
    load_library().ham_destroy(model)


class HamRuntime:
    """Allocates the library's three buffers as torch tensors on one device and
    binds them (``ham_init_weights``).  Device memory and the stream are torch's;
    the computation is the library's."""

    def __init__(self, cfg: HamConfig, seed: int, device: str = "cuda:0", stream=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = torch.device(device)
        self.stream = stream or torch.cuda.current_stream(self.device)
        nb = [ham_weights_bytes(cfg), ham_state_bytes(cfg), ham_workspace_bytes(cfg)]
        if 0 in nb:
            raise HamError(HAM_EINVAL, "invalid configuration")
        self.weights, self.state, self.workspace = (
            torch.empty(n, dtype=torch.uint8, device=self.device) for n in nb)
        self.handle = ham_init_weights(cfg, seed, self.weights, self.state, self.workspace,
                                       self.stream.cuda_stream)
        B = cfg.max_batch
        self.out_tokens = torch.full((B, 4), -1, dtype=torch.int32, device=self.device)
        self.out_lens = torch.zeros(B, dtype=torch.int32, device=self.device)
        self.batch = 0

    def prefill(self, prompt, max_new, forced=None, teacher=None):
        self.batch = prompt.shape[0]
        ham_prefill(self.handle, prompt.shape[0], prompt, prompt.shape[1], max_new, forced, teacher,
                    self.out_tokens, self.out_lens)

    def prefill_embeds(self, embeds, positions, max_new, forced=None, teacher=None):
        self.batch = embeds.shape[0]
        ham_prefill_embeds(self.handle, embeds, positions, max_new, forced, teacher, self.out_tokens, self.out_lens)

    def kv_cache(self, layer: int, n_slots: int):
        """K and V of base layer ``layer``, slots [0, n_slots) of the current batch, as
        float32 [batch][n_kv_heads][n_slots][head_dim] tensors (a copy)."""
        torch = self.torch
        info = ham_state_info(self.cfg, layer)
        c = self.cfg
        es = 2 if c.dtype == HAM_BF16 else 4
        B, Hk, S, hd = c.max_batch, c.n_kv_heads, info["slots"], c.head_dim
        n = B * Hk * S * hd

        def view(off):
            raw = self.state[off: off + n * es]
            if es == 2:  # bf16 bits -> float32
                return (raw.view(torch.int16).to(torch.int32) << 16).view(torch.float32)
            return raw.view(torch.float32)
        K = view(info["k_offset"]).view(B, Hk, S, hd)[: self.batch, :, :n_slots]
        V = view(info["v_offset"]).view(B, Hk, S // 32, hd, 32).permute(0, 1, 2, 4, 3).reshape(B, Hk, S, hd)
        return K.clone(), V[: self.batch, :, :n_slots].clone()

    def macro_step(self, forced=None, teacher=None):
        ham_macro_step(self.handle, forced, teacher, self.out_tokens, self.out_lens)

    def save_state(self, buf) -> None:
        """Copy the decode state (KV cache + counters) into ``buf`` (uint8, >= state bytes)."""
        _check(load_library().ham_state_save(self.handle, buf.data_ptr(), buf.numel() * buf.element_size()))

    def restore_state(self, buf) -> None:
        """Continue from the point of the last save_state (its copy in ``buf``)."""
        _check(load_library().ham_state_restore(self.handle, buf.data_ptr(), buf.numel() * buf.element_size()))

    def set_graph(self, enable: bool) -> None:
        _check(load_library().ham_set_graph(self.handle, 1 if enable else 0))

    def kv_stats(self):
        return ham_kv_stats(self.handle, self.batch)

    def tensor(self, tensor_id: int):
        """A generated tensor [rows][cols] in logical row-major order (bf16 as int16 bits)."""
        torch = self.torch
        t = ham_tensor_info(self.cfg, tensor_id)
        es = 2 if self.cfg.dtype == HAM_BF16 else 4
        dt = torch.int16 if es == 2 else torch.float32
        R, K = t["mat_rows"], t["cols"]
        flat = self.weights[t["offset"]: t["offset"] + R * K * es].view(dt)
        if t["tiled"]:   # undo the fragment tiling: [tile][frag][group][row][elem] -> [tile][row][frag][group][elem]
            epl = 16 // es
            flat = flat.view(R // 16, K // (4 * epl), 4, 16, epl).permute(0, 3, 1, 2, 4)
        mat = flat.reshape(R, K)
        r = torch.arange(t["rows"], device=mat.device)
        if t["interleave"]:
            idx = 16 * (r // 8) + r % 8 + (8 if t["interleave"] == 2 else 0)
        else:
            idx = r + t["row_off"]
        return mat[idx]

    def close(self):
        if self.handle:
            ham_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
