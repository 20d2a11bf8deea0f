"""Float64 oracle of the HAMburger decode loop.

Test infrastructure only (see the package docstring).

Numeric contract (bf16 models): the weights and the KV cache are bf16 (K and V
are rounded to bf16 when stored, ``_rnd``); every activation, including the
operands of the matrix products, the residual stream, norms, softmax, logits and
the stop logit, is kept at full precision (here float64).  For fp32 models
``_rnd`` is the identity and everything is float64.
"""
from __future__ import annotations

import dataclasses
import math
import time
from typing import Callable, List, Optional, Sequence

import numpy as np

import synth
from synth.configs import BF16, STOP_FORCED, STOP_FORCED_TOKEN, STOP_HEAD, STOP_TOKEN, HamShape


# ----------------------------------------------------------------------------
# rounding of activations (the contract's rounding points)
# ----------------------------------------------------------------------------
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16 through float32 (nearest even at both steps), as float64."""
    f = np.asarray(x, dtype=np.float32)
    b = np.ascontiguousarray(f).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)) << np.uint32(16)
    return r.view(np.float32).astype(np.float64)


def _bits_to_f64(u: np.ndarray) -> np.ndarray:
    return (u.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, n_valid: Sequence[int], n_kv_heads: int) -> np.ndarray:
    """GQA softmax attention: q [T][H][hd]; K, V [S][Hkv][hd]; row t sees slots < n_valid[t];
    q-head h reads kv-head h // (H / Hkv); scores scaled by 1/sqrt(hd)."""
    T, H, hd = q.shape
    grp = H // n_kv_heads
    out = np.zeros((T, H, hd))
    scale = 1.0 / math.sqrt(hd)
    n_valid = np.asarray(n_valid, dtype=np.int64).reshape(T)
    # Rows are independent: they are taken in groups only to bound the size of
    # the score matrix.  Within a row, a slot j counts iff j < n_valid[t].
    ROWS = 512
    for t0 in range(0, T, ROWS):
        t1 = min(T, t0 + ROWS)
        n = int(n_valid[t0:t1].max(initial=0))
        if n == 0:
            continue
        seen = np.arange(n)[None, :] < n_valid[t0:t1, None]         # [rows][n]
        live = n_valid[t0:t1] > 0
        for h in range(H):
            Kh = K[:n, h // grp, :].astype(np.float64)               # [n][hd]
            Vh = V[:n, h // grp, :].astype(np.float64)
            sc = np.where(seen, (q[t0:t1, h, :] @ Kh.T) * scale, -np.inf)
            m = np.where(live, sc.max(axis=1), 0.0)[:, None]
            a = np.exp(sc - m)
            a /= np.where(live, a.sum(axis=1), 1.0)[:, None]
            out[t0:t1, h, :] = a @ Vh
    return out


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------
class _Mat:
    """One generated matrix, kept compact (bf16 bits or float32) and expanded on use."""

    def __init__(self, data: np.ndarray, rows: int, cols: int, bf16: bool):
        self.data = data.reshape(rows, cols)
        self.rows, self.cols, self.bf16 = rows, cols, bf16
        self._f64 = None

    def f64(self, r0: int = 0, r1: Optional[int] = None) -> np.ndarray:
        if self._f64 is not None:
            return self._f64[r0:r1]
        d = self.data[r0:r1]
        return _bits_to_f64(d) if self.bf16 else d.astype(np.float64)

    def cache(self) -> None:
        self._f64 = self.f64()

    def matvec(self, x: np.ndarray, chunk: int = 16384) -> np.ndarray:
        """y = x @ W^T for x of shape [T][cols] (float64)."""
        if self._f64 is not None or self.rows <= chunk:
            return x @ self.f64().T
        out = np.empty(x.shape[:-1] + (self.rows,), dtype=np.float64)
        for r0 in range(0, self.rows, chunk):
            r1 = min(self.rows, r0 + chunk)
            out[..., r0:r1] = x @ self.f64(r0, r1).T
        return out


def _gen(seed: int, tid: int, rows: int, cols: int, bf16: bool) -> _Mat:
    return _Mat(synth.normal_tensor(seed, tid, rows * cols, bf16), rows, cols, bf16)


@dataclasses.dataclass
class _Layer:
    wq: _Mat
    wk: _Mat
    wv: _Mat
    wo: _Mat
    wg: _Mat
    wu: _Mat
    wd: _Mat
    g1: np.ndarray
    g2: np.ndarray


@dataclasses.dataclass
class Decision:
    """One token decision (greedy, Sec. 4.1) with its stop logit (Sec. 3.3)."""
    step: int          # 0 = prefill group, s = s-th macro-step
    k: int             # micro index (0 = from the base model, Sec. 3.4)
    token: int
    stop_logit: float
    h: Optional[np.ndarray] = None        # normed hidden (before rounding)
    logits: Optional[np.ndarray] = None   # float32 copy, when recording


@dataclasses.dataclass
class SeqResult:
    groups: List[List[int]]
    kv_len: int
    prompt_slots: int
    gen_slots: int
    tokens: int
    decisions: List[Decision]


# ----------------------------------------------------------------------------
# the model
# ----------------------------------------------------------------------------
class OracleHam:
    """HAMburger = compositional embedder + base decoder + micro-step decoder.

    ``shape`` gives the architecture, ``seed`` the weights (see :mod:`synth`).
    """

    def __init__(self, shape: HamShape, seed: int, cache_f64: Optional[bool] = None):
        s = shape
        self.s = s
        self.bf16 = s.dtype == BF16
        bf = self.bf16
        d, hd, H, Hk, F, V = s.d_model, s.head_dim, s.n_heads, s.n_kv_heads, s.ffn_dim, s.vocab
        self.E = _gen(seed, synth.T_EMBED, V, d, bf)
        self.P = _gen(seed, synth.T_RELPOS, 4, d, bf)
        self.Aq = _gen(seed, synth.T_AQ, H * hd, d, bf)
        self.Ak = _gen(seed, synth.T_AK, H * hd, d, bf)
        self.Av = _gen(seed, synth.T_AV, H * hd, d, bf)
        self.Ao = _gen(seed, synth.T_AO, d, H * hd, bf)
        self.Alin = _gen(seed, synth.T_ALIN, d, d, bf)
        self.Wlm = _gen(seed, synth.T_LMHEAD, V, d, bf)
        self.ws = _gen(seed, synth.T_STOP, 1, d, bf)
        self.layers: List[_Layer] = []
        for j in range(s.n_layers + s.micro_layers):
            t = lambda k: synth.layer_tensor_id(j, k)  # noqa: E731
            self.layers.append(_Layer(
                wq=_gen(seed, t(synth.L_WQ), H * hd, d, bf),
                wk=_gen(seed, t(synth.L_WK), Hk * hd, d, bf),
                wv=_gen(seed, t(synth.L_WV), Hk * hd, d, bf),
                wo=_gen(seed, t(synth.L_WO), d, H * hd, bf),
                wg=_gen(seed, t(synth.L_WG), F, d, bf),
                wu=_gen(seed, t(synth.L_WU), F, d, bf),
                wd=_gen(seed, t(synth.L_WD), d, F, bf),
                g1=np.ones(d), g2=np.ones(d)))
        self.g_final = np.ones(d)
        self.g_micro_final = np.ones(d)
        n_params = (V * d * 2 + 4 * d + 5 * d * d + d
                    + (s.n_layers + s.micro_layers) * (2 * d * H * hd + 2 * d * Hk * hd + 3 * d * F))
        if cache_f64 is None:
            cache_f64 = n_params <= 64_000_000
        if cache_f64:
            for m in self._all_mats():
                m.cache()
        # RoPE tables: theta_i(p) = p * rho^(-2i/hd); cos/sin in float64, rounded to fp32
        self._inv_freq = s.rope_theta ** (-2.0 * np.arange(hd // 2, dtype=np.float64) / hd)
        # stop threshold on the stop logit: continue iff 1 - sigmoid(s) >= c
        c = s.stop_conf
        self.tau = math.inf if c <= 0.0 else (-math.inf if c >= 1.0 else math.log((1.0 - c) / c))

    def _all_mats(self):
        yield from (self.E, self.P, self.Aq, self.Ak, self.Av, self.Ao, self.Alin, self.Wlm, self.ws)
        for L in self.layers:
            yield from (L.wq, L.wk, L.wv, L.wo, L.wg, L.wu, L.wd)

    # ------------------------------------------------------------------ pieces
    def _rnd(self, x: np.ndarray) -> np.ndarray:
        return round_bf16(x) if self.bf16 else np.asarray(x, dtype=np.float64)

    def rmsnorm(self, x: np.ndarray, g: np.ndarray) -> np.ndarray:
        """g * x / sqrt(mean(x^2) + eps) over the last axis."""
        ms = np.mean(x * x, axis=-1, keepdims=True)
        return x / np.sqrt(ms + self.s.norm_eps) * g

    def rope_cos_sin(self, pos: np.ndarray):
        ang = np.asarray(pos, dtype=np.float64)[:, None] * self._inv_freq[None, :]
        return (np.cos(ang).astype(np.float32).astype(np.float64),
                np.sin(ang).astype(np.float32).astype(np.float64))

    def rope(self, v: np.ndarray, pos: np.ndarray) -> np.ndarray:
        """Rotate-half RoPE of v [T][heads][hd] at positions pos [T]."""
        half = self.s.head_dim // 2
        c, sn = self.rope_cos_sin(pos)
        c, sn = c[:, None, :], sn[:, None, :]
        a, b = v[..., :half], v[..., half:]
        return np.concatenate([a * c - b * sn, b * c + a * sn], axis=-1)

    def embed_rows(self, ids: Sequence[int]) -> np.ndarray:
        return np.stack([self.E.f64(int(t), int(t) + 1)[0] for t in ids])

    def attend(self, q: np.ndarray, K: np.ndarray, V: np.ndarray, n_valid: Sequence[int]) -> np.ndarray:
        """Softmax attention: q [T][H][hd]; K, V [S][Hkv][hd]; row t sees slots < n_valid[t]."""
        return attend(q, K, V, n_valid, self.s.n_kv_heads)

    def forward_rows(self, layers: Sequence[_Layer], X: np.ndarray, pos: np.ndarray,
                     caches: list, capture: Sequence[int] = ()):
        """Causal forward of new rows X [T][d] at positions ``pos`` through ``layers``.

        ``caches[i]`` = [K, V] arrays [S][Hkv][hd] of layer i, grown in place by T
        slots (one per row).  Returns the residual outputs and, for each 1-based
        layer index in ``capture``, the residual output of that layer.
        """
        s = self.s
        T = X.shape[0]
        H, Hk, hd = s.n_heads, s.n_kv_heads, s.head_dim
        kv_dtype = np.float32 if self.bf16 else np.float64
        captured = {}
        X = X.astype(np.float64).copy()
        for li, L in enumerate(layers):
            u = self.rmsnorm(X, L.g1)
            q = L.wq.matvec(u).reshape(T, H, hd)
            k = L.wk.matvec(u).reshape(T, Hk, hd)
            v = L.wv.matvec(u).reshape(T, Hk, hd)
            q = self.rope(q, pos)
            k = self._rnd(self.rope(k, pos))
            v = self._rnd(v)
            Kc, Vc = caches[li]
            S0 = Kc.shape[0]
            Kc = np.concatenate([Kc, k.astype(kv_dtype)], axis=0)
            Vc = np.concatenate([Vc, v.astype(kv_dtype)], axis=0)
            caches[li] = [Kc, Vc]
            o = self.attend(q, Kc, Vc, [S0 + t + 1 for t in range(T)])
            o = o.reshape(T, H * hd)
            X = X + L.wo.matvec(o)
            w = self.rmsnorm(X, L.g2)
            g = L.wg.matvec(w)
            up = L.wu.matvec(w)
            act = g / (1.0 + np.exp(-g)) * up
            X = X + L.wd.matvec(act)
            if (li + 1) in capture:
                captured[li + 1] = X.copy()
        return X, captured

    def new_caches(self, n_layers: int) -> list:
        s = self.s
        dt = np.float32 if self.bf16 else np.float64
        z = np.zeros((0, s.n_kv_heads, s.head_dim), dtype=dt)
        return [[z, z] for _ in range(n_layers)]

    def decide(self, x_row: np.ndarray, g: np.ndarray, record: bool):
        """Normed hidden -> (argmax token, stop logit); lowest index wins ties."""
        h = self.rmsnorm(x_row, g)
        logits = self.Wlm.matvec(h[None, :])[0]
        t = int(np.argmax(logits))
        st = float(self.ws.f64()[0] @ h)
        return t, st, h, (logits.astype(np.float32) if record else None)

    def embed_group(self, group: Sequence[int]) -> np.ndarray:
        """Compositional embedder (Sec. 3.2): one vector for an ordered token group."""
        n = len(group)
        if n == 1:  # bypass (Fig. 2a, Sec. 3.4)
            return self.embed_rows(group)[0]
        s = self.s
        H, hd = s.n_heads, s.head_dim
        e = self.embed_rows(group) + self.P.f64(0, n)       # learned relative positions 0..n-1
        qbar = e.mean(axis=0)                                # query = mean of the inputs
        Q = self.Aq.matvec(qbar[None, :])[0].reshape(H, hd)
        K = self.Ak.matvec(e).reshape(n, H, hd)
        Vv = self.Av.matvec(e).reshape(n, H, hd)
        o = np.zeros((H, hd))
        for h in range(H):
            sc = K[:, h, :] @ Q[h] / math.sqrt(hd)
            a = np.exp(sc - sc.max())
            a /= a.sum()
            o[h] = a @ Vv[:, h, :]
        y = self.Ao.matvec(o.reshape(1, H * hd))[0]
        return self.Alin.matvec(y[None, :])[0]

    # ------------------------------------------------------------------ loop
    def _stop_after(self, k: int, stop_logit: float, forced_len: int) -> bool:
        mode = self.s.stop_mode
        if mode == STOP_HEAD:
            return stop_logit > self.tau
        if mode == STOP_FORCED:
            return k + 1 >= forced_len
        return False  # TOKEN mode decides through the reserved id instead

    def micro_loop(self, ctx: List[np.ndarray], t0: int, s0: float, h0, lg0, step: int,
                   emitted: int, budget: int, forced_len: int, record: bool,
                   decisions: List[Decision]) -> List[int]:
        """Micro-step decoder (Sec. 3.3): the group emitted at this macro-step."""
        s = self.s
        G = s.max_group
        decisions.append(Decision(step, 0, t0, s0, h0 if record else None, lg0))
        group = [t0]
        emitted += 1
        if (self._stop_after(0, s0, forced_len) or len(group) >= G
                or (budget > 0 and emitted >= budget)):
            return group
        C = len(ctx)
        micro = self.layers[s.n_layers:]
        caches = self.new_caches(len(micro))
        Y = np.concatenate([np.stack(ctx), self.embed_rows([t0])], axis=0)
        X, _ = self.forward_rows(micro, Y, np.arange(C + 1), caches)
        for k in range(1, G):
            t, st, h, lg = self.decide(X[-1], self.g_micro_final, record)
            decisions.append(Decision(step, k, t, st, h if record else None, lg))
            if s.stop_mode == STOP_TOKEN and t == s.stop_id:
                break  # reserved stop token: not emitted (Sec. 4.4 variant)
            if s.stop_mode == STOP_FORCED_TOKEN and k >= forced_len:
                break  # the forced length's reserved-token decision: not emitted (Sec. 4.4 variant)
            group.append(t)
            emitted += 1
            if (self._stop_after(k, st, forced_len) or len(group) >= G
                    or (budget > 0 and emitted >= budget)):
                break
            X, _ = self.forward_rows(micro, self.embed_rows([t]), np.array([C + k]), caches)
        return group

    def generate(self, prompt: Sequence[int], budget: int, macro_steps: int,
                 forced: Optional[Callable[[int], int]] = None, record: bool = False,
                 inputs: Optional[List[np.ndarray]] = None, timing: Optional[dict] = None) -> SeqResult:
        """Prefill then ``macro_steps`` macro-steps (or until the budget is spent).

        ``forced(step)`` gives the forced group length (FORCED stop mode).
        If ``inputs`` is a list, the base-model input vectors and their positions
        are appended to it (for the prefill-versus-incremental check).  If
        ``timing`` is a dict it receives the wall time of prefill and of the
        macro-steps (``prefill_s``, ``decode_s``).
        """
        t_start = time.perf_counter()
        s = self.s
        forced = forced or (lambda step: s.max_group)
        P = len(prompt)
        base = self.layers[:s.n_layers]
        caches = self.new_caches(s.n_layers)
        ctx_l = s.ctx_layers
        decisions: List[Decision] = []
        # prefill: prompt tokens are not fused, one KV slot each (Fig. 2b)
        X0 = self.embed_rows(prompt)
        pos = np.arange(P)
        X, cap = self.forward_rows(base, X0, pos, caches, capture=ctx_l)
        if inputs is not None:
            inputs.append((X0, pos))
        t0, s0, h0, lg0 = self.decide(X[-1], self.g_final, record)
        ctx = [cap[l][-1] for l in ctx_l]
        group = self.micro_loop(ctx, t0, s0, h0, lg0, 0, 0, budget, forced(0), record, decisions)
        groups = [group]
        emitted = len(group)
        pos_last = P - 1
        step = 0
        t_prefill = time.perf_counter()
        while True:
            if budget > 0 and emitted >= budget:
                break
            if macro_steps > 0 and step >= macro_steps:
                break
            if budget == 0 and macro_steps == 0:
                break
            step += 1
            n = len(group)
            pos_last += n   # the fused entry sits at its last token's position (Sec. 3.2)
            z = self.embed_group(group)
            if inputs is not None:
                inputs.append((z[None, :], np.array([pos_last])))
            X, cap = self.forward_rows(base, z[None, :], np.array([pos_last]), caches, capture=ctx_l)
            t0, s0, h0, lg0 = self.decide(X[-1], self.g_final, record)
            ctx = [cap[l][-1] for l in ctx_l]
            group = self.micro_loop(ctx, t0, s0, h0, lg0, step, emitted, budget, forced(step),
                                    record, decisions)
            groups.append(group)
            emitted += len(group)
        if timing is not None:
            timing["prefill_s"] = t_prefill - t_start
            timing["decode_s"] = time.perf_counter() - t_prefill
        self.last_caches = caches
        kv_len = caches[0][0].shape[0]
        return SeqResult(groups=groups, kv_len=kv_len, prompt_slots=P, gen_slots=kv_len - P,
                         tokens=sum(len(g) for g in groups), decisions=decisions)
