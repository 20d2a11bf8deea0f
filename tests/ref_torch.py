"""An independent second reading of the decode loop, used to pin the oracle.

Written separately from ``oracle/`` on purpose: torch library primitives
(``scaled_dot_product_attention``, ``multi_head_attention_forward``, complex
rotation for RoPE) and *full recomputation* of every forward instead of KV
caches.  Float64 throughout; in bf16 models only the stored K and V are rounded,
through torch's own bfloat16 conversion.  Slow (quadratic); tiny shapes only.
"""
from __future__ import annotations

import math

import numpy as np
import torch
import torch.nn.functional as F

import synth
from synth.configs import BF16, STOP_FORCED, STOP_HEAD, STOP_TOKEN, HamShape


def _w(seed, tid, rows, cols, bf16):
    v = synth.normal_tensor(seed, tid, rows * cols, bf16)
    if bf16:
        v = synth.bf16_bits_to_f32(v)
    return torch.from_numpy(v.astype(np.float64)).reshape(rows, cols)


class RefHam:
    def __init__(self, shape: HamShape, seed: int):
        s = shape
        self.s = s
        bf = s.dtype == BF16
        self.bf = bf
        d, H, Hk, hd, Fd, V = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim, s.vocab
        self.E = _w(seed, synth.T_EMBED, V, d, bf)
        self.P = _w(seed, synth.T_RELPOS, 4, d, bf)
        self.Aq, self.Ak, self.Av = (_w(seed, t, H * hd, d, bf) for t in (synth.T_AQ, synth.T_AK, synth.T_AV))
        self.Ao = _w(seed, synth.T_AO, d, H * hd, bf)
        self.Alin = _w(seed, synth.T_ALIN, d, d, bf)
        self.Wlm = _w(seed, synth.T_LMHEAD, V, d, bf)
        self.ws = _w(seed, synth.T_STOP, 1, d, bf)[0]
        self.layers = []
        for j in range(s.n_layers + s.micro_layers):
            tid = lambda t: synth.layer_tensor_id(j, t)  # noqa: E731
            self.layers.append(dict(
                q=_w(seed, tid(synth.L_WQ), H * hd, d, bf), k=_w(seed, tid(synth.L_WK), Hk * hd, d, bf),
                v=_w(seed, tid(synth.L_WV), Hk * hd, d, bf), o=_w(seed, tid(synth.L_WO), d, H * hd, bf),
                g=_w(seed, tid(synth.L_WG), Fd, d, bf), u=_w(seed, tid(synth.L_WU), Fd, d, bf),
                dn=_w(seed, tid(synth.L_WD), d, Fd, bf)))

    def rnd(self, t):
        return t.to(torch.float32).to(torch.bfloat16).to(torch.float64) if self.bf else t

    def norm(self, x):
        return F.rms_norm(x, (x.shape[-1],), eps=self.s.norm_eps)

    def rope(self, x, pos):
        # complex form: (x_i + j x_{i+hd/2}) * exp(j p rho^(-2i/hd)), cos/sin taken in fp32
        hd = self.s.head_dim
        half = hd // 2
        inv = torch.tensor([self.s.rope_theta ** (-2.0 * i / hd) for i in range(half)], dtype=torch.float64)
        ang = pos.to(torch.float64)[:, None] * inv[None, :]
        rot = torch.complex(torch.cos(ang).float().double(), torch.sin(ang).float().double())
        z = torch.complex(x[..., :half], x[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    def stack_forward(self, layers, X, pos):
        """Full causal forward over all rows; returns the residual output of every layer."""
        s = self.s
        T = X.shape[0]
        H, Hk, hd = s.n_heads, s.n_kv_heads, s.head_dim
        outs = []
        for L in layers:
            u = self.norm(X)
            q = self.rope((u @ L["q"].T).view(T, H, hd), pos)
            k = self.rnd(self.rope((u @ L["k"].T).view(T, Hk, hd), pos))
            v = self.rnd((u @ L["v"].T).view(T, Hk, hd))
            rep = H // Hk
            kk = k.repeat_interleave(rep, dim=1).transpose(0, 1)
            vv = v.repeat_interleave(rep, dim=1).transpose(0, 1)
            o = F.scaled_dot_product_attention(q.transpose(0, 1), kk, vv, is_causal=True)
            o = o.transpose(0, 1).reshape(T, H * hd)
            X = X + o @ L["o"].T
            w = self.norm(X)
            X = X + (F.silu(w @ L["g"].T) * (w @ L["u"].T)) @ L["dn"].T
            outs.append(X)
        return outs

    def decide(self, x):
        h = self.norm(x)
        logits = self.Wlm @ h
        return int(torch.argmax(logits)), float(self.ws @ h), logits

    def embed(self, group):
        if len(group) == 1:
            return self.E[group[0]].clone()
        s = self.s
        n = len(group)
        e = self.E[list(group)] + self.P[:n]
        qbar = e.mean(0)
        o, _ = F.multi_head_attention_forward(
            qbar.view(1, 1, -1), e.view(n, 1, -1), e.view(n, 1, -1),
            s.d_model, s.n_heads, None, None, None, None, False, 0.0,
            torch.eye(s.d_model, dtype=torch.float64), None, training=False, need_weights=False,
            use_separate_proj_weight=True, q_proj_weight=self.Aq, k_proj_weight=self.Ak,
            v_proj_weight=self.Av)
        # the identity out-projection above leaves the concatenated heads; A_o then A_lin follow
        return self.Alin @ (self.Ao @ o.view(-1))

    def generate(self, prompt, budget, macro_steps, forced=None, record=None):
        """Groups per step; ``record`` (a list) receives (token, stop logit, logits) per decision."""
        s = self.s
        G = s.max_group
        c = s.stop_conf
        tau = math.inf if c <= 0 else (-math.inf if c >= 1 else math.log((1 - c) / c))
        forced = forced or (lambda step: G)
        base = self.layers[:s.n_layers]
        micro = self.layers[s.n_layers:]
        inputs = [self.E[int(t)] for t in prompt]
        positions = list(range(len(prompt)))
        groups, emitted, step = [], 0, 0
        while True:
            outs = self.stack_forward(base, torch.stack(inputs), torch.tensor(positions))
            t0, s0, lg = self.decide(outs[-1][-1])
            if record is not None:
                record.append((t0, s0, lg.numpy()))
            group = [t0]
            emitted += 1
            L = forced(step)

            def stops(k, st):
                if s.stop_mode == STOP_HEAD:
                    return st > tau
                if s.stop_mode == STOP_FORCED:
                    return k + 1 >= L
                return False

            if not (stops(0, s0) or G <= 1 or (budget and emitted >= budget)):
                rows = [outs[l - 1][-1] for l in s.ctx_layers] + [self.E[t0]]
                for k in range(1, G):
                    mo = self.stack_forward(micro, torch.stack(rows), torch.arange(len(rows)))
                    t, st, lg = self.decide(mo[-1][-1])
                    if record is not None:
                        record.append((t, st, lg.numpy()))
                    if s.stop_mode == STOP_TOKEN and t == s.stop_id:
                        break
                    group.append(t)
                    emitted += 1
                    if stops(k, st) or len(group) >= G or (budget and emitted >= budget):
                        break
                    rows.append(self.E[t])
            groups.append(group)
            if budget and emitted >= budget:
                break
            if macro_steps and step >= macro_steps:
                break
            step += 1
            inputs.append(self.embed(group))
            positions.append(positions[-1] + len(group))
        return groups


def plain_greedy(ref: RefHam, prompt, n_new):
    """Textbook greedy decoding of the base model alone: one forward and one KV per token."""
    toks = [int(t) for t in prompt]
    out = []
    for _ in range(n_new):
        X = ref.E[toks]
        outs = ref.stack_forward(ref.layers[:ref.s.n_layers], X, torch.arange(len(toks)))
        t, _, _ = ref.decide(outs[-1][-1])
        out.append(t)
        toks.append(t)
    return out
