"""Pins of the oracle's building blocks against library routines, closed forms and invariants."""
import dataclasses
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import OracleHam
from oracle.ham import round_bf16
from synth.configs import BF16, F32, TINY

SMALL = dataclasses.replace(TINY, vocab=96, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96)


@pytest.fixture(scope="module")
def om():
    return OracleHam(SMALL, 77)


def test_round_bf16_matches_torch():
    x = np.random.default_rng(1).standard_normal(50000) * 5
    ref = torch.from_numpy(x).float().bfloat16().double().numpy()
    assert np.array_equal(round_bf16(x), ref)


def test_rmsnorm_unit_rms(om):
    x = np.random.default_rng(2).standard_normal((5, 64)) * 7
    y = om.rmsnorm(x, np.ones(64))
    rms = np.sqrt((y * y).mean(-1))
    assert np.allclose(rms, 1.0 / np.sqrt(1 + om.s.norm_eps / (x * x).mean(-1)), rtol=1e-12)
    ref = F.rms_norm(torch.from_numpy(x), (64,), eps=om.s.norm_eps).numpy()
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_rope_identity_at_zero_and_relative(om):
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, 16))
    k = rng.standard_normal((1, 1, 16))
    assert np.array_equal(om.rope(q, np.array([0])), q)
    dots = []
    for a, b in [(5, 2), (13, 10), (1003, 1000)]:
        dots.append(float((om.rope(q, np.array([a])) * om.rope(k, np.array([b]))).sum()))
    # depends only on a - b (up to the fp32 rounding of the cos/sin tables)
    assert max(dots) - min(dots) < 1e-6
    # rotation preserves the norm of every (i, i + hd/2) pair
    r = om.rope(q, np.array([77]))
    assert np.allclose(q[..., :8] ** 2 + q[..., 8:] ** 2, r[..., :8] ** 2 + r[..., 8:] ** 2, rtol=1e-6)


def test_rope_matches_complex_rotation(om):
    rng = np.random.default_rng(4)
    v = rng.standard_normal((3, 2, 16))
    pos = np.array([0, 9, 4000])
    inv = om.s.rope_theta ** (-np.arange(8) * 2.0 / 16)
    rot = np.exp(1j * pos[:, None] * inv[None, :])
    z = (v[..., :8] + 1j * v[..., 8:]) * rot[:, None, :]
    assert np.allclose(om.rope(v, pos), np.concatenate([z.real, z.imag], -1), atol=1e-6)


def test_attention_special_cases_and_sdpa(om):
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 4, 16))
    K = rng.standard_normal((9, 2, 16))
    V = rng.standard_normal((9, 2, 16))
    # one slot: the output is that slot's value, exactly
    o1 = om.attend(q, K[:1], V[:1], [1])
    assert np.array_equal(o1[0, 0], V[0, 0]) and np.array_equal(o1[0, 3], V[0, 1])
    # identical keys: uniform weights, the mean of the values
    Ku = np.repeat(K[:1], 9, axis=0)
    assert np.allclose(om.attend(q, Ku, V, [9])[0, 1], V[:, 0].mean(0), rtol=1e-12)
    # library routine with GQA head sharing (heads 0,1 -> kv 0; 2,3 -> kv 1), ragged lengths
    qs = rng.standard_normal((3, 4, 16))
    n_valid = [2, 9, 5]
    ours = om.attend(qs, K, V, n_valid)
    for t, n in enumerate(n_valid):
        kk = torch.from_numpy(K[:n]).repeat_interleave(2, dim=1).transpose(0, 1)
        vv = torch.from_numpy(V[:n]).repeat_interleave(2, dim=1).transpose(0, 1)
        ref = F.scaled_dot_product_attention(torch.from_numpy(qs[t])[:, None, :], kk, vv)[:, 0, :]
        assert np.allclose(ours[t], ref.numpy(), rtol=1e-12, atol=1e-12)


def test_embedder_bypass_is_exact(om):
    assert np.array_equal(om.embed_group([17]), om.E.f64(17, 18)[0])


def test_embedder_closed_form_identical_tokens(om):
    # all rows equal and P = 0: attention returns that row, z = A_lin A_o A_v E[t]
    saved = om.P._f64
    om.P._f64 = np.zeros_like(saved)
    try:
        z = om.embed_group([5, 5, 5])
        e = om.E.f64(5, 6)[0]
        ref = om.Alin.f64() @ (om.Ao.f64() @ (om.Av.f64() @ e))
        assert np.allclose(z, ref, rtol=1e-12, atol=1e-14)
        # P = 0: permutation invariant
        assert np.allclose(om.embed_group([3, 8, 11]), om.embed_group([11, 3, 8]), rtol=1e-12, atol=1e-14)
    finally:
        om.P._f64 = saved
    # learned relative positions make the embedding permutation-variant (at random init the
    # attention is nearly uniform, so the effect is small but far above float64 rounding)
    a, b = om.embed_group([3, 8, 11]), om.embed_group([11, 3, 8])
    assert np.abs(a - b).max() > 1e-9 * np.abs(a).max()


def test_embedder_matches_torch_mha(om):
    from tests.ref_torch import RefHam
    ref = RefHam(SMALL, 77)
    for g in ([1, 2], [9, 9, 40], [5, 6, 7, 8], [95, 0, 3, 3]):
        assert np.allclose(om.embed_group(g), ref.embed(g).numpy(), rtol=1e-10, atol=1e-13)


def test_embedder_bf16_matches_torch_mha():
    from tests.ref_torch import RefHam
    shp = dataclasses.replace(SMALL, dtype=BF16)
    om16, ref = OracleHam(shp, 78), RefHam(shp, 78)
    for g in ([1, 2], [5, 6, 7, 8]):
        assert np.allclose(om16.embed_group(g), ref.embed(g).numpy(), rtol=1e-9, atol=1e-12)


def test_decide_lowest_index_wins_ties(om):
    saved = om.Wlm._f64
    W = np.zeros_like(saved)
    W[10, 0] = W[40, 0] = 1.0   # two identical maximal logits
    om.Wlm._f64 = W
    try:
        x = np.zeros(64)
        x[0] = 3.0
        t, _, _, _ = om.decide(x, np.ones(64), False)
        assert t == 10
    finally:
        om.Wlm._f64 = saved


def test_stop_threshold_readings():
    # continue the micro steps iff 1 - sigmoid(s) >= c, i.e. stop iff s > ln((1-c)/c)
    for c in (0.5, 0.6, 0.9, 1.0, 0.0):
        om = OracleHam(dataclasses.replace(SMALL, stop_conf=c), 1)
        for s in (-2.0, -0.3, 0.0, 0.4, 3.0):
            cont = (1.0 - 1.0 / (1.0 + math.exp(-s))) >= c
            if abs(s - om.tau) > 1e-9:
                assert cont == (s <= om.tau), (c, s)
    assert OracleHam(dataclasses.replace(SMALL, stop_conf=1.0), 1).tau == -math.inf
    assert OracleHam(dataclasses.replace(SMALL, stop_conf=0.0), 1).tau == math.inf


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("rows,chunk", [(40000, 16384), (50, 7), (16384, 16384), (16385, 16384)])
def test_uncached_matvec_row_chunks_match_the_plain_product(bf16, rows, chunk):
    # Matrices too large to keep in float64 (the LM head at vocabulary 128256) are
    # multiplied a block of rows at a time; the result must be the plain x @ W^T
    # for every row, including a ragged last block.  W is expanded independently
    # here (torch's bfloat16 view of the bit patterns).
    from oracle.ham import _Mat
    rng = np.random.default_rng(rows + 13 * bf16)
    cols = 24
    vals = rng.standard_normal(rows * cols).astype(np.float32)
    if bf16:
        data = torch.from_numpy(vals).bfloat16().view(torch.int16).numpy().view(np.uint16)
        W = torch.from_numpy(data.view(np.int16)).view(torch.bfloat16).double().numpy().reshape(rows, cols)
    else:
        data = vals
        W = vals.astype(np.float64).reshape(rows, cols)
    m = _Mat(data.copy(), rows, cols, bf16)
    assert m._f64 is None
    x = rng.standard_normal((3, cols))
    got = m.matvec(x, chunk=chunk)
    ref = (torch.from_numpy(x) @ torch.from_numpy(W).T).numpy()
    assert got.shape == (3, rows)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
    # a planted slicing mistake (a block shifted by one row) would move whole rows
    assert np.array_equal(np.argmax(got, axis=1), np.argmax(ref, axis=1))
