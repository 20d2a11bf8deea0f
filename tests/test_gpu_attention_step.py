"""The fused decode-attention step (the kernel every base layer of a macro-step
launches) against the oracle, at the cache lengths of the batched and
long-context workloads, through ``ham_op_attention_step``.

The op picks its slot split exactly as a macro-step over the same number of
sequences with the same slot bound does, so each case runs the launch shape of
that workload: 4 sequences near 33K slots (8 splits, each wave looping over
about 16 key blocks after its first chunk), 32 ragged sequences near 2.3K slots
(one workgroup per sequence and kv head, each wave about 10 blocks), and small
fp32 / head-dim-64 cases.  Per row: RoPE of q and k with the row's factors,
k and v rounded to the cache type and appended at the row's new slot, then
softmax attention over every slot up to and including the new one (Sec. 3.1:
one KV entry per fused group; the oracle's ``attend``).

Marked ``gpu``: needs an MI355X and ``libham.so`` built in-tree.
"""
import dataclasses

import numpy as np
import pytest

from oracle import OracleHam
from oracle.ham import attend
from synth.configs import BF16, F32, TINY
from tests.gpu_util import from_act, tiled_v, untiled_v

pytestmark = pytest.mark.gpu

CASES = {
    # name: dtype, H, Hk, hd, prompt, steps (slot bound = prompt + steps - 1), kv_len after the append per row
    "c5_long_b4": (BF16, 32, 8, 128, 32768, 1024, [33314, 32769, 33792, 1000]),
    "c4_ragged_b32": (BF16, 32, 8, 128, 2048, 512, None),
    "hd64_b1_split": (BF16, 32, 8, 64, 512, 512, [785]),
    "fp32_b3": (F32, 4, 2, 64, 64, 129, [1, 70, 193]),
}


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


@pytest.mark.parametrize("case", sorted(CASES))
def test_attention_step_against_oracle(torch_cuda, case):
    torch = torch_cuda
    from paper_2505_20438_amd import ham
    dtype, H, Hk, hd, P, steps, lens = CASES[case]
    rng = np.random.default_rng(101 + sorted(CASES).index(case))
    S = (P + steps + 63) // 64 * 64
    kv_cap = P + steps - 1
    if lens is None:
        lens = list(rng.integers(P + 1, P + steps + 1, 30)) + [1, P + steps]
    R = len(lens)
    enable = [1] * R
    new_slot = [n - 1 for n in lens]
    if R >= 4:
        enable[3] = 0              # a finished sequence: writes nothing, zeros out
    if R >= 8:
        new_slot[5] = lens[5] - 2  # an inconsistent row: error bit 8, nothing written, zeros out
    splits = ham.ham_op_attention_step_splits(dtype, R, Hk, hd, kv_cap)
    print(case, "rows", R, "slots", S, "kv_cap", kv_cap, "splits", splits, flush=True)
    # the tiny oracle instance provides RoPE (same head dim and base) and rounding
    om = OracleHam(dataclasses.replace(TINY, n_heads=H, n_kv_heads=Hk, head_dim=hd, d_model=64, ffn_dim=64,
                                       vocab=64, n_layers=1, dtype=dtype), 1)
    pos = rng.integers(0, 200000, R)
    cos, sin = om.rope_cos_sin(pos)
    qkv = rng.standard_normal((R, (H + 2 * Hk) * hd)).astype(np.float32)
    K = rng.standard_normal((R, Hk, S, hd)).astype(np.float32)
    V = rng.standard_normal((R, Hk, S, hd)).astype(np.float32)
    dev = "cuda:0"
    tdt = torch.bfloat16 if dtype == BF16 else torch.float32
    Kt = torch.from_numpy(K).to(dev).to(tdt)
    VTt = tiled_v(torch, torch.from_numpy(V).to(dev).to(tdt))
    Kf = Kt.float().cpu().numpy()   # the stored (rounded) cache both sides start from
    Vf = untiled_v(torch, VTt).float().cpu().numpy()
    out = torch.zeros((R, H * hd * (2 if dtype == BF16 else 1)), dtype=tdt, device=dev)
    err = torch.zeros(R, dtype=torch.int32, device=dev)
    ws = torch.empty(ham.ham_op_attention_workspace_bytes(R, H, Hk, hd), dtype=torch.uint8, device=dev)
    i32 = lambda v: torch.tensor(v, dtype=torch.int32, device=dev)  # noqa: E731
    ham.ham_op_attention_step(dtype, torch.from_numpy(qkv).to(dev), torch.from_numpy(cos.astype(np.float32)).to(dev),
                              torch.from_numpy(sin.astype(np.float32)).to(dev), Kt, VTt, i32(lens), i32(new_slot),
                              i32(enable), kv_cap, err, out, ws, torch.cuda.current_stream().cuda_stream, H, Hk, hd, S)
    torch.cuda.synchronize()
    got = from_act(torch, out, H * hd, dtype).cpu().numpy().reshape(R, H, hd)
    Kg = Kt.float().cpu().numpy()
    Vg = untiled_v(torch, VTt).float().cpu().numpy()
    errs = err.cpu().numpy()
    tol = 2e-3 if dtype == BF16 else 1e-5
    worst = 0.0
    for r in range(R):
        ok = enable[r] and new_slot[r] == lens[r] - 1
        if not ok:
            assert np.all(got[r] == 0), r
            assert errs[r] == (8 if enable[r] else 0), (r, errs[r])
            # the cache is untouched for this row
            assert np.array_equal(Kg[r], Kf[r]) and np.array_equal(Vg[r], Vf[r]), r
            continue
        assert errs[r] == 0, r
        s = new_slot[r]
        x = qkv[r].astype(np.float64)
        q = om.rope(x[:H * hd].reshape(1, H, hd), pos[r:r + 1])[0]
        k = om._rnd(om.rope(x[H * hd:(H + Hk) * hd].reshape(1, Hk, hd), pos[r:r + 1])[0])
        v = om._rnd(x[(H + Hk) * hd:].reshape(Hk, hd))
        # appended entry: v exactly; k within one rounding step of the stored type plus
        # the fp32 rounding of the rotation (the kernel rotates in fp32, the oracle in float64)
        assert np.array_equal(Vg[r][:, s], v.astype(np.float32)), r
        kr = x[H * hd:(H + Hk) * hd].reshape(Hk, hd)
        mag = np.abs(kr[:, :hd // 2]) + np.abs(kr[:, hd // 2:])
        bound = (np.abs(k) * (2.0 ** -7 if dtype == BF16 else 2.0 ** -23)
                 + 4 * 2.0 ** -24 * np.concatenate([mag, mag], axis=1))
        assert np.all(np.abs(Kg[r][:, s] - k) <= bound), r
        # every other slot untouched
        Kr, Vr = Kf[r].copy(), Vf[r].copy()
        Kr[:, s], Vr[:, s] = k, v
        assert np.array_equal(np.delete(Kg[r], s, axis=1), np.delete(Kf[r], s, axis=1)), r
        ref = attend(q[None], Kr.transpose(1, 0, 2), Vr.transpose(1, 0, 2), [lens[r]], Hk)[0]
        e = float(np.max(np.abs(got[r] - ref)))
        worst = max(worst, e)
        assert e <= tol, (case, r, lens[r], e)
    print(case, "max abs error", worst, flush=True)
