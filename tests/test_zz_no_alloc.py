"""The allocation-free attention step (``ham_op_attention_step_noalloc``)
against the entry point it varies (``ham_op_attention_step``), through the C ABI.

Two calls in a row on the same GPU, the second with a smaller input (fewer
rows, a shorter cache, fewer splits), so the second reads the library's shared
scratch array after the first has filled it.  Both entry points run the same
kernels on the same inputs: outputs, appended cache entries and error flags
must be bitwise equal.

Marked ``gpu``: needs an MI355X and ``libham.so`` built in-tree.
"""
import numpy as np
import pytest

from synth.configs import BF16
from tests.gpu_util import tiled_v

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2505_20438_amd import ham
    ham.load_library()
    return torch


def _inputs(torch, rng, R, H, Hk, hd, S, lens):
    dev = "cuda:0"
    qkv = torch.from_numpy(rng.standard_normal((R, (H + 2 * Hk) * hd)).astype(np.float32)).to(dev)
    ang = rng.uniform(0, 6.3, (R, hd // 2))
    cos = torch.from_numpy(np.cos(ang).astype(np.float32)).to(dev)
    sin = torch.from_numpy(np.sin(ang).astype(np.float32)).to(dev)
    K = torch.from_numpy(rng.standard_normal((R, Hk, S, hd)).astype(np.float32)).to(dev).to(torch.bfloat16)
    VT = tiled_v(torch, torch.from_numpy(rng.standard_normal((R, Hk, S, hd)).astype(np.float32)).to(dev)
                 .to(torch.bfloat16))
    i32 = lambda v: torch.tensor(v, dtype=torch.int32, device=dev)  # noqa: E731
    return qkv, cos, sin, K, VT, i32(lens), i32([n - 1 for n in lens]), i32([1] * R)


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_workspace_entry_point_twice(torch_cuda, order):
    torch = torch_cuda
    from paper_2505_20438_amd import ham
    rng = np.random.default_rng(7)
    H, Hk, hd = 32, 8, 128
    stream = torch.cuda.current_stream().cuda_stream
    assert ham.load_library().ham_op_attention_step_noalloc_max_bytes() == 4 << 20
    # (rows, slots, kv_cap, kv lengths): the long-context launch, then a smaller one
    cases = [(4, 33792, 33791, [33314, 32769, 33792, 30000]), (2, 2048, 1500, [1501, 900])]
    for R, S, kv_cap, lens in cases:
        splits = ham.ham_op_attention_step_splits(BF16, R, Hk, hd, kv_cap)
        print("rows", R, "slots", S, "kv_cap", kv_cap, "splits", splits, flush=True)
        assert splits > 1   # the split records (the scratch) are in use
        qkv, cos, sin, K, VT, kv_len, new_slot, enable = _inputs(torch, rng, R, H, Hk, hd, S, lens)
        K2, VT2 = K.clone(), VT.clone()
        out_ws = torch.zeros((R, 2 * H * hd), dtype=torch.bfloat16, device="cuda:0")
        out_na = torch.full_like(out_ws, 7.0)
        err_ws = torch.zeros(R, dtype=torch.int32, device="cuda:0")
        err_na = torch.zeros_like(err_ws)
        ws = torch.empty(ham.ham_op_attention_workspace_bytes(R, H, Hk, hd), dtype=torch.uint8, device="cuda:0")
        ham.ham_op_attention_step(BF16, qkv, cos, sin, K, VT, kv_len, new_slot, enable, kv_cap, err_ws, out_ws, ws,
                                  stream, H, Hk, hd, S)
        ham.ham_op_attention_step_noalloc(BF16, qkv, cos, sin, K2, VT2, kv_len, new_slot, enable, kv_cap, err_na,
                                          out_na, stream, H, Hk, hd, S)
        torch.cuda.synchronize()
        assert torch.equal(out_ws.view(torch.int16), out_na.view(torch.int16))
        assert torch.equal(err_ws, err_na) and int(err_ws.abs().sum()) == 0
        assert torch.equal(K.view(torch.int16), K2.view(torch.int16))
        assert torch.equal(VT.view(torch.int16), VT2.view(torch.int16))
        assert float(out_na.float().abs().sum()) > 0
