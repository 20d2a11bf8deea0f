"""The C ABI on the CPU: the library loads, exports what include/*.h declares,
and rejects bad configurations and calls before touching the GPU."""
import ctypes
import os
import re

import pytest

from paper_2505_20438_amd import ham
from synth.configs import SHAPE_1B, SHAPE_8B, TINY, WORKLOADS
from tests.gpu_util import config_for

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ham.LIB_PATH):
        pytest.skip("libham.so not built")
    return ham.load_library()


def _declared():
    names = set()
    for h in ("ham.h", "ham_ops.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(ham_[a-z_0-9]+)\s*\(", text))
    return names


def test_every_declared_symbol_is_exported(lib):
    declared = _declared()
    assert {"ham_init_weights", "ham_prefill", "ham_macro_step", "ham_kv_stats"} <= declared
    for n in declared:
        assert hasattr(lib, n), n
    assert declared == set(ham.EXPORTED)


def test_binding_constants_match_header():
    # every #define of the header that the binding names has the same value there
    text = open(os.path.join(ROOT, "include", "ham.h")).read()
    defines = dict(re.findall(r"^#define (HAM_\w+) \(?(-?\d+)\)?", text, re.M))
    named = [k for k in defines if hasattr(ham, k)]
    assert len(named) >= 23 and {"HAM_PROF_NORM", "HAM_PROF_KINDS", "HAM_BF16", "HAM_ECAP"} <= set(named)
    for k in named:
        assert getattr(ham, k) == int(defines[k]), k


def test_size_queries(lib):
    for w in WORKLOADS.values():
        cfg = config_for(w.shape, w.batch, w.prompt_len, max(w.max_new, w.macro_steps))
        assert ham.ham_weights_bytes(cfg) > 0 and ham.ham_state_bytes(cfg) > 0
        assert ham.ham_workspace_bytes(cfg) > 0
    # the weights buffer holds at least every parameter once
    cfg = config_for(SHAPE_8B, 1, 16, 16)
    s = SHAPE_8B
    layer = (2 * s.d_model * s.n_heads * s.head_dim + 2 * s.d_model * s.n_kv_heads * s.head_dim
             + 3 * s.d_model * s.ffn_dim)
    params = (s.n_layers + s.micro_layers) * layer + 2 * s.vocab * s.d_model + 5 * s.d_model ** 2
    assert ham.ham_weights_bytes(cfg) >= 2 * params
    # the smashed KV cache holds max_prompt + max_steps slots per sequence and layer
    cfg = config_for(SHAPE_1B, 2, 100, 28)
    kv = 2 * SHAPE_1B.n_layers * 2 * SHAPE_1B.n_kv_heads * 128 * SHAPE_1B.head_dim * 2
    assert ham.ham_state_bytes(cfg) >= kv


@pytest.mark.parametrize("field,value", [
    ("head_dim", 96), ("n_kv_heads", 3), ("n_heads", 32), ("max_group", 5), ("max_group", 0), ("stop_mode", 7),
    ("dtype", 3), ("max_batch", 0), ("max_batch", 65), ("ffn_dim", 700), ("d_model", 100), ("vocab", 1),
    ("stop_conf", 1.5), ("micro_layers", 0), ("max_prompt", 0), ("norm_eps", 0.0)])
def test_invalid_configs_are_rejected(lib, field, value):
    cfg = config_for(TINY, 1, 8, 4)
    setattr(cfg, field, value)
    assert ham.ham_weights_bytes(cfg) == 0
    h = ctypes.c_void_p()
    rc = lib.ham_init_weights(ctypes.byref(cfg), 1, 256, 1 << 30, 256, 1 << 30, 256, 1 << 30, None, ctypes.byref(h))
    assert rc == ham.HAM_EINVAL and h.value is None
    assert len(lib.ham_last_error()) > 0


@pytest.mark.parametrize("n,layers,ok", [
    (0, [], True), (1, [2], True), (2, [1, 2], True), (2, [2, 1], False), (2, [1, 1], False),
    (1, [0], False), (1, [3], False), (9, [1] * 8, False), (-1, [], False)])
def test_context_layer_sets_are_validated(lib, n, layers, ok):
    # the micro decoder's context layers (Sec. 3.3): 1-based, strictly increasing, within the base depth
    cfg = config_for(TINY, 1, 8, 4)   # two base layers
    cfg.n_ctx_layers = n
    for i, l in enumerate(layers):
        cfg.ctx_layers[i] = l
    assert (ham.ham_weights_bytes(cfg) > 0) == ok


def test_embedder_is_one_layer(lib):
    cfg = config_for(TINY, 1, 8, 4)
    for v, ok in ((0, True), (1, True), (2, False)):
        cfg.embed_layers = v
        assert (ham.ham_weights_bytes(cfg) > 0) == ok


def test_more_context_layers_grow_the_micro_workspace(lib):
    base = config_for(SHAPE_1B, 4, 64, 8)
    more = config_for(SHAPE_1B, 4, 64, 8)
    more.n_ctx_layers = 8
    for i in range(8):
        more.ctx_layers[i] = 2 * i + 1
    assert ham.ham_workspace_bytes(more) > ham.ham_workspace_bytes(base)


def test_op_attention_step_rejects_bad_shapes(lib):
    ws = ham.ham_op_attention_workspace_bytes(4, 32, 8, 128)
    assert ham.ham_op_attention_step_splits(1, 4, 8, 128, 33791) == 8
    assert ham.ham_op_attention_step_splits(1, 32, 8, 128, 2559) == 1
    assert ham.ham_op_attention_step_splits(1, 1, 8, 64, 1023) == 16
    assert ham.ham_op_attention_step_splits(5, 1, 8, 64, 1023) == 0
    args = lambda rows, hd, S, cap, wsb: (1, rows, 32, 8, hd, S, *([256] * 8), cap, 256, 256, 256, wsb, None)  # noqa: E731
    assert lib.ham_op_attention_step(*args(4, 96, 33792, 100, ws)) == ham.HAM_EINVAL        # head dim
    assert lib.ham_op_attention_step(*args(4, 128, 100, 10, ws)) == ham.HAM_EINVAL          # slots not /64
    assert lib.ham_op_attention_step(*args(4, 128, 33792, 33792, ws)) == ham.HAM_EINVAL     # kv_cap >= slots
    assert lib.ham_op_attention_step(*args(65, 128, 33792, 100, ws)) == ham.HAM_EINVAL      # rows
    assert lib.ham_op_attention_step(*args(4, 128, 33792, 100, 16)) == ham.HAM_ENOMEM       # workspace
    a = list(args(4, 128, 33792, 100, ws))
    a[8] = None   # no sin table
    assert lib.ham_op_attention_step(*a) == ham.HAM_EINVAL


def test_token_mode_stop_id_must_be_in_vocab(lib):
    cfg = config_for(TINY, 1, 8, 4)
    cfg.stop_id = TINY.vocab
    assert ham.ham_weights_bytes(cfg) == 0


def test_null_and_small_buffers(lib):
    cfg = config_for(TINY, 1, 8, 4)
    h = ctypes.c_void_p()
    assert lib.ham_init_weights(ctypes.byref(cfg), 1, None, 0, None, 0, None, 0, None, ctypes.byref(h)) == ham.HAM_EINVAL
    rc = lib.ham_init_weights(ctypes.byref(cfg), 1, 256, 16, 256, 16, 256, 16, None, ctypes.byref(h))
    assert rc == ham.HAM_ENOMEM
    assert b"too small" in lib.ham_last_error()
    rc = lib.ham_init_weights(ctypes.byref(cfg), 1, 257, 1 << 40, 256, 1 << 40, 256, 1 << 40, None, ctypes.byref(h))
    assert rc == ham.HAM_EINVAL  # misaligned


def test_calls_on_null_handle(lib):
    assert lib.ham_macro_step(None, None, None, None, None) == ham.HAM_EINVAL
    assert lib.ham_prefill(None, 1, None, 1, None, None, None, None, None) == ham.HAM_EINVAL
    assert lib.ham_kv_stats(None, None) == ham.HAM_EINVAL
    assert lib.ham_prefill_embeds(None, 1, None, None, 1, None, None, None, None, None) == ham.HAM_EINVAL
    assert lib.ham_set_graph(None, 1) == ham.HAM_EINVAL
    assert lib.ham_steps_done(None) == -1
    lib.ham_destroy(None)


def test_tensor_info_layout(lib):
    cfg = config_for(TINY, 1, 8, 4)
    total = ham.ham_weights_bytes(cfg)
    ids = list(range(9)) + [16 + 8 * j + t for j in range(TINY.n_layers + TINY.micro_layers) for t in range(7)]
    info = {tid: ham.ham_tensor_info(cfg, tid) for tid in ids}
    for tid, t in info.items():
        assert t["offset"] % 256 == 0
        assert t["offset"] + t["mat_rows"] * t["cols"] * 4 <= total
        assert t["row_off"] + t["rows"] <= t["mat_rows"] or t["interleave"]
    assert (info[0]["rows"], info[0]["cols"], info[0]["tiled"]) == (TINY.vocab, TINY.d_model, 0)
    assert info[7]["tiled"] == 1 and info[8]["row_off"] == TINY.vocab      # stop head = extra LM-head row
    wg, wu = info[16 + 4], info[16 + 5]
    assert wg["offset"] == wu["offset"] and (wg["interleave"], wu["interleave"]) == (1, 2)
    assert wg["mat_rows"] == 2 * TINY.ffn_dim
    with pytest.raises(ham.HamError):
        ham.ham_tensor_info(cfg, 12)
    with pytest.raises(ham.HamError):
        ham.ham_tensor_info(cfg, 16 + 8 * 3)


def test_op_attention_rejects_bad_shapes(lib):
    assert ham.ham_op_attention_workspace_bytes(1, 32, 8, 128) > 0
    ws = 1 << 20
    rc = lib.ham_op_decode_attention(1, 1, 32, 8, 96, 64, 256, 256, 256, 256, 256, 8, 256, 256, ws, None)
    assert rc == ham.HAM_EINVAL
    rc = lib.ham_op_decode_attention(1, 1, 32, 8, 128, 100, 256, 256, 256, 256, 256, 8, 256, 256, ws, None)
    assert rc == ham.HAM_EINVAL
    rc = lib.ham_op_decode_attention(1, 4, 32, 8, 128, 4096, 256, 256, 256, 256, 256, 8, 256, 256, 16, None)
    assert rc == ham.HAM_ENOMEM


def test_state_info_layout(lib):
    cfg = config_for(TINY, 2, 64, 128)
    total = ham.ham_state_bytes(cfg)
    es = 4  # fp32 model
    infos = [ham.ham_state_info(cfg, l) for l in range(TINY.n_layers)]
    S = infos[0]["slots"]
    assert S % 64 == 0 and S >= 64 + 128
    per_layer = 2 * TINY.n_kv_heads * S * TINY.head_dim * es
    spans = []
    for i in infos:
        assert i["slots"] == S and i["k_offset"] % 256 == 0 and i["v_offset"] % 256 == 0
        spans += [(i["k_offset"], i["k_offset"] + per_layer), (i["v_offset"], i["v_offset"] + per_layer)]
    spans.sort()
    assert spans[-1][1] <= total
    assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))   # K and V of all layers are disjoint
    with pytest.raises(ham.HamError):
        ham.ham_state_info(cfg, TINY.n_layers)
    with pytest.raises(ham.HamError):
        ham.ham_state_info(cfg, -1)
