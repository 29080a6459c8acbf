"""Host-side checks of the C ABI: exports, canonical weights, config validation.

These load the real libclover.so but make no compute calls (no GPU needed).
"""
import ctypes
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2405_00263_amd", "libclover.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libclover.so not built")


def _declared():
    txt = open(os.path.join(ROOT, "include", "clover.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(clover_[a-z_0-9]+)\s*\(", txt)))


def test_every_declared_symbol_is_exported():
    import paper_2405_00263_amd as P
    L = P.lib()
    names = _declared()
    assert len(names) >= 25
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(P.EXPORTS)


VARIANTS = [(n, {}) for n in synth.CONFIGS] + [
    ("tiny_fp32", {"regressive": "mlp"}), ("llama7b_b1", {"regressive": "mlp", "ab": "none"}),
    ("tiny_fp32", {"ad_per_head": True}), ("large_gqa_b1", {"ab": "attn"}),
    ("llama7b_b1_medusa", {"medusa_lm": "per_head"}), ("tiny_fp32_medusa", {"medusa_lm": "per_head", "ab": "full"})]


@pytest.mark.parametrize("name,kw", VARIANTS)
def test_weight_list_matches_synth(name, kw):
    import paper_2405_00263_amd as P
    cfg = synth.get_config(name).with_(**kw)
    c = P.make_config(cfg)
    specs = synth.weight_specs(cfg)
    assert P.weight_names(c) == [n for n, _ in specs]
    assert P.weight_shapes(c) == [tuple(s) for _, s in specs]
    es = 2 if cfg.dtype == "bf16" else 4
    L = P.lib()
    for i, (_, shp) in enumerate(specs):
        n = 1
        for s in shp:
            n *= s
        assert L.clover_packed_bytes(ctypes.byref(c), i) == n * es


def test_workspace_sizes_fit_one_device():
    import paper_2405_00263_amd as P
    for name in synth.CONFIGS:
        cfg = synth.get_config(name)
        ws = P.workspace_bytes(P.make_config(cfg))
        assert 0 < ws < 100 * 2 ** 30, (name, ws)


@pytest.mark.parametrize("field,value", [("head_dim", 48), ("n_kv_heads", 3), ("d_model", 100),
                                         ("tree_tokens", 200), ("vocab", 1000), ("kv_block", 32),
                                         ("ffn_dim", 40), ("max_batch", 0), ("prefill_chunk", 100),
                                         ("draft_mode", 2), ("draft_mode", -1)])
def test_invalid_config_rejected(field, value):
    import paper_2405_00263_amd as P
    c = P.make_config(synth.get_config("tiny_fp32"))
    setattr(c, field, value)
    L = P.lib()
    assert L.clover_check_config(ctypes.byref(c)) == 1
    assert L.clover_last_error(None)
    assert L.clover_workspace_bytes(ctypes.byref(c)) == 0


def test_tree_larger_than_candidates_rejected():
    import paper_2405_00263_amd as P
    c = P.make_config(synth.get_config("tiny_fp32").with_(topk=(2, 2), tree_tokens=8))
    assert P.lib().clover_check_config(ctypes.byref(c)) == 1
    c = P.make_config(synth.get_config("tiny_fp32").with_(topk=(2, 2), tree_tokens=7))
    assert P.lib().clover_check_config(ctypes.byref(c)) == 0


def test_init_rejects_bad_arguments_before_device_work():
    import paper_2405_00263_amd as P
    L = P.lib()
    c = P.make_config(synth.get_config("tiny_fp32"))
    ctx = ctypes.c_void_p()
    assert L.clover_init(ctypes.byref(c), None, None, 0, None, ctypes.byref(ctx)) == 1
    n = L.clover_weight_count(ctypes.byref(c))
    ptrs = (ctypes.c_void_p * n)(*([1] * n))
    # workspace too small: capacity error, no device call made
    assert L.clover_init(ctypes.byref(c), ptrs, ctypes.c_void_p(1), 16, None, ctypes.byref(ctx)) == 2
    assert b"workspace" in L.clover_last_error(None)
    assert not ctx.value


def test_op_entry_points_validate():
    import paper_2405_00263_amd as P
    L = P.lib()
    assert L.clover_op_scratch_bytes(1, 64, 4096, 4096) > 0
    assert L.clover_op_scratch_bytes(1, 64, 4100, 4096) == 0      # N not a multiple of 16
    assert L.clover_op_scratch_bytes(1, 64, 4096, 4016) == 0      # K not a multiple of 32
    assert L.clover_packed_matrix_bytes(0, 32, 48) == 32 * 48 * 4
    assert L.clover_op_attention_scratch_bytes(1, 100, 64, 32, 8, 128) > 0
    assert L.clover_op_attention_scratch_bytes(1, 100, 64, 32, 7, 128) == 0
    assert L.clover_op_topk(None, 1, 10, 3, None, None, None, None) == 1
    assert L.clover_op_topk_scratch_bytes(4, 125696, 16) > 0
    assert L.clover_op_topk_scratch_bytes(4, 125696, 17) == 0
    # gated MLP: sizes a model may take, no null operands; rejected before any device call
    one = ctypes.c_void_p(1)
    assert L.clover_op_swiglu(1, one, 64, 4096, one, one, 11008 + 16, one, None) == 1  # F not a multiple of 32 (bf16)
    assert L.clover_op_swiglu(1, one, 64, 4016, one, one, 11008, one, None) == 1       # K not a multiple of 32
    assert L.clover_op_swiglu(0, one, 0, 256, one, one, 688, one, None) == 1           # no rows
    assert L.clover_op_swiglu(1, one, 64, 4096, None, one, 11008, one, None) == 1      # null gate
    assert L.clover_op_swiglu(2, one, 64, 4096, one, one, 11008, one, None) == 1       # unknown dtype
    assert b"op_swiglu" in L.clover_last_error(None)
