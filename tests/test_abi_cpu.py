"""The C-ABI library on the CPU: it loads, exports every function that
include/axon.h declares, and rejects every malformed configuration and weight
map on the host (validation runs before any HIP call, so these tests need no
GPU)."""
import ctypes
import os
import re
import subprocess

import pytest
import torch

from paper_2608_19889_amd import axon
from synthetic import small_shape, weight_shapes

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(axon_\w+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    lib = axon.lib()
    declared = _declared_functions()
    assert {"axon_init_model", "axon_prefill", "axon_decode_step", "axon_free"} <= declared
    for name in declared:
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", axon.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\b(axon_\w+)$", out, flags=re.M))
    assert declared == exported, (declared ^ exported)


def test_struct_layout_matches_header():
    assert ctypes.sizeof(axon.AxonConfig) == 112
    assert axon.AxonConfig.n_experts.offset == 72 and axon.AxonConfig.norm_topk_prob.offset == 92
    assert axon.AxonConfig.sliding_window.offset == 96 and axon.AxonConfig.max_positions.offset == 104
    assert axon.AxonConfig.rope_theta.offset == 32
    assert ctypes.sizeof(axon.AxonWeight) == 48


def test_struct_layout_matches_the_c_compiler(tmp_path):
    """Offsets of every axon_config / axon_weight field as gcc lays out the
    header, against the ctypes mirror."""
    fields = {"axon_config": [f for f, _ in axon.AxonConfig._fields_],
              "axon_weight": [f for f, _ in axon.AxonWeight._fields_]}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "axon.h"', "int main(void) {"]
    for st, names in fields.items():
        lines.append(f'  printf("{st} size %zu\\n", sizeof({st}));')
        lines += [f'  printf("{st} {n} %zu\\n", offsetof({st}, {n}));' for n in names]
    lines.append("  return 0;\n}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {tuple(line.split()[:2]): int(line.split()[2]) for line in out if line}
    for st, cls in (("axon_config", axon.AxonConfig), ("axon_weight", axon.AxonWeight)):
        assert got[(st, "size")] == ctypes.sizeof(cls)
        for n in fields[st]:
            assert got[(st, n)] == getattr(cls, n).offset, (st, n)


def _shape():
    s = small_shape("7b", layers=2, vocab=256, intermediate=128, hidden=128, dtype="bf16")
    s.update(num_attention_heads=4, num_key_value_heads=2, head_dim=64)
    return s


def _fake_weights(shape, dtype=torch.bfloat16):
    # validation never reads weight data: tiny placeholder buffers suffice
    return {n: torch.empty(shp, dtype=dtype) for n, shp in weight_shapes(shape).items()}


def _status(shape, weights, **cap):
    cfg = axon.make_config(shape, cap.get("max_batch", 2), cap.get("max_seq", 64),
                           page_size=cap.get("page_size", 0), num_pages=cap.get("num_pages", 0))
    for k, v in cap.get("override", {}).items():
        setattr(cfg, k, v)
    return axon.init_status(cfg, weights)


@pytest.mark.parametrize("field,value,fragment", [
    ("hidden", 100, "hidden"), ("hidden", 0, "hidden"), ("n_layers", 0, "n_layers"),
    ("n_heads", 5, "multiple of n_kv_heads"), ("n_kv_heads", 0, "n_kv_heads"),
    ("head_dim", 96, "head_dim"), ("intermediate", 100, "intermediate"), ("vocab", 0, "vocab"),
    ("rms_eps", 0.0, "rms_eps"), ("rope_theta", 1.0, "rope_theta"), ("dtype", 7, "dtype"),
    ("max_batch", 0, "max_batch"), ("max_seq", 0, "max_seq"), ("max_tokens", -1, "max_tokens"),
    ("kv_page_size", 8, "kv_page_size"), ("qkv_bias", 2, "qkv_bias")])
def test_bad_config_is_rejected(field, value, fragment):
    s = _shape()
    rc, msg = _status(s, _fake_weights(s), override={field: value})
    assert rc == axon.AXON_E_INVALID and fragment in msg, (rc, msg)


def test_group_size_limit_and_paged_needs_pages():
    s = _shape()
    rc, msg = _status(s, _fake_weights(s), override={"n_heads": 34, "n_kv_heads": 2})
    assert rc == axon.AXON_E_INVALID and "<= 16" in msg
    # 13 query heads of 128 dims per kv head: within 16 heads, past 1536 dims
    rc, msg = _status(s, _fake_weights(s), override={"n_heads": 26, "n_kv_heads": 2, "head_dim": 128})
    assert rc == axon.AXON_E_INVALID and "1536" in msg
    rc, msg = _status(s, _fake_weights(s), page_size=16, num_pages=0)
    assert rc == axon.AXON_E_INVALID and "kv_num_pages" in msg


def test_missing_weight():
    s = _shape()
    w = _fake_weights(s)
    del w["model.layers.1.self_attn.k_proj.bias"]
    rc, msg = _status(s, w)
    assert rc == axon.AXON_E_MISSING and "model.layers.1.self_attn.k_proj.bias" in msg


def test_unknown_and_duplicate_weight():
    s = _shape()
    w = _fake_weights(s)
    w["model.layers.0.self_attn.o_proj.bias"] = torch.empty(128, dtype=torch.bfloat16)
    rc, msg = _status(s, w)
    assert rc == axon.AXON_E_MISSING and "unknown" in msg and "o_proj.bias" in msg
    # a tied model must not carry lm_head.weight
    t = dict(s, tie_word_embeddings=True)
    w = _fake_weights(dict(s, tie_word_embeddings=False))
    rc, msg = _status(t, w)
    assert rc == axon.AXON_E_MISSING and "lm_head.weight" in msg and "tie" in msg
    # duplicates: pass the same name twice through the raw array
    w = _fake_weights(s)
    arr, keep = axon.make_weights(w)
    arr2 = (axon.AxonWeight * (len(w) + 1))(*arr, arr[0])
    cfg = axon.make_config(s, 2, 64)
    h = ctypes.c_void_p()
    rc = axon.lib().axon_init_model(ctypes.byref(cfg), arr2, len(w) + 1, None, ctypes.byref(h))
    assert rc == axon.AXON_E_MISSING and "duplicate" in axon.last_error()
    assert not h.value


@pytest.mark.parametrize("name,bad", [
    ("model.layers.0.self_attn.q_proj.weight", (4 * 64, 127)),
    ("model.layers.1.mlp.down_proj.weight", (128, 128 * 2)),
    ("model.embed_tokens.weight", (255, 128)),
    ("model.norm.weight", (128, 1)),
])
def test_wrong_shape_names_tensor_and_shapes(name, bad):
    s = _shape()
    w = _fake_weights(s)
    w[name] = torch.empty(bad, dtype=torch.bfloat16)
    rc, msg = _status(s, w)
    assert rc == axon.AXON_E_SHAPE and name in msg and "expected" in msg, msg


def test_wrong_dtype():
    s = _shape()
    w = _fake_weights(s)
    w["model.layers.0.mlp.up_proj.weight"] = torch.empty((128, 128), dtype=torch.float32)
    rc, msg = _status(s, w)
    assert rc == axon.AXON_E_DTYPE and "up_proj" in msg


def test_null_arguments():
    s = _shape()
    cfg = axon.make_config(s, 2, 64)
    h = ctypes.c_void_p()
    L = axon.lib()
    assert L.axon_init_model(None, None, 0, None, ctypes.byref(h)) == axon.AXON_E_INVALID
    assert L.axon_init_model(ctypes.byref(cfg), None, 0, None, None) == axon.AXON_E_INVALID
    assert L.axon_init_model(ctypes.byref(cfg), None, -1, None, ctypes.byref(h)) == axon.AXON_E_INVALID
    assert L.axon_prefill(None, 1, None, None, None, None, 0, 0, None, None, None) == axon.AXON_E_INVALID
    assert L.axon_decode_step(None, 1, None, None, None, None) == axon.AXON_E_INVALID
    assert L.axon_decode_step_noalloc(None, 1, None, None, None, None) == axon.AXON_E_INVALID
    assert L.axon_slot_lengths(None, None, 0) == axon.AXON_E_INVALID
    L.axon_free(None)  # NULL-safe
    w = _fake_weights(s)
    w["model.norm.weight"] = torch.empty(0, dtype=torch.bfloat16)
    arr, keep = axon.make_weights(w)
    for i in range(len(w)):
        if arr[i].name == b"model.norm.weight":
            arr[i].shape[0] = 128
            arr[i].data = None
    rc = L.axon_init_model(ctypes.byref(cfg), arr, len(w), None, ctypes.byref(h))
    assert rc == axon.AXON_E_INVALID and "NULL data" in axon.last_error()


def test_no_cpu_fallback_in_binding():
    """The binding only marshals arguments: it contains no torch compute."""
    src = open(os.path.join(ROOT, "paper_2608_19889_amd", "axon.py")).read()
    for forbidden in ("oracle", "torch.matmul", "softmax", "F.linear", "@ "):
        assert forbidden not in src, forbidden


def test_step_and_reset_reject_a_null_model():
    """The continuous-batching calls validate on the host before touching a GPU."""
    lib = axon.lib()
    cu = (ctypes.c_int32 * 2)(0, 1)
    sl = (ctypes.c_int32 * 1)(0)
    rc = lib.axon_step(None, 1, sl, None, None, None, cu, None, 0, None, None, None)
    assert rc == axon.AXON_E_INVALID and "NULL" in axon.last_error()
    assert lib.axon_reset_slot(None, 0) == axon.AXON_E_INVALID


def _moe_shape(**kw):
    s = _shape()
    s.update(n_routed_experts=4, num_experts_per_tok=2, moe_intermediate_size=64, n_shared_experts=1,
             first_k_dense_replace=1, norm_topk_prob=False)
    s.update(kw)
    return s


@pytest.mark.parametrize("field,value,fragment", [
    ("n_experts", 1, "n_experts"), ("n_experts", 300, "n_experts"), ("top_k", 0, "top_k"),
    ("top_k", 5, "top_k"), ("moe_intermediate", 96, "moe_intermediate"), ("n_shared_experts", -1, "n_shared"),
    ("first_moe_layer", 3, "first_moe_layer"), ("norm_topk_prob", 2, "norm_topk_prob"), ("dtype", 2, "AXON_BF16")])
def test_bad_moe_config_is_rejected(field, value, fragment):
    s = _moe_shape()
    rc, msg = _status(s, _fake_weights(s), override={field: value})
    assert rc == axon.AXON_E_INVALID and fragment in msg, (rc, msg)


def test_moe_weight_map_is_checked():
    s = _moe_shape()
    w = _fake_weights(s)
    assert "model.layers.1.mlp.experts.3.up_proj.weight" in w and "model.layers.0.mlp.up_proj.weight" in w
    missing = dict(w)
    del missing["model.layers.1.mlp.experts.3.up_proj.weight"]
    rc, msg = _status(s, missing)
    assert rc == axon.AXON_E_MISSING and "experts.3.up_proj" in msg
    bad = dict(w)
    bad["model.layers.1.mlp.shared_experts.down_proj.weight"] = torch.empty((128, 128), dtype=torch.bfloat16)
    rc, msg = _status(s, bad)
    assert rc == axon.AXON_E_SHAPE and "shared_experts.down_proj" in msg and "[128, 64]" in msg, msg
    dense_names = dict(w)
    dense_names["model.layers.1.mlp.gate_proj.weight"] = torch.empty((128, 128), dtype=torch.bfloat16)
    rc, msg = _status(s, dense_names)
    assert rc == axon.AXON_E_MISSING and "unknown" in msg and "layers.1.mlp.gate_proj" in msg


def _gpt2_shape(**kw):
    s = dict(model_type="gpt2", hidden_size=128, num_hidden_layers=2, num_attention_heads=2, num_key_value_heads=2,
             head_dim=64, intermediate_size=512, vocab_size=256, max_position_embeddings=64,
             tie_word_embeddings=True, attention_bias=True, layer_norm_epsilon=1e-5, dtype="bf16")
    s.update(kw)
    return s


@pytest.mark.parametrize("field,value,fragment", [
    ("n_kv_heads", 1, "n_kv_heads == n_heads"), ("qkv_bias", 0, "qkv_bias == 1"),
    ("tie_embeddings", 0, "tie_embeddings == 1"), ("dtype", 2, "AXON_BF16"), ("max_positions", 32, "max_positions"),
    ("arch", 5, "arch"), ("sliding_window", -1, "sliding_window")])
def test_bad_gpt2_config_is_rejected(field, value, fragment):
    s = _gpt2_shape()
    rc, msg = _status(s, _fake_weights(s), override={field: value})
    assert rc == axon.AXON_E_INVALID and fragment in msg, (rc, msg)


def test_gpt2_weight_map_is_checked():
    s = _gpt2_shape()
    w = _fake_weights(s)
    assert w["transformer.h.1.attn.c_attn.weight"].shape == (128, 384)  # Conv1D [in, out]
    missing = dict(w)
    del missing["transformer.h.1.mlp.c_fc.bias"]
    rc, msg = _status(s, missing)
    assert rc == axon.AXON_E_MISSING and "mlp.c_fc.bias" in msg
    bad = dict(w)
    bad["transformer.h.0.attn.c_attn.weight"] = torch.empty((384, 128), dtype=torch.bfloat16)  # [out, in]
    rc, msg = _status(s, bad)
    assert rc == axon.AXON_E_SHAPE and "c_attn.weight" in msg and "[128, 384]" in msg, msg
    extra = dict(w)
    extra["lm_head.weight"] = torch.empty((256, 128), dtype=torch.bfloat16)  # the head is tied
    rc, msg = _status(s, extra)
    assert rc == axon.AXON_E_MISSING and "lm_head.weight" in msg
    llama_names = dict(w)
    llama_names["model.norm.weight"] = torch.empty(128, dtype=torch.bfloat16)
    rc, msg = _status(s, llama_names)
    assert rc == axon.AXON_E_MISSING and "unknown" in msg


def test_loss_and_grads_rejects_null_arguments():
    """The backward entry point validates on the host before any GPU work."""
    lib = axon.lib()
    cu = (ctypes.c_int32 * 2)(0, 4)
    rc = lib.axon_loss_and_grads(None, 1, None, None, cu, None, None, None, 0, None)
    assert rc == axon.AXON_E_INVALID and "NULL" in axon.last_error()
