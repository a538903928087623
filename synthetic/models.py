"""Decoder shapes, synthetic random-init weights, prompts and page tables.

Model shapes are the decoder-only Llama/Qwen-style families that the paper's
compiler emits and benchmarks (Results, Experimental Setup; the Python-overhead
study in the Technical Supplement uses Qwen2.5-0.5B and Pleias-3b).  There are
no checkpoints here: every tensor is drawn from a per-tensor seeded generator.

Recipe (also stated in the design notes):
  * a tensor named ``name`` uses the seed ``crc32(name) ^ (seed << 32)``;
  * linear, embedding and bias tensors are 0.02 * N(0, 1);
  * RMSNorm and LayerNorm gains are 1 + 0.02 * N(0, 1) (a literal N(0, 0.02) gain would
    shrink every activation fifty-fold and make the logits nearly constant);
  * values are drawn in float32 with ``torch.randn`` on the requested device
    and rounded to bfloat16 (round-to-nearest-even) for the bf16 models; that
    rounded value is the weight for both the oracle and the GPU path;
  * prompts are uniform token ids, ``torch.randint`` with seed 0 on the CPU.

``torch.randn`` draws different streams on CPU and GPU for one seed, so a test
draws a model once, on one device, and copies it to wherever it is needed.
"""
from __future__ import annotations

import zlib

import torch

# HF-style keys, matching the ``Config.dim @@hidden_size`` lookups of the
# paper's built-in Config module.
MODEL_SHAPES = {
    "135m": dict(hidden_size=576, num_hidden_layers=30, num_attention_heads=9,
                 num_key_value_heads=3, head_dim=64, intermediate_size=1536,
                 vocab_size=49152, tie_word_embeddings=True, attention_bias=False,
                 rms_norm_eps=1e-5, rope_theta=10000.0, dtype="f32"),
    "1b": dict(hidden_size=2048, num_hidden_layers=16, num_attention_heads=32,
               num_key_value_heads=8, head_dim=64, intermediate_size=8192,
               vocab_size=128256, tie_word_embeddings=True, attention_bias=False,
               rms_norm_eps=1e-5, rope_theta=500000.0, dtype="bf16"),
    "7b": dict(hidden_size=3584, num_hidden_layers=28, num_attention_heads=28,
               num_key_value_heads=4, head_dim=128, intermediate_size=18944,
               vocab_size=152064, tie_word_embeddings=False, attention_bias=True,
               rms_norm_eps=1e-6, rope_theta=1000000.0, dtype="bf16"),
    "32b": dict(hidden_size=5120, num_hidden_layers=64, num_attention_heads=40,
                num_key_value_heads=8, head_dim=128, intermediate_size=27648,
                vocab_size=152064, tie_word_embeddings=False, attention_bias=True,
                rms_norm_eps=1e-6, rope_theta=1000000.0, dtype="bf16"),
    # DeepSeek-MoE-16B-shaped (the MoE model of the paper's 4-32B benchmark):
    # layer 0 dense (intermediate 10944), layers 1..27 with 64 routed experts
    # (top 6, intermediate 1408, no renormalization) + 2 shared experts
    "moe16b": dict(hidden_size=2048, num_hidden_layers=28, num_attention_heads=16,
                   num_key_value_heads=16, head_dim=128, intermediate_size=10944,
                   vocab_size=102400, tie_word_embeddings=False, attention_bias=False,
                   rms_norm_eps=1e-6, rope_theta=10000.0, dtype="bf16",
                   n_routed_experts=64, num_experts_per_tok=6, moe_intermediate_size=1408,
                   n_shared_experts=2, first_k_dense_replace=1, norm_topk_prob=False),
    # the GPT-2 definition of the paper's complete-model listing (LayerNorm,
    # learned positions, fused c_attn, GELU MLP, biases, tied head), XL size
    "gpt2xl": dict(model_type="gpt2", hidden_size=1600, num_hidden_layers=48, num_attention_heads=25,
                   num_key_value_heads=25, head_dim=64, intermediate_size=6400, vocab_size=50257,
                   max_position_embeddings=1024, tie_word_embeddings=True, attention_bias=True,
                   layer_norm_epsilon=1e-5, dtype="bf16"),
    "gpt2": dict(model_type="gpt2", hidden_size=768, num_hidden_layers=12, num_attention_heads=12,
                 num_key_value_heads=12, head_dim=64, intermediate_size=3072, vocab_size=50257,
                 max_position_embeddings=1024, tie_word_embeddings=True, attention_bias=True,
                 layer_norm_epsilon=1e-5, dtype="bf16"),
    # Mistral-7B-shaped: sliding-window attention over the last 4096 keys
    "mistral7b": dict(hidden_size=4096, num_hidden_layers=32, num_attention_heads=32,
                      num_key_value_heads=8, head_dim=128, intermediate_size=14336,
                      vocab_size=32000, tie_word_embeddings=False, attention_bias=False,
                      rms_norm_eps=1e-5, rope_theta=10000.0, dtype="bf16", sliding_window=4096),
}


def is_gpt2(shape: dict) -> bool:
    return shape.get("model_type") == "gpt2"


def is_moe_layer(shape: dict, i: int) -> bool:
    return bool(shape.get("n_routed_experts")) and i >= int(shape.get("first_k_dense_replace") or 0)

# The five workloads: model shape, batch, prompt length, greedy decode steps,
# KV-cache kind.  "7b_paged" has per-sequence prompt lengths drawn uniformly in
# [64, 4096] and a randomly permuted page table with 16-token pages.
WORKLOADS = {
    "135m": dict(model="135m", batch=1, prompt_len=32, steps=16, paged=False),
    "1b": dict(model="1b", batch=8, prompt_len=512, steps=128, paged=False),
    "7b": dict(model="7b", batch=16, prompt_len=2048, steps=256, paged=False),
    "7b_paged": dict(model="7b", batch=64, prompt_len=None, len_range=(64, 4096),
                     steps=128, paged=True, page_size=16),
    "32b": dict(model="32b", batch=32, prompt_len=1024, steps=256, paged=False),
    # the DeepSeek-MoE-16B shape: routed experts through grouped GEMMs
    "moe16b": dict(model="moe16b", batch=32, prompt_len=1024, steps=128, paged=False),
    # a training step (forward, mean next-token cross-entropy, every weight's
    # gradient) over the 1B workload's 8 x 512 prompts
    "1b_train": dict(model="1b", batch=8, prompt_len=512, steps=0, paged=False, train=True),
    # GPT-2 XL (the largest checkpoint of the paper's GPT-2 listing), the 1B
    # workload's batch, prompt and decode lengths
    "gpt2xl": dict(model="gpt2xl", batch=8, prompt_len=512, steps=128, paged=False),
    # Mistral-7B shape with its 4096-key sliding window: prompts twice the
    # window, so prefill attention and every decode step see the window
    "mistral7b": dict(model="mistral7b", batch=16, prompt_len=8192, steps=128, paged=False),
    # the 7b_paged requests served by continuous batching: every step carries
    # the running sequences' decode tokens plus prompt chunks of the waiting
    # ones, up to a token budget
    "7b_serve": dict(model="7b", batch=64, prompt_len=None, len_range=(64, 4096),
                     steps=128, paged=True, page_size=16, serve=True, step_tokens=8192),
}


def small_shape(base: str, layers: int, vocab: int, intermediate: int | None = None,
                hidden: int | None = None, dtype: str | None = None) -> dict:
    """A reduced copy of a named shape: fewer layers, a smaller vocabulary,
    optionally a narrower MLP/hidden size, every head geometry kept."""
    s = dict(MODEL_SHAPES[base])
    s["num_hidden_layers"] = layers
    s["vocab_size"] = vocab
    if intermediate is not None:
        s["intermediate_size"] = intermediate
    if hidden is not None:
        s["hidden_size"] = hidden
    if dtype is not None:
        s["dtype"] = dtype
    return s


def weight_names(shape: dict) -> list[str]:
    """Flat, path-keyed weight names (the ``_param("layers.0.self_attn...")``
    convention of the generated code), HF Llama/Qwen2 layout, or HF GPT-2's."""
    if is_gpt2(shape):
        names = ["transformer.wte.weight", "transformer.wpe.weight"]
        for i in range(shape["num_hidden_layers"]):
            p = f"transformer.h.{i}."
            for part in ("ln_1", "attn.c_attn", "attn.c_proj", "ln_2", "mlp.c_fc", "mlp.c_proj"):
                names += [p + part + ".weight", p + part + ".bias"]
        return names + ["transformer.ln_f.weight", "transformer.ln_f.bias"]
    names = ["model.embed_tokens.weight"]
    for i in range(shape["num_hidden_layers"]):
        p = f"model.layers.{i}."
        names += [p + "input_layernorm.weight"]
        for x in ("q", "k", "v"):
            names.append(p + f"self_attn.{x}_proj.weight")
            if shape["attention_bias"]:
                names.append(p + f"self_attn.{x}_proj.bias")
        names += [p + "self_attn.o_proj.weight", p + "post_attention_layernorm.weight"]
        if is_moe_layer(shape, i):
            names.append(p + "mlp.gate.weight")
            for e in range(shape["n_routed_experts"]):
                names += [p + f"mlp.experts.{e}.{x}_proj.weight" for x in ("gate", "up", "down")]
            if shape.get("n_shared_experts"):
                names += [p + f"mlp.shared_experts.{x}_proj.weight" for x in ("gate", "up", "down")]
        else:
            names += [p + "mlp.gate_proj.weight", p + "mlp.up_proj.weight", p + "mlp.down_proj.weight"]
    names.append("model.norm.weight")
    if not shape["tie_word_embeddings"]:
        names.append("lm_head.weight")
    return names


def _gpt2_shape(n: str, D: int, I: int, V: int, P: int) -> tuple:
    # Conv1D weights are stored [in, out]
    if n == "transformer.wte.weight":
        return (V, D)
    if n == "transformer.wpe.weight":
        return (P, D)
    part = n.rsplit(".", 2)[-2] if n.endswith(".weight") or n.endswith(".bias") else ""
    full = n.rsplit(".", 1)[0]
    ins, outs = {"c_attn": (D, 3 * D), "c_fc": (D, I)}.get(part, (None, None))
    if full.endswith("mlp.c_proj"):
        ins, outs = I, D
    elif full.endswith("attn.c_proj"):
        ins, outs = D, D
    if ins is None:  # ln_1, ln_2, ln_f
        return (D,)
    return (ins, outs) if n.endswith(".weight") else (outs,)


def weight_shapes(shape: dict) -> dict[str, tuple]:
    D, H, KV = shape["hidden_size"], shape["num_attention_heads"], shape["num_key_value_heads"]
    hd, I, V = shape["head_dim"], shape["intermediate_size"], shape["vocab_size"]
    if is_gpt2(shape):
        return {n: _gpt2_shape(n, D, I, V, shape["max_position_embeddings"]) for n in weight_names(shape)}
    out = {}
    for n in weight_names(shape):
        if n.endswith("embed_tokens.weight") or n == "lm_head.weight":
            out[n] = (V, D)
        elif n.endswith("layernorm.weight") or n == "model.norm.weight":
            out[n] = (D,)
        elif n.endswith("q_proj.weight"):
            out[n] = (H * hd, D)
        elif n.endswith("k_proj.weight") or n.endswith("v_proj.weight"):
            out[n] = (KV * hd, D)
        elif n.endswith("q_proj.bias"):
            out[n] = (H * hd,)
        elif n.endswith("k_proj.bias") or n.endswith("v_proj.bias"):
            out[n] = (KV * hd,)
        elif n.endswith("o_proj.weight"):
            out[n] = (D, H * hd)
        elif n.endswith("mlp.gate.weight"):
            out[n] = (shape["n_routed_experts"], D)
        elif n.endswith("gate_proj.weight") or n.endswith("up_proj.weight") or n.endswith("down_proj.weight"):
            ii = I
            if ".mlp.experts." in n:
                ii = shape["moe_intermediate_size"]
            elif ".mlp.shared_experts." in n:
                ii = shape["moe_intermediate_size"] * shape["n_shared_experts"]
            out[n] = (D, ii) if n.endswith("down_proj.weight") else (ii, D)
        else:  # pragma: no cover
            raise KeyError(n)
    return out


def _is_gain(name: str) -> bool:
    """Norm gains (1 + 0.02 N): RMSNorm weights and LayerNorm weights (the
    LayerNorm biases are drawn like any bias)."""
    return (name.endswith("layernorm.weight") or name == "model.norm.weight"
            or (".ln_" in name and name.endswith(".weight")))


def _seed(name: str, seed: int) -> int:
    return (zlib.crc32(name.encode()) ^ (seed << 32)) & ((1 << 63) - 1)


def model_weights(shape: dict, seed: int = 0, device: str = "cpu") -> dict[str, torch.Tensor]:
    """Random-init weights for ``shape`` as torch tensors in the model dtype
    (bfloat16 or float32) on ``device``."""
    dt = torch.bfloat16 if shape["dtype"] == "bf16" else torch.float32
    out = {}
    for name, shp in weight_shapes(shape).items():
        g = torch.Generator(device=device)
        g.manual_seed(_seed(name, seed))
        w = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
        w.mul_(0.02)
        if _is_gain(name):
            w.add_(1.0)
        out[name] = w.to(dt)
    return out


def prompts(batch: int, length: int, vocab: int, seed: int = 0) -> torch.Tensor:
    """Uniform random token ids, int32 [batch, length], drawn on the CPU."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return torch.randint(0, vocab, (batch, length), generator=g, dtype=torch.int64).to(torch.int32)


def paged_workload(batch: int, len_lo: int, len_hi: int, steps: int, vocab: int,
                   page_size: int, seed: int = 0, spare_pages: int = 0):
    """Variable-length prompts and a randomly permuted page table.

    Returns (list of int32 prompt tensors, block_table int32 [batch, max_blocks]
    with -1 padding, number of pages in the pool).  Each sequence gets exactly
    enough pages for its prompt plus ``steps`` decode tokens; the pool is a
    random permutation of all pages, dealt out to the logical blocks in order.
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    lens = torch.randint(len_lo, len_hi + 1, (batch,), generator=g, dtype=torch.int64)
    seqs = [torch.randint(0, vocab, (int(n),), generator=g, dtype=torch.int64).to(torch.int32)
            for n in lens]
    need = [-(-(int(n) + steps) // page_size) for n in lens]
    pool = sum(need) + spare_pages
    perm = torch.randperm(pool, generator=g, dtype=torch.int64)
    max_blocks = max(need)
    table = torch.full((batch, max_blocks), -1, dtype=torch.int32)
    k = 0
    for b, nb in enumerate(need):
        table[b, :nb] = perm[k:k + nb].to(torch.int32)
        k += nb
    return seqs, table, pool
