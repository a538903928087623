"""Pins of the CPU oracle to facts outside itself.

Each test checks the oracle against a closed form, an invariant of the model
family, brute force on tiny inputs, or an independent library routine (torch's
RMSNorm/SiLU/SDPA, HF transformers' Llama and Qwen2 causal LMs in float64), so
that a dropped term, a wrong sign or index, or a transposed operand anywhere in
the oracle fails at least one of them.  CPU only.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.decoder import OracleDecoder, generate_greedy, teacher_forced
from synthetic import model_weights, small_shape

RNG = np.random.default_rng(1234)


# ----------------------------------------------------------------- RMSNorm

def test_rmsnorm_constant_row_closed_form():
    c, eps = 0.37, 1e-5
    g = RNG.standard_normal(8)
    x = np.full((3, 8), c)
    np.testing.assert_allclose(oracle.rms_norm(x, g, eps), np.broadcast_to(g * c / math.sqrt(c * c + eps), (3, 8)),
                               rtol=1e-14)


def test_rmsnorm_matches_torch_and_is_scale_invariant():
    x = RNG.standard_normal((5, 64))
    g = 1 + 0.1 * RNG.standard_normal(64)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), weight=torch.from_numpy(g), eps=1e-6)
    np.testing.assert_allclose(oracle.rms_norm(x, g, 1e-6), ref.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.rms_norm(7.5 * x, g, 0.0), oracle.rms_norm(x, g, 0.0), rtol=1e-12)
    # eps matters: a tiny-magnitude row is not blown up to unit RMS
    tiny = 1e-4 * x[:1]
    assert np.sqrt(np.mean(oracle.rms_norm(tiny, np.ones(64), 1e-5) ** 2)) < 0.1


# ----------------------------------------------------------------- RoPE

def _rot(x, pos, hd, theta=10000.0):
    c, s = oracle.rope_cos_sin(np.asarray(pos), hd, theta)
    return oracle.apply_rope(x, c, s)


def test_rope_identities():
    hd = 16
    q = RNG.standard_normal((1, 1, hd))
    k = RNG.standard_normal((1, 1, hd))
    np.testing.assert_allclose(_rot(q, [0], hd), q, rtol=0, atol=0)
    for m in (1, 5, 123, 4000):
        np.testing.assert_allclose(np.linalg.norm(_rot(q, [m], hd)), np.linalg.norm(q), rtol=1e-13)
    # R(m) R(n) = R(m + n)
    np.testing.assert_allclose(_rot(_rot(q, [7], hd), [11], hd), _rot(q, [18], hd), atol=1e-13)
    # <R(m) q, R(n) k> = <R(m - n) q, k>
    for m, n in ((9, 4), (100, 37), (4096, 17)):
        lhs = np.sum(_rot(q, [m], hd) * _rot(k, [n], hd))
        rhs = np.sum(_rot(q, [m - n], hd) * k)
        assert abs(lhs - rhs) < 1e-11 * max(1.0, abs(lhs))


def test_rope_matches_transformers_rotate_half():
    """Pairing (i, i + HD/2) and inv_freq = theta^(-2i/HD), as HF's Llama."""
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    hd, theta = 32, 500000.0
    S = 9
    pos = np.arange(3, 3 + S)
    q = RNG.standard_normal((S, 2, hd))
    k = RNG.standard_normal((S, 1, hd))
    inv = theta ** (-np.arange(0, hd, 2, dtype=np.float64) / hd)
    ang = np.outer(pos, inv)
    emb = np.concatenate([ang, ang], axis=-1)
    cos, sin = torch.from_numpy(np.cos(emb))[None], torch.from_numpy(np.sin(emb))[None]
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).permute(1, 0, 2)[None]
    qr, kr = apply_rotary_pos_emb(qt, kt, cos, sin)
    np.testing.assert_allclose(_rot(q, pos, hd, theta), qr[0].permute(1, 0, 2).numpy(), atol=1e-13)
    np.testing.assert_allclose(_rot(k, pos, hd, theta), kr[0].permute(1, 0, 2).numpy(), atol=1e-13)


# ----------------------------------------------------------------- attention

def _brute_attention(q, k, v, q_pos):
    """Explicit loops, one query and head at a time (MHA/GQA by index math)."""
    sq, H, hd = q.shape
    KV = k.shape[1]
    out = np.zeros_like(q)
    for i in range(sq):
        for h in range(H):
            kvh = h * KV // H
            scores = []
            for j in range(q_pos[i] + 1):
                scores.append(sum(q[i, h, d] * k[j, kvh, d] for d in range(hd)) / math.sqrt(hd))
            m = max(scores)
            e = [math.exp(s - m) for s in scores]
            z = sum(e)
            for d in range(hd):
                out[i, h, d] = sum(e[j] / z * v[j, kvh, d] for j in range(len(e)))
    return out


@pytest.mark.parametrize("H,KV,sq,sk", [(4, 2, 5, 9), (3, 3, 4, 4), (6, 2, 1, 7), (2, 1, 9, 9)])
def test_attention_brute_force(H, KV, sq, sk):
    hd = 8
    q = RNG.standard_normal((sq, H, hd))
    k = RNG.standard_normal((sk, KV, hd))
    v = RNG.standard_normal((sk, KV, hd))
    q_pos = np.arange(sk - sq, sk)
    np.testing.assert_allclose(oracle.causal_gqa_attention(q, k, v, q_pos),
                               _brute_attention(q, k, v, q_pos), atol=1e-12)


def test_softmax_rows_sum_to_one_and_special_cases():
    s = RNG.standard_normal((6, 11)) * 30
    s[:, 7:] = -np.inf
    p = oracle.softmax(s)
    assert np.all(np.abs(p.sum(-1) - 1) < 1e-12)
    assert np.all(p[:, 7:] == 0)
    H, KV, S, hd = 4, 2, 7, 8
    q = RNG.standard_normal((S, H, hd))
    k = RNG.standard_normal((S, KV, hd))
    v = RNG.standard_normal((S, KV, hd))
    pos = np.arange(S)
    o = oracle.causal_gqa_attention(q, k, v, pos)
    # the first query sees only key 0: o = v_0 exactly
    np.testing.assert_array_equal(o[0], v[0][np.arange(H) * KV // H])
    # v == 1 everywhere gives 1 (probabilities sum to one)
    np.testing.assert_allclose(oracle.causal_gqa_attention(q, k, np.ones_like(v), pos), 1.0, atol=1e-13)
    # q == 0 gives uniform weights: the running mean of v
    o0 = oracle.causal_gqa_attention(np.zeros_like(q), k, v, pos)
    cm = np.cumsum(v, axis=0) / np.arange(1, S + 1)[:, None, None]
    np.testing.assert_allclose(o0, cm[:, np.arange(H) * KV // H], atol=1e-13)


def test_attention_matches_torch_sdpa_gqa():
    H, KV, S, hd = 6, 2, 13, 16
    q = RNG.standard_normal((S, H, hd))
    k = RNG.standard_normal((S, KV, hd))
    v = RNG.standard_normal((S, KV, hd))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(0, 1)[None], torch.from_numpy(k).transpose(0, 1)[None],
        torch.from_numpy(v).transpose(0, 1)[None], is_causal=True, enable_gqa=True)
    np.testing.assert_allclose(oracle.causal_gqa_attention(q, k, v, np.arange(S)),
                               ref[0].transpose(0, 1).numpy(), atol=1e-12)


def _mha(q, k, v):
    """Separate multi-head routine: one kv head per query head."""
    S, H, hd = q.shape
    out = np.zeros_like(q)
    for h in range(H):
        s = q[:, h] @ k[:, h].T / np.sqrt(hd)
        s[np.triu_indices(S, 1)] = -np.inf
        p = np.exp(s - s.max(-1, keepdims=True))
        out[:, h] = (p / p.sum(-1, keepdims=True)) @ v[:, h]
    return out


def test_gqa_with_kv_equal_heads_is_mha():
    S, H, hd = 10, 5, 8
    q, k, v = (RNG.standard_normal((S, H, hd)) for _ in range(3))
    np.testing.assert_allclose(oracle.causal_gqa_attention(q, k, v, np.arange(S)), _mha(q, k, v),
                               atol=1e-12)


# ----------------------------------------------------------------- MLP

def test_silu_and_swiglu():
    z = np.linspace(-20, 20, 401)
    np.testing.assert_allclose(oracle.silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(),
                               rtol=1e-14, atol=1e-300)
    assert oracle.silu(np.zeros(1))[0] == 0.0
    D, I = 6, 10
    h = RNG.standard_normal((3, D))
    wg, wu, wd = RNG.standard_normal((I, D)), RNG.standard_normal((I, D)), RNG.standard_normal((D, I))
    np.testing.assert_allclose(oracle.swiglu_mlp(h, wg, np.zeros_like(wu), wd), 0.0)
    ref = ((h @ wg.T) / (1 + np.exp(-(h @ wg.T))) * (h @ wu.T)) @ wd.T
    np.testing.assert_allclose(oracle.swiglu_mlp(h, wg, wu, wd), ref, rtol=1e-13)


def test_bf16_rounding_matches_torch():
    x = np.concatenate([RNG.standard_normal(10000) * 10.0 ** RNG.integers(-8, 8, 10000),
                        [0.0, -0.0, 1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -9]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_to_bf16(x), ref)


def test_greedy_ties_go_to_lowest_index():
    lg = np.array([[0.0, 3.0, 1.0, 3.0], [5.0, 5.0, 5.0, 5.0]])
    np.testing.assert_array_equal(oracle.greedy(lg), [1, 0])


# ----------------------------------------------------------------- whole model

def _tiny(kind: str, dtype="f32", layers=2):
    base = {"llama": "1b", "qwen": "7b"}[kind]
    shp = small_shape(base, layers=layers, vocab=97, intermediate=48, hidden=48, dtype=dtype)
    shp.update(num_attention_heads=6, num_key_value_heads=2, head_dim=8)
    return shp


def _np_weights(shp, seed=0):
    return {k: v.float().numpy().astype(np.float64) for k, v in model_weights(shp, seed).items()}


@pytest.mark.parametrize("kind", ["llama", "qwen"])
def test_incremental_decode_equals_full_recompute(kind):
    shp = _tiny(kind)
    w = _np_weights(shp)
    seq = RNG.integers(0, shp["vocab_size"], 12)
    full = OracleDecoder(shp, w).prefill([seq], all_logits=True)[0]
    m = OracleDecoder(shp, w)
    first = m.prefill([seq[:5]], all_logits=True)[0]
    rest = [m.decode([t])[0] for t in seq[5:]]
    np.testing.assert_allclose(np.concatenate([first, np.stack(rest)]), full, atol=1e-10)
    # chunked extension of a cache gives the same logits as well
    m2 = OracleDecoder(shp, w)
    m2.prefill([seq[:3]])
    np.testing.assert_allclose(m2.extend(0, seq[3:]), full[3:], atol=1e-10)


def test_slot_reset_and_admission_equal_fresh_sequences():
    """Continuous batching on the oracle: a slot that is reset and fed a new
    prompt in chunks gives the logits of a fresh prefill of that prompt, and
    the other slots are unaffected by it."""
    shp = _tiny("qwen")
    w = _np_weights(shp)
    a = RNG.integers(0, shp["vocab_size"], 10)
    b = RNG.integers(0, shp["vocab_size"], 7)
    c = RNG.integers(0, shp["vocab_size"], 9)
    fresh_b = OracleDecoder(shp, w).prefill([b], all_logits=True)[0]
    fresh_c = OracleDecoder(shp, w).prefill([c], all_logits=True)[0]
    full_a = OracleDecoder(shp, w).prefill([a], all_logits=True)[0]
    m = OracleDecoder(shp, w)
    m.prefill([a[:4], b])
    m.reset(1)                       # evict b
    got_c1 = m.extend(1, c[:5])      # admit c in its slot, in two chunks
    got_a = m.extend(0, a[4:])       # slot 0 continues meanwhile
    got_c2 = m.extend(1, c[5:])
    np.testing.assert_allclose(np.concatenate([got_c1, got_c2]), fresh_c, atol=1e-12)
    np.testing.assert_allclose(got_a, full_a[4:], atol=1e-12)
    got_b = m.extend(3, b)           # a slot never used before starts empty
    np.testing.assert_allclose(got_b, fresh_b, atol=1e-12)
    assert m.lengths() == [len(a), len(c), 0, len(b)]


@pytest.mark.parametrize("kind", ["llama", "qwen"])
def test_causal_prefix_invariance_and_batch_independence(kind):
    shp = _tiny(kind)
    w = _np_weights(shp)
    a = RNG.integers(0, shp["vocab_size"], 9)
    b = RNG.integers(0, shp["vocab_size"], 4)
    long = OracleDecoder(shp, w).prefill([np.concatenate([a, b])], all_logits=True)[0]
    short = OracleDecoder(shp, w).prefill([a], all_logits=True)[0]
    np.testing.assert_allclose(long[:9], short, atol=1e-12)
    # a sequence's logits do not depend on the other sequences of the batch
    both = OracleDecoder(shp, w).prefill([a, b], all_logits=True)
    np.testing.assert_allclose(both[0], short, atol=1e-12)


def test_gqa_model_equals_mha_model_with_repeated_kv_weights():
    """Pins the kv-head mapping h -> h // (H/KV) at the model level."""
    shp = _tiny("qwen")
    w = _np_weights(shp)
    H, KV, hd = shp["num_attention_heads"], shp["num_key_value_heads"], shp["head_dim"]
    g = H // KV
    mha = dict(shp, num_key_value_heads=H)
    w2 = dict(w)
    for n in list(w):
        if n.endswith(("k_proj.weight", "v_proj.weight")):
            w2[n] = np.repeat(w[n].reshape(KV, hd, -1), g, axis=0).reshape(H * hd, -1)
        if n.endswith(("k_proj.bias", "v_proj.bias")):
            w2[n] = np.repeat(w[n].reshape(KV, hd), g, axis=0).reshape(H * hd)
    seq = RNG.integers(0, shp["vocab_size"], 7)
    np.testing.assert_allclose(OracleDecoder(mha, w2).prefill([seq], all_logits=True)[0],
                               OracleDecoder(shp, w).prefill([seq], all_logits=True)[0], atol=1e-11)


def _hf_model(kind, shp, w):
    import transformers
    common = dict(hidden_size=shp["hidden_size"], num_hidden_layers=shp["num_hidden_layers"],
                  num_attention_heads=shp["num_attention_heads"],
                  num_key_value_heads=shp["num_key_value_heads"],
                  intermediate_size=shp["intermediate_size"], vocab_size=shp["vocab_size"],
                  rms_norm_eps=shp["rms_norm_eps"], max_position_embeddings=256,
                  tie_word_embeddings=shp["tie_word_embeddings"], hidden_act="silu")
    if kind == "llama":
        cfg = transformers.LlamaConfig(head_dim=shp["head_dim"], attention_bias=False,
                                       rope_parameters={"rope_type": "default",
                                                        "rope_theta": shp["rope_theta"]},
                                       **common)
        model = transformers.LlamaForCausalLM(cfg)
    else:
        cfg = transformers.Qwen2Config(rope_parameters={"rope_type": "default",
                                                        "rope_theta": shp["rope_theta"]},
                                       **common)
        model = transformers.Qwen2ForCausalLM(cfg)
    model = model.to(torch.float64).eval()
    sd = {k: torch.from_numpy(v) for k, v in w.items()}
    if shp["tie_word_embeddings"]:
        sd["lm_head.weight"] = sd["model.embed_tokens.weight"]
    missing, unexpected = model.load_state_dict(sd, strict=False)
    assert not unexpected, unexpected
    assert all("rotary" in m for m in missing), missing
    assert model.config.rope_parameters["rope_theta"] == shp["rope_theta"]
    return model


@pytest.mark.parametrize("kind", ["llama", "qwen"])
def test_whole_model_matches_transformers_fp64(kind):
    """The paper's baseline library (Results, Experimental Setup) runs the same
    state dict in float64: prefill logits at every position, then greedy decode
    with its KV cache."""
    shp = _tiny(kind, layers=3)
    assert shp["hidden_size"] == shp["num_attention_heads"] * shp["head_dim"]
    w = _np_weights(shp, seed=3)
    model = _hf_model(kind, shp, w)
    ids = RNG.integers(0, shp["vocab_size"], (2, 11))
    with torch.no_grad():
        ref = model(torch.from_numpy(ids)).logits.numpy()
    orc = OracleDecoder(shp, w).prefill(list(ids), all_logits=True)
    # HF evaluates the rotary angles in float32 even for a float64 model, so
    # agreement is ~1e-7; a wrong pairing, sign, head map or operand order
    # gives differences of order 0.1.
    for b in range(2):
        np.testing.assert_allclose(orc[b], ref[b], atol=1e-6, rtol=0)
    # greedy generation with the KV cache
    steps = 6
    toks, _ = generate_greedy(OracleDecoder(shp, w), list(ids), steps)
    with torch.no_grad():
        out = model.generate(torch.from_numpy(ids), max_new_tokens=steps + 1, do_sample=False,
                             pad_token_id=0, eos_token_id=None)
    np.testing.assert_array_equal(toks, out[:, ids.shape[1]:].numpy())


def test_teacher_forced_equals_free_running_on_own_tokens():
    shp = _tiny("llama")
    w = _np_weights(shp)
    seqs = [RNG.integers(0, shp["vocab_size"], 6) for _ in range(3)]
    toks, lg = generate_greedy(OracleDecoder(shp, w), seqs, 4)
    lg2 = teacher_forced(OracleDecoder(shp, w), seqs, toks[:, :4])
    np.testing.assert_array_equal(lg, lg2)


def test_io_round_mode_stays_close_to_exact():
    shp = _tiny("qwen", dtype="bf16")
    w = _np_weights(shp)
    seq = RNG.integers(0, shp["vocab_size"], 8)
    a = OracleDecoder(shp, w).prefill([seq], all_logits=True)[0]
    b = OracleDecoder(shp, w, io_round="bf16").prefill([seq], all_logits=True)[0]
    assert 0 < np.max(np.abs(a - b)) < 2e-2


def test_io_round_sites_are_the_documented_ones_and_each_is_live():
    """The bf16-storage mode rounds at exactly the documented sites (the GPU's
    bf16 storage points: normed projection inputs, rotated q and k, v, the
    attention output, the gated activation, the final norm; float32 residual
    stream).  Each bf16 site alone moves the logits away from the exact ones,
    removing any one changes the result, and the error of the full mode is the
    sum of the single sites' errors (as variances of independent rounding
    errors, within 25%): nothing outside the listed sites adds error, so the
    tolerance band that this mode sets is made of these roundings only.  With
    every site removed the mode is the exact oracle."""
    from oracle.decoder import BF16_SITES, F32_SITES
    every = set(BF16_SITES) | set(F32_SITES)
    shp = _tiny("qwen", dtype="bf16")
    shp.update(num_attention_heads=8, num_key_value_heads=2, head_dim=16)
    w = _np_weights(shp)
    seqs = [np.random.default_rng(5).integers(0, shp["vocab_size"], 24) for _ in range(2)]

    def run(skip):
        o = OracleDecoder(shp, w, io_round="bf16", io_skip=skip)
        out = np.concatenate(o.prefill(seqs, all_logits=True))
        assert o.io_applied == every - set(skip)
        return out

    exact = np.concatenate(OracleDecoder(shp, w).prefill(seqs, all_logits=True))
    np.testing.assert_array_equal(run(every), exact)
    full = run(set())
    mse_full = np.mean((full - exact) ** 2)
    parts = 0.0
    for site in BF16_SITES:
        assert not np.array_equal(run({site}), full), f"rounding site {site} has no effect"
        only = np.mean((run(every - {site}) - exact) ** 2)
        assert only > 0, site
        parts += only
    assert 0.75 < parts / mse_full < 1.25, parts / mse_full
    with pytest.raises(ValueError):
        OracleDecoder(shp, w, io_round="bf16", io_skip={"residual_bf16"})


# ----------------------------------------------------------- mixture of experts

def _moe_weights(D, E, I, shared_I, seed):
    r = np.random.default_rng(seed)
    router = r.standard_normal((E, D)) * 0.3
    ex = [tuple(r.standard_normal(shp) * 0.2 for shp in ((I, D), (I, D), (D, I))) for _ in range(E)]
    sh = tuple(r.standard_normal(shp) * 0.2 for shp in ((shared_I, D), (shared_I, D), (D, shared_I))) \
        if shared_I else None
    return router, ex, sh


def test_moe_block_matches_transformers_deepseek_v2():
    """DeepSeek-MoE semantics (the paper's MoE benchmark model): softmax router,
    greedy top-k without renormalization, ungated shared experts.  Pinned to
    transformers' DeepseekV2Moe block in float64 (its router runs in float32,
    so agreement is ~1e-7; a wrong selection, weight or sum differs by ~0.1)."""
    from transformers import DeepseekV2Config
    from transformers.models.deepseek_v2.modeling_deepseek_v2 import DeepseekV2Moe
    D, E, I, K, S = 32, 8, 16, 3, 11
    cfg = DeepseekV2Config(hidden_size=D, moe_intermediate_size=I, n_routed_experts=E, num_experts_per_tok=K,
                           n_shared_experts=2, topk_method="greedy", routed_scaling_factor=1.0, n_group=1,
                           topk_group=1, hidden_act="silu")
    blk = DeepseekV2Moe(cfg).double()
    router, ex, sh = _moe_weights(D, E, I, 2 * I, seed=5)
    with torch.no_grad():
        blk.gate.weight.copy_(torch.from_numpy(router))
        blk.experts.gate_up_proj.copy_(torch.from_numpy(np.stack([np.concatenate([g, u]) for g, u, _ in ex])))
        blk.experts.down_proj.copy_(torch.from_numpy(np.stack([d for _, _, d in ex])))
        blk.shared_experts.gate_proj.weight.copy_(torch.from_numpy(sh[0]))
        blk.shared_experts.up_proj.weight.copy_(torch.from_numpy(sh[1]))
        blk.shared_experts.down_proj.weight.copy_(torch.from_numpy(sh[2]))
    h = RNG.standard_normal((S, D))
    with torch.no_grad():
        ref = blk(torch.from_numpy(h)[None]).numpy()[0]
    got = oracle.decoder.moe_mlp(h, router, ex, sh, K, False)
    np.testing.assert_allclose(got, ref, atol=1e-6, rtol=0)
    # the shared experts matter, and so does the routing
    assert np.abs(got - oracle.decoder.moe_mlp(h, router, ex, None, K, False)).max() > 1e-2
    assert np.abs(got - oracle.decoder.moe_mlp(h, router[::-1].copy(), ex, sh, K, False)).max() > 1e-2


def test_moe_block_matches_transformers_qwen3_moe_renormalized():
    """The renormalized variant (weights of the chosen experts divided by their
    sum), pinned to transformers' Qwen3MoeSparseMoeBlock."""
    from transformers import Qwen3MoeConfig
    from transformers.models.qwen3_moe.modeling_qwen3_moe import Qwen3MoeSparseMoeBlock
    D, E, I, K, S = 32, 8, 16, 2, 9
    cfg = Qwen3MoeConfig(hidden_size=D, moe_intermediate_size=I, num_experts=E, num_experts_per_tok=K,
                         norm_topk_prob=True, hidden_act="silu")
    blk = Qwen3MoeSparseMoeBlock(cfg).double()
    router, ex, _ = _moe_weights(D, E, I, 0, seed=6)
    with torch.no_grad():
        blk.gate.weight.copy_(torch.from_numpy(router))
        blk.experts.gate_up_proj.copy_(torch.from_numpy(np.stack([np.concatenate([g, u]) for g, u, _ in ex])))
        blk.experts.down_proj.copy_(torch.from_numpy(np.stack([d for _, _, d in ex])))
    h = RNG.standard_normal((S, D))
    with torch.no_grad():
        ref = blk(torch.from_numpy(h)[None]).numpy()[0]
    np.testing.assert_allclose(oracle.decoder.moe_mlp(h, router, ex, None, K, True), ref, atol=1e-6, rtol=0)


def test_moe_router_ties_go_to_the_lowest_expert():
    """Experts 2 and 5 tie for the last of 3 places: expert 2 is chosen."""
    D, E, I = 4, 6, 3
    v = np.array([1.0, 0.0, 0.0, 0.0])
    c = np.array([3.0, 0.0, 1.0, 0.0, 2.0, 1.0])
    router = 0.25 * c[:, None] * v[None, :]
    _, ex, _ = _moe_weights(D, E, I, 0, seed=7)
    h = v[None, :] * 2.0  # logits 0.5 c
    got = oracle.decoder.moe_mlp(h, router, ex, None, 3, False)
    p = np.exp(0.5 * c) / np.exp(0.5 * c).sum()
    want = sum(p[e] * oracle.decoder.swiglu_mlp(h, *ex[e]) for e in (0, 4, 2))
    np.testing.assert_allclose(got, want, atol=1e-14)
    other = sum(p[e] * oracle.decoder.swiglu_mlp(h, *ex[e]) for e in (0, 4, 5))
    assert np.abs(got - other).max() > 1e-3


def test_moe_model_layers_and_decode_invariants():
    """A small MoE decoder: layer 0 dense, later layers MoE; incremental decode
    equals full recompute (routing is per token, so it does not depend on the
    other tokens of the call)."""
    shp = _tiny("llama")
    shp.update(n_routed_experts=6, num_experts_per_tok=2, moe_intermediate_size=16, n_shared_experts=1,
               first_k_dense_replace=1, norm_topk_prob=False)
    w = _np_weights(shp)
    assert "model.layers.0.mlp.gate_proj.weight" in w and "model.layers.1.mlp.experts.5.down_proj.weight" in w
    seq = RNG.integers(0, shp["vocab_size"], 10)
    full = OracleDecoder(shp, w).prefill([seq], all_logits=True)[0]
    m = OracleDecoder(shp, w)
    m.prefill([seq[:4]])
    np.testing.assert_allclose(m.extend(0, seq[4:]), full[4:], atol=1e-10)
    dense = OracleDecoder(dict(shp, n_routed_experts=0), {**w, **{
        k.replace("mlp.shared_experts.", "mlp."): v for k, v in w.items() if ".mlp.shared_experts." in k}})
    assert np.abs(dense.prefill([seq], all_logits=True)[0] - full).max() > 1e-3  # the routed experts contribute


def test_moe_of_identical_experts_equals_the_dense_model():
    """Every routed expert a copy of one SwiGLU MLP, renormalized top-k weights
    and no shared expert: each token's mixture is that MLP times weights that
    sum to one, so the MoE model equals the dense model with that MLP (a
    dropped weight, a wrong expert slice or an unnormalized sum breaks it)."""
    dense_shp = _tiny("qwen", layers=3)
    w = _np_weights(dense_shp, seed=5)
    moe_shp = dict(dense_shp, n_routed_experts=5, num_experts_per_tok=3,
                   moe_intermediate_size=dense_shp["intermediate_size"], n_shared_experts=0,
                   first_k_dense_replace=1, norm_topk_prob=True)
    rng = np.random.default_rng(9)
    mw = {}
    for k, v in w.items():
        if ".mlp." in k and not k.startswith("model.layers.0."):
            p, name = k.split(".mlp.")
            for e in range(5):
                mw[f"{p}.mlp.experts.{e}.{name}"] = v
            mw[f"{p}.mlp.gate.weight"] = rng.standard_normal((5, dense_shp["hidden_size"]))
        else:
            mw[k] = v
    seq = RNG.integers(0, dense_shp["vocab_size"], 9)
    ref = OracleDecoder(dense_shp, w).prefill([seq], all_logits=True)[0]
    got = OracleDecoder(moe_shp, mw).prefill([seq], all_logits=True)[0]
    np.testing.assert_allclose(got, ref, atol=1e-12)
    # without renormalization the weights sum to less than one: the models differ
    un = OracleDecoder(dict(moe_shp, norm_topk_prob=False), mw).prefill([seq], all_logits=True)[0]
    assert np.abs(un - ref).max() > 1e-4
    # a routing override (another valid top-k set for some tokens) keeps the
    # weights summing to one, so it leaves this model equal to the dense one
    force = {(0, 1, 2): (4, 0, 1), (0, 2, 5): (3, 2, 4), (0, 1, 8): (0, 1, 2)}
    got = OracleDecoder(moe_shp, mw, route_override=force).prefill([seq], all_logits=True)[0]
    np.testing.assert_allclose(got, ref, atol=1e-12)


def test_moe_route_override():
    """Forcing each token's own top-k set changes nothing (bit for bit);
    forcing another set changes that token's logits and, through the KV cache,
    only the later positions'."""
    shp = dict(_tiny("llama", layers=2), n_routed_experts=6, num_experts_per_tok=2, moe_intermediate_size=16,
               n_shared_experts=1, first_k_dense_replace=0, norm_topk_prob=False)
    w = _np_weights(shp, seed=8)
    seq = RNG.integers(0, shp["vocab_size"], 7)
    base = OracleDecoder(shp, w).prefill([seq], all_logits=True)[0]
    own = {}
    orig = oracle.decoder.moe_mlp
    calls = []

    def spy(h, w_router, experts, shared, top_k, norm_topk, rnd=None, force=None):
        p = oracle.decoder.softmax(h @ w_router.T)
        calls.append(np.argsort(-p, axis=-1, kind="stable")[:, :top_k])
        return orig(h, w_router, experts, shared, top_k, norm_topk, rnd, force)

    oracle.decoder.moe_mlp = spy
    try:
        OracleDecoder(shp, w).prefill([seq], all_logits=True)
    finally:
        oracle.decoder.moe_mlp = orig
    for layer, idx in enumerate(calls):
        for pos in range(len(seq)):
            own[(0, layer, pos)] = tuple(int(e) for e in idx[pos])
    same = OracleDecoder(shp, w, route_override=own).prefill([seq], all_logits=True)[0]
    np.testing.assert_array_equal(same, base)
    alt = dict(own)
    e0, e1 = own[(0, 1, 4)]
    alt[(0, 1, 4)] = (e0, next(e for e in range(6) if e not in (e0, e1)))
    moved = OracleDecoder(shp, w, route_override=alt).prefill([seq], all_logits=True)[0]
    np.testing.assert_array_equal(moved[:4], base[:4])
    assert np.abs(moved[4] - base[4]).max() > 1e-6


# ------------------------------------------------- GPT-2 family and sliding windows

def test_layernorm_closed_forms_and_torch():
    eps = 1e-5
    g, b = RNG.standard_normal(6), RNG.standard_normal(6)
    # a constant row has no deviation: the output is the bias
    np.testing.assert_allclose(oracle.layer_norm(np.full((2, 6), 3.7), g, b, eps), np.broadcast_to(b, (2, 6)),
                               atol=1e-12)
    # mean 0, variance 1: x / sqrt(1 + eps) * g + b
    x = np.array([[1.0, -1.0, 1.0, -1.0, 1.0, -1.0]])
    np.testing.assert_allclose(oracle.layer_norm(x, g, b, eps), x / math.sqrt(1 + eps) * g + b, rtol=1e-14)
    # invariant to shifting a row; torch's layer_norm (biased variance)
    x = RNG.standard_normal((4, 6)) * 3
    np.testing.assert_allclose(oracle.layer_norm(x + 5.0, g, b, eps), oracle.layer_norm(x, g, b, eps), atol=1e-12)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (6,), torch.from_numpy(g), torch.from_numpy(b), eps)
    np.testing.assert_allclose(oracle.layer_norm(x, g, b, eps), ref.numpy(), atol=1e-13)


def test_gelu_tanh_against_torch_and_identities():
    z = np.linspace(-8, 8, 401)
    ref = torch.nn.functional.gelu(torch.from_numpy(z), approximate="tanh").numpy()
    np.testing.assert_allclose(oracle.gelu_tanh(z), ref, atol=1e-14)
    # gelu(z) - gelu(-z) = z (the tanh form keeps this property of z Phi(z))
    np.testing.assert_allclose(oracle.gelu_tanh(z) - oracle.gelu_tanh(-z), z, atol=1e-13)
    # within 1e-3 of the exact z Phi(z)
    exact = 0.5 * z * (1 + np.vectorize(math.erf)(z / math.sqrt(2)))
    assert np.max(np.abs(oracle.gelu_tanh(z) - exact)) < 1e-3


def _tiny_gpt2(layers=2, **kw):
    s = dict(model_type="gpt2", hidden_size=48, num_hidden_layers=layers, num_attention_heads=6,
             num_key_value_heads=6, head_dim=8, intermediate_size=192, vocab_size=97,
             max_position_embeddings=40, tie_word_embeddings=True, attention_bias=True,
             layer_norm_epsilon=1e-5, dtype="f32")
    s.update(kw)
    return s


def test_gpt2_matches_transformers_fp64():
    """The complete GPT-2 definition against transformers' GPT2LMHeadModel in
    float64 with the same state dict: logits at every position, then greedy
    generation through its KV cache."""
    import transformers
    shp = _tiny_gpt2(layers=3)
    w = _np_weights(shp, seed=11)
    cfg = transformers.GPT2Config(n_embd=48, n_layer=3, n_head=6, n_inner=192, vocab_size=97, n_positions=40,
                                  activation_function="gelu_new", layer_norm_epsilon=1e-5, resid_pdrop=0.0,
                                  embd_pdrop=0.0, attn_pdrop=0.0)
    model = transformers.GPT2LMHeadModel(cfg).to(torch.float64).eval()
    sd = {k: torch.from_numpy(v) for k, v in w.items()}
    sd["lm_head.weight"] = sd["transformer.wte.weight"]
    missing, unexpected = model.load_state_dict(sd, strict=False)
    assert not unexpected and not missing, (missing, unexpected)
    ids = RNG.integers(0, 97, (2, 13))
    with torch.no_grad():
        ref = model(torch.from_numpy(ids)).logits.numpy()
    orc = OracleDecoder(shp, w).prefill(list(ids), all_logits=True)
    for b in range(2):
        np.testing.assert_allclose(orc[b], ref[b], atol=1e-10, rtol=0)
    steps = 6
    toks, _ = generate_greedy(OracleDecoder(shp, w), list(ids), steps)
    with torch.no_grad():
        # an explicit mask: generate() otherwise takes every prompt token equal
        # to pad_token_id for padding and shifts the learned positions
        out = model.generate(torch.from_numpy(ids), attention_mask=torch.ones(ids.shape, dtype=torch.long),
                             max_new_tokens=steps + 1, do_sample=False, pad_token_id=0, eos_token_id=None)
    np.testing.assert_array_equal(toks, out[:, ids.shape[1]:].numpy())


def test_gpt2_incremental_decode_and_positions():
    shp = _tiny_gpt2()
    w = _np_weights(shp, seed=12)
    seq = RNG.integers(0, 97, 11)
    full = OracleDecoder(shp, w).prefill([seq], all_logits=True)[0]
    m = OracleDecoder(shp, w)
    m.prefill([seq[:4]])
    np.testing.assert_allclose(m.extend(0, seq[4:7]), full[4:7], atol=1e-10)
    np.testing.assert_allclose(np.stack([m.decode([t])[0] for t in seq[7:]]), full[7:], atol=1e-10)
    # the learned positions matter: the same token at two positions differs
    a = OracleDecoder(shp, w).prefill([[5, 5]], all_logits=True)[0]
    assert np.abs(a[0] - a[1]).max() > 1e-3
    # the table ends at max_position_embeddings
    with pytest.raises(AssertionError):
        OracleDecoder(shp, w).prefill([RNG.integers(0, 97, 41)])


def test_sliding_window_attention_special_cases():
    S, H, KV, hd = 9, 4, 2, 8
    q = RNG.standard_normal((S, H, hd))
    k = RNG.standard_normal((S, KV, hd))
    v = RNG.standard_normal((S, KV, hd))
    pos = np.arange(S)
    full = oracle.causal_gqa_attention(q, k, v, pos)
    # a window at least as long as the context changes nothing
    np.testing.assert_array_equal(oracle.causal_gqa_attention(q, k, v, pos, window=S), full)
    # a window of one key: each query sees only its own key, so the output is v
    one = oracle.causal_gqa_attention(q, k, v, pos, window=1)
    np.testing.assert_allclose(one, np.repeat(v, H // KV, axis=1), atol=1e-14)
    # brute force for W = 3: keys pos-2 .. pos
    W = 3
    got = oracle.causal_gqa_attention(q, k, v, pos, window=W)
    for i in range(S):
        keys = np.arange(max(0, i - W + 1), i + 1)
        for h in range(H):
            s = q[i, h] @ k[keys, h * KV // H].T / math.sqrt(hd)
            p = np.exp(s - s.max())
            np.testing.assert_allclose(got[i, h], (p / p.sum()) @ v[keys, h * KV // H], atol=1e-13)


def test_sliding_window_matches_transformers_mistral_fp64():
    """A Mistral-style model (window shorter than the sequence) against
    transformers' MistralForCausalLM in float64 with eager attention; decode
    past the window through the cache equals full recompute."""
    import transformers
    shp = dict(_tiny("llama", layers=2), sliding_window=4, tie_word_embeddings=False)
    w = _np_weights(shp, seed=13)
    cfg = transformers.MistralConfig(hidden_size=48, num_hidden_layers=2, num_attention_heads=6,
                                     num_key_value_heads=2, head_dim=8, intermediate_size=48, vocab_size=97,
                                     rms_norm_eps=shp["rms_norm_eps"], max_position_embeddings=64,
                                     tie_word_embeddings=False, sliding_window=4,
                                     rope_parameters={"rope_type": "default", "rope_theta": shp["rope_theta"]},
                                     attn_implementation="eager")
    model = transformers.MistralForCausalLM(cfg).to(torch.float64).eval()
    missing, unexpected = model.load_state_dict({k: torch.from_numpy(v) for k, v in w.items()}, strict=False)
    assert not unexpected and all("rotary" in m for m in missing), (missing, unexpected)
    ids = RNG.integers(0, 97, (2, 12))
    with torch.no_grad():
        ref = model(torch.from_numpy(ids)).logits.numpy()
    orc = OracleDecoder(shp, w).prefill(list(ids), all_logits=True)
    for b in range(2):
        np.testing.assert_allclose(orc[b], ref[b], atol=1e-6, rtol=0)
    # the window matters here
    nowin = OracleDecoder(dict(shp, sliding_window=None), w).prefill(list(ids), all_logits=True)
    assert np.abs(nowin[0] - orc[0]).max() > 1e-3
    m = OracleDecoder(shp, w)
    m.prefill([ids[0, :3]])
    np.testing.assert_allclose(np.stack([m.decode([t])[0] for t in ids[0, 3:]]), orc[0][3:], atol=1e-10)


# ----------------------------------------------------------------- backward pass

def test_rmsnorm_backward_against_torch_autograd():
    x = RNG.standard_normal((5, 12))
    g = 1 + 0.1 * RNG.standard_normal(12)
    dy = RNG.standard_normal((5, 12))
    xt = torch.from_numpy(x).requires_grad_()
    gt = torch.from_numpy(g).requires_grad_()
    y = xt / torch.sqrt(torch.mean(xt * xt, -1, keepdim=True) + 1e-5) * gt
    y.backward(torch.from_numpy(dy))
    dx, dg = oracle.rms_norm_backward(x, g, 1e-5, dy)
    np.testing.assert_allclose(dx, xt.grad.numpy(), atol=1e-13)
    np.testing.assert_allclose(dg, gt.grad.numpy(), atol=1e-13)


@pytest.mark.parametrize("kind", ["llama", "qwen"])
def test_loss_and_grads_match_transformers_autograd_fp64(kind):
    """The paper trains through the framework's autograd: transformers' model
    in float64 with labels = the tokens (its loss shifts them by one) gives
    the same mean cross-entropy and the same gradient for every weight (HF
    evaluates the rotary angles in float32, hence the 1e-6 scale)."""
    shp = _tiny(kind, layers=2)
    w = _np_weights(shp, seed=21)
    model = _hf_model(kind, shp, w)
    ids = RNG.integers(0, shp["vocab_size"], (2, 10))
    out = model(torch.from_numpy(ids), labels=torch.from_numpy(ids))
    out.loss.backward()
    targets = [np.append(s[1:], -1) for s in ids]
    loss, grads = oracle.loss_and_grads(shp, w, list(ids), targets)
    assert abs(loss - out.loss.item()) < 1e-6
    params = dict(model.named_parameters())
    for name, g in grads.items():
        ref = params[name].grad.numpy()
        np.testing.assert_allclose(g, ref, atol=1e-6 * max(1.0, np.abs(ref).max()), rtol=0, err_msg=name)
        assert np.abs(ref).max() > 0, name  # every weight matters here


def test_loss_and_grads_against_finite_differences():
    """Central differences of the oracle's own loss, for entries of every
    kind of weight (independent of any library): a dropped term, wrong sign
    or transposed operand in the reverse pass shows up as a mismatch."""
    shp = _tiny("qwen", layers=2)
    w = _np_weights(shp, seed=22)
    seqs = [RNG.integers(0, shp["vocab_size"], 7), RNG.integers(0, shp["vocab_size"], 4)]
    targets = [RNG.integers(0, shp["vocab_size"], 7), np.array([3, -1, 5, 9])]
    _, grads = oracle.loss_and_grads(shp, w, seqs, targets)
    r = np.random.default_rng(5)
    h = 1e-5
    for name in ["model.embed_tokens.weight", "lm_head.weight", "model.norm.weight",
                 "model.layers.0.input_layernorm.weight", "model.layers.0.self_attn.q_proj.weight",
                 "model.layers.1.self_attn.k_proj.weight", "model.layers.0.self_attn.v_proj.weight",
                 "model.layers.1.self_attn.q_proj.bias", "model.layers.0.self_attn.k_proj.bias",
                 "model.layers.1.self_attn.o_proj.weight", "model.layers.0.post_attention_layernorm.weight",
                 "model.layers.1.mlp.gate_proj.weight", "model.layers.0.mlp.up_proj.weight",
                 "model.layers.1.mlp.down_proj.weight"]:
        for _ in range(3):
            idx = tuple(r.integers(0, n) for n in w[name].shape)
            if name == "model.embed_tokens.weight":  # a row some token uses
                idx = (int(seqs[0][r.integers(0, 7)]),) + idx[1:]
            wp = dict(w)
            wp[name] = w[name].copy()
            wp[name][idx] += h
            lp, _ = oracle.loss_and_grads(shp, wp, seqs, targets)
            wp[name][idx] -= 2 * h
            lm, _ = oracle.loss_and_grads(shp, wp, seqs, targets)
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grads[name][idx]) < 1e-7 + 1e-5 * abs(fd), (name, idx, fd, grads[name][idx])
