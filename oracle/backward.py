"""CPU oracle of the backward pass: mean next-token cross-entropy and its
gradient with respect to every weight of a Llama-family decoder.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package; the product path never does.  It shares no code with the GPU path.

The paper trains its generated models through the framework's automatic
differentiation (Results, "Training with Axon Derived Models": the only change
to the generated model is enabling gradients).  This module writes that
derivative out by hand, in float64, as the reverse of the forward pass in
``decoder.py`` (same readings: RMSNorm with eps inside the root, rotate-half
RoPE, grouped-query causal attention with scale 1/sqrt(HD), SwiGLU MLP,
optional q/k/v biases, optionally tied head):

  loss = (1 / N) * sum over positions t with target[t] >= 0 of
         logsumexp(logits[t]) - logits[t][target[t]]

N is the number of such positions over all sequences.  Every step below is
the chain rule applied to one forward step, in reverse order.
"""
from __future__ import annotations

import numpy as np

from .decoder import _to_f64, apply_rope, rms_norm, rope_cos_sin, silu, softmax


def rms_norm_backward(x: np.ndarray, gain: np.ndarray, eps: float, dy: np.ndarray):
    """y = x r g with r = (mean(x^2) + eps)^(-1/2) per row.  Returns (dx, dgain):
    dgain = sum_t dy x r; dx = r (g dy) - x r^3 mean(g dy x)."""
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    gdy = gain * dy
    dx = r * gdy - x * r ** 3 * np.mean(gdy * x, axis=-1, keepdims=True)
    return dx, np.sum(dy * x * r, axis=0)


def _layer_forward(w, p, x, pos, H, KV, hd, eps, theta, bias):
    """One layer's forward over a sequence, keeping what the backward reads."""
    s = x.shape[0]
    c = {"x": x}
    h = rms_norm(x, w[p + "input_layernorm.weight"], eps)
    c["h"] = h
    q = h @ w[p + "self_attn.q_proj.weight"].T
    k = h @ w[p + "self_attn.k_proj.weight"].T
    v = h @ w[p + "self_attn.v_proj.weight"].T
    if bias:
        q = q + w[p + "self_attn.q_proj.bias"]
        k = k + w[p + "self_attn.k_proj.bias"]
        v = v + w[p + "self_attn.v_proj.bias"]
    cos, sin = rope_cos_sin(pos, hd, theta)
    c["cos"], c["sin"] = cos, sin
    qr = apply_rope(q.reshape(s, H, hd), cos, sin)
    kr = apply_rope(k.reshape(s, KV, hd), cos, sin)
    vv = v.reshape(s, KV, hd)
    group = H // KV
    scale = 1.0 / np.sqrt(hd)
    masked = np.arange(s)[None, :] > np.arange(s)[:, None]
    P = np.empty((H, s, s))
    o = np.empty((s, H, hd))
    for hh in range(H):
        sc = (qr[:, hh, :] @ kr[:, hh // group, :].T) * scale
        P[hh] = softmax(np.where(masked, -np.inf, sc))
        o[:, hh, :] = P[hh] @ vv[:, hh // group, :]
    c.update(qr=qr, kr=kr, v=vv, P=P, o=o.reshape(s, H * hd))
    x = x + c["o"] @ w[p + "self_attn.o_proj.weight"].T
    c["x2"] = x
    h2 = rms_norm(x, w[p + "post_attention_layernorm.weight"], eps)
    g = h2 @ w[p + "mlp.gate_proj.weight"].T
    u = h2 @ w[p + "mlp.up_proj.weight"].T
    a = silu(g) * u
    c.update(h2=h2, g=g, u=u, a=a)
    return x + a @ w[p + "mlp.down_proj.weight"].T, c


def _layer_backward(w, p, c, dx, grads, H, KV, hd, eps, bias):
    """Reverse of ``_layer_forward``: returns the gradient at the layer's
    input x, accumulating weight gradients into ``grads``."""
    s = dx.shape[0]
    group = H // KV
    scale = 1.0 / np.sqrt(hd)
    # MLP: x_out = x2 + a Wd^T, a = silu(g) u
    grads[p + "mlp.down_proj.weight"] += dx.T @ c["a"]
    da = dx @ w[p + "mlp.down_proj.weight"]
    sg = 1.0 / (1.0 + np.exp(-c["g"]))
    dg = da * c["u"] * sg * (1.0 + c["g"] * (1.0 - sg))  # d silu(g) / dg = s (1 + g (1 - s))
    du = da * silu(c["g"])
    grads[p + "mlp.gate_proj.weight"] += dg.T @ c["h2"]
    grads[p + "mlp.up_proj.weight"] += du.T @ c["h2"]
    dh2 = dg @ w[p + "mlp.gate_proj.weight"] + du @ w[p + "mlp.up_proj.weight"]
    dxn, dgain = rms_norm_backward(c["x2"], w[p + "post_attention_layernorm.weight"], eps, dh2)
    grads[p + "post_attention_layernorm.weight"] += dgain
    dx = dx + dxn
    # attention output projection: x2 = x + o Wo^T
    grads[p + "self_attn.o_proj.weight"] += dx.T @ c["o"]
    do = (dx @ w[p + "self_attn.o_proj.weight"]).reshape(s, H, hd)
    # attention: o = P v, P = softmax(qr kr^T scale) (masked entries have P = 0)
    dqr = np.zeros_like(c["qr"])
    dkr = np.zeros_like(c["kr"])
    dv = np.zeros_like(c["v"])
    for hh in range(H):
        kh = hh // group
        P = c["P"][hh]
        dv[:, kh, :] += P.T @ do[:, hh, :]
        dP = do[:, hh, :] @ c["v"][:, kh, :].T
        dS = P * (dP - np.sum(dP * P, axis=-1, keepdims=True))
        dqr[:, hh, :] = dS @ c["kr"][:, kh, :] * scale
        dkr[:, kh, :] += dS.T @ c["qr"][:, hh, :] * scale
    # RoPE is a rotation per pair: its transpose rotates by the opposite angle
    dq = apply_rope(dqr, c["cos"], -c["sin"]).reshape(s, H * hd)
    dk = apply_rope(dkr, c["cos"], -c["sin"]).reshape(s, KV * hd)
    dv = dv.reshape(s, KV * hd)
    for name, d in (("q", dq), ("k", dk), ("v", dv)):
        grads[p + f"self_attn.{name}_proj.weight"] += d.T @ c["h"]
        if bias:
            grads[p + f"self_attn.{name}_proj.bias"] += np.sum(d, axis=0)
    dh = dq @ w[p + "self_attn.q_proj.weight"] + dk @ w[p + "self_attn.k_proj.weight"] \
        + dv @ w[p + "self_attn.v_proj.weight"]
    dxn, dgain = rms_norm_backward(c["x"], w[p + "input_layernorm.weight"], eps, dh)
    grads[p + "input_layernorm.weight"] += dgain
    return dx + dxn


def loss_and_grads(cfg: dict, weights: dict, seqs, targets):
    """Mean cross-entropy of ``targets`` (one int per token of each sequence,
    -1 = not counted) under the model, and the gradient of that mean with
    respect to every weight (float64 arrays keyed like ``weights``).
    Sequences are independent (each starts at position 0)."""
    assert not cfg.get("n_routed_experts") and cfg.get("model_type") != "gpt2" and not cfg.get("sliding_window")
    w = {k: _to_f64(v) for k, v in weights.items()}
    H, KV, hd = cfg["num_attention_heads"], cfg["num_key_value_heads"], cfg["head_dim"]
    eps, theta, bias = float(cfg["rms_norm_eps"]), float(cfg["rope_theta"]), bool(cfg["attention_bias"])
    L = cfg["num_hidden_layers"]
    tied = bool(cfg["tie_word_embeddings"])
    head_name = "model.embed_tokens.weight" if tied else "lm_head.weight"
    grads = {k: np.zeros_like(v) for k, v in w.items()}
    n_total = sum(int(np.sum(np.asarray(t) >= 0)) for t in targets)
    assert n_total > 0
    loss = 0.0
    for ids, tgt in zip(seqs, targets):
        ids = np.asarray(ids, dtype=np.int64)
        tgt = np.asarray(tgt, dtype=np.int64)
        pos = np.arange(len(ids))
        x = w["model.embed_tokens.weight"][ids]
        caches = []
        for i in range(L):
            x, c = _layer_forward(w, f"model.layers.{i}.", x, pos, H, KV, hd, eps, theta, bias)
            caches.append(c)
        hf = rms_norm(x, w["model.norm.weight"], eps)
        logits = hf @ w[head_name].T
        # loss and its gradient at the logits
        m = np.max(logits, axis=-1, keepdims=True)
        lse = (m + np.log(np.sum(np.exp(logits - m), axis=-1, keepdims=True)))[:, 0]
        valid = tgt >= 0
        loss += float(np.sum((lse - logits[np.arange(len(ids)), np.maximum(tgt, 0)])[valid])) / n_total
        dlogits = softmax(logits)
        dlogits[np.arange(len(ids)), np.maximum(tgt, 0)] -= 1.0
        dlogits = np.where(valid[:, None], dlogits, 0.0) / n_total
        # head and final norm
        grads[head_name] += dlogits.T @ hf
        dhf = dlogits @ w[head_name]
        dx, dgain = rms_norm_backward(x, w["model.norm.weight"], eps, dhf)
        grads["model.norm.weight"] += dgain
        for i in reversed(range(L)):
            dx = _layer_backward(w, f"model.layers.{i}.", caches[i], dx, grads, H, KV, hd, eps, bias)
        np.add.at(grads["model.embed_tokens.weight"], ids, dx)
    return loss, grads
