"""CPU oracle of the decoder-only forward pass (prefill + greedy decode).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package; the product path never does.  It shares no code with the GPU path.

What it computes is the plain definition of the pass that the paper's compiler
emits for Llama/Qwen-style causal LMs, written out in float64 with NumPy:

* the pre-norm residual block ``x + f(rmsnorm(x))`` (the ``block`` example in
  the Axon Language section, Syntax paragraph, and the layer body of the
  complete GPT-2 definition in the Technical Supplement, with RMSNorm in place
  of LayerNorm);
* q/k/v/o projections under the attention scope (Technical Supplement,
  "Scoped parameter binding" listing), rotary positions from
  ``past_length + arange(S)`` (Built-In Libraries, "Positions and cache
  management" listing);
* scaled dot-product attention with scale ``1/sqrt(HD)`` (Built-In Libraries,
  "Tensor and math built-ins" listing), causal masking, grouped-query heads
  (Built-In Libraries, "Attention and masking");
* the gated MLP ``linear@up |> swiglu |> linear@down`` (Technical Supplement,
  "Bare calls, pipes" listing);
* final norm followed by the (optionally tied) output linear (complete GPT-2
  definition), greedy argmax over the logits (Results, Measures: generated
  tokens are produced by ``generate()``).

The paper leaves several details open; the readings taken here are:
RMSNorm ``g * x / sqrt(mean(x^2) + eps)``; rotate-half RoPE pairing (i, i+HD/2)
with ``inv_freq_i = theta^(-2i/HD)`` and no frequency scaling; kv head of query
head h is ``h // (H/KV)``; biases (when present) on q, k, v only, added before
the rotation; SiLU applied to the gate projection, times the up projection;
greedy ties go to the lowest index.

``io_round="bf16"`` is a diagnostic mode that rounds to bfloat16 at the points
where the GPU path stores bf16 (normed activations, rotated q/k, v, attention
output, gated MLP activation) and keeps the residual stream in float32.  The
reference mode is ``io_round=None`` (everything float64).  Each rounding point
is a named site (``BF16_SITES``, ``F32_SITES``); ``io_skip`` leaves the named
sites unrounded and ``io_applied`` records the sites a run actually rounded,
so that the set of rounding points can be checked and each one's share of the
error measured.
"""
from __future__ import annotations

import numpy as np

# Rounding sites of the bf16-storage mode: bf16 where the GPU stores an
# activation in bf16 (the RMSNorm / LayerNorm outputs that feed a projection,
# the rotated query and key and the value as stored in the KV cache, the
# attention output, the gated MLP activation, the final norm's output), float32
# for the residual stream (the embedding row and the stream after each residual
# add).
BF16_SITES = ("norm_in", "q", "k", "v", "attn_out", "norm_post", "mlp_act", "final_norm")
F32_SITES = ("resid",)


# --------------------------------------------------------------------------
# rounding helpers for the diagnostic mode
# --------------------------------------------------------------------------

def round_to_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> float32 -> bfloat16 (round to nearest even) -> float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# building blocks
# --------------------------------------------------------------------------

def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """Built-in ``NN.rmsnorm``: scale each row by the inverse root of its mean
    square (eps inside the root), then multiply by the learned gain."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def layer_norm(x: np.ndarray, gain: np.ndarray, bias: np.ndarray, eps: float) -> np.ndarray:
    """Built-in ``NN.layernorm`` (the GPT-2 definition's ln_1 / ln_2 / ln_f):
    subtract each row's mean, divide by the root of its (biased) variance
    plus eps, then scale by the gain and add the bias."""
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gain + bias


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    """``gelu_new`` of the GPT-2 definition: the tanh form of GELU,
    0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))."""
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def rope_inv_freq(head_dim: int, theta: float) -> np.ndarray:
    i = np.arange(head_dim // 2, dtype=np.float64)
    return theta ** (-2.0 * i / head_dim)


def rope_cos_sin(positions: np.ndarray, head_dim: int, theta: float):
    """cos/sin of the rotation angles ``pos * inv_freq_i``, shape [S, HD/2]."""
    ang = np.outer(np.asarray(positions, dtype=np.float64), rope_inv_freq(head_dim, theta))
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate each pair (x_i, x_{i+HD/2}) by its angle.  ``x`` is [S, heads, HD],
    ``cos``/``sin`` are [S, HD/2]."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s: np.ndarray) -> np.ndarray:
    """Row softmax; masked entries are -inf and get probability 0."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                         q_pos: np.ndarray, window: int | None = None) -> np.ndarray:
    """Scaled dot-product attention with a causal mask and grouped KV heads.

    q: [Sq, H, HD] at absolute positions ``q_pos``; k, v: [Sk, KV, HD] for
    positions 0..Sk-1.  Query i sees keys j <= q_pos[i], and with a sliding
    ``window`` W only the last W of them, j > q_pos[i] - W (the masking
    built-in's ``window`` argument).  Head h reads kv head h // (H / KV).
    Returns [Sq, H, HD].
    """
    sq, n_heads, hd = q.shape
    n_kv = k.shape[1]
    group = n_heads // n_kv
    scale = 1.0 / np.sqrt(hd)
    keys = np.arange(k.shape[0])
    masked = keys[None, :] > np.asarray(q_pos)[:, None]
    if window:
        masked |= keys[None, :] <= np.asarray(q_pos)[:, None] - window
    out = np.empty_like(q)
    for h in range(n_heads):
        kvh = h // group
        s = (q[:, h, :] @ k[:, kvh, :].T) * scale
        s = np.where(masked, -np.inf, s)
        out[:, h, :] = softmax(s) @ v[:, kvh, :]
    return out


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def swiglu_mlp(h: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray,
               rnd=None) -> np.ndarray:
    """``linear@up |> swiglu |> linear@down`` with the SiLU on the gate branch."""
    a = silu(h @ w_gate.T) * (h @ w_up.T)
    if rnd is not None:
        a = rnd(a)
    return a @ w_down.T


def gelu_mlp(h: np.ndarray, w_fc: np.ndarray, b_fc: np.ndarray, w_proj: np.ndarray, b_proj: np.ndarray,
             rnd=None) -> np.ndarray:
    """The GPT-2 MLP, ``linear@c_fc |> gelu_new |> linear@c_proj`` with biases;
    the weights are stored [in, out] (the definition's ``transpose=true``)."""
    a = gelu_tanh(h @ w_fc + b_fc)
    if rnd is not None:
        a = rnd(a)
    return a @ w_proj + b_proj


def moe_mlp(h: np.ndarray, w_router: np.ndarray, experts: list, shared, top_k: int, norm_topk: bool,
            rnd=None, force: dict | None = None) -> np.ndarray:
    """Mixture-of-experts MLP (the MoE built-in's softmax top-k router followed
    by the routed experts; Built-In Libraries, "Activations and specialized
    modules").  Per token: router probabilities = softmax over the experts of
    h W_router^T; the top_k experts by probability (ties to the lowest expert
    index); their probabilities are the mixing weights (divided by their sum
    when ``norm_topk``); each chosen expert is a SwiGLU MLP; ``shared`` (a
    (gate, up, down) triple or None) is an always-active SwiGLU MLP added
    without a weight.  ``experts`` is a list of (gate, up, down) triples.
    ``force`` (row -> top_k expert ids) replaces the chosen set of the given
    rows (their weights are still their probabilities): where two experts'
    probabilities lie within rounding of each other either choice is a valid
    result, and this evaluates the other one."""
    p = softmax(h @ w_router.T)
    idx = np.argsort(-p, axis=-1, kind="stable")[:, :top_k]
    for row, chosen in (force or {}).items():
        idx[row] = np.asarray(chosen, dtype=idx.dtype)
    wts = np.take_along_axis(p, idx, axis=-1)
    if norm_topk:
        wts = wts / np.sum(wts, axis=-1, keepdims=True)
    out = np.zeros_like(h)
    for e, (wg, wu, wd) in enumerate(experts):
        rows, slots = np.nonzero(idx == e)
        if rows.size:
            out[rows] += wts[rows, slots][:, None] * swiglu_mlp(h[rows], wg, wu, wd, rnd=rnd)
    if shared is not None:
        out = out + swiglu_mlp(h, *shared, rnd=rnd)
    return out


# --------------------------------------------------------------------------
# the model
# --------------------------------------------------------------------------

class OracleDecoder:
    """Float64 decoder with a per-sequence KV cache.

    ``cfg`` uses HF-style keys (hidden_size, num_hidden_layers,
    num_attention_heads, num_key_value_heads, head_dim, intermediate_size,
    vocab_size, rms_norm_eps, rope_theta, attention_bias, tie_word_embeddings).
    ``weights`` maps the flat checkpoint names to arrays (any float dtype, or
    torch tensors); they are held as float64.  Mixture-of-experts models add
    n_routed_experts, num_experts_per_tok, moe_intermediate_size,
    n_shared_experts, first_k_dense_replace (leading layers with a dense MLP)
    and norm_topk_prob (DeepSeek-MoE-style keys); their MoE layers read
    ``mlp.gate.weight`` (the router), ``mlp.experts.{e}.*`` and
    ``mlp.shared_experts.*``.

    ``model_type == "gpt2"`` selects the GPT-2 definition of the Technical
    Supplement ("A Complete Model Definition"): LayerNorm with bias
    (layer_norm_epsilon), learned positions added to the token embedding
    (max_position_embeddings rows), one fused ``c_attn`` projection with bias
    giving q, k, v, multi-head attention without rotation, ``c_proj`` with
    bias, the GELU MLP with biases, and the head tied to the token embedding;
    weights under ``transformer.*`` in the [in, out] layout.  ``sliding_window``
    (any model) limits each query to its last W keys.
    """

    def __init__(self, cfg: dict, weights: dict, io_round: str | None = None, io_skip=(),
                 route_override: dict | None = None):
        self.cfg = cfg
        self.D = cfg["hidden_size"]
        self.L = cfg["num_hidden_layers"]
        self.H = cfg["num_attention_heads"]
        self.KV = cfg["num_key_value_heads"]
        self.hd = cfg["head_dim"]
        self.gpt2 = cfg.get("model_type") == "gpt2"
        self.eps = float(cfg["layer_norm_epsilon"] if self.gpt2 else cfg["rms_norm_eps"])
        self.theta = None if self.gpt2 else float(cfg["rope_theta"])
        self.bias = bool(cfg["attention_bias"])
        self.window = int(cfg.get("sliding_window") or 0) or None
        self.w = {k: _to_f64(v) for k, v in weights.items()}
        if self.gpt2:
            self.lm_head = self.w["transformer.wte.weight"]
        else:
            self.lm_head = self.w["model.embed_tokens.weight"] if cfg["tie_word_embeddings"] \
                else self.w["lm_head.weight"]
        if io_round not in (None, "bf16"):
            raise ValueError(io_round)
        unknown = set(io_skip) - set(BF16_SITES) - set(F32_SITES)
        if unknown:
            raise ValueError(f"unknown rounding sites {sorted(unknown)}")
        self.io_round = io_round
        self.io_skip = frozenset(io_skip)
        self.io_applied: set[str] = set()
        self.caches: list[list[tuple[np.ndarray, np.ndarray]]] = []
        # (sequence, layer, position) -> the top-k expert set that token takes
        # in that layer instead of its own choice (mixture-of-experts models)
        self.route_override = dict(route_override or {})
        self._seq = 0
        self.n_experts = int(cfg.get("n_routed_experts") or 0)
        self.first_moe = int(cfg.get("first_k_dense_replace") or 0)

    # ---- rounding at the GPU's storage points (bf16-storage mode only) ----
    def _r(self, a: np.ndarray, site: str) -> np.ndarray:
        if self.io_round is None or site in self.io_skip:
            return a
        self.io_applied.add(site)
        return round_to_bf16(a)

    def _rx(self, a: np.ndarray) -> np.ndarray:
        if self.io_round is None or "resid" in self.io_skip:
            return a
        self.io_applied.add("resid")
        return round_to_f32(a)

    def _r_act(self, a: np.ndarray) -> np.ndarray:
        return self._r(a, "mlp_act")

    # ---- one layer over the new tokens of one sequence ----
    def _layer(self, i: int, x: np.ndarray, pos: np.ndarray, cache: list) -> np.ndarray:
        p = f"model.layers.{i}."
        w = self.w
        s = x.shape[0]
        h = self._r(rms_norm(x, w[p + "input_layernorm.weight"], self.eps), "norm_in")
        q = h @ w[p + "self_attn.q_proj.weight"].T
        k = h @ w[p + "self_attn.k_proj.weight"].T
        v = h @ w[p + "self_attn.v_proj.weight"].T
        if self.bias:
            q = q + w[p + "self_attn.q_proj.bias"]
            k = k + w[p + "self_attn.k_proj.bias"]
            v = v + w[p + "self_attn.v_proj.bias"]
        q = q.reshape(s, self.H, self.hd)
        k = k.reshape(s, self.KV, self.hd)
        v = v.reshape(s, self.KV, self.hd)
        cos, sin = rope_cos_sin(pos, self.hd, self.theta)
        q = self._r(apply_rope(q, cos, sin), "q")
        k = self._r(apply_rope(k, cos, sin), "k")
        v = self._r(v, "v")
        kc, vc = cache[i]
        kc = np.concatenate([kc, k], axis=0)
        vc = np.concatenate([vc, v], axis=0)
        cache[i] = (kc, vc)
        o = self._r(causal_gqa_attention(q, kc, vc, pos, self.window), "attn_out").reshape(s, self.H * self.hd)
        x = self._rx(x + o @ w[p + "self_attn.o_proj.weight"].T)
        h2 = self._r(rms_norm(x, w[p + "post_attention_layernorm.weight"], self.eps), "norm_post")
        if self.n_experts and i >= self.first_moe:
            c = self.cfg
            ex = [tuple(w[p + f"mlp.experts.{e}.{n}_proj.weight"] for n in ("gate", "up", "down"))
                  for e in range(self.n_experts)]
            sh = tuple(w[p + f"mlp.shared_experts.{n}_proj.weight"] for n in ("gate", "up", "down")) \
                if c.get("n_shared_experts") else None
            force = {r: self.route_override[(self._seq, i, int(q))] for r, q in enumerate(pos)
                     if (self._seq, i, int(q)) in self.route_override}
            mlp = moe_mlp(h2, w[p + "mlp.gate.weight"], ex, sh, int(c["num_experts_per_tok"]),
                          bool(c.get("norm_topk_prob")), rnd=self._r_act, force=force)
        else:
            mlp = swiglu_mlp(h2, w[p + "mlp.gate_proj.weight"], w[p + "mlp.up_proj.weight"],
                             w[p + "mlp.down_proj.weight"], rnd=self._r_act)
        return self._rx(x + mlp)

    def _layer_gpt2(self, i: int, x: np.ndarray, pos: np.ndarray, cache: list) -> np.ndarray:
        p = f"transformer.h.{i}."
        w = self.w
        s, D = x.shape
        h = self._r(layer_norm(x, w[p + "ln_1.weight"], w[p + "ln_1.bias"], self.eps), "norm_in")
        qkv = h @ w[p + "attn.c_attn.weight"] + w[p + "attn.c_attn.bias"]
        q = self._r(qkv[:, :D].reshape(s, self.H, self.hd), "q")
        k = self._r(qkv[:, D:2 * D].reshape(s, self.KV, self.hd), "k")
        v = self._r(qkv[:, 2 * D:].reshape(s, self.KV, self.hd), "v")
        kc, vc = cache[i]
        kc = np.concatenate([kc, k], axis=0)
        vc = np.concatenate([vc, v], axis=0)
        cache[i] = (kc, vc)
        o = self._r(causal_gqa_attention(q, kc, vc, pos, self.window), "attn_out").reshape(s, D)
        x = self._rx(x + o @ w[p + "attn.c_proj.weight"] + w[p + "attn.c_proj.bias"])
        h2 = self._r(layer_norm(x, w[p + "ln_2.weight"], w[p + "ln_2.bias"], self.eps), "norm_post")
        mlp = gelu_mlp(h2, w[p + "mlp.c_fc.weight"], w[p + "mlp.c_fc.bias"], w[p + "mlp.c_proj.weight"],
                       w[p + "mlp.c_proj.bias"], rnd=self._r_act)
        return self._rx(x + mlp)

    def _forward_seq(self, b: int, ids: np.ndarray, all_logits: bool) -> np.ndarray:
        self._seq = b
        cache = self.caches[b]
        past = cache[0][0].shape[0]
        pos = past + np.arange(len(ids))
        ids = np.asarray(ids, dtype=np.int64)
        if self.gpt2:
            assert pos[-1] < self.cfg["max_position_embeddings"], "position past the learned table"
            x = self._rx(self.w["transformer.wte.weight"][ids] + self.w["transformer.wpe.weight"][pos])
            for i in range(self.L):
                x = self._layer_gpt2(i, x, pos, cache)
        else:
            x = self._rx(self.w["model.embed_tokens.weight"][ids])
            for i in range(self.L):
                x = self._layer(i, x, pos, cache)
        if not all_logits:
            x = x[-1:]
        if self.gpt2:
            hf = self._r(layer_norm(x, self.w["transformer.ln_f.weight"], self.w["transformer.ln_f.bias"], self.eps), "final_norm")
        else:
            hf = self._r(rms_norm(x, self.w["model.norm.weight"], self.eps), "final_norm")
        return hf @ self.lm_head.T

    def _empty_cache(self):
        z = np.zeros((0, self.KV, self.hd))
        return [(z, z) for _ in range(self.L)]

    # ---- public API ----
    def prefill(self, seqs, all_logits: bool = False):
        """Start fresh sequences (slot b <- seqs[b]).  Returns, per sequence,
        logits [S_b, V] if ``all_logits`` else [V] for the last position."""
        self.caches = [self._empty_cache() for _ in seqs]
        out = []
        for b, ids in enumerate(seqs):
            lg = self._forward_seq(b, np.asarray(ids), all_logits)
            out.append(lg if all_logits else lg[0])
        return out

    def extend(self, b: int, ids, all_logits: bool = True) -> np.ndarray:
        """Feed more tokens to slot b (positions continue after its cache; a
        slot never used before starts empty)."""
        while len(self.caches) <= b:
            self.caches.append(self._empty_cache())
        lg = self._forward_seq(b, np.asarray(ids), all_logits)
        return lg if all_logits else lg[0]

    def reset(self, b: int):
        """Drop the sequence of slot b: its cache becomes empty, so the next
        tokens fed to it start at position 0 (admission of a new sequence in
        continuous batching)."""
        while len(self.caches) <= b:
            self.caches.append(self._empty_cache())
        self.caches[b] = self._empty_cache()

    def decode(self, tokens) -> np.ndarray:
        """One token per active slot; returns logits [B, V]."""
        return np.stack([self._forward_seq(b, np.asarray([t]), False)[0]
                         for b, t in enumerate(tokens)])

    def lengths(self):
        return [c[0][0].shape[0] for c in self.caches]


def greedy(logits: np.ndarray) -> np.ndarray:
    """Greedy next token: the first index of the maximum along the last axis."""
    return np.argmax(logits, axis=-1)


def generate_greedy(model: OracleDecoder, seqs, steps: int):
    """Prefill, then ``steps`` greedy decode steps with a fixed step count
    (random-init models have no end-of-sequence token).

    Returns (tokens int64 [B, steps+1], logits float64 [steps+1, B, V]): entry 0
    is the prefill's last-position prediction, entry s the prediction of decode
    step s.  Decode step s consumes the token chosen at entry s-1.
    """
    logits = [np.stack(model.prefill(seqs))]
    toks = [greedy(logits[0])]
    for _ in range(steps):
        lg = model.decode(toks[-1])
        logits.append(lg)
        toks.append(greedy(lg))
    return np.stack(toks, axis=1), np.stack(logits)


def teacher_forced(model: OracleDecoder, seqs, forced: np.ndarray):
    """Prefill, then decode feeding ``forced[:, s]`` at step s (instead of the
    model's own choice).  Returns logits [steps+1, B, V]."""
    logits = [np.stack(model.prefill(seqs))]
    for s in range(forced.shape[1]):
        logits.append(model.decode(forced[:, s]))
    return np.stack(logits)


def _to_f64(t) -> np.ndarray:
    """float64 view of a weight; float64 arrays are used as given (no copy), so
    several oracle instances can share one converted weight map."""
    if hasattr(t, "detach"):
        t = t.detach().to("cpu")
        import torch  # local: only to read torch inputs
        return t.to(torch.float64).numpy()
    return np.asarray(t, dtype=np.float64)


def weights_f64(weights: dict) -> dict:
    """Convert a weight map once, for sharing between oracle instances."""
    return {k: _to_f64(v) for k, v in weights.items()}
