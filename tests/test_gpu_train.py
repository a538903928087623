"""The backward pass on the GPU against the float64 oracle.

Loss and the gradient of every weight (embedding with the tied head, norm
gains, q/k/v weights and biases back through RoPE and the grouped-row layout,
O, the interleaved gate/up, down) for ragged batches with uncounted
positions, including sequences of 1 token, of exact multiples of the
attention backward's 32-position blocks and one position past a block.

The GPU stores activations and gradients in bf16 between kernels (float32
accumulation, float32 residual stream and residual gradient).  Each such
rounding has relative error up to 2^-9, and a gradient element passes through
several of them (the head's gradient, the bf16 input gradient of every GEMM,
P in attention), so its error is a sum of several independent rounding
errors of the size of the tensor's entries.  dS in attention is a bf16 pair
(hi + lo): its rows sum to zero, so dQ = dS K and dK = dS^T Q cancel, and a
single bf16 rounding of dS left the q / k gradients with relative L2 errors
near 1e-2.  Bars, per tensor with reference r:
  * every element: |g - r| <= 32 * 2^-8 * scale + 4 * 2^-8 * |r|, the scale
    being the tensor's rms or, where larger, its row's.  Measured errors
    reach 8% of the scale (a gradient row dominated by one token whose input
    gradient cancels in its bf16 dot product), so the bar is 12.5%: a wrong
    row, column or block, or a missing or doubled token contribution to a
    row, fails it;
  * every embedding row of an input token (that token's own gradient,
    flowing back through every layer, so an error confined to a few
    positions or keys shows there undiluted): relative L2 error < 5e-2;
  * relative L2 error < 3e-2;
  * loss within 2e-3 (about 8 here).
"""
import numpy as np
import pytest
import torch

import oracle
from parity_util import gpu_model, pack
from synthetic import model_weights, prompts, small_shape

pytestmark = pytest.mark.gpu

CASES = {
    # tied head, head_dim 64, group 4
    "llama_hd64_tied": ("1b", dict(layers=2, vocab=3000, hidden=512, intermediate=1024), [37, 130, 65, 5]),
    # untied head, q/k/v biases, head_dim 128, group 7
    "qwen_hd128_bias": ("7b", dict(layers=2, vocab=2048, hidden=896, intermediate=1792), [100, 33, 71]),
    # 600 tokens: the narrow projections (hidden 512) have fewer than 160
    # output tiles of 256 and split K (float32 partials summed in order)
    "llama_hd64_split_k": ("1b", dict(layers=2, vocab=3000, hidden=512, intermediate=1024), [200, 310, 90]),
    # block edges of the attention backward: 1 token, exact multiples of 32,
    # one past a multiple
    "llama_hd64_block_edges": ("1b", dict(layers=2, vocab=3000, hidden=512, intermediate=1024), [1, 32, 64, 33]),
    "qwen_hd128_block_edges": ("7b", dict(layers=2, vocab=2048, hidden=896, intermediate=1792), [33, 1, 96, 32]),
}

ULP = 2.0 ** -8


def check_gradient(name: str, g: np.ndarray, r: np.ndarray):
    """Element-wise and relative-L2 bars of one gradient tensor; returns
    (relative L2 error, largest |g - r| / scale).  The scale of an element is
    the tensor's rms, or its row's rms where that is larger (row i of a
    matrix gradient sums the products of output feature i's gradient, so its
    errors follow that row's magnitude: the tied embedding's rows of input
    tokens also carry the gradient that flows back through every layer)."""
    assert np.all(np.isfinite(g)), name
    scale = np.full(r.shape, float(np.sqrt(np.mean(r * r))))
    if r.ndim == 2:
        scale = np.maximum(scale, np.sqrt(np.mean(r * r, axis=1, keepdims=True)))
    err = np.abs(g - r)
    bound = 32 * ULP * scale + 4 * ULP * np.abs(r)
    bad = np.argwhere(err > bound)
    assert bad.size == 0, (f"{name}: {len(bad)} elements beyond the bar, first at {tuple(bad[0])}: "
                           f"got {g[tuple(bad[0])]:.4e}, oracle {r[tuple(bad[0])]:.4e}, "
                           f"scale {scale[tuple(bad[0])]:.3e}")
    rel = float(np.linalg.norm(g - r) / np.linalg.norm(r))
    assert rel < 3e-2, (name, rel)
    return rel, float((err / scale).max())


def check_token_rows(g: np.ndarray, r: np.ndarray, tokens: np.ndarray):
    """Relative L2 error of the embedding gradient's rows of the input tokens."""
    worst = 0.0
    for v in np.unique(tokens):
        nr = float(np.linalg.norm(r[v]))
        if nr == 0.0:  # a token no counted position depends on: exactly zero
            assert float(np.abs(g[v]).max()) == 0.0, f"embedding row of token {v} should be zero"
            continue
        e = float(np.linalg.norm(g[v] - r[v])) / nr
        worst = max(worst, e)
        assert e < 5e-2, f"embedding row of token {v}: relative L2 error {e:.3e}"
    return worst


def _targets(seqs, vocab, seed):
    r = np.random.default_rng(seed)
    out = []
    for s in seqs:
        t = np.append(s[1:], -1).astype(np.int64)
        t[r.random(len(t)) < 0.1] = -1  # some positions are not counted
        out.append(t)
    return out


@pytest.mark.parametrize("case", list(CASES))
def test_loss_and_grads_against_oracle(case):
    base, ov, lens = CASES[case]
    shape = small_shape(base, **ov)
    w = model_weights(shape, seed=71)
    ids = prompts(len(lens), max(lens), shape["vocab_size"], seed=72).numpy()
    seqs = [ids[i, :n] for i, n in enumerate(lens)]
    tg = _targets(seqs, shape["vocab_size"], seed=73)
    ref_loss, ref = oracle.loss_and_grads(shape, oracle.weights_f64(w), seqs, tg)
    m = gpu_model(shape, w, max_batch=len(lens), max_seq=max(lens))
    flat, cu = pack(seqs)
    targets = torch.as_tensor(np.concatenate(tg).astype(np.int32)).to("cuda")
    grads = {k: torch.full(tuple(v.shape), float("nan"), dtype=torch.float32, device="cuda") for k, v in w.items()}
    loss = m.loss_and_grads(flat, cu, targets, grads)
    torch.cuda.synchronize()
    got = float(loss.item())
    print(f"{case}: loss {got:.6f} vs oracle {ref_loss:.6f}")
    assert abs(got - ref_loss) < 2e-3
    worst, worst_name, worst_el, worst_el_name = 0.0, "", 0.0, ""
    for name, r in ref.items():
        rel, el = check_gradient(name, grads[name].cpu().double().numpy(), r)
        print(f"  {name}: relative L2 {rel:.2e}, largest element error {el:.2e} x scale")
        if rel > worst:
            worst, worst_name = rel, name
        if el > worst_el:
            worst_el, worst_el_name = el, name
    print(f"{case}: largest relative L2 gradient error {worst:.3e} ({worst_name}); largest element error "
          f"{worst_el:.3e} x scale ({worst_el_name})")
    emb = "model.embed_tokens.weight"
    tr = check_token_rows(grads[emb].cpu().double().numpy(), ref[emb], np.concatenate(seqs))
    print(f"{case}: largest relative L2 error of an input token's embedding row {tr:.3e}")
    # a second call on another batch overwrites every gradient
    loss2 = m.loss_and_grads(*pack(seqs[:2]), targets[:sum(lens[:2])], grads)
    ref_loss2, ref2 = oracle.loss_and_grads(shape, oracle.weights_f64(w), seqs[:2], tg[:2])
    torch.cuda.synchronize()
    assert abs(float(loss2.item()) - ref_loss2) < 2e-3
    for name, r in ref2.items():
        check_gradient(name, grads[name].cpu().double().numpy(), r)
    check_token_rows(grads[emb].cpu().double().numpy(), ref2[emb], np.concatenate(seqs[:2]))
    m.close()


def test_backward_rejects_other_model_kinds():
    from paper_2608_19889_amd import axon as ax
    shape = dict(small_shape("1b", layers=1, vocab=500, hidden=256, intermediate=512), sliding_window=16)
    w = model_weights(shape, seed=74)
    m = gpu_model(shape, w, max_batch=1, max_seq=32)
    flat, cu = pack([np.arange(8)])
    grads = {k: torch.zeros(tuple(v.shape), dtype=torch.float32, device="cuda") for k, v in w.items()}
    with pytest.raises(ax.AxonError, match="backward pass covers"):
        m.loss_and_grads(flat, cu, flat.clone(), grads)
    m.close()


def test_gradient_map_is_validated_and_uncounted_batches_give_zero():
    from paper_2608_19889_amd import axon as ax
    shape = small_shape("1b", layers=1, vocab=500, hidden=256, intermediate=512)
    w = model_weights(shape, seed=75)
    m = gpu_model(shape, w, max_batch=2, max_seq=32)
    flat, cu = pack([np.arange(9), np.arange(5)])
    grads = {k: torch.full(tuple(v.shape), 7.0, dtype=torch.float32, device="cuda") for k, v in w.items()}
    # no position counted: loss 0 and every gradient 0 (overwritten, not left as 7)
    none = torch.full((14,), -1, dtype=torch.int32, device="cuda")
    loss = m.loss_and_grads(flat, cu, none, grads)
    torch.cuda.synchronize()
    assert float(loss.item()) == 0.0
    for name, g in grads.items():
        assert float(g.abs().max().item()) == 0.0, name
    # the map must match the weights exactly: dtype, names, shapes, device buffers
    bad = dict(grads)
    bad["model.norm.weight"] = torch.zeros(256, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ax.AxonError, match="AXON_F32"):
        m.loss_and_grads(flat, cu, none, bad)
    bad = dict(grads)
    del bad["model.layers.0.mlp.up_proj.weight"]
    with pytest.raises(ax.AxonError, match="missing gradient"):
        m.loss_and_grads(flat, cu, none, bad)
    bad = dict(grads)
    bad["model.layers.0.self_attn.o_proj.weight"] = torch.zeros((256, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(ax.AxonError, match="o_proj"):
        m.loss_and_grads(flat, cu, none, bad)
    bad = dict(grads)
    bad["model.norm.weight"] = torch.zeros(256, dtype=torch.float32)  # host memory
    with pytest.raises(ax.AxonError, match="device buffer"):
        m.loss_and_grads(flat, cu, none, bad)
    m.close()
