"""The GPT-2 family on the GPU against the float64 oracle.

The complete GPT-2 definition of the Technical Supplement: LayerNorm with bias,
learned positions, the fused c_attn projection with bias (identity rotation
through the shared QKV epilogue), c_proj with bias into the residual stream,
the tanh-GELU MLP with biases, and the head tied to the token embedding.
Cases cover the narrow fused decode projections (<= 16 tokens), the
row-splitting and K-split ones (17..64), decode batches above 64 (GEMMs), an
XL-like geometry (25 heads of 64, hidden 1600), the paged cache, chunked
prefill and graph-replayed continuous-batching steps.
"""
import numpy as np
import pytest
import torch

import oracle
from parity_util import check_argmax, check_bf16, gpu_model, oracle_bf16_storage, oracle_greedy, pack, \
    run_teacher_forced
from synthetic import model_weights, paged_workload, prompts

pytestmark = pytest.mark.gpu


def gpt2_shape(hidden=512, heads=8, layers=2, vocab=3000, inter=None, positions=512):
    return dict(model_type="gpt2", hidden_size=hidden, num_hidden_layers=layers, num_attention_heads=heads,
                num_key_value_heads=heads, head_dim=hidden // heads, intermediate_size=inter or 4 * hidden,
                vocab_size=vocab, max_position_embeddings=positions, tie_word_embeddings=True, attention_bias=True,
                layer_norm_epsilon=1e-5, dtype="bf16")


CASES = {
    # name: (shape, prompt lengths, decode steps, absolute bf16-storage bar)
    "small_hd64": (gpt2_shape(), [37, 130, 300, 5], 6, True),
    # at hidden 1600 bf16 storage alone already moves the logits by a mean of
    # 2.8e-3 (logit std 0.8): held to the band around the exact oracle, as
    # every model of that width
    "xl_geometry_h25": (gpt2_shape(hidden=1600, heads=25, vocab=2000, positions=400), [61, 200, 9], 4, False),
    "batch40_split": (gpt2_shape(), [2 + (i * 29) % 61 for i in range(40)], 4, True),
    "batch80_gemm": (gpt2_shape(), [3 + (i * 37) % 45 for i in range(80)], 3, True),
}


def _ragged(vocab, lens, seed):
    ids = prompts(len(lens), max(lens), vocab, seed=seed).numpy()
    return [ids[i, :n] for i, n in enumerate(lens)]


@pytest.mark.parametrize("case", list(CASES))
def test_gpt2_against_oracle(case):
    shape, lens, steps, absolute = CASES[case]
    w = model_weights(shape, seed=61)
    seqs = _ragged(shape["vocab_size"], lens, seed=62)
    ref_tok, ref_lg = oracle_greedy(shape, w, seqs, steps)
    ref_b = oracle_bf16_storage(shape, w, seqs, ref_tok[:, :steps])
    m = gpu_model(shape, w, max_batch=len(lens), max_seq=max(lens) + steps + 3)
    lg, _ = run_teacher_forced(m, seqs, ref_tok[:, :steps])
    mx = check_bf16(lg, ref_lg, ref_b, case, absolute=absolute)
    check_argmax(lg, ref_lg, mx, case)
    m.close()


def test_gpt2_paged_equals_contiguous():
    shape = gpt2_shape()
    w = model_weights(shape, seed=63)
    steps = 4
    seqs, table, pool = paged_workload(4, 20, 200, steps, shape["vocab_size"], 16, seed=64, spare_pages=3)
    seqs = [s.numpy() for s in seqs]
    ref_tok, ref_lg = oracle_greedy(shape, w, seqs, steps)
    ref_b = oracle_bf16_storage(shape, w, seqs, ref_tok[:, :steps])
    mp = gpu_model(shape, w, max_batch=4, max_seq=208, page_size=16, num_pages=pool)
    lg_p, _ = run_teacher_forced(mp, seqs, ref_tok[:, :steps], block_table=table)
    mx = check_bf16(lg_p, ref_lg, ref_b, "gpt2 paged")
    check_argmax(lg_p, ref_lg, mx, "gpt2 paged")
    mc = gpu_model(shape, w, max_batch=4, max_seq=208)
    lg_c, _ = run_teacher_forced(mc, seqs, ref_tok[:, :steps])
    np.testing.assert_array_equal(lg_p, lg_c)
    mp.close()
    mc.close()


def test_gpt2_chunked_prefill_equals_one_shot_bitwise():
    """Learned positions continue from the chunk's base position."""
    shape = gpt2_shape()
    w = model_weights(shape, seed=65)
    ids = prompts(2, 150, shape["vocab_size"], seed=66).numpy()
    a, b = ids[0], ids[1, :70]
    one = gpu_model(shape, w, max_batch=2, max_seq=160)
    flat, cu = pack([a, b])
    ref, _ = one.prefill(flat, cu)
    ref = ref.cpu().numpy()
    one.close()
    m = gpu_model(shape, w, max_batch=2, max_seq=160)
    m.step(*pack([a[:60], b[:25]]), [0, 1], [1, 1])
    lg1, _ = m.step(*pack([a[60:120], b[25:]]), [0, 1], [0, 0])
    lg2, _ = m.step(*pack([a[120:]]), [0], [0])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lg2.cpu().numpy()[0], ref[0])
    np.testing.assert_array_equal(lg1.cpu().numpy()[1], ref[1])
    m.close()


def test_gpt2_step_admission_then_graph_decode():
    """Sequences admitted by steps (slots scrambled) continue through the
    graph-replayed decode step and through decode-only steps."""
    shape = gpt2_shape(hidden=384, heads=6, vocab=1500)
    w = model_weights(shape, seed=67)
    ids = prompts(3, 70, shape["vocab_size"], seed=68).numpy()
    seqs = [ids[0, :70], ids[1, :33], ids[2, :5]]
    steps = 4
    w64 = oracle.weights_f64(w)
    ref_tok, ref_lg = oracle.generate_greedy(oracle.OracleDecoder(shape, w64), seqs, steps)
    ref_b = oracle.teacher_forced(oracle.OracleDecoder(shape, w64, io_round="bf16"), seqs, ref_tok[:, :steps])
    m = gpu_model(shape, w, max_batch=3, max_seq=96)
    lg_0, _ = m.step(*pack([seqs[2], seqs[0][:40]]), [2, 0], [1, 1])
    lg_1, _ = m.step(*pack([seqs[0][40:], seqs[1]]), [0, 1], [0, 1])
    got = np.zeros((steps + 1, 3, shape["vocab_size"]))
    got[0, 2] = lg_0[0].cpu().double().numpy()
    got[0, 0] = lg_1[0].cpu().double().numpy()
    got[0, 1] = lg_1[1].cpu().double().numpy()
    for s in range(steps):
        if s % 2 == 0:  # the graph-replayed decode step
            tok = torch.as_tensor(ref_tok[:, s].astype(np.int32)).to("cuda")
            lg = torch.empty((3, shape["vocab_size"]), dtype=torch.float32, device="cuda")
            m.decode_step(tok, logits=lg)
            got[s + 1] = lg.cpu().double().numpy()
        else:  # a decode-only continuous-batching step, slots in another order
            order = [1, 2, 0]
            flat, cu = pack([[int(ref_tok[b, s])] for b in order])
            lg, _ = m.step(flat, cu, order, [0, 0, 0])
            for i, b in enumerate(order):
                got[s + 1, b] = lg[i].cpu().double().numpy()
    torch.cuda.synchronize()
    assert m.lengths() == [70 + steps, 33 + steps, 5 + steps]
    mx = check_bf16(got, ref_lg, ref_b, "gpt2 step admission + decode")
    check_argmax(got, ref_lg, mx, "gpt2 step admission + decode")
    m.close()
