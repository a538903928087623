"""Sliding-window attention on the GPU against the float64 oracle.

A query at position p attends to keys p - W + 1 .. p (the masking built-in's
window; Mistral-style).  The cases put the window's lower edge inside 64-key
prefill tiles and 32-key decode chunks (W not a multiple of either), cross it
in prefill query tiles of 128, split decode keys over workgroups with the
window starting inside the first split, and run it through the paged cache,
the float32 check mode and chunked prefill.
"""
import numpy as np
import pytest
import torch

from parity_util import (F32_MAX, check_argmax, check_bf16, check_logits, gpu_model, oracle_bf16_storage,
                         oracle_greedy, pack, run_teacher_forced)
from synthetic import model_weights, paged_workload, prompts, small_shape

pytestmark = pytest.mark.gpu

CASES = {
    # name: (base shape, overrides, window, prompt lengths, decode steps)
    "llama_hd64_w48": ("1b", dict(layers=2, vocab=3000, hidden=512, intermediate=1024), 48, [37, 130, 300, 5], 6),
    "qwen_hd128_w200": ("7b", dict(layers=2, vocab=2048, hidden=896, intermediate=1792), 200, [129, 400, 77], 5),
    # two sequences of four kv heads: the decode keys are split in two, and
    # the window starts inside the first split
    "qwen_hd128_w1000_split": ("7b", dict(layers=2, vocab=1500, hidden=640, intermediate=1280), 1000,
                               [1500, 1210], 3),
}


def _shape(base, ov, window):
    s = small_shape(base, **ov)
    s["sliding_window"] = window
    return s


def _ragged(vocab, lens, seed):
    ids = prompts(len(lens), max(lens), vocab, seed=seed).numpy()
    return [ids[i, :n] for i, n in enumerate(lens)]


@pytest.mark.parametrize("case", list(CASES))
def test_window_against_oracle(case):
    base, ov, W, lens, steps = CASES[case]
    shape = _shape(base, ov, W)
    w = model_weights(shape, seed=51)
    seqs = _ragged(shape["vocab_size"], lens, seed=52)
    ref_tok, ref_lg = oracle_greedy(shape, w, seqs, steps)
    ref_b = oracle_bf16_storage(shape, w, seqs, ref_tok[:, :steps])
    m = gpu_model(shape, w, max_batch=len(lens), max_seq=max(lens) + steps + 3)
    lg, _ = run_teacher_forced(m, seqs, ref_tok[:, :steps])
    mx = check_bf16(lg, ref_lg, ref_b, case)
    check_argmax(lg, ref_lg, mx, case)
    m.close()


def test_window_paged_equals_contiguous():
    shape = _shape("7b", dict(layers=2, vocab=2048, hidden=896, intermediate=1792), 90)
    w = model_weights(shape, seed=53)
    steps = 5
    seqs, table, pool = paged_workload(4, 40, 260, steps, shape["vocab_size"], 16, seed=54, spare_pages=5)
    seqs = [s.numpy() for s in seqs]
    ref_tok, ref_lg = oracle_greedy(shape, w, seqs, steps)
    ref_b = oracle_bf16_storage(shape, w, seqs, ref_tok[:, :steps])
    mp = gpu_model(shape, w, max_batch=4, max_seq=272, page_size=16, num_pages=pool)
    lg_p, _ = run_teacher_forced(mp, seqs, ref_tok[:, :steps], block_table=table)
    mx = check_bf16(lg_p, ref_lg, ref_b, "window, paged")
    check_argmax(lg_p, ref_lg, mx, "window, paged")
    mc = gpu_model(shape, w, max_batch=4, max_seq=272)
    lg_c, _ = run_teacher_forced(mc, seqs, ref_tok[:, :steps])
    np.testing.assert_array_equal(lg_p, lg_c)
    mp.close()
    mc.close()


def test_window_f32_check_mode():
    shape = _shape("7b", dict(layers=2, vocab=2048, hidden=896, intermediate=1792), 37)
    shape["dtype"] = "f32"
    w = {k: v.float() for k, v in model_weights(dict(shape, dtype="bf16"), seed=55).items()}
    seqs = _ragged(shape["vocab_size"], [20, 90], seed=56)
    steps = 6
    ref_tok, ref_lg = oracle_greedy(shape, w, seqs, steps)
    m = gpu_model(shape, w, max_batch=2, max_seq=100)
    lg, _ = run_teacher_forced(m, seqs, ref_tok[:, :steps])
    check_logits(lg, ref_lg, F32_MAX, None, "window, f32 check mode")
    m.close()


def test_window_chunked_prefill_equals_one_shot_bitwise():
    """Chunks continue a slot from position base > 0, so the window's lower
    edge falls before the chunk: the same keys in the same tile order."""
    shape = _shape("1b", dict(layers=2, vocab=3000, hidden=512, intermediate=1024), 70)
    w = model_weights(shape, seed=57)
    ids = prompts(2, 260, shape["vocab_size"], seed=58).numpy()
    a, b = ids[0], ids[1, :150]
    one = gpu_model(shape, w, max_batch=2, max_seq=270)
    flat, cu = pack([a, b])
    ref, _ = one.prefill(flat, cu)
    ref = ref.cpu().numpy()
    one.close()
    m = gpu_model(shape, w, max_batch=2, max_seq=270)
    m.step(*pack([a[:100], b[:45]]), [0, 1], [1, 1])
    lg1, _ = m.step(*pack([a[100:190], b[45:]]), [0, 1], [0, 0])
    lg2, _ = m.step(*pack([a[190:]]), [0], [0])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lg2.cpu().numpy()[0], ref[0])
    np.testing.assert_array_equal(lg1.cpu().numpy()[1], ref[1])
    m.close()
