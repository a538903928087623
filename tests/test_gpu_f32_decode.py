"""The float32 decode step (check mode and the 135M-shaped float32 model)
against the float64 oracle: the fused float32 projections (RMSNorm folded into
the projections that read the normed rows, bias + RoPE + KV write, SiLU gate,
residual, head with argmax partials), and both attention paths: attention
recomputed inside every O-projection workgroup (contexts up to 128 keys, at
most 4 sequences) and the grouped float32 decode attention kernel beyond.

Each case: logits within 1e-4 of the oracle at every teacher-forced step, and
free-running greedy tokens identical to the oracle's.
"""
import numpy as np
import pytest

from parity_util import F32_MAX, check_logits, gpu_model, oracle_greedy, run_free, run_teacher_forced
from synthetic import model_weights, prompts, small_shape

pytestmark = pytest.mark.gpu

CASES = {
    # name: (base, overrides, prompt lengths, decode steps, max_seq, sliding window)
    # head_dim 64, group of 3: attention inside the O projection, 2 key chunks
    "hd64_fused_two_chunks": ("135m", dict(layers=2, vocab=1000), [5, 60, 110], 6, 120, 0),
    # the same model with a capacity above 128 keys: the attention kernel
    # (4 wavefronts, several 64-key chunks, merged)
    "hd64_kernel_long": ("135m", dict(layers=2, vocab=1000), [5, 140, 290], 6, 300, 0),
    # head_dim 128, group of 7 with QKV biases, 4 sequences, fused
    "hd128_fused_bias": ("7b", dict(layers=2, vocab=1024, hidden=896, intermediate=1792), [3, 33, 64, 97], 5, 104, 0),
    # a sliding window shorter than the contexts, fused and not
    "hd64_fused_window": ("135m", dict(layers=2, vocab=1000), [30, 100], 6, 110, 40),
    "hd128_kernel_window": ("7b", dict(layers=2, vocab=1024, hidden=896, intermediate=1792), [70, 200], 5, 210, 90),
    # 16 sequences (the widest float32 fused projection), attention kernel
    "hd64_batch16": ("135m", dict(layers=2, vocab=1000), [3 + (i * 13) % 50 for i in range(16)], 4, 60, 0),
}


@pytest.mark.parametrize("case", list(CASES))
def test_f32_decode_against_oracle(case):
    base, ov, lens, steps, max_seq, window = CASES[case]
    print(f"[f32 decode] {case}", flush=True)
    shape = small_shape(base, **ov)
    shape["dtype"] = "f32"
    if window:
        shape["sliding_window"] = window
    w = {k: v.float() for k, v in model_weights(dict(shape, dtype="bf16"), seed=61).items()}
    ids = prompts(len(lens), max(lens), shape["vocab_size"], seed=62).numpy()
    seqs = [ids[i, :n] for i, n in enumerate(lens)]
    ref_tok, ref_lg = oracle_greedy(shape, w, seqs, steps)
    m = gpu_model(shape, w, max_batch=len(lens), max_seq=max_seq)
    lg, _ = run_teacher_forced(m, seqs, ref_tok[:, :steps])
    check_logits(lg, ref_lg, F32_MAX, None, case)
    np.testing.assert_array_equal(run_free(m, seqs, steps), ref_tok)
    m.close()
