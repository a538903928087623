"""Shared helpers of the GPU parity tests (imported by test modules only)."""
from __future__ import annotations

import math
import sys
import time

import numpy as np
import torch

import oracle
from paper_2608_19889_amd.axon import Model

# Tolerances on logits.  bf16 path: max-abs 2e-2 and mean-abs 2e-3 against the
# oracle evaluated at the paper's primary precision (bfloat16 storage of every
# activation the GPU stores: normed inputs, q/k/v and the KV cache, attention
# output, gated MLP activation; float32 residual stream), and against the exact
# float64 oracle no more than BAND times the error that this bf16 storage alone
# causes.  float32 check mode: 1e-4 max-abs against the exact float64 oracle.
BF16_MAX, BF16_MEAN = 2e-2, 2e-3
BAND = 1.5
F32_MAX = 1e-4
# A greedy decision may differ from the oracle's only where the oracle's
# margin between the two tokens is below GREEDY_SIGMAS x the root-mean-square
# logit error of that decision's own row (the errors of one row are spread
# alike over the vocabulary: the head multiplies one error vector by random
# rows, so a flip past 6 sigma has probability ~1e-5).
GREEDY_SIGMAS = 6.0


def progress(msg: str):
    """A progress line on the real stderr (not captured by pytest), so a long
    oracle run shows that it is advancing."""
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", file=sys.__stderr__, flush=True)


def gpu_model(shape, weights, max_batch, max_seq, **kw) -> Model:
    return Model(shape, {k: v.to("cuda") for k, v in weights.items()}, max_batch=max_batch, max_seq=max_seq, **kw)


def pack(seqs):
    flat = torch.cat([torch.as_tensor(np.asarray(s), dtype=torch.int32) for s in seqs]).to("cuda")
    cu = [0]
    for s in seqs:
        cu.append(cu[-1] + len(s))
    return flat, cu


def run_teacher_forced(m: Model, seqs, forced: np.ndarray, block_table=None):
    """GPU prefill, then decode feeding forced[:, s]; returns logits [steps+1, B, V]
    and the GPU's own argmax tokens [B, steps+1]."""
    flat, cu = pack(seqs)
    lg, nxt = m.prefill(flat, cu, block_table=block_table)
    out, toks = [lg], [nxt.clone()]
    B = len(seqs)
    for s in range(forced.shape[1]):
        tok = torch.as_tensor(forced[:, s].astype(np.int32)).to("cuda")
        lg = torch.empty((B, m.vocab), dtype=torch.float32, device="cuda")
        _, nx = m.decode_step(tok, logits=lg)
        out.append(lg)
        toks.append(nx.clone())
    torch.cuda.synchronize()
    return (torch.stack(out).cpu().double().numpy(), torch.stack(toks, 1).cpu().numpy())


def run_free(m: Model, seqs, steps: int, block_table=None):
    """GPU greedy generation: tokens [B, steps+1] (entry 0 from the prefill)."""
    flat, cu = pack(seqs)
    _, nxt = m.prefill(flat, cu, block_table=block_table, want_logits=False)
    toks = [nxt.clone()]
    a = nxt
    b = torch.empty_like(nxt)
    for _ in range(steps):
        m.decode_step(a, next_tokens=b)
        toks.append(b.clone())
        a, b = b, a
    torch.cuda.synchronize()
    return torch.stack(toks, 1).cpu().numpy()



def check_logits(gpu: np.ndarray, ref: np.ndarray, max_tol: float, mean_tol: float | None, what: str):
    err = np.abs(gpu - ref)
    mx, mean = float(err.max()), float(err.mean())
    print(f"{what}: max|dlogit| = {mx:.3e}, mean = {mean:.3e}, logit std = {ref.std():.3f}")
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite logits"
    assert mx < max_tol, f"{what}: max abs error {mx:.3e} >= {max_tol}"
    if mean_tol is not None:
        assert mean < mean_tol, f"{what}: mean abs error {mean:.3e} >= {mean_tol}"
    return mx


def check_greedy(gpu: np.ndarray, exact: np.ndarray, what: str, b16: np.ndarray | None = None,
                 strict: bool = False):
    """Greedy decisions, one per row of [steps+1, B, V] logits (teacher-forced,
    so every row has the oracle's history).

    Every decision where the GPU's argmax differs from the exact oracle's is
    listed with the oracle's margin between the two tokens, that row's RMS and
    max logit error, and the choice of the bf16-storage oracle at the same
    decision (where ``b16`` covers that row).  A flip is accepted only if its
    margin is below GREEDY_SIGMAS x the row's RMS error, and the number of
    flips may not exceed what those errors explain: the expected count
    sum over rows and the 8 strongest rivals of P(N(0, 2 rms^2) > gap), plus 4
    standard deviations and 2.  ``strict``: no flip at all (float32 check
    mode).  Returns the flipped (step, sequence) pairs."""
    S, B, V = gpu.shape
    g_all = np.argmax(gpu, -1)
    r_all = np.argmax(exact, -1)
    flips, expected = [], 0.0
    for s in range(S):
        for b in range(B):
            row_g, row_r = gpu[s, b], exact[s, b]
            err = row_g - row_r
            rms = float(np.sqrt(np.mean(err * err)))
            r = int(r_all[s, b])
            rivals = np.partition(row_r, V - 9)[V - 9:] if V > 9 else np.sort(row_r)
            gaps = row_r[r] - np.sort(rivals)[:-1]
            if rms > 0:
                expected += float(sum(0.5 * math.erfc(gp / (2.0 * rms)) for gp in gaps))
            g = int(g_all[s, b])
            if g == r:
                continue
            margin = float(row_r[r] - row_r[g])
            verdict = "not computed"
            if b16 is not None and s < b16.shape[0]:
                c = int(np.argmax(b16[s, b]))
                verdict = "the GPU's token" if c == g else ("the oracle's token" if c == r else f"token {c}")
            flips.append((s, b))
            print(f"{what}: flip at step {s}, sequence {b}: oracle {r} vs GPU {g}, oracle margin {margin:.3e} "
                  f"= {margin / rms:.2f} x row rms error {rms:.3e} (row max {np.abs(err).max():.3e}); "
                  f"bf16-storage oracle chooses {verdict}")
            assert not strict, f"{what}: greedy token differs at step {s}, sequence {b}"
            assert margin < GREEDY_SIGMAS * rms, \
                f"{what}: flip at step {s}, sequence {b} with margin {margin:.3e} > {GREEDY_SIGMAS} x rms {rms:.3e}"
    bound = expected + 4.0 * math.sqrt(expected) + 2.0
    print(f"{what}: {len(flips)} flips of {S * B} greedy decisions (expected from the row errors {expected:.2f}, "
          f"bound {bound:.1f})")
    assert len(flips) <= bound, f"{what}: {len(flips)} flips, more than the row errors explain ({bound:.1f})"
    return flips


def check_free_running(free: np.ndarray, oracle_tokens: np.ndarray, forced_gpu: np.ndarray, what: str):
    """Free-running GPU greedy tokens [B, steps+1] against the oracle's.  Up to
    its first divergence a sequence has the same history in the free run as
    in the teacher-forced run, so it must follow the oracle exactly until the
    first teacher-forced flip (``forced_gpu``: the GPU's argmax under teacher
    forcing) and, at that step, choose the token the teacher-forced run chose
    (a flip already held to the margin bar).  Without a flip every token must
    be the oracle's."""
    B, n = free.shape
    for b in range(B):
        diff = np.nonzero(free[b] != oracle_tokens[b])[0]
        tf = np.nonzero(forced_gpu[b] != oracle_tokens[b])[0]
        first = int(diff[0]) if diff.size else n
        first_tf = int(tf[0]) if tf.size else n
        print(f"{what}: sequence {b} follows the oracle for {first} of {n} greedy tokens"
              + (f" (first teacher-forced flip at step {first_tf})" if tf.size else ""))
        assert first == first_tf, f"{what}: sequence {b} diverges at {first}, teacher-forced flip at {first_tf}"
        if first < n:
            assert free[b, first] == forced_gpu[b, first], f"{what}: sequence {b} diverged to another token"


def check_argmax(gpu_logits: np.ndarray, ref_logits: np.ndarray, max_err: float, what: str):
    """Greedy decisions of any stack of logit rows [..., V], each decision held
    to its own row's error by check_greedy (``max_err``, the largest error over
    all rows, is only printed)."""
    V = gpu_logits.shape[-1]
    print(f"{what}: largest logit error over all rows {max_err:.3e}")
    return check_greedy(gpu_logits.reshape(-1, 1, V), ref_logits.reshape(-1, 1, V), what)


def oracle_greedy(shape, weights, seqs, steps, io_round=None):
    return oracle.generate_greedy(oracle.OracleDecoder(shape, weights, io_round=io_round), seqs, steps)


def oracle_bf16_storage(shape, weights, seqs, forced):
    """Oracle logits at bf16 storage precision, teacher-forced on ``forced``."""
    return oracle.teacher_forced(oracle.OracleDecoder(shape, weights, io_round="bf16"), seqs, forced)


def check_bf16(gpu: np.ndarray, exact: np.ndarray, bf16_ref: np.ndarray, what: str, absolute: bool = True):
    """bf16-path logits: no further from the exact oracle than BAND x the error
    that bf16 storage alone causes (the bf16-storage oracle's distance from
    the exact one), and -- where ``absolute`` -- within 2e-2 / 2e-3 of the
    bf16-storage oracle.  ``bf16_ref`` may cover only the first steps (rows
    of the leading axis): the storage error is then measured on those and the
    band applied to every step, the absolute bar to the covered ones."""
    k = bf16_ref.shape[0]
    if k < gpu.shape[0]:
        inherent = np.abs(bf16_ref - exact[:k])
        err = np.abs(gpu - exact)
        print(f"{what}: vs exact max {err.max():.3e} mean {err.mean():.3e} over {gpu.shape[0]} steps; bf16 storage "
              f"alone (first {k} steps) max {inherent.max():.3e} mean {inherent.mean():.3e}")
        assert np.all(np.isfinite(gpu)), f"{what}: non-finite logits"
        assert err.max() <= BAND * inherent.max() + 1e-3, (err.max(), inherent.max())
        assert err.mean() <= BAND * inherent.mean() + 1e-4, (err.mean(), inherent.mean())
        if absolute:
            check_logits(gpu[:k], bf16_ref, BF16_MAX, BF16_MEAN, what + " vs bf16-storage oracle")
        return float(err.max())
    inherent = np.abs(bf16_ref - exact)
    err = np.abs(gpu - exact)
    vs_b = np.abs(gpu - bf16_ref)
    print(f"{what}: vs exact max {err.max():.3e} mean {err.mean():.3e}; bf16 storage alone max "
          f"{inherent.max():.3e} mean {inherent.mean():.3e}; vs bf16-storage oracle max {vs_b.max():.3e} "
          f"mean {vs_b.mean():.3e}; logit std {exact.std():.3f}")
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite logits"
    assert err.max() <= BAND * inherent.max() + 1e-3, (err.max(), inherent.max())
    assert err.mean() <= BAND * inherent.mean() + 1e-4, (err.mean(), inherent.mean())
    if absolute:
        check_logits(gpu, bf16_ref, BF16_MAX, BF16_MEAN, what + " vs bf16-storage oracle")
    return float(err.max())
