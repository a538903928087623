"""Shared helpers of the GPU parity tests (imported by test modules only)."""
from __future__ import annotations

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


def top2_gap(lg: np.ndarray) -> np.ndarray:
    part = np.sort(lg, axis=-1)
    return part[..., -1] - part[..., -2]


def check_logits(gpu: np.ndarray, ref: np.ndarray, max_tol: float, mean_tol: float | None, what: str):
    err = np.abs(gpu - ref)
    mx, mean = float(err.max()), float(err.mean())
    print(f"{what}: max|dlogit| = {mx:.3e}, mean = {mean:.3e}, logit std = {ref.std():.3f}")
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite logits"
    assert mx < max_tol, f"{what}: max abs error {mx:.3e} >= {max_tol}"
    if mean_tol is not None:
        assert mean < mean_tol, f"{what}: mean abs error {mean:.3e} >= {mean_tol}"
    return mx


def check_argmax(gpu_logits: np.ndarray, ref_logits: np.ndarray, max_err: float, what: str):
    """Greedy decisions must agree wherever the oracle's top-2 gap exceeds what
    the measured logit error can flip (2 x max error)."""
    g = np.argmax(gpu_logits, -1)
    r = np.argmax(ref_logits, -1)
    gap = top2_gap(ref_logits)
    bad = (g != r) & (gap >= 2 * max_err)
    flips = int((g != r).sum())
    print(f"{what}: {flips} near-tie flips of {g.size} decisions")
    assert not bad.any(), f"{what}: argmax differs at gaps {gap[bad]}"


def oracle_greedy(shape, weights, seqs, steps, io_round=None):
    return oracle.generate_greedy(oracle.OracleDecoder(shape, weights, io_round=io_round), seqs, steps)


def oracle_bf16_storage(shape, weights, seqs, forced):
    """Oracle logits at bf16 storage precision, teacher-forced on ``forced``."""
    return oracle.teacher_forced(oracle.OracleDecoder(shape, weights, io_round="bf16"), seqs, forced)


def check_bf16(gpu: np.ndarray, exact: np.ndarray, bf16_ref: np.ndarray, what: str, absolute: bool = True):
    """bf16-path logits: no further from the exact oracle than BAND x the error
    that bf16 storage alone causes (the bf16-storage oracle's distance from
    the exact one), and -- where ``absolute`` -- within 2e-2 / 2e-3 of the
    bf16-storage oracle."""
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
