"""GPU properties at the workloads' sizes that hold without the oracle.

Checked bit for bit where the arithmetic is identical: the paged cache equals
the contiguous one (7B shape, ragged prompts, permuted pages); a sequence's
logits do not depend on the other sequences of its batch; the graph-replayed
decode step equals the eager one.  Across kernels, the decode step's logits
agree with the all-positions prefill of the same tokens.  Capacity errors are
reported without side effects.  (Oracle parity at the workloads' own sizes is
in test_gpu_atsize.py.)
"""
import numpy as np
import pytest
import torch

from paper_2608_19889_amd.axon import AxonError, Model
from parity_util import BF16_MAX, BF16_MEAN, F32_MAX, check_logits, pack
from synthetic import MODEL_SHAPES, model_weights, paged_workload, prompts, small_shape

pytestmark = pytest.mark.gpu


def test_7b_paged_equals_contiguous_bitwise():
    shape = MODEL_SHAPES["7b"]
    steps = 4
    w = model_weights(shape, seed=1, device="cuda")
    seqs, table, pool = paged_workload(6, 64, 4096, steps, shape["vocab_size"], 16, seed=11)
    max_seq = max(len(s) for s in seqs) + steps
    flat, cu = pack([s.numpy() for s in seqs])
    outs = []
    for kw in (dict(page_size=16, num_pages=pool), {}):
        m = Model(shape, w, max_batch=6, max_seq=max_seq, max_tokens=cu[-1], **kw)
        lg, nxt = m.prefill(flat, cu, block_table=table if kw else None)
        res = [lg.cpu()]
        for _ in range(steps):
            lg = torch.empty((6, shape["vocab_size"]), dtype=torch.float32, device="cuda")
            _, nxt = m.decode_step(nxt, logits=lg)
            res.append(lg.cpu())
        torch.cuda.synchronize()
        outs.append(torch.stack(res))
        m.close()
    assert torch.isfinite(outs[0]).all()
    assert torch.equal(outs[0], outs[1])


def test_batch_composition_invariance_bitwise():
    """Slot 1 holds the same sequence in two batches of the same size."""
    shape = MODEL_SHAPES["1b"]
    w = model_weights(shape, seed=2, device="cuda")
    ids = prompts(5, 200, shape["vocab_size"], seed=4).numpy()
    batches = [[ids[0, :50], ids[1, :120], ids[2, :200]], [ids[3, :190], ids[1, :120], ids[4, :7]]]
    res = []
    for seqs in batches:
        m = Model(shape, w, max_batch=3, max_seq=256)
        flat, cu = pack(seqs)
        lg, nxt = m.prefill(flat, cu)
        out = [lg[1].cpu()]
        tok = nxt
        for _ in range(3):
            lg = torch.empty((3, shape["vocab_size"]), dtype=torch.float32, device="cuda")
            _, tok = m.decode_step(tok, logits=lg)
            out.append(lg[1].cpu())
        torch.cuda.synchronize()
        res.append(torch.stack(out))
        m.close()
    assert torch.equal(res[0], res[1])


def test_graph_replay_equals_eager(monkeypatch):
    shape = MODEL_SHAPES["1b"]
    w = model_weights(shape, seed=5, device="cuda")
    ids = prompts(4, 64, shape["vocab_size"], seed=6).numpy()
    flat, cu = pack(list(ids))
    res = []
    for eager in ("0", "1"):
        monkeypatch.setenv("AXON_NO_GRAPH", eager)
        m = Model(shape, w, max_batch=4, max_seq=80)
        lg, tok = m.prefill(flat, cu)
        out = [lg.cpu()]
        for _ in range(4):
            lg = torch.empty((4, shape["vocab_size"]), dtype=torch.float32, device="cuda")
            _, tok = m.decode_step(tok, logits=lg)
            out.append(lg.cpu())
        torch.cuda.synchronize()
        res.append(torch.stack(out))
        m.close()
    assert torch.equal(res[0], res[1])


@pytest.mark.parametrize("mode", ["f32_full_depth", "bf16_2_layers"])
def test_decode_logits_agree_with_all_positions_prefill(mode):
    """Causal consistency across kernels: decoding tokens one by one gives the
    logits that a prefill of the whole sequence gives at those positions (the
    GEMM and the decode projections, prefill and decode attention)."""
    if mode == "f32_full_depth":
        shape = dict(MODEL_SHAPES["1b"], dtype="f32")
        w = {k: v.float() for k, v in model_weights(MODEL_SHAPES["1b"], seed=7, device="cuda").items()}
    else:
        # two bf16 pipelines (prefill GEMM + RMSNorm kernel vs decode projections
        # with the norm folded in) round at different points; at this width their
        # difference stays inside the absolute bf16 tolerance
        shape = small_shape("1b", layers=2, vocab=4096, hidden=512, intermediate=1024)
        w = model_weights(shape, seed=7, device="cuda")
    ids = prompts(2, 40, shape["vocab_size"], seed=8).numpy()
    P, extra = 30, 10
    m = Model(shape, w, max_batch=2, max_seq=64)
    flat, cu = pack([ids[0], ids[1]])
    full, _ = m.prefill(flat, cu, all_logits=True)
    full = full.cpu().double().numpy()
    flat, cu = pack([ids[0, :P], ids[1, :P]])
    lg, _ = m.prefill(flat, cu)
    got = [lg.cpu().double().numpy()]
    for s in range(extra - 1):
        tok = torch.as_tensor(ids[:, P + s].astype(np.int32)).cuda()
        lg = torch.empty((2, shape["vocab_size"]), dtype=torch.float32, device="cuda")
        m.decode_step(tok, logits=lg)
        got.append(lg.cpu().double().numpy())
    torch.cuda.synchronize()
    got = np.stack(got)  # [extra, 2, V]: positions P-1 .. P+extra-2
    want = np.stack([full[40 * b + P - 1:40 * b + P - 1 + extra] for b in range(2)], axis=1)
    if mode == "f32_full_depth":
        check_logits(got, want, F32_MAX, None, "decode vs all-positions prefill (f32)")
    else:
        check_logits(got, want, BF16_MAX, BF16_MEAN, "decode vs all-positions prefill (bf16)")
    m.close()


def test_capacity_errors_are_reported_without_side_effects():
    shape = dict(MODEL_SHAPES["1b"], num_hidden_layers=1, vocab_size=512)
    w = model_weights(shape, seed=9, device="cuda")
    m = Model(shape, w, max_batch=2, max_seq=8)
    flat, cu = pack([np.arange(7), np.arange(3)])
    with pytest.raises(AxonError) as e:
        m.prefill(torch.arange(9, dtype=torch.int32, device="cuda"), [0, 9])
    assert e.value.code == -5
    _, tok = m.prefill(flat, cu)
    _, tok = m.decode_step(tok)  # slot 0 reaches 8 = max_seq
    with pytest.raises(AxonError) as e:
        m.decode_step(tok)
    assert e.value.code == -5 and "full" in str(e.value)
    assert m.lengths() == [8, 4]
    with pytest.raises(AxonError) as e:
        m.decode_step(torch.zeros(3, dtype=torch.int32, device="cuda"))
    assert e.value.code == -5
    torch.cuda.synchronize()
    m.close()
    # paged: a slot without a page for its next position
    m = Model(shape, w, max_batch=1, max_seq=64, page_size=16, num_pages=4)
    table = torch.tensor([[2, -1, -1, -1]], dtype=torch.int32)
    _, tok = m.prefill(torch.arange(16, dtype=torch.int32, device="cuda"), [0, 16], block_table=table)
    with pytest.raises(AxonError) as e:
        m.decode_step(tok)
    assert e.value.code == -5 and "page" in str(e.value)
    with pytest.raises(AxonError) as e:
        m.prefill(torch.arange(16, dtype=torch.int32, device="cuda"), [0, 16],
                  block_table=torch.tensor([[4, -1, -1, -1]], dtype=torch.int32))
    assert e.value.code == -5
    with pytest.raises(AxonError) as e:
        m.prefill(torch.arange(20, dtype=torch.int32, device="cuda"), [0, 20],
                  block_table=torch.tensor([[1, 1, -1, -1]], dtype=torch.int32))
    assert e.value.code == -1 and "twice" in str(e.value)
    torch.cuda.synchronize()
    m.close()
