"""Continuous batching (axon_step) on the GPU against the float64 oracle.

A scripted serving schedule admits sequences into free slots with prompt
chunks, mixes those chunks with decode tokens of running sequences in one
step, evicts a sequence and reuses its slot (and, paged, its pages).  Each
entry's last-token logits are compared with the oracle fed the same tokens
slot by slot (decode tokens are the oracle's own greedy choices, so a near-tie
flip never cascades).  Chunked prefill is also checked bit for bit against a
one-shot prefill of the same prompts: the same kernels see the same keys in
the same order.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_19889_amd.axon import AXON_E_CAPACITY, AXON_E_INVALID, AxonError
from parity_util import F32_MAX, check_argmax, check_bf16, check_logits, gpu_model, pack
from synthetic import model_weights, prompts, small_shape

pytestmark = pytest.mark.gpu

PAGE = 16


class Pages:
    """Page allocator of the test: a randomly permuted pool, rows per slot."""

    def __init__(self, num_pages, stride, seed=0):
        self.free = list(np.random.default_rng(seed).permutation(num_pages))
        self.rows = {}
        self.stride = stride

    def admit(self, slot, tokens):
        self.release(slot)
        need = (tokens + PAGE - 1) // PAGE
        self.rows[slot] = [int(self.free.pop()) for _ in range(need)]

    def release(self, slot):
        self.free.extend(self.rows.pop(slot, []))

    def table(self, slots):
        t = np.full((len(slots), self.stride), -1, dtype=np.int32)
        for i, s in enumerate(slots):
            r = self.rows[s]
            t[i, :len(r)] = r
        return torch.from_numpy(t)


# (slot, fresh, tokens): tokens is a prompt length, or "d" for a decode token;
# "reset" evicts slots before the step's entries
SCHEDULE = [
    {"entries": [(0, 1, 37), (2, 1, 130)]},
    {"entries": [(0, 0, 20), (2, 0, "d"), (5, 1, 9)]},
    {"entries": [(0, 0, "d"), (2, 0, "d"), (5, 0, 64)]},
    {"reset": [2], "entries": [(2, 1, 50), (0, 0, "d"), (5, 0, "d")]},
    {"entries": [(0, 0, "d"), (5, 0, "d"), (2, 0, "d"), (1, 1, 1)]},
    {"entries": [(1, 0, "d"), (0, 0, "d"), (2, 0, "d"), (5, 0, "d")]},
    # decode-only steps of the same size replay one recorded graph with other
    # slot assignments; then a smaller one
    {"entries": [(2, 0, "d"), (5, 0, "d"), (1, 0, "d"), (0, 0, "d")]},
    {"entries": [(5, 0, "d"), (0, 0, "d"), (1, 0, "d")]},
    {"entries": [(0, 0, "d"), (1, 0, "d"), (2, 0, "d"), (5, 0, "d")]},
]
BUDGET = 12  # decode tokens reserved per admitted sequence (pages)


def run_schedule(shape, w, paged, with_b16=True):
    """Returns (gpu logits [entries, V], exact oracle logits, bf16-storage oracle
    logits or None)."""
    V = shape["vocab_size"]
    max_seq = 160
    w64 = oracle.weights_f64(w)
    exact = oracle.OracleDecoder(shape, w64)
    b16 = oracle.OracleDecoder(shape, w64, io_round="bf16") if with_b16 else None
    kw = {}
    pages = None
    if paged:
        pages = Pages(64, (max_seq + PAGE - 1) // PAGE, seed=3)
        kw = dict(page_size=PAGE, num_pages=64)
    m = gpu_model(shape, w, max_batch=6, max_seq=max_seq, **kw)
    rng = np.random.default_rng(11)
    last, gpu_out, ref_out, refb_out = {}, [], [], []
    for step in SCHEDULE:
        for slot in step.get("reset", []):
            m.reset_slot(slot)
            exact.reset(slot)
            if b16:
                b16.reset(slot)
            if pages:
                pages.release(slot)
        slots, fresh, seqs = [], [], []
        for slot, fr, n in step["entries"]:
            toks = np.array([last[slot]]) if n == "d" else rng.integers(0, V, n)
            if fr:
                exact.reset(slot)
                if b16:
                    b16.reset(slot)
                if pages:
                    pages.admit(slot, min(max_seq, len(toks) + 80 + BUDGET))
            lg = exact.extend(slot, toks, all_logits=False)
            ref_out.append(lg)
            if b16:
                refb_out.append(b16.extend(slot, toks, all_logits=False))
            last[slot] = int(np.argmax(lg))
            slots.append(slot)
            fresh.append(fr)
            seqs.append(toks)
        flat, cu = pack(seqs)
        rows = pages.table(slots) if pages else None
        lg, _ = m.step(flat, cu, slots, fresh, block_rows=rows)
        gpu_out.append(lg.cpu().double().numpy())
        for i, s in enumerate(slots):
            assert m.lengths()[s] == exact.lengths()[s]
    torch.cuda.synchronize()
    m.close()
    return (np.concatenate(gpu_out), np.stack(ref_out), np.stack(refb_out) if b16 else None)


@pytest.mark.parametrize("paged", [False, True], ids=["contiguous", "paged"])
def test_continuous_batching_schedule_bf16(paged):
    shape = small_shape("7b", layers=2, vocab=2048, hidden=896, intermediate=1792)
    w = model_weights(shape, seed=21)
    gpu, exact, b16 = run_schedule(shape, w, paged)
    mx = check_bf16(gpu, exact, b16, f"continuous batching bf16 ({'paged' if paged else 'contiguous'})")
    check_argmax(gpu, exact, mx, "continuous batching bf16")


def test_continuous_batching_schedule_f32_check_mode():
    shape = small_shape("1b", layers=2, vocab=3000, hidden=512, intermediate=1024)
    w = {k: v.float() for k, v in model_weights(shape, seed=22).items()}
    shape = dict(shape, dtype="f32")
    gpu, exact, _ = run_schedule(shape, w, paged=True, with_b16=False)
    check_logits(gpu, exact, F32_MAX, None, "continuous batching f32")
    np.testing.assert_array_equal(np.argmax(gpu, -1), np.argmax(exact, -1))


@pytest.mark.parametrize("paged", [False, True], ids=["contiguous", "paged"])
def test_chunked_prefill_equals_one_shot_bitwise(paged):
    shape = small_shape("1b", layers=2, vocab=3000, hidden=512, intermediate=1024)
    w = model_weights(shape, seed=23)
    ids = prompts(2, 100, shape["vocab_size"], seed=24).numpy()
    a, b = ids[0], ids[1, :37]
    kw = dict(page_size=PAGE, num_pages=32) if paged else {}
    pages = Pages(32, 8, seed=5) if paged else None
    if pages:
        pages.admit(0, 100)
        pages.admit(1, 37)
    one = gpu_model(shape, w, max_batch=2, max_seq=128, **kw)
    flat, cu = pack([a, b])
    ref, _ = one.prefill(flat, cu, block_table=pages.table([0, 1]) if pages else None)
    ref = ref.cpu().numpy()
    one.close()
    m = gpu_model(shape, w, max_batch=2, max_seq=128, **kw)
    rows = pages.table([0, 1]) if pages else None
    flat, cu = pack([a[:30], b[:2]])
    m.step(flat, cu, [0, 1], [1, 1], block_rows=rows)
    flat, cu = pack([a[30:70], b[2:]])
    lg1, _ = m.step(flat, cu, [0, 1], [0, 0])
    flat, cu = pack([a[70:]])
    lg2, _ = m.step(flat, cu, [0], [0])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lg2.cpu().numpy()[0], ref[0])
    np.testing.assert_array_equal(lg1.cpu().numpy()[1], ref[1])
    assert m.lengths()[:2] == [100, 37]
    m.close()


def test_step_admission_then_graph_decode():
    """Sequences admitted by steps continue with the graph-replayed decode step."""
    shape = small_shape("32b", layers=2, vocab=1500, hidden=640, intermediate=1280)
    w = model_weights(shape, seed=25)
    ids = prompts(3, 70, shape["vocab_size"], seed=26).numpy()
    seqs = [ids[0, :70], ids[1, :33], ids[2, :5]]
    steps = 4
    w64 = oracle.weights_f64(w)
    ref_tok, ref_lg = oracle.generate_greedy(oracle.OracleDecoder(shape, w64), seqs, steps)
    ref_b = oracle.teacher_forced(oracle.OracleDecoder(shape, w64, io_round="bf16"), seqs, ref_tok[:, :steps])
    m = gpu_model(shape, w, max_batch=3, max_seq=96)
    # prompts in two chunk steps, slot order scrambled
    flat, cu = pack([seqs[2], seqs[0][:40]])
    lg_0, _ = m.step(flat, cu, [2, 0], [1, 1])
    flat, cu = pack([seqs[0][40:], seqs[1]])
    lg_1, _ = m.step(flat, cu, [0, 1], [0, 1])
    got = np.zeros((steps + 1, 3, shape["vocab_size"]))
    # last-prompt-token logits: slot 2 from the first step, slots 0 and 1 from the second
    got[0, 2] = lg_0[0].cpu().double().numpy()
    got[0, 0] = lg_1[0].cpu().double().numpy()
    got[0, 1] = lg_1[1].cpu().double().numpy()
    for s in range(steps):
        tok = torch.as_tensor(ref_tok[:, s].astype(np.int32)).to("cuda")
        lg = torch.empty((3, shape["vocab_size"]), dtype=torch.float32, device="cuda")
        m.decode_step(tok, logits=lg)
        got[s + 1] = lg.cpu().double().numpy()
    torch.cuda.synchronize()
    assert m.lengths() == [70 + steps, 33 + steps, 5 + steps]
    mx = check_bf16(got, ref_lg, ref_b, "step admission + graph decode")
    check_argmax(got, ref_lg, mx, "step admission + graph decode")
    m.close()


def test_step_validation_leaves_state_unchanged():
    shape = small_shape("1b", layers=1, vocab=1000, hidden=512, intermediate=1024)
    w = model_weights(shape, seed=27)
    m = gpu_model(shape, w, max_batch=3, max_seq=40, page_size=PAGE, num_pages=8)
    pages = Pages(8, 3, seed=1)
    pages.admit(0, 30)
    pages.admit(1, 10)
    flat, cu = pack([np.arange(20), np.arange(5)])
    m.step(flat, cu, [0, 1], [1, 1], block_rows=pages.table([0, 1]))
    torch.cuda.synchronize()
    before = m.lengths()

    def expect(code, fn):
        with pytest.raises(AxonError) as e:
            fn()
        assert e.value.code == code, str(e.value)
        assert m.lengths() == before

    one = pack([np.arange(3)])
    two = pack([np.arange(3), np.arange(2)])
    expect(AXON_E_INVALID, lambda: m.step(two[0], two[1], [1, 1], [0, 0]))                  # repeated slot
    expect(AXON_E_INVALID, lambda: m.step(one[0], one[1], [3], [1]))                       # slot out of range
    expect(AXON_E_CAPACITY, lambda: m.step(*pack([np.arange(25)]), [0], [0]))              # 20 + 25 > max_seq
    expect(AXON_E_CAPACITY, lambda: m.step(*pack([np.arange(12)]), [1], [0]))              # no page for block 1
    moved = pages.table([0])
    moved[0, 0] = int(pages.free[0])
    expect(AXON_E_INVALID, lambda: m.step(one[0], one[1], [0], [0], block_rows=moved))    # moves cached page
    taken = pages.table([1])
    taken[0, 1] = pages.rows[0][0]
    expect(AXON_E_INVALID, lambda: m.step(*pack([np.arange(12)]), [1], [0], block_rows=taken))  # page twice
    # an evicted slot cannot decode, and its pages can go to another slot
    m.reset_slot(1)
    before = m.lengths()
    expect(AXON_E_INVALID, lambda: m.decode_step(torch.zeros(2, dtype=torch.int32, device="cuda")))
    freed = pages.rows[1]
    pages.release(1)
    pages.rows[2] = freed
    m.step(*pack([np.arange(4)]), [2], [1], block_rows=pages.table([2]))
    torch.cuda.synchronize()
    assert m.lengths() == [20, 0, 4]
    m.close()
