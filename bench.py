#!/usr/bin/env python3
"""Throughput of the decoder forward pass on one MI355X.

One step = one whole greedy generate on the workload: prefill of every
prompt, then ``decode_steps`` graph-replayed decode steps (tokens stay on the
device).  Prints ONE JSON line on stdout; progress goes to stderr.

value = generated tokens / wall time (the paper's throughput measure:
Results, "Measures"), generated = batch x (decode_steps + 1) because the
prefill already yields each sequence's first token.  Prefill tokens/s, decode
tokens/s and decode HBM bandwidth are reported beside it; ``roofline`` covers
the kernel class with the most device time, measured with HIP events around
each of its launches in an instrumented repeat of the step; ``cpu_baseline``
times the float64 CPU oracle on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
F32_PEAK_TFLOPS = 157.3     # MI355X fp32 vector

METRIC = "prefill & decode tokens/s + decode HBM GB/s fraction, 1B and 7B shapes"
COUNTER_DECODE_STEPS = 4    # decode steps of the hardware-counter runs


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def weight_bytes(shape, esz):
    from synthetic import weight_shapes
    tot = 0
    for n, shp in weight_shapes(shape).items():
        k = 1
        for d in shp:
            k *= d
        tot += k * esz
    return tot


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="1b", choices=["1b", "7b", "135m", "7b_paged", "32b", "7b_serve", "moe16b",
                                                         "gpt2xl", "mistral7b", "1b_train"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--no-7b", action="store_true",
                    help="with the 1b workload: leave out the 7B workload's object in the JSON line")
    ap.add_argument("--decode-steps", type=int, default=None,
                    help="override the workload's decode step count (hardware-counter runs only)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="finish with one 1 GiB device-to-device copy (a known-size reference for HBM counters)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, WRITE_SIZE) of a "
                         "--copy-calibration run into profiles/decode_gemv_<workload>_traffic.json and exit")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="time the vendor library's GEMM (torch.matmul, bf16) on the workload's prefill projection "
                         "shapes instead of the workload, as a reference for the hand-written kernels, and exit")
    args = ap.parse_args()
    if args.summarize_counters:
        summarize_counters(args.summarize_counters[0], args.summarize_counters[1], args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(this build has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2608_19889_amd import axon as ax
    if not os.path.exists(ax.LIB_PATH):
        from paper_2608_19889_amd.build import build
        build()
    from synthetic import MODEL_SHAPES, WORKLOADS

    wl = dict(WORKLOADS[args.workload])
    shape = MODEL_SHAPES[wl["model"]]
    if args.vendor_gemm:
        return vendor_gemm(shape, wl)
    if wl.get("train"):
        return train_bench(args, wl, shape)
    out, lens, steps = measure_generate(args, args.workload, args.steps, args.warmup)
    # the metric covers the 1B and the 7B shapes: the 7B workload's figures go
    # into the same line (1 warmup + up to 2 timed generates)
    if args.workload == "1b" and not args.no_7b:
        out["workloads"] = {"7b": workload_summary(measure_generate(args, "7b", min(args.steps, 2), 1)[0])}
    if args.copy_calibration:
        src = torch.empty(1 << 29, dtype=torch.int16, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] calibration copy: 1 GiB read + 1 GiB written")
        del src, dst
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, wl, lens, steps, wl["batch"])
    print(json.dumps(out), flush=True)


def measure_generate(args, workload, n_steps, n_warmup):
    """Time ``n_steps`` whole greedy generates of ``workload`` after
    ``n_warmup`` untimed ones; returns (result dict, prompt lengths, decode
    steps)."""
    import numpy as np
    import torch

    from paper_2608_19889_amd import axon as ax
    from synthetic import MODEL_SHAPES, WORKLOADS, model_weights, paged_workload, prompts
    wl = dict(WORKLOADS[workload])
    shape = MODEL_SHAPES[wl["model"]]
    esz = 2 if shape["dtype"] == "bf16" else 4
    B, steps = wl["batch"], wl["steps"] if args.decode_steps is None else args.decode_steps
    L, D, V = shape["num_hidden_layers"], shape["hidden_size"], shape["vocab_size"]
    KV, hd = shape["num_key_value_heads"], shape["head_dim"]
    dev = "cuda"
    torch.cuda.set_device(0)

    # ---- synthetic inputs, resident on the GPU before timing
    t0 = time.time()
    w = model_weights(shape, seed=0, device=dev)
    if wl["paged"]:
        seqs, table, pool = paged_workload(B, wl["len_range"][0], wl["len_range"][1], steps, V,
                                           wl["page_size"], seed=0)
        lens = [len(s) for s in seqs]
        flat = torch.cat(seqs).to(dev)
        seqs = [x.to(dev) for x in seqs]
        max_seq = max(lens) + steps
        page_kw = dict(page_size=wl["page_size"], num_pages=pool)
    else:
        P = wl["prompt_len"]
        ids = prompts(B, P, V, seed=0)
        lens = [P] * B
        flat = ids.reshape(-1).to(dev)
        table = None
        max_seq = P + steps
        page_kw = {}
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    max_tokens = cu[-1] if not wl.get("serve") else wl["step_tokens"] + B
    m = ax.Model(shape, w, max_batch=B, max_seq=max_seq, max_tokens=max_tokens, **page_kw)
    log(f"[bench] model + inputs ready in {time.time() - t0:.1f}s "
        f"(weights {weight_bytes(shape, esz) / 1e9:.2f} GB, prompt tokens {cu[-1]})")

    nt = [torch.empty(B, dtype=torch.int32, device=dev) for _ in range(2)]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    serve_plan = make_serve_plan(lens, steps, wl["step_tokens"]) if wl.get("serve") else None

    serve_ev = []
    serve_state = {}

    def generate(record=False):
        if serve_plan is not None:
            return serve(m, serve_plan, seqs, table, B, serve_ev if record else None, serve_state)
        if record:
            ev[0].record()
        m.prefill(flat, cu, block_table=table, want_logits=False, next_tokens=nt[0])
        if record:
            ev[1].record()
        a, b = nt
        for _ in range(steps):
            m.decode_step(a, next_tokens=b)
            a, b = b, a
        if record:
            ev[2].record()

    for i in range(n_warmup):
        generate()
        log(f"[bench] warmup {i + 1}/{n_warmup} done")
    torch.cuda.synchronize()
    pre_ms, dec_ms = [], []
    t_start = time.perf_counter()
    for i in range(n_steps):
        generate(record=True)
        torch.cuda.synchronize()
        if serve_plan is not None:
            p, d = serve_split_ms(serve_plan, serve_ev)
            pre_ms.append(p)
            dec_ms.append(d)
            log(f"[bench] step {i + 1}/{n_steps}: steps with prompt chunks {p:.2f} ms, decode-only steps "
                f"{d:.2f} ms ({len(serve_plan)} scheduler steps)")
        else:
            pre_ms.append(ev[0].elapsed_time(ev[1]))
            dec_ms.append(ev[1].elapsed_time(ev[2]))
            log(f"[bench] step {i + 1}/{n_steps}: prefill {pre_ms[-1]:.2f} ms, decode {dec_ms[-1]:.2f} ms")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = wall * 1e3 / n_steps
    gen_tokens = B * (steps + 1)
    value = gen_tokens / (ms_per_step / 1e3)
    prefill_ms, decode_ms = float(np.mean(pre_ms)), float(np.mean(dec_ms))

    # algorithmic decode bytes: every weight except the embedding table (B rows
    # of it), the KV cache read over each step's context and the new KV written
    # (a tied head reads the embedding table in full; an untied model reads
    # only B rows of the table and the separate head matrix)
    wb = weight_bytes(shape, esz)
    emb = V * D * esz
    # (decode steps, decode tokens, KV positions read) of the timed decode phase:
    # every step of a static generate; the decode-only steps of a served run
    dsteps = [[n + s for n in lens] for s in range(steps)] if serve_plan is None else \
        [[lens[b] + start for b, start, c in st] for st in serve_plan if all(c == 0 for _, _, c in st)]
    # keys a query at position pos attends to (a sliding window keeps the last W)
    W = shape.get("sliding_window") or 0
    keys = (lambda pos: min(pos + 1, W)) if W else (lambda pos: pos + 1)  # noqa: E731
    kv_read = sum(2 * L * KV * hd * keys(pos) * esz for st in dsteps for pos in st)
    dtok = sum(len(st) for st in dsteps)
    kv_write = dtok * 2 * L * KV * hd * esz
    # a mixture-of-experts step reads the experts its tokens choose: counted as
    # the expectation under uniform routing, E (1 - (1 - k/E)^tokens) per layer
    moe_b, moe_frac = 0, (lambda n: 1.0)
    if shape.get("n_routed_experts"):
        E, k, Ie = shape["n_routed_experts"], shape["num_experts_per_tok"], shape["moe_intermediate_size"]
        n_moe = L - shape.get("first_k_dense_replace", 0)
        moe_b = n_moe * E * 3 * D * Ie * esz
        moe_frac = lambda n: 1.0 - (1.0 - k / E) ** n  # noqa: E731
    # GPT-2's learned-position table: only the step's rows are read
    wpe = shape.get("max_position_embeddings", 0) * D * esz if shape.get("model_type") == "gpt2" else 0
    rows_per_token = 2 if wpe else 1  # embedding rows gathered per token (token, and position)
    decode_bytes = sum(wb - moe_b + moe_b * moe_frac(len(st)) - (0 if shape["tie_word_embeddings"] else emb)
                       - wpe + rows_per_token * len(st) * D * esz for st in dsteps) + kv_read + kv_write
    decode_gbs = decode_bytes / (decode_ms / 1e3) / 1e9

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "generated tokens/s",
        "n_gpus": 1,
        "steps": n_steps,
        "warmup": n_warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape["dtype"],
        "data": "synthetic (random-init N(0,0.02) weights, uniform random prompt ids)",
        "config": {"workload": f"{workload}-shaped decoder: batch {B}, "
                               + (f"prompts {wl['prompt_len']}" if not wl["paged"] else
                                  f"prompts U[{wl['len_range'][0]},{wl['len_range'][1]}] (sum {cu[-1]})")
                               + f", {steps} greedy decode steps, "
                               + ("paged KV (16-token pages)" if wl["paged"] else "contiguous KV")
                               + (f", continuous batching: {wl['step_tokens']}-token steps of decode tokens and "
                                  f"prompt chunks, {len(serve_plan)} steps" if serve_plan is not None else ""),
                   "batch": B, "prompt_tokens": cu[-1], "decode_steps": steps,
                   "layers": L, "hidden": D, "vocab": V},
        "prefill_tok_s": round(cu[-1] / (prefill_ms / 1e3), 1),
        "prefill_ms": round(prefill_ms, 3),
        "decode_tok_s": round(dtok / (decode_ms / 1e3), 1),
        "decode_ms_per_token_step": round(decode_ms / max(1, len(dsteps)), 4),
        "decode_hbm_gbs": round(decode_gbs, 1),
        "decode_hbm_frac": round(decode_gbs / HBM_PEAK_GBS, 4),
    }

    if not args.no_roofline:
        out.update(roofline_pass(m, generate, shape, esz, lens))
        out["roofline"]["traffic"] = measured_traffic(out["roofline"], workload)
        att = out["kernels"].get("decode attention (+ split merge)")
        if att is not None:
            att["traffic_per_layer"] = measured_attention_traffic(workload)
    m.close()
    del w
    torch.cuda.empty_cache()
    return out, lens, steps


def workload_summary(o):
    """The figures of a second workload's measurement that go into the main
    JSON line: throughput, prefill and decode rates, decode HBM fraction and
    each kernel class's roofline."""
    keys = ("value", "ms_per_step", "steps", "warmup", "prefill_tok_s", "prefill_ms", "decode_tok_s",
            "decode_ms_per_token_step", "decode_hbm_gbs", "decode_hbm_frac")
    r = {"workload": o["config"]["workload"], "unit": o["unit"]}
    r.update({k: o[k] for k in keys if k in o})
    r["generated_tok_s"] = r.pop("value")
    k = o.get("kernels", {})
    for name, key in (("prefill projection GEMM (MFMA)", "prefill_gemm"), ("prefill flash attention", "prefill_attention"),
                      ("decode projection GEMM (weight streaming)", "decode_projections"),
                      ("decode attention (+ split merge)", "decode_attention")):
        if name in k:
            r[key] = {f: k[name][f] for f in ("bound", "achieved", "peak", "unit", "frac", "avg_us", "total_ms",
                                              "traffic_per_layer") if f in k[name]}
    if "roofline" in o:
        r["roofline"] = o["roofline"]
    return r


def vendor_gemm(shape, wl):
    """Time torch.matmul (the vendor BLAS library) on the prefill projection
    shapes of the workload's model (QKV, O, gate/up, down; M = the prompt
    tokens of one prefill), bf16 operands and output, X ~ N(0, 1), W ~ N(0,
    0.02).  A reference point for the hand-written GEMMs only: nothing of it
    runs in the measured path."""
    import torch
    D, H, KV, hd = shape["hidden_size"], shape["num_attention_heads"], shape["num_key_value_heads"], shape["head_dim"]
    I = shape["intermediate_size"]
    M = wl["batch"] * wl["prompt_len"] if wl.get("prompt_len") else wl["batch"] * sum(wl["len_range"]) // 2
    shapes = {"qkv": ((H + 2 * KV) * hd, D), "o": (D, H * hd), "gate/up": (2 * I, D), "down": (D, I)}
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda").manual_seed(0)
    out = {}
    for name, (N, K) in shapes.items():
        W = (torch.randn(N, K, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
        X = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
        for _ in range(3):
            Y = X @ W.t()
        torch.cuda.synchronize()
        reps = 5
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            Y = X @ W.t()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        out[name] = {"N": N, "K": K, "M": M, "ms": round(ms, 4), "tflops": round(2.0 * M * N * K / ms / 1e9, 1)}
        log(f"vendor GEMM {name} N={N} K={K} M={M}: {ms:.3f} ms, {out[name]['tflops']} TFLOP/s")
        del W, X, Y
    print(json.dumps({"vendor_gemm": out, "workload": wl["model"]}))


def train_bench(args, wl, shape):
    """One training step per timed step: the forward pass keeping its
    activations, the mean next-token cross-entropy and every weight's
    gradient (axon_loss_and_grads) over batch x prompt_len synthetic tokens."""
    import numpy as np
    import torch

    from paper_2608_19889_amd import axon as ax
    from synthetic import model_weights, prompts
    dev = "cuda"
    torch.cuda.set_device(0)
    B, P = wl["batch"], wl["prompt_len"]
    V, D, L = shape["vocab_size"], shape["hidden_size"], shape["num_hidden_layers"]
    H, hd = shape["num_attention_heads"], shape["head_dim"]
    t0 = time.time()
    w = model_weights(shape, seed=0, device=dev)
    ids = prompts(B, P, V, seed=0)
    flat = ids.reshape(-1).to(dev)
    tg = torch.cat([ids[:, 1:], torch.full((B, 1), -1, dtype=ids.dtype)], 1).reshape(-1).to(dev)
    cu = [b * P for b in range(B + 1)]
    T = B * P
    m = ax.Model(shape, w, max_batch=B, max_seq=P, max_tokens=T)
    grads = {k: torch.empty(tuple(v.shape), dtype=torch.float32, device=dev) for k, v in w.items()}
    loss = torch.empty((1,), dtype=torch.float32, device=dev)
    log(f"[bench] model + inputs ready in {time.time() - t0:.1f}s (weights {weight_bytes(shape, 2) / 1e9:.2f} GB, "
        f"{T} training tokens)")

    def step():
        m.loss_and_grads(flat, cu, tg, grads, loss=loss)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done (loss {loss.item():.4f})")
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_start = time.perf_counter()
    e0.record()
    for i in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms = wall * 1e3 / args.steps
    log(f"[bench] {args.steps} steps: {ms:.2f} ms per step (events {e0.elapsed_time(e1) / args.steps:.2f} ms), "
        f"loss {loss.item():.4f}")
    # algorithmic FLOPs of a step: 6 x (matmul parameters) per token (forward
    # 2, backward 4), attention 4 hd per (query, key, head) forward and 10 hd
    # backward (probabilities recomputed)
    mm = 0
    for n, shp in w.items():
        if len(shp) == 2 and n != "model.embed_tokens.weight":
            mm += shp[0] * shp[1]
    if shape["tie_word_embeddings"]:
        mm += V * D
    pairs = B * P * (P + 1) / 2
    flops = 6.0 * mm * T + 14.0 * hd * H * pairs * L
    out = {
        "metric": "training tokens/s (forward + next-token cross-entropy + every weight's gradient)",
        "value": round(T / (ms / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (random-init N(0,0.02) weights, uniform random token ids, next-token targets)",
        "config": {"workload": f"{wl['model']}-shaped decoder training step: batch {B} x {P} tokens",
                   "batch": B, "seq_len": P, "tokens": T, "layers": L, "hidden": D, "vocab": V},
        "loss": round(float(loss.item()), 5),
        "step_tflops": round(flops / (ms / 1e3) / 1e12, 1),
    }
    if not args.no_roofline:
        m.timing(True)
        step()
        torch.cuda.synchronize()
        recs = m.timing_records()
        m.timing(False)
        agg = {}
        for c, (d0, d1, d2), t_ms in recs:
            a = agg.setdefault(c, {"ms": 0.0, "n": 0, "flops": 0.0})
            a["ms"] += t_ms
            a["n"] += 1
            if c == ax.T_GEMM:
                a["flops"] += 2.0 * d0 * d1 * d2
        if ax.T_ATTN_PREFILL in agg:
            agg[ax.T_ATTN_PREFILL]["flops"] = 4.0 * H * hd * pairs * L
        if ax.T_ATTN_BWD in agg:
            agg[ax.T_ATTN_BWD]["flops"] = 10.0 * H * hd * pairs * L
        names = {ax.T_GEMM: ("forward and backward projection GEMMs (MFMA)", "mfma", BF16_PEAK_TFLOPS),
                 ax.T_ATTN_PREFILL: ("forward flash attention (MFMA)", "mfma", BF16_PEAK_TFLOPS),
                 ax.T_ATTN_BWD: ("attention backward (MFMA)", "mfma", BF16_PEAK_TFLOPS)}
        kernels = {}
        for c, a in agg.items():
            if c not in names:
                continue
            nm, bound, peak = names[c]
            ach = a["flops"] / (a["ms"] / 1e3) / 1e12
            kernels[nm] = {"bound": bound, "achieved": round(ach, 1), "peak": peak, "unit": "TFLOP/s",
                           "frac": round(ach / peak, 4), "launches": a["n"], "total_ms": round(a["ms"], 3),
                           "avg_us": round(1e3 * a["ms"] / a["n"], 2)}
        dom = max((c for c in agg if c in names), key=lambda c: agg[c]["ms"])
        r = dict(kernels[names[dom][0]])
        r["kernel"] = names[dom][0]
        r["traffic"] = None
        out["roofline"] = r
        out["kernels"] = kernels
    m.close()
    print(json.dumps(out), flush=True)


def make_serve_plan(lens, steps, budget):
    """First-come-first-served continuous-batching schedule, host only (the
    tokens themselves are produced on the device).  Every sequence needs its
    prompt, fed in chunks, then ``steps`` decode tokens.  A step first gives
    each running sequence (prompt complete, decode tokens left) one decode
    token, then fills the rest of the token budget with prompt chunks in
    arrival order.  Returns the steps as lists of (sequence, start, count):
    count > 0 prompt tokens from ``start``; count == 0 a decode token, with
    ``start`` the number of decode tokens the sequence has already fed."""
    B = len(lens)
    fed, dec = [0] * B, [0] * B
    plan = []
    while True:
        entries, used = [], 0
        for b in range(B):
            if fed[b] == lens[b] and dec[b] < steps:
                entries.append((b, dec[b], 0))
                used += 1
        for b in range(B):
            if fed[b] < lens[b] and used < budget:
                c = min(lens[b] - fed[b], budget - used)
                entries.append((b, fed[b], c))
                used += c
        if not entries:
            return plan
        for b, _, c in entries:
            if c == 0:
                dec[b] += 1
            else:
                fed[b] += c
        plan.append(entries)


def serve(m, plan, seqs, table, B, events, state):
    """Run a continuous-batching schedule through axon_step.  Sequence b lives
    in slot b; a sequence's decode token is its own previous greedy output,
    gathered on the device (no host synchronization inside the run).  Token,
    cu_seqlens and output buffers keep their addresses from step to step, so
    decode-only steps replay one recorded graph per entry count."""
    import torch
    dev = seqs[0].device
    if not state:
        cap = max(sum(c if c else 1 for _, _, c in st) for st in plan)
        state.update(tok=torch.empty(cap, dtype=torch.int32, device=dev),
                     cu=torch.empty(B + 1, dtype=torch.int32, device=dev),
                     nxt=torch.empty(B, dtype=torch.int32, device=dev),
                     last=torch.zeros(B, dtype=torch.int32, device=dev))
    tok, nxt, last = state["tok"], state["nxt"], state["last"]
    if events is not None:
        events.clear()
    for st in plan:
        slots = [b for b, _, _ in st]
        fresh = [1 if c > 0 and start == 0 else 0 for _, start, c in st]
        dec = [b for b, _, c in st if c == 0]
        parts = [last.index_select(0, torch.tensor(dec, dtype=torch.int64).to(dev, non_blocking=True))] if dec else []
        parts += [seqs[b][start:start + c] for b, start, c in st if c > 0]
        cu = [0]
        for _, _, c in st:
            cu.append(cu[-1] + (c if c else 1))
        torch.cat(parts, out=tok[:cu[-1]])
        rows = table[slots] if any(fresh) else None
        if events is not None:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
        m.step(tok[:cu[-1]], cu, slots, fresh, block_rows=rows, next_tokens=nxt[:len(st)], want_logits=False,
               cu_device=state["cu"])
        if events is not None:
            e1.record()
            events.append((e0, e1))
        last.index_copy_(0, torch.tensor(slots, dtype=torch.int64).to(dev, non_blocking=True), nxt[:len(st)])


def serve_split_ms(plan, events):
    """(ms of the steps that carry prompt chunks, ms of the decode-only steps)."""
    mixed = dec = 0.0
    for st, (e0, e1) in zip(plan, events):
        t = e0.elapsed_time(e1)
        if all(c == 0 for _, _, c in st):
            dec += t
        else:
            mixed += t
    return mixed, dec


def roofline_pass(m, generate, shape, esz, lens):
    """Instrumented repeat of one step: HIP events around every launch of the
    projection GEMMs and attention kernels, on the stream they run on."""
    import torch
    from paper_2608_19889_amd import axon as ax
    m.timing(True)
    generate()
    torch.cuda.synchronize()
    recs = m.timing_records()
    m.timing(False)
    hd, KV, H = shape["head_dim"], shape["num_key_value_heads"], shape["num_attention_heads"]
    peak_mm = BF16_PEAK_TFLOPS if esz == 2 else F32_PEAK_TFLOPS
    W = shape.get("sliding_window") or 0
    # causal (query, key) pairs; a sliding window keeps min(i + 1, W) keys of query i
    sq = sum(n * (n + 1) / 2 if not W or n <= W else W * (W + 1) / 2 + (n - W) * W for n in lens)
    # grouped expert launches stream every expert some token chose: the
    # expectation under uniform routing, E (1 - (1 - k/E)^tokens) experts
    E_r, k_r = shape.get("n_routed_experts") or 1, shape.get("num_experts_per_tok") or 1
    cls_name = {ax.T_GEMV: "decode projection GEMM (weight streaming)",
                ax.T_GEMV_GROUPED: "decode grouped experts (weight streaming)",
                ax.T_GEMM: "prefill projection GEMM (MFMA)",
                ax.T_ATTN_DECODE: "decode attention (+ split merge)",
                ax.T_ATTN_PREFILL: "prefill flash attention"}
    agg = {}
    for c, (d0, d1, d2), ms in recs:
        a = agg.setdefault(c, {"ms": 0.0, "n": 0, "bytes": 0.0, "flops": 0.0})
        a["ms"] += ms
        a["n"] += 1
        if c == ax.T_GEMV:
            N, M, K = d0, d1, d2
            a["bytes"] += N * K * esz + M * K * esz + M * N * 4
            a["flops"] += 2.0 * N * M * K
        elif c == ax.T_GEMV_GROUPED:
            N, M, K = d0, d1, d2
            active = E_r * (1.0 - (1.0 - k_r / E_r) ** M)
            a["bytes"] += active * N * K * esz + M * K * esz + M * k_r * N * 4
            a["flops"] += 2.0 * N * M * k_r * K
        elif c == ax.T_GEMM:
            N, M, K = d0, d1, d2
            a["flops"] += 2.0 * N * M * K
            a["bytes"] += N * K * esz + M * K * esz + M * N * 4
        elif c == ax.T_ATTN_DECODE:
            ctx = d2
            a["bytes"] += 2 * KV * hd * esz * ctx + 2 * d1 * H * hd * esz
            a["flops"] += 4.0 * H * hd * ctx
        # prefill attention: the workload's causal total is added below (one
        # launch per layer for a prefill, several for chunked prompts)
    if ax.T_ATTN_PREFILL in agg:
        agg[ax.T_ATTN_PREFILL]["flops"] = 4.0 * H * hd * sq * shape["num_hidden_layers"]
    # per-shape breakdown of the decode projections (stderr): (N, K) -> time, bandwidth
    shapes = {}
    for c, (d0, d1, d2), ms in recs:
        if c != ax.T_GEMV:
            continue
        b = shapes.setdefault((d0, d2), {"ms": 0.0, "n": 0, "bytes": 0.0})
        b["ms"] += ms
        b["n"] += 1
        b["bytes"] += d0 * d2 * esz + d1 * d2 * esz + d1 * d0 * 4
    for (N, K), b in sorted(shapes.items(), key=lambda kv: -kv[1]["ms"]):
        log(f"decode projection N={N} K={K}: {b['n']} launches, avg {1e3 * b['ms'] / b['n']:.2f} us, "
            f"{b['bytes'] / (b['ms'] / 1e3) / 1e9:.0f} GB/s")
    # and of the prefill GEMMs: (N, K) -> time, TFLOP/s
    gshapes = {}
    for c, (d0, d1, d2), ms in recs:
        if c != ax.T_GEMM:
            continue
        b = gshapes.setdefault((d0, d2), {"ms": 0.0, "n": 0, "flops": 0.0, "rows": 0})
        b["ms"] += ms
        b["n"] += 1
        b["flops"] += 2.0 * d0 * d1 * d2
        b["rows"] += d1
    for (N, K), b in sorted(gshapes.items(), key=lambda kv: -kv[1]["ms"]):
        log(f"prefill GEMM N={N} K={K}: {b['n']} launches, {b['rows'] // b['n']} rows each, "
            f"{b['ms']:.2f} ms, {b['flops'] / (b['ms'] / 1e3) / 1e12:.0f} TFLOP/s")
    kernels = {}
    for c, a in agg.items():
        hbm = c in (ax.T_GEMV, ax.T_GEMV_GROUPED, ax.T_ATTN_DECODE)
        ach = (a["bytes"] / (a["ms"] / 1e3) / 1e9) if hbm else (a["flops"] / (a["ms"] / 1e3) / 1e12)
        peak = HBM_PEAK_GBS if hbm else peak_mm
        kernels[cls_name[c]] = {"bound": "hbm" if hbm else "mfma", "achieved": round(ach, 1),
                                "peak": peak, "unit": "GB/s" if hbm else "TFLOP/s",
                                "frac": round(ach / peak, 4), "launches": a["n"],
                                "total_ms": round(a["ms"], 3), "avg_us": round(1e3 * a["ms"] / a["n"], 2)}
    dom = max(agg, key=lambda c: agg[c]["ms"])
    r = dict(kernels[cls_name[dom]])
    r["kernel"] = cls_name[dom]
    r["traffic"] = None
    return {"roofline": r, "kernels": kernels}


def kernel_source_digest():
    """Digest of the decode projection kernels' sources: k_gemv.hip, common.h
    and, of kernels.h, the part from the projection epilogue enum through the
    argument struct (declarations elsewhere in that header do not change the
    kernels)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_19889_amd", "csrc")
    for f in ("k_gemv.hip", "common.h"):
        h.update(open(os.path.join(csrc, f), "rb").read())
    hdr = open(os.path.join(csrc, "kernels.h")).read()
    a = hdr.index("enum GvEpi")
    h.update(hdr[a:hdr.index("};", hdr.index("struct GemvArgs", a)) + 2].encode())
    return h.hexdigest()[:16]


def attention_source_digest():
    """Digest of the decode attention kernels' source (k_attn.hip, common.h)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_19889_amd", "csrc")
    for f in ("k_attn.hip", "common.h"):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def measured_attention_traffic(workload):
    """HBM bytes per layer of the decode attention (with its split merge) from
    the committed counter runs, or None when they were taken on other kernel
    sources."""
    path = os.path.join(ROOT, "profiles", f"decode_gemv_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    att = rec.get("decode_attention")
    if not att or rec.get("attention_source_digest") != attention_source_digest():
        return None
    return att.get("hbm_bytes_per_layer")


def measured_traffic(roof, workload):
    """HBM bytes per launch of the decode projection kernels from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE runs (scaled by the counters' reading of
    a 1 GiB copy), or None when those counters were taken on other kernel
    sources or another workload."""
    path = os.path.join(ROOT, "profiles", f"decode_gemv_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_source_digest") != kernel_source_digest():
        return None
    return rec.get("hbm_bytes_per_launch")


def summarize_counters(fetch_csv, write_csv, workload):
    """HBM bytes per decode-projection launch from FETCH_SIZE / WRITE_SIZE
    (KiB per dispatch).  Each counter is scaled by what it reads for the 1 GiB
    calibration copy (the largest __amd_rocclr_copyBuffer dispatch).  Every
    fused-projection dispatch gets a role from its epilogue template argument
    and its place in dispatch order (the residual projection after QKV is O,
    the one after gate/up is down); per-role averages are then weighted by the
    launch mix of one generate on the workload (per decode step: QKV, O,
    gate/up and down of every layer plus the head; plus the prefill's head)."""
    import csv
    from synthetic import MODEL_SHAPES, WORKLOADS
    wl = WORKLOADS[workload]
    L, steps = MODEL_SHAPES[wl["model"]]["num_hidden_layers"], wl["steps"]

    def per_role(path):
        rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
        cal = max(float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"])
        scale = (1 << 30) / (cal * 1024.0)
        agg, names, after = {}, {}, None
        for r in rows:
            name = r["Kernel_Name"]
            if "attn_decode_bf16_kernel" in name or "attn_combine_kernel" in name:  # (older builds: a merge kernel)
                a = agg.setdefault("attention" if "attn_decode" in name else "attention merge", [0, 0.0])
                a[0] += 1
                a[1] += float(r["Counter_Value"]) * 1024.0 * scale
                continue
            if "gemv_fused_kernel" not in name:
                continue
            targs = name[name.index("gemv_fused_kernel<") + 18:name.index(">")].split(",")
            norm, epi = targs[3].strip() == "true", int(targs[4])
            if epi == 3:
                role = after = "qkv"
            elif epi == 2:
                role = after = "gate/up"
            elif epi == 1:
                role = "o" if after == "qkv" else "down"
            else:
                role = "head (decode)" if norm else "head (prefill)"
            a = agg.setdefault(role, [0, 0.0])
            a[0] += 1
            a[1] += float(r["Counter_Value"]) * 1024.0 * scale
            names.setdefault(role, name[name.index("gemv_fused_kernel"):name.index(">") + 1])
        # one generate of this workload alone: each projection once per layer
        # and decode step (a run that also held another model would mix them)
        want = COUNTER_DECODE_STEPS * L
        for role in ("qkv", "o", "gate/up", "down"):
            if agg.get(role, [0])[0] != want:
                raise SystemExit(f"{path}: {agg.get(role, [0])[0]} '{role}' dispatches, expected {want} "
                                 f"({COUNTER_DECODE_STEPS} decode steps x {L} layers of the {workload} workload)")
        return scale, {k: v[1] / v[0] for k, v in agg.items()}, names

    fs, fetch, names = per_role(fetch_csv)
    ws, write, _ = per_role(write_csv)
    per = {k: fetch[k] + write.get(k, 0.0) for k in fetch}
    # decode attention: HBM bytes of one layer's launch (with its split merge,
    # when there is one) against its algorithmic bytes (K and V of every key
    # each sequence attends to, q read and o written), averaged over the
    # COUNTER_DECODE_STEPS decode steps of the counter run
    shape = MODEL_SHAPES[wl["model"]]
    KV, hd, H = shape["num_key_value_heads"], shape["head_dim"], shape["num_attention_heads"]
    W = shape.get("sliding_window") or 0
    if wl["paged"]:
        from synthetic import paged_workload
        seqs, _, _ = paged_workload(wl["batch"], wl["len_range"][0], wl["len_range"][1], steps,
                                    shape["vocab_size"], wl["page_size"], seed=0)
        lens = [len(x) for x in seqs]
    else:
        lens = [wl["prompt_len"]] * wl["batch"]
    alg = 0.0
    for st in range(COUNTER_DECODE_STEPS):
        keys = sum(min(n + st + 1, W) if W else n + st + 1 for n in lens)
        alg += 2 * KV * hd * 2 * keys + 2 * len(lens) * H * hd * 2
    alg /= COUNTER_DECODE_STEPS
    attention = None
    if "attention" in per:
        hbm = per["attention"] + per.get("attention merge", 0.0)
        attention = {"hbm_bytes_per_layer": round(hbm), "algorithmic_bytes_per_layer": round(alg),
                     "ratio": round(hbm / alg, 4), "kernel_bytes": round(per["attention"]),
                     "merge_bytes": round(per.get("attention merge", 0.0))}
    for k in ("attention", "attention merge"):
        per.pop(k, None)
    step_bytes = L * sum(per[k] for k in ("qkv", "o", "gate/up", "down")) + per["head (decode)"]
    launches = steps * (4 * L + 1) + 1
    total = steps * step_bytes + per["head (prefill)"]
    rec = {"workload": workload, "kernel_source_digest": kernel_source_digest(),
           "attention_source_digest": attention_source_digest(),
           "fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
           "hbm_bytes_per_launch_by_role": {k: round(v) for k, v in per.items()},
           "kernel_by_role": names,
           "hbm_bytes_per_launch": round(total / launches),
           "launch_mix": f"{steps} decode steps x ({L} layers x 4 projections + head) + prefill head = {launches}",
           "decode_attention": attention,
           "commands": [f"rocprofv3 --pmc {c} --kernel-include-regex "
                        f"'gemv_fused|attn_decode|attn_combine|copyBuffer|elementwise_kernel' "
                        f"-f csv -d <dir> -o run -- python3 bench.py --workload {workload} --steps 1 --warmup 0 "
                        f"--decode-steps {COUNTER_DECODE_STEPS} --no-cpu-baseline --no-roofline --copy-calibration"
                        + (" --no-7b" if workload == "1b" else "")
                        for c in ("FETCH_SIZE", "WRITE_SIZE")]}
    out = os.path.join(ROOT, "profiles", f"decode_gemv_{workload}_traffic.json")
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec, indent=1))


def host_description():
    """The host the oracle ran on: logical CPUs, CPU model name and RAM, read
    from /proc."""
    model, mem_kb = "unknown", 0
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal:"):
                mem_kb = int(line.split()[1])
                break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model, "ram_gb": round(mem_kb / 2 ** 20, 1),
            "blas_threads_env": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(shape, wl, lens, steps, B, seqs_sample=2):
    """The float64 oracle on the host cores, on a bounded sample of the same
    workload: the first ``seqs_sample`` sequences run in full (prefill of the
    real prompt, then every greedy decode step).  The oracle processes one
    sequence at a time, so generated tokens / wall time over the sample is its
    throughput on the whole batch."""
    import numpy as np
    import oracle
    from synthetic import model_weights, paged_workload, prompts
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [os.cpu_count()])
    except Exception:
        threads = os.cpu_count()
    t0 = time.time()
    w = model_weights(shape, seed=0, device="cpu")
    orc = oracle.OracleDecoder(shape, w)
    del w
    log(f"[bench] oracle weights ready in {time.time() - t0:.1f}s")
    if wl["paged"]:
        seqs, _, _ = paged_workload(B, wl["len_range"][0], wl["len_range"][1], steps, shape["vocab_size"],
                                    wl["page_size"], seed=0)
        seqs = [s.numpy() for s in seqs[:seqs_sample]]
    else:
        seqs = list(prompts(B, wl["prompt_len"], shape["vocab_size"], seed=0).numpy()[:seqs_sample])
    t1 = time.perf_counter()
    toks, _ = oracle.generate_greedy(orc, seqs, steps)
    t2 = time.perf_counter()
    gen = toks.size
    value = gen / (t2 - t1)
    log(f"[bench] oracle sample: {gen} tokens in {t2 - t1:.1f}s")
    return {"value": round(value, 4), "unit": "generated tokens/s", "cores": threads, "kind": "oracle",
            "host": host_description(),
            "sample": f"{len(seqs)} of the {B} sequences, complete (prefill of {[len(x) for x in seqs]} prompt "
                      f"tokens + {steps} greedy decode steps each), float64, {t2 - t1:.1f}s"}


if __name__ == "__main__":
    main()
