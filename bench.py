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
    ap.add_argument("--workload", default="1b", choices=["1b", "7b", "135m", "7b_paged", "32b"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-roofline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(this build has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_19889_amd import axon as ax
    if not os.path.exists(ax.LIB_PATH):
        from paper_2608_19889_amd.build import build
        build()
    from synthetic import MODEL_SHAPES, WORKLOADS, model_weights, paged_workload, prompts

    wl = dict(WORKLOADS[args.workload])
    shape = MODEL_SHAPES[wl["model"]]
    esz = 2 if shape["dtype"] == "bf16" else 4
    B, steps = wl["batch"], wl["steps"]
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
    m = ax.Model(shape, w, max_batch=B, max_seq=max_seq, max_tokens=cu[-1], **page_kw)
    log(f"[bench] model + inputs ready in {time.time() - t0:.1f}s "
        f"(weights {weight_bytes(shape, esz) / 1e9:.2f} GB, prompt tokens {cu[-1]})")

    nt = [torch.empty(B, dtype=torch.int32, device=dev) for _ in range(2)]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]

    def generate(record=False):
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

    for i in range(args.warmup):
        generate()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    pre_ms, dec_ms = [], []
    t_start = time.perf_counter()
    for i in range(args.steps):
        generate(record=True)
        torch.cuda.synchronize()
        pre_ms.append(ev[0].elapsed_time(ev[1]))
        dec_ms.append(ev[1].elapsed_time(ev[2]))
        log(f"[bench] step {i + 1}/{args.steps}: prefill {pre_ms[-1]:.2f} ms, decode {dec_ms[-1]:.2f} ms")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = wall * 1e3 / args.steps
    gen_tokens = B * (steps + 1)
    value = gen_tokens / (ms_per_step / 1e3)
    prefill_ms, decode_ms = float(np.mean(pre_ms)), float(np.mean(dec_ms))

    # algorithmic decode bytes: every weight except the embedding table (B rows
    # of it), the KV cache read over each step's context and the new KV written
    # (a tied head reads the embedding table in full; an untied model reads
    # only B rows of the table and the separate head matrix)
    wb = weight_bytes(shape, esz)
    emb = V * D * esz
    kv_read = 0
    for s in range(steps):
        for n in lens:
            kv_read += 2 * L * KV * hd * (n + s + 1) * esz
    kv_write = steps * B * 2 * L * KV * hd * esz
    per_step_weights = wb - (0 if shape["tie_word_embeddings"] else emb) + B * D * esz
    decode_bytes = steps * per_step_weights + kv_read + kv_write
    decode_gbs = decode_bytes / (decode_ms / 1e3) / 1e9

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "generated tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape["dtype"],
        "data": "synthetic (random-init N(0,0.02) weights, uniform random prompt ids)",
        "config": {"workload": f"{args.workload}-shaped decoder: batch {B}, "
                               + (f"prompts {wl['prompt_len']}" if not wl["paged"] else
                                  f"prompts U[{wl['len_range'][0]},{wl['len_range'][1]}] (sum {cu[-1]})")
                               + f", {steps} greedy decode steps, "
                               + ("paged KV (16-token pages)" if wl["paged"] else "contiguous KV"),
                   "batch": B, "prompt_tokens": cu[-1], "decode_steps": steps,
                   "layers": L, "hidden": D, "vocab": V},
        "prefill_tok_s": round(cu[-1] / (prefill_ms / 1e3), 1),
        "prefill_ms": round(prefill_ms, 3),
        "decode_tok_s": round(B * steps / (decode_ms / 1e3), 1),
        "decode_ms_per_token_step": round(decode_ms / steps, 4),
        "decode_hbm_gbs": round(decode_gbs, 1),
        "decode_hbm_frac": round(decode_gbs / HBM_PEAK_GBS, 4),
    }

    if not args.no_roofline:
        out.update(roofline_pass(m, generate, shape, esz, lens))
    m.close()
    del w
    torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, wl, lens, steps, B)
    print(json.dumps(out), flush=True)


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
    sq = sum(n * (n + 1) / 2 for n in lens)
    cls_name = {ax.T_GEMV: "decode projection GEMM (weight streaming)",
                ax.T_GEMM: "prefill projection GEMM (MFMA)",
                ax.T_ATTN_DECODE: "decode attention (split-K + combine)",
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
        elif c == ax.T_GEMM:
            N, M, K = d0, d1, d2
            a["flops"] += 2.0 * N * M * K
            a["bytes"] += N * K * esz + M * K * esz + M * N * 4
        elif c == ax.T_ATTN_DECODE:
            ctx = d2
            a["bytes"] += 2 * KV * hd * esz * ctx + 2 * d1 * H * hd * esz
            a["flops"] += 4.0 * H * hd * ctx
        else:
            a["flops"] += 4.0 * H * hd * sq
    kernels = {}
    for c, a in agg.items():
        hbm = c in (ax.T_GEMV, ax.T_ATTN_DECODE)
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


def cpu_baseline(shape, wl, lens, steps, B):
    """The float64 oracle on the host cores, on a bounded sample: one sequence,
    a short prefill and a few decode steps; its per-token costs are scaled to
    the workload's generated tokens/s."""
    import numpy as np
    import torch
    import oracle
    from synthetic import model_weights, prompts
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
    P_s, S_s = 64, 3
    ids = prompts(1, P_s, shape["vocab_size"], seed=0)[0].numpy()
    t1 = time.perf_counter()
    lg = orc.prefill([ids])
    t2 = time.perf_counter()
    tok = [int(np.argmax(lg[0]))]
    for _ in range(S_s):
        tok = [int(np.argmax(orc.decode(tok)[0]))]
    t3 = time.perf_counter()
    pre_tok_s = P_s / (t2 - t1)
    dec_step_s = (t3 - t2) / S_s
    # workload time on the oracle: prefill all prompt tokens, then every
    # sequence's decode steps one at a time (the oracle has no batching)
    total_s = sum(lens) / pre_tok_s + B * steps * dec_step_s
    value = B * (steps + 1) / total_s
    log(f"[bench] oracle sample: prefill {pre_tok_s:.1f} tok/s, decode {dec_step_s:.3f} s/token")
    return {"value": round(value, 4), "unit": "generated tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"1 sequence: {P_s}-token prefill ({t2 - t1:.1f}s) + {S_s} decode steps "
                      f"({t3 - t2:.1f}s) of the same model in float64; scaled to the workload "
                      f"({sum(lens)} prompt tokens, {B}x{steps} decode tokens)",
            "prefill_tok_s": round(pre_tok_s, 2), "decode_s_per_token": round(dec_step_s, 4)}


if __name__ == "__main__":
    main()
