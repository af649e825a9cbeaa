"""Population decode benchmark on one MI355X.

Default workload: 8B-class dense decoder (36 layers, hidden 4096, 32/8 heads x
128, FFN 12288 SwiGLU, vocab 151936, bf16 weights, random init), population
N = 64 candidates, each an aggregation context of K = 4 candidates with
16k-32k cached tokens (uniform), 16-token pages in a shuffled page table.
A step = one decode step of the whole population (embedding, 36 layers of
RMSNorm / QKV / QK-norm + RoPE + KV append / paged attention / O / SwiGLU FFN,
final norm, LM head, log-softmax + Gumbel-max sampling) followed by the
host-side bookkeeping done on device (next tokens, positions + 1).

--workload moe30b_pop64_agg4 runs the same step on a 30B-A3B-class
mixture-of-experts decoder (48 layers, hidden 2048, 32/4 heads x 128, 128
experts of FFN 768, top-8 routing, vocab 151936) at the same population and
contexts.

Prints one JSON line: tokens/s of the population, the roofline of the dominant
kernel (the split-KV attention kernel, HIP events around each of its launches
in the last timed step) and the oracle's throughput on a bounded sample of the
same workload on the host cores (cpu_baseline).
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
# sources of the attention split kernel; the HBM-counter traffic recorded under
# profiles/ is reported only while they are unchanged
ATTN_SOURCES = ["paper_2604_07725_amd/csrc/attn_decode.hip", "paper_2604_07725_amd/csrc/common.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_split_mfma_kernel_traffic.json")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def attention_bytes(lengths, hkv, hq, d):
    """Algorithmic bytes of one attention launch: every cached key and value of
    every candidate once (bf16), q and o (bf16) and the page-table entries."""
    lengths = np.asarray(lengths, np.int64)
    kv = int(lengths.sum()) * hkv * d * 2 * 2
    pages = int(((lengths + 15) // 16).sum())
    n = len(lengths)
    return kv + 2 * n * hq * d * 2 + pages * 4


def expected_distinct_experts(shape, n):
    """Experts a layer touches when n tokens each pick top_k of n_experts
    uniformly at random: E (1 - (1 - k / E)^n)."""
    E, k = shape.n_experts, shape.top_k
    return E * (1.0 - (1.0 - k / E) ** n)


def peak_fracs(achieved, peak):
    """achieved GB/s as fractions of the measured read ceilings (None if not measured)."""
    if not peak:
        return {"frac_of_measured_sequential": None, "frac_of_measured_pages": None}
    return {"frac_of_measured_sequential": achieved / peak["sequential_GBs"],
            "frac_of_measured_pages": achieved / peak["pages_8KB_GBs"]}


def attention_main(args, w, peak):
    """Attention-only workload (split-KV attention + combine of one layer):
    `reps` timed calls rotating 4 independent KV pools (each larger than the
    256 MB Infinity Cache), HIP events around every split launch."""
    import torch
    from paper_2604_07725_amd import device_inputs as di
    from paper_2604_07725_amd import sevo, synth
    shape = w.shape
    reps = 100 if args.steps is None else args.steps
    pop = synth.workload_population(w)
    dev = torch.device("cuda:0")
    pools = [di.device_pools(shape, w.seed + 1000 * r, pop.n_pages, dev, layers=[0])[0]
             for r in range(4)]
    q = di.device_q(shape, w.seed, pop.n, dev)
    lens = torch.from_numpy(pop.lengths.astype(np.int32)).to(dev)
    pt = torch.from_numpy(pop.page_table).to(dev)
    S = args.num_splits or sevo.sevo_attn_plan_splits(pop.n, shape.n_kv_heads, pop.max_pages)
    ws = torch.empty(sevo.sevo_attn_workspace_bytes(pop.n, shape.n_q_heads, shape.n_kv_heads,
                                                    shape.head_dim, pop.max_pages, S),
                     dtype=torch.uint8, device=dev)
    out = torch.empty(pop.n, shape.n_q_heads, shape.head_dim, dtype=torch.bfloat16, device=dev)
    call = lambda r: sevo.sevo_attn_decode(q, pools[r % 4], pt, lens, num_splits=S,  # noqa: E731
                                           out=out, workspace=ws)
    for r in range(args.warmup + 4):
        call(r)
    torch.cuda.synchronize()
    sevo.sevo_profile_begin(reps, ("attn_split", "attn_combine"))
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for r in range(reps):
        call(r)
    b.record()
    torch.cuda.synchronize()
    prof = sevo.sevo_profile_end()
    total_ms = a.elapsed_time(b)
    byts = attention_bytes(pop.lengths, shape.n_kv_heads, shape.n_q_heads, shape.head_dim)
    split_ms = prof["attn_split"][0] / max(prof["attn_split"][1], 1)
    comb_ms = prof["attn_combine"][0] / max(prof["attn_combine"][1], 1)
    achieved = byts / (split_ms * 1e-3) / 1e9
    res = {
        "metric": "attention HBM GB/s", "value": byts / ((split_ms + comb_ms) * 1e-3) / 1e9,
        "unit": "GB/s", "n_gpus": 1, "steps": reps, "warmup": args.warmup,
        "ms_per_step": total_ms / reps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded)",
        "config": {"workload": w.name, "heads": f"{shape.n_q_heads}/{shape.n_kv_heads}x"
                   f"{shape.head_dim}", "population": pop.n, "aggregation_k": w.aggregation_k,
                   "context_tokens": [int(pop.lengths.min()), int(pop.lengths.max())],
                   "page_size": 16, "num_splits": S, "kv_pools_rotated": 4,
                   "parallelism": "none (1 GPU)"},
        "roofline": {"kernel": f"{attn_kernel_name(shape)} (paged split-KV GQA attention)",
                     "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "bytes_per_launch": byts, "avg_launch_ms": split_ms,
                     "combine_avg_ms": comb_ms, **peak_fracs(achieved, peak)},
        "read_peak": peak,
    }
    if not args.no_cpu_baseline:
        log("timing the oracle on a bounded sample (host cores)")
        res["cpu_baseline"] = attention_cpu_baseline(shape, w.seed, pop)
    print(json.dumps(res), flush=True)


def attention_cpu_baseline(shape, seed, pop, n_sample=4):
    """The oracle's dense float64 attention (all heads) for the first n_sample
    candidates over their full contexts; GB/s of their algorithmic bytes."""
    from oracle import decoder as od
    from paper_2604_07725_amd import synth
    from threadpoolctl import threadpool_info
    qh = synth.host_values(synth.q_spec(shape, seed, pop.n)).reshape(pop.n, shape.n_q_heads,
                                                                      shape.head_dim)
    spec = synth.kv_spec(shape, seed, 0, pop.n_pages)
    kv = []
    for i in range(n_sample):
        n = int(pop.lengths[i])
        pool = synth.pool_pages(spec, pop.page_table[i, :(n + 15) // 16])
        kv.append(od.gather_kv(pool, np.arange(pool.shape[0]), n))
    t0 = time.perf_counter()
    for i in range(n_sample):
        od.attention_dense(qh[i], kv[i][0], kv[i][1], shape.head_dim ** -0.5)
    dt = time.perf_counter() - t0
    byts = attention_bytes(pop.lengths[:n_sample], shape.n_kv_heads, shape.n_q_heads,
                           shape.head_dim)
    blas = threadpool_info()
    return {"value": byts / dt / 1e9, "unit": "GB/s", "kind": "oracle",
            "cores": int(max([b.get("num_threads", 1) for b in blas] or [1])),
            "sample": f"oracle float64 attention of {n_sample} of {pop.n} candidates "
                      f"({int(pop.lengths[:n_sample].sum())} cached tokens), {dt:.2f} s",
            "host_cpus": len(os.sched_getaffinity(0))}


def attn_kernel_name(shape):
    g = shape.n_q_heads // shape.n_kv_heads
    kern = "attn_split_mfma_kernel" if g >= 4 else "attn_split_kernel"
    return f"{kern}<{shape.head_dim},{g}>"


def model_name(shape):
    if shape.is_moe:
        return (f"MoE decoder ({shape.n_experts} experts, top-{shape.top_k}, "
                f"{shape.weight_bytes() / 2e9:.1f}B stored / "
                f"{shape.weight_bytes(shape.top_k) / 2e9:.1f}B active parameters)")
    return f"dense {shape.weight_bytes() / 2e9:.0f}B-class decoder"


def ffn_config(shape):
    if shape.is_moe:
        return {"experts": shape.n_experts, "experts_per_token": shape.top_k,
                "expert_ffn": shape.expert_ffn}
    return {"ffn": shape.ffn}


def kernel_table(shape, n, kprof, attn_bytes):
    """Average time per launch of each kernel kind of the step, with the
    projections' weight-streaming rate and matrix-core utilisation (algorithmic
    bytes: weights + activations in + outputs out; flops 2 M N K).  The MoE
    experts row counts the weights of the experts a layer is expected to touch
    under uniform routing, each once."""
    H, F, V = shape.hidden, shape.ffn, shape.vocab
    qd = shape.n_q_heads * shape.head_dim
    qkvd = qd + 2 * shape.n_kv_heads * shape.head_dim
    gemms = {"qkv": (qkvd, H, 4), "attn_out": (H, qd, 4), "gate_up": (2 * F, H, None),
             "down": (H, F, 4), "lm_head": (V, H, 4)}
    table = {}
    for kind, (ms, cnt) in kprof.items():
        avg = ms / cnt
        row = {"avg_us": avg * 1e3, "launches": cnt}
        byts = flops = None
        if kind in gemms:
            N, K, ob = gemms[kind]
            out_bytes = n * (F * 2 if ob is None else N * ob)
            byts = N * K * 2 + n * K * 2 + out_bytes
            flops = 2.0 * n * N * K
        elif kind == "moe_experts" and shape.is_moe:
            Fe, k = shape.expert_ffn, shape.top_k
            ne = expected_distinct_experts(shape, n)
            # gate/up: weights, gathered rows in, SwiGLU rows out (bf16);
            # down: weights, SwiGLU rows in, weighted fp32 partials out
            byts = (ne * 3 * Fe * H * 2 + n * k * (H * 2 + Fe * 2) + n * k * (Fe * 2 + H * 4))
            flops = 2.0 * n * k * 3 * Fe * H
            row["expected_distinct_experts"] = ne
        if byts is not None:
            row.update({"GB_s": byts / (avg * 1e-3) / 1e9,
                        "hbm_frac": byts / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS,
                        "TFLOP_s": flops / (avg * 1e-3) / 1e12,
                        "mfma_frac": flops / (avg * 1e-3) / 1e12 / BF16_PEAK_TFLOPS})
        elif kind == "attn_split":
            row["GB_s"] = attn_bytes / (avg * 1e-3) / 1e9
        table[kind] = row
    return table


def measure_read_peak(dev, gib=8, grid=32768, reps=10):
    """The measured HBM read ceiling on this machine (sevo_hbm_read_probe): a
    sequential read and random whole 8 KB pages (the decode attention's
    pattern) of a {gib} GiB buffer, GB/s by events over `reps` reads each."""
    import torch
    from paper_2604_07725_amd import sevo
    buf = torch.empty(gib << 30, dtype=torch.uint8, device=dev)
    order = torch.randperm((gib << 30) // 8192, device=dev, dtype=torch.int32)
    sink = torch.empty(grid * 16, dtype=torch.uint8, device=dev)
    out = {"buffer_bytes": buf.numel(), "grid": grid}
    for name, po in (("sequential_GBs", None), ("pages_8KB_GBs", order)):
        for _ in range(2):
            sevo.sevo_hbm_read_probe(buf, po, grid, sink)
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            sevo.sevo_hbm_read_probe(buf, po, grid, sink)
        b.record()
        torch.cuda.synchronize()
        out[name] = buf.numel() * reps / (a.elapsed_time(b) * 1e-3) / 1e9
    del buf, order, sink
    torch.cuda.empty_cache()
    return out


def measured_traffic(workload):
    """HBM bytes per attention launch from the rocprofv3 FETCH_SIZE / WRITE_SIZE
    passes (copy-kernel calibrated) recorded under profiles/, or None when they
    were taken on another workload or the kernel sources changed since."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if rec.get("source_sha256") != h.hexdigest() or rec.get("workload") != workload:
        return None
    return rec


def cpu_baseline(w, pop, n_sample, budget_s=30.0):
    """The oracle, as it stands, on a bounded sample of the workload: layer 0
    of the model for the first n_sample candidates (attention over their full
    contexts + that layer's projections), then the final norm, LM head and
    sampler for them.  Inputs are generated before the clock starts.  The
    per-token time extrapolates the layer time to the model's depth."""
    from oracle import decoder as od
    from paper_2604_07725_amd import synth
    from threadpoolctl import threadpool_info
    shape = w.shape
    idx = np.arange(n_sample)
    lengths = pop.lengths[idx].astype(np.int64)
    # compact host pools holding only the sampled candidates' pages
    need = (lengths + 1 + 15) // 16
    pt = np.full((n_sample, int(need.max())), -1, np.int64)
    spec = synth.kv_spec(shape, w.seed, 0, pop.n_pages)
    kvp = np.empty((int(need.sum()),) + tuple(spec.shape[1:]), np.float32)
    c = 0
    for j, i in enumerate(idx):
        pages = pop.page_table[i, :need[j]]
        kvp[c:c + need[j]] = synth.pool_pages(spec, pages)
        pt[j, :need[j]] = np.arange(c, c + need[j])
        c += need[j]
    hw = synth.host_weights(shape, w.seed, lazy=True)
    lw = hw["layers"][0]
    x = np.asarray(hw["embed"][pop.tokens[idx]], np.float64)
    lm_head = hw["lm_head"][0:shape.vocab]
    t0 = time.perf_counter()
    x1 = od.decoder_layer(shape, lw, x, lengths, kvp, pt, mirror=True)
    t1 = time.perf_counter()
    logits = od.lm_logits(shape, hw["final_norm"], lm_head, x1, mirror=True)
    od.logprob_sample(logits, 1.0, 1234, pop.uids[idx], lengths)
    t2 = time.perf_counter()
    t_layer, t_head = t1 - t0, t2 - t1
    step_s = shape.n_layers * t_layer + t_head
    blas = threadpool_info()
    threads = max([b.get("num_threads", 1) for b in blas] or [1])
    return {
        "value": n_sample / step_s, "unit": "tokens/s", "cores": int(threads),
        "kind": "oracle",
        "sample": (f"oracle decoder layer 0 + LM head + sampler for {n_sample} of {pop.n} "
                   f"candidates (contexts {int(lengths.min())}-{int(lengths.max())} tokens); "
                   f"layer time x {shape.n_layers} layers + head time = {step_s:.2f} s per "
                   f"step of {n_sample} tokens (measured {t_layer:.2f} s layer, {t_head:.2f} s "
                   f"head; extrapolated in depth only)"),
        "host_cpus": len(os.sched_getaffinity(0)),
        "blas": [b.get("internal_api") for b in blas],
    }


PREFILL_GEMM_KINDS = ("qkv", "attn_out", "gate_up", "down", "moe_route", "moe_experts")
# the paper's confidence-engine latency for Qwen3-30B-A3B (the shapes of the MoE
# stand-in), seconds per request at each length: another machine's figures
PAPER_ENGINE_S_QWEN3_30B_A3B = {40960: 1.58, 81920: 4.42, 122880: 8.41}


def prefill_flops(shape, T, R):
    """Algorithmic flops of one request of T tokens from position 0 with R
    scored rows: causal attention (2 flops per multiply-add, q.k and p.v over
    keys 0..t for every token and head), the projections (2 M N K) and the LM
    head on the scored rows."""
    hq, d, H, F = shape.n_q_heads, shape.head_dim, shape.hidden, shape.ffn
    attn = 4.0 * hq * d * T * (T + 1) / 2
    per_layer = {"qkv": 2.0 * T * shape.qkv_dim * H, "attn_out": 2.0 * T * H * shape.q_dim}
    if shape.is_moe:
        # router GEMM; the selected experts' gate/up + down for every token
        per_layer["moe_route"] = 2.0 * T * shape.n_experts * H
        per_layer["moe_experts"] = 2.0 * T * shape.top_k * 3 * shape.expert_ffn * H
    else:
        per_layer["gate_up"] = 2.0 * T * 2 * F * H
        per_layer["down"] = 2.0 * T * H * F
    return attn, per_layer, 2.0 * R * shape.vocab * H


def prefill_cpu_baseline(shape, seed, n_tokens=256):
    """The oracle on a bounded sample: layer 0 of the prefill over one
    n_tokens sequence, then final norm + LM head + confidence for its rows;
    extrapolated to the model's depth (the per-layer time is for that length)."""
    from oracle import decoder as od
    from paper_2604_07725_amd import synth
    from threadpoolctl import threadpool_info
    hw = synth.host_weights(shape, seed, lazy=True)
    lw = hw["layers"][0]
    rng = np.random.default_rng(seed)
    toks = rng.integers(0, shape.vocab, n_tokens)
    pages = (n_tokens + 15) // 16
    pool = np.zeros((pages, shape.n_kv_heads, 2, 16 * shape.head_dim))
    pt = np.arange(pages)[None]
    row, pos = od.prefill_index([0, n_tokens])
    x = np.asarray(hw["embed"][toks], np.float64)
    t0 = time.perf_counter()
    x = od.decoder_layer(shape, lw, x, pos, pool, pt[row], mirror=True)
    t1 = time.perf_counter()
    logits = od.lm_logits(shape, hw["final_norm"], hw["lm_head"][0:shape.vocab], x, mirror=True)
    od.token_confidence(logits, 20)
    t2 = time.perf_counter()
    per_req = shape.n_layers * (t1 - t0) + (t2 - t1)
    blas = threadpool_info()
    return {"value": n_tokens / per_req, "unit": "tokens/s", "cores":
            int(max([b.get("num_threads", 1) for b in blas] or [1])), "kind": "oracle",
            "sample": (f"oracle prefill of one {n_tokens}-token sequence: layer 0 "
                       f"({t1 - t0:.2f} s) x {shape.n_layers} layers + LM head and confidence "
                       f"of every row ({t2 - t1:.2f} s) = {per_req:.1f} s; extrapolated in "
                       f"depth only, at this length")}


def prefill_main(args):
    """The confidence engine (prefill-only scoring pass) on the 8B-class model,
    or on the 30B-A3B-class MoE model with --workload moe30b_pop64_agg4: one
    request at a time of each length, every row scored (Eq. 1 c, K_l = 20),
    one C per request returned; per-kernel times from HIP events."""
    import torch
    from paper_2604_07725_amd import device_inputs as di
    from paper_2604_07725_amd import sevo, synth
    w = synth.WORKLOADS[args.workload]
    moe = w.shape.is_moe
    shape = w.shape if moe else synth.DENSE_8B
    seed = w.seed if moe else 2
    lengths = [int(v) for v in args.prefill_tokens.split(",")]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t = time.time()
    tensors = di.device_weights(shape, seed, dev)
    model = sevo.sevo_init_model(shape, tensors, max_position=max(lengths) + 1)
    torch.cuda.synchronize()
    log(f"prefill: weights resident in {time.time() - t:.1f} s")
    results = []
    for T in lengths:
        pages = (T + 15) // 16
        pool = torch.empty(pages, shape.n_kv_heads, 2, 16 * shape.head_dim, dtype=torch.bfloat16,
                           device=dev)   # one pool for every layer: the cache is not kept
        perm = np.random.default_rng(T).permutation(pages).astype(np.int32)
        pt = torch.from_numpy(perm[None]).to(dev)
        toks = torch.from_numpy(np.random.default_rng(T + 1).integers(
            0, shape.vocab, T).astype(np.int32)).to(dev)
        ss = torch.tensor([0, T], dtype=torch.int32, device=dev)
        rows = torch.arange(T, dtype=torch.int32, device=dev)
        buf = sevo.PrefillBuffers(model, toks, ss, pt, pool, rows, 20, T, keep_row_conf=False)
        buf.run()                      # warm-up
        torch.cuda.synchronize()
        reps = args.steps if args.steps < 16 else 2
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(reps):
            buf.run()
        stop.record()
        torch.cuda.synchronize()
        sec = start.elapsed_time(stop) / reps / 1e3
        # per-kernel times: one more request with every launch bracketed
        sevo.sevo_profile_begin(4096, sevo.PROF_KINDS)
        buf.run()
        torch.cuda.synchronize()
        kp = sevo.sevo_profile_end()
        attn_f, gemm_f, head_f = prefill_flops(shape, T, T)
        kern = {}
        for k, (ms, cnt) in kp.items():
            row = {"ms": ms, "launches": cnt}
            f = None
            if k == "attn_prefill":
                f = attn_f * shape.n_layers
            elif k in gemm_f:
                f = gemm_f[k] * shape.n_layers
            elif k == "lm_head":
                f = head_f
            if f:
                row["TFLOP_s"] = f / (ms * 1e-3) / 1e12
                row["mfma_frac"] = row["TFLOP_s"] / BF16_PEAK_TFLOPS
            kern[k] = row
        conf = float(buf.out_conf.cpu()[0])
        log(f"prefill {T} tokens: {sec:.3f} s per request; C = {conf:.4f}")
        results.append({"tokens": T, "s_per_request": sec, "tokens_per_s": T / sec,
                        "confidence": conf, "kernels": kern})
        del buf, pool
        torch.cuda.empty_cache()
    model.close()
    big = results[-1]
    tot_gemm = sum(big["kernels"][k]["ms"] for k in PREFILL_GEMM_KINDS if k in big["kernels"])
    gemm_flops = sum(prefill_flops(shape, big["tokens"], big["tokens"])[1].values()) * shape.n_layers
    out = {
        "metric": "confidence-engine prefill latency per request (s)",
        "value": big["s_per_request"], "unit": "s", "higher_is_better": False,
        "n_gpus": 1, "steps": args.steps if args.steps < 16 else 2, "warmup": 1,
        "dtype": "bf16", "data": "synthetic (seeded; random-init weights)",
        "vs_baseline": (big["s_per_request"] / PAPER_ENGINE_S_QWEN3_30B_A3B[big["tokens"]]
                        if moe and big["tokens"] in PAPER_ENGINE_S_QWEN3_30B_A3B else None),
        "config": {"workload": "confidence_engine_" + ("moe30b" if moe else "dense8b"),
                   "model": model_name(shape), "layers": shape.n_layers,
                   "hidden": shape.hidden,
                   "heads": f"{shape.n_q_heads}/{shape.n_kv_heads}x{shape.head_dim}",
                   **ffn_config(shape), "vocab": shape.vocab, "batch": 1,
                   "tokens": [r["tokens"] for r in results], "scored_rows": "all",
                   "conf_topk": 20},
        "roofline": {"kernel": f"attn_prefill_kernel<{shape.head_dim}> (causal GQA prefill "
                               "attention)",
                     "bound": "mfma", "achieved": big["kernels"]["attn_prefill"]["TFLOP_s"],
                     "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": big["kernels"]["attn_prefill"]["mfma_frac"], "traffic": None},
        "gemm_roofline": {"bound": "mfma", "achieved": gemm_flops / (tot_gemm * 1e-3) / 1e12,
                          "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                          "frac": gemm_flops / (tot_gemm * 1e-3) / 1e12 / BF16_PEAK_TFLOPS},
        "per_length": results,
    }
    if not args.no_cpu_baseline:
        log("timing the oracle on a bounded prefill sample (host cores)")
        out["cpu_baseline"] = prefill_cpu_baseline(shape, seed)
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default: the workload's own count, 16 for the default)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="dense8b_pop64_agg4")
    ap.add_argument("--num-splits", type=int, default=0)
    ap.add_argument("--cpu-sample", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step as one captured HIP graph (same kernels, same work)")
    ap.add_argument("--no-read-peak", action="store_true",
                    help="skip the streaming-read measurement of the HBM ceiling")
    ap.add_argument("--temperature", type=float, default=1.0)
    ap.add_argument("--top-k", type=int, default=0, help="0 = full-vocabulary sampling")
    ap.add_argument("--top-p", type=float, default=1.0)
    ap.add_argument("--min-p", type=float, default=0.0)
    ap.add_argument("--conf-topk", type=int, default=0,
                    help="also compute the per-token self-confidence (top-K log-probs) each step")
    ap.add_argument("--mode", choices=("decode", "prefill"), default="decode",
                    help="decode: the population decode step (default); prefill: the "
                         "cross-model confidence engine at the prefill-benchmark lengths")
    ap.add_argument("--prefill-tokens", default="40960,81920,122880",
                    help="prefill mode: request lengths (tokens), one request at a time")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (3 times), to scale HBM counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the population decode step needs no collectives "
              "and this build runs on a single MI355X; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")   # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": src.numel() * 4, "copies": 3}), flush=True)
        return
    if args.mode == "prefill":
        if args.steps is None:
            args.steps = 16
        return prefill_main(args)
    from paper_2604_07725_amd import device_inputs as di
    from paper_2604_07725_amd import sevo, synth

    w = synth.WORKLOADS[args.workload]
    shape = w.shape
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    peak = None if args.no_read_peak else measure_read_peak(dev)
    if peak:
        log(f"measured read ceiling: sequential {peak['sequential_GBs']:.0f} GB/s, random 8 KB "
            f"pages {peak['pages_8KB_GBs']:.0f} GB/s")
    if w.attention_only:
        return attention_main(args, w, peak)
    if args.steps is None:
        args.steps = w.steps
    # key slots every step appends: warm-up, timed, (graph mode: as many eager
    # steps again for the attention timing), the 2 kernel-table steps
    n_steps_total = args.warmup + args.steps * (2 if args.graph else 1) + 2
    extra = n_steps_total + 1
    pop = synth.workload_population(w, extra_tokens=extra)
    kv_bytes_total = 2 * shape.n_layers * pop.n_pages * shape.n_kv_heads * 16 * shape.head_dim * 2
    free, total = torch.cuda.mem_get_info()
    need = kv_bytes_total + shape.weight_bytes() + 2 * shape.vocab * shape.hidden + (2 << 30)
    log(f"workload {w.name}: N={pop.n} contexts {pop.lengths.min()}-{pop.lengths.max()} "
        f"pages {pop.n_pages}; KV {kv_bytes_total / 1e9:.1f} GB, weights "
        f"{shape.weight_bytes() / 1e9:.2f} GB; free {free / 1e9:.1f} of {total / 1e9:.1f} GB")
    if need > free:
        raise SystemExit(f"not enough device memory: need {need / 1e9:.1f} GB")
    t = time.time()
    tensors = di.device_weights(shape, w.seed, dev)
    kvp = di.device_pools(shape, w.seed, pop.n_pages, dev)
    d = di.device_population(pop, dev)
    model = sevo.sevo_init_model(shape, tensors, max_position=int(pop.lengths.max()) + extra + 1)
    torch.cuda.synchronize()
    log(f"inputs resident in HBM in {time.time() - t:.1f} s")

    tokens = d["tokens"].clone()
    positions = d["lengths"].clone()
    conf_sum = torch.zeros(pop.n, dtype=torch.float32, device=dev) if args.conf_topk else None
    buf = sevo.StepBuffers(model, tokens, positions, d["page_table"], kvp, d["uids"],
                           seed=20260412, temperature=args.temperature,
                           num_splits=args.num_splits, conf_topk=args.conf_topk,
                           conf_sum=conf_sum, top_k=args.top_k, top_p=args.top_p,
                           min_p=args.min_p)

    def step():
        ids, _ = buf.run()
        tokens.copy_(ids)
        positions.add_(1)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done")
    eager_step = step
    if args.graph:
        # one step captured as a graph (every launch of sevo_decode_step and the
        # bookkeeping reads and writes the same device buffers each step)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()   # capture does not run the step
        step = graph.replay

    # HIP events around the attention launches of the last timed step only: a
    # recorded event holds the next launch back until the previous kernel's
    # end is stamped (about 4.5 us idle per event, three per layer), which on
    # every step would slow the steps the clock measures by 1.5-4.5%.  The
    # event pool is created before the clock starts.
    if not args.graph:
        sevo.sevo_profile_begin(shape.n_layers, ("attn_split", "attn_combine"))
        sevo.sevo_profile_end()
    # one event per step boundary (median and spread of the step time)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    marks[0].record()
    for i in range(args.steps):
        if not args.graph and i == args.steps - 1:
            sevo.sevo_profile_begin(shape.n_layers, ("attn_split", "attn_combine"))
        step()
        marks[i + 1].record()
    torch.cuda.synchronize()
    total_ms = marks[0].elapsed_time(marks[-1])
    step_ms = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)])
    if args.graph:
        # the replayed graph records no per-launch events: time the attention
        # launches over one eager step
        sevo.sevo_profile_begin(shape.n_layers, ("attn_split", "attn_combine"))
        eager_step()
        torch.cuda.synchronize()
    prof = sevo.sevo_profile_end()
    split_ms, launches = prof["attn_split"]
    attn_ms = split_ms + prof["attn_combine"][0]
    ms_per_step = total_ms / args.steps

    # per-kernel breakdown: two more steps with every launch of the step timed
    # (outside the timed region: the extra event records cost a little time)
    sevo.sevo_profile_begin(400 * 2, sevo.PROF_KINDS)
    for _ in range(2):
        eager_step()
    torch.cuda.synchronize()
    kprof = sevo.sevo_profile_end()
    log(f"{args.steps} steps: {ms_per_step:.3f} ms/step; attention launches {launches}")

    # algorithmic bytes of the timed attention launches (lengths grow by one per
    # step): those of the last timed step (graph mode: the eager step after them)
    lens_timed = pop.lengths.astype(np.int64) + args.warmup + 1 + (args.steps if args.graph
                                                                    else args.steps - 1)
    attn_bytes_per_launch = float(attention_bytes(lens_timed, shape.n_kv_heads, shape.n_q_heads,
                                                  shape.head_dim))
    # the step's bytes: the mean over the timed steps
    base = pop.lengths.astype(np.int64) + args.warmup + 1
    step_attn_bytes = float(np.mean([attention_bytes(base + s, shape.n_kv_heads, shape.n_q_heads,
                                                     shape.head_dim) for s in range(args.steps)]))
    split_avg_ms = split_ms / max(launches, 1)
    attn_avg_ms = attn_ms / max(launches, 1)
    achieved = attn_bytes_per_launch / (split_avg_ms * 1e-3) / 1e9
    active = expected_distinct_experts(shape, pop.n) if shape.is_moe else None
    step_bytes = shape.n_layers * step_attn_bytes + shape.weight_bytes(active)
    tr = measured_traffic(w.name)
    out = {
        "metric": "population decode tokens/s/GPU",
        "value": pop.n / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_median": float(np.median(step_ms)),
        "ms_per_step_min_max": [float(step_ms.min()), float(step_ms.max())],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded; random-init weights)",
        "config": {"workload": w.name, "model": model_name(shape), "layers": shape.n_layers,
                   "hidden": shape.hidden, "heads": f"{shape.n_q_heads}/{shape.n_kv_heads}x"
                   f"{shape.head_dim}", "vocab": shape.vocab, **ffn_config(shape),
                   "population": pop.n, "aggregation_k": w.aggregation_k,
                   "context_tokens": [int(pop.lengths.min()), int(pop.lengths.max())],
                   "page_size": 16, "parallelism": "none (1 GPU)",
                   "num_splits": int(buf.args.num_splits) or
                   sevo.sevo_attn_plan_splits(pop.n, shape.n_kv_heads, pop.max_pages),
                   "temperature": args.temperature,
                   "sampling": ("full vocabulary" if args.top_k == 0 else
                                f"top-k {args.top_k}, top-p {args.top_p}, min-p {args.min_p}"),
                   "self_confidence_topk": args.conf_topk,
                   "launch": "hip graph replay" if args.graph else "stream launches"},
        "roofline": {"kernel": f"{attn_kernel_name(shape)} (paged split-KV GQA attention)",
                     "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": None if tr is None else tr["traffic_bytes_per_launch"],
                     "traffic_over_algorithmic": None if tr is None else
                     tr["traffic_bytes_per_launch"] / tr["algorithmic_bytes_per_launch"],
                     "bytes_per_launch": attn_bytes_per_launch,
                     "avg_launch_ms": split_avg_ms,
                     "with_combine_GBs": attn_bytes_per_launch / (attn_avg_ms * 1e-3) / 1e9,
                     **peak_fracs(achieved, peak)},
        "read_peak": peak,
        "step_roofline": {"bound": "hbm", "bytes_per_step": step_bytes,
                          "achieved": step_bytes / (ms_per_step * 1e-3) / 1e9,
                          "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
                          "attention_ms_per_step": attn_ms},
    }
    out["kernels"] = kernel_table(shape, pop.n, kprof, attn_bytes_per_launch)
    if not args.no_cpu_baseline:
        log("timing the oracle on a bounded sample (host cores)")
        out["cpu_baseline"] = cpu_baseline(w, pop, args.cpu_sample)
    model.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
