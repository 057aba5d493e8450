#!/usr/bin/env python3
"""Benchmark of the SEED draft-verify decode loop on one MI355X.

Workload: the 4B-scale model (36 layers = 34 encoder + 2 decoder, hidden 2560, GQA 32/8 x 128,
SwiGLU 9728, vocab 151936, tied head), bf16 weights and KV cache, random-init N(0, 0.02),
1024-token uniform-random prompt, draft length k = 4, batch 1. A step is one draft-verify round
(k decoder-only draft steps, one verification of k+1 rows, acceptance and commit).

Prints ONE JSON line. ``value`` is decoded tokens/s over the timed rounds (inputs resident in
HBM, rounds replayed from a HIP graph). Also reported: verify- and draft-step latency and
algorithmic HBM GB/s, throughput at forced acceptance lengths 0..k and for plain greedy
decoding, per-kernel HIP-event timings, the roofline entry of the dominant kernel, and the CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2609_36590_amd import binding, synth  # noqa: E402

METRIC = "decoded tokens/sec at batch 1 (4B-scale, k=4); verify/draft step HBM GB/s"
PEAK_BF16 = 2.5e15   # dense bf16 MFMA, MI355X
PEAK_HBM = 8.0e12   # MI355X HBM3E, bytes/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------------------------------------
# algorithmic bytes
# ------------------------------------------------------------------------------------------
def kernel_bytes(cfg, op, M, L):
    """Algorithmic HBM bytes of one launch: weights + activations in/out (+ KV for attention).
    M rows; L = KV positions each row sees (mean); bf16 weights/KV, fp32 activations."""
    H, QD, KVD, F, V = cfg.hidden, cfg.q_dim, cfg.kv_dim, cfg.ffn, cfg.vocab
    es = 2 if cfg.dtype == "bf16" else 4
    if op == binding.OP_QKV:
        return (QD + 2 * KVD) * H * es + M * H * 4 + M * QD * 4 + M * 2 * KVD * es
    if op == binding.OP_O:
        return H * QD * es + M * QD * 4 + M * H * 8
    if op == binding.OP_GATEUP:
        return 2 * F * H * es + M * H * 4 + M * F * 4
    if op == binding.OP_DOWN:
        return H * F * es + M * F * 4 + M * H * 8
    if op == binding.OP_HEAD:
        return V * H * es + M * H * 4
    if op == binding.OP_ATTN:
        return L * 2 * KVD * es + M * QD * 4
    return 0


def attention_span(max_ctx, max_batch):
    """Positions per attention group for a context and batch capacity (the runtime's rule)."""
    small = 4096 if max_batch == 1 else 2048
    return 64 if max_ctx <= small else (128 if max_ctx <= 8192 else 256)


def combine_bytes(cfg, M, L, group):
    """Group partials read (o, m, l per query vector and group) + output written."""
    groups = (L + group - 1) // group
    return groups * M * cfg.n_heads * (cfg.head_dim + 2) * 4 + M * cfg.q_dim * 4


def step_bytes(cfg, M, L, layers):
    per_layer = sum(kernel_bytes(cfg, op, M, L) for op in
                    (binding.OP_QKV, binding.OP_ATTN, binding.OP_O, binding.OP_GATEUP, binding.OP_DOWN))
    return layers * per_layer + kernel_bytes(cfg, binding.OP_HEAD, M, L)


# ------------------------------------------------------------------------------------------
# HBM traffic from rocprofv3 counters (FETCH_SIZE / WRITE_SIZE), measured offline
# ------------------------------------------------------------------------------------------
KERNEL_SOURCES = ("linear.hip", "attention.hip", "misc.hip", "device_common.h", "kernels.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_4B-36L_k4_b1.md")


def kernel_source_hash():
    """sha256 over the HIP kernel sources: counters taken with other kernels do not apply."""
    import hashlib

    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_36590_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of ``kernel`` from the committed counter summary: FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch) each scaled by what the same counter reads for a plain copy of
    known size. None when the summary is missing, covers another kernel, or was taken with
    kernel sources that differ from the current ones."""
    try:
        with open(TRAFFIC_FILE) as fh:
            lines = [ln for ln in fh if ln.startswith("traffic-json:")]
        rec = json.loads(lines[-1].split(":", 1)[1])
    except (OSError, IndexError, ValueError):
        return None
    if rec.get("kernel") != kernel or rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return rec["fetch_kib"] * 1024 * rec["fetch_scale"] + rec["write_kib"] * 1024 * rec["write_scale"]


def copy_calibration(torch):
    """A plain device-to-device copy of 1 GiB (4 launches): the reference for the counters."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 4}), flush=True)


# ------------------------------------------------------------------------------------------
# every workload at measured and forced acceptance
# ------------------------------------------------------------------------------------------
SWEEP = (("tiny-4L-h256", (4,)), ("28L-h2048", (4,)), ("4B-36L-h2560", (2, 4, 6)),
         ("4B-36L-h2560-b8", (4,)), ("4B-36L-h2560-16k", (4,)))


def step_latency(dec, k, torch, n=8):
    """Median verify latency and per-draft-step latency (HIP events) at the current state."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ver, dr = [], []
    for _ in range(n):
        ev[0].record(dec.stream)
        if k:
            dec.draft(k)
        ev[1].record(dec.stream)
        dec.verify(k)
        ev[2].record(dec.stream)
        dec.stream.synchronize()
        if k:
            dr.append(ev[0].elapsed_time(ev[1]) / k)
        ver.append(ev[1].elapsed_time(ev[2]))
    return statistics.median(ver), (statistics.median(dr) if dr else 0.0)


def measure_config(cfg, k, weights, torch):
    lens = synth.make_prompt_lengths(cfg)
    prompts = synth.make_prompts(cfg, lengths=lens)
    B, gen = len(prompts), cfg.gen_len
    dec = binding.Decoder(cfg, max_batch=B, max_ctx=max(lens) + gen + 2 * 7 + 2, max_draft=max(k, 1))
    dec.load_weights(weights)
    res = {"workload": cfg.name, "batch": B, "k": k, "prompt_lens": lens if B > 1 else lens[0], "gen": gen}
    out0, _, st0 = dec.generate(prompts, 0, gen, use_graph=True)
    res["greedy_tokens_per_s"] = round(B * gen / (st0["decode_ms"] * 1e-3), 2)
    out, cnt, st = dec.generate(prompts, k, gen, use_graph=True)
    res["measured"] = {"tokens_per_s": round(int(cnt.sum()) / (st["decode_ms"] * 1e-3), 2),
                       "mean_accept": round(st["accepted"] / max(1, st["rounds"] * B), 4),
                       "output_equals_greedy": bool(np.array_equal(out, out0))}
    # step latencies inside the replayed rounds of the measured-acceptance run (kernel-stamped
    # device clock, medians over its rounds); the eager step-by-step figures beside them
    t_ver, t_dr = st["verify_ms"], st["draft_ms"]
    dec.prefill(prompts)
    e_ver, e_dr = step_latency(dec, k, torch)
    res["eager_verify_ms"], res["eager_draft_step_ms"] = round(e_ver, 4), round(e_dr, 4)
    Lm = int(np.mean(lens)) + gen // 2
    vb = step_bytes(cfg, B * (k + 1), Lm, cfg.n_layers) + (B - 1) * cfg.n_layers * kernel_bytes(
        cfg, binding.OP_ATTN, 0, Lm)
    db = step_bytes(cfg, B, Lm, cfg.n_dec_layers) + (B - 1) * cfg.n_dec_layers * kernel_bytes(
        cfg, binding.OP_ATTN, 0, Lm)
    res["verify_ms"], res["draft_step_ms"] = round(t_ver, 4), round(t_dr, 4)
    res["verify_gbps"] = round(vb / (t_ver * 1e-3) / 1e9, 1)
    res["verify_frac"] = round(vb / (t_ver * 1e-3) / PEAK_HBM, 4)
    if k:
        res["draft_gbps"] = round(db / (t_dr * 1e-3) / 1e9, 1)
        res["draft_frac"] = round(db / (t_dr * 1e-3) / PEAK_HBM, 4)
    forced = {}
    for a in range(k + 1):
        o, c, sa = dec.generate(prompts, k, gen, sim_accept=a, forced_trace=out0, use_graph=True)
        meas = int(c.sum()) / (sa["decode_ms"] * 1e-3)
        # cost model of the Computational Cost Analysis appendix with the measured step latencies:
        # B (a+1) tokens per round of k draft steps and one verification
        pred = B * (a + 1) / ((k * t_dr + t_ver) * 1e-3)
        forced[str(a)] = {"tokens_per_s": round(meas, 2), "model_tokens_per_s": round(pred, 2),
                          "output_equals_greedy": bool(np.array_equal(o, out0))}
    res["forced_acceptance"] = forced
    dec.close()
    return res


_ORACLE_MODEL = {}


def cpu_config_baseline(cfg, k, weights, rounds=6):
    """The oracle (fp32 NumPy) on one workload, on this host's cores: prefill and a bounded number
    of rounds of Algorithm 2 (the 64-token tiny workload whole). Batched workloads run their
    sequences one after another (the oracle has no batching), so the batch rate is one sequence's;
    the median-length sequence is timed. A 16k-token prompt is not prefilled (20+ minutes): its
    cache is filled with random keys/values of the same shape and the rounds are timed on it."""
    from oracle import model as om
    from oracle import seed as os_

    cores = len(os.sched_getaffinity(0))
    if _ORACLE_MODEL.get("weights") is not weights:   # widen each model's weights once
        _ORACLE_MODEL.clear()
        _ORACLE_MODEL.update(weights=weights, model=om.Model(cfg, synth.weights_as_f32(cfg, weights), np.float32))
    model = _ORACLE_MODEL["model"]
    lens = synth.make_prompt_lengths(cfg)
    prompts = synth.make_prompts(cfg, lengths=lens)
    b = int(np.argsort(lens)[len(lens) // 2])
    prompt = [int(x) for x in prompts[b]]
    if cfg.gen_len <= 64:
        rounds = cfg.gen_len
    cap = len(prompt) + (k + 1) * rounds + 2
    notes = []
    if len(prompt) > 4096:
        st = os_.State(model, prompt, cap)
        rng = np.random.default_rng(0)
        n = len(prompt) - 1
        for layer in range(cfg.n_layers):
            kv = rng.standard_normal((2, n, cfg.n_kv_heads, cfg.head_dim), dtype=np.float32)
            st.cache.K[layer, :n] = om.round_to_bf16(kv[0]) if model.kv_bf16 else kv[0]
            st.cache.V[layer, :n] = om.round_to_bf16(kv[1]) if model.kv_bf16 else kv[1]
        st.cache.valid[:] = n
        t_prefill = None
        notes.append(f"extrapolated: no {len(prompt)}-token prefill; a cache of random keys/values of that length")
    else:
        t0 = time.perf_counter()
        st = os_.prefill(model, prompt, cap)
        t_prefill = time.perf_counter() - t0
    if len(lens) > 1:
        notes.append(f"{len(lens)} sequences decoded one after another: the batch rate is one sequence's "
                     f"(timed: the median-length one, {len(prompt)} tokens)")
    before = st.t
    t_draft, t_verify = [], []
    t0 = time.perf_counter()
    for _ in range(rounds):
        a = time.perf_counter()
        d, _ = os_.draft(st, k)
        c1 = time.perf_counter()
        n_acc, bonus = os_.accept(d, os_.verify(st, d))
        os_.commit(st, d, n_acc, bonus)
        c2 = time.perf_counter()
        if k:
            t_draft.append((c1 - a) / k)
        t_verify.append(c2 - c1)
    dt = time.perf_counter() - t0
    return {"tokens_per_s": round((st.t - before) / dt, 3), "cores": cores, "rounds": rounds,
            "verify_ms": round(statistics.median(t_verify) * 1e3, 1),
            "draft_step_ms": round(statistics.median(t_draft) * 1e3, 1) if t_draft else 0.0,
            "prefill_s": round(t_prefill, 2) if t_prefill is not None else None, "notes": "; ".join(notes)}


def config_sweep(torch, out_md):
    results, cache = [], {}
    t0 = time.perf_counter()
    for name, ks in SWEEP:
        cfg = synth.CONFIGS[name]
        key = (cfg.n_layers, cfg.hidden, cfg.ffn, cfg.vocab, cfg.dtype)
        if key not in cache:
            cache.clear()
            log(f"[sweep] weights for {name}")
            cache[key] = synth.make_weights(cfg)
        for k in ks:
            log(f"[sweep] {name} k={k}")
            r = measure_config(cfg, k, cache[key], torch)
            torch.cuda.empty_cache()
            log(f"[sweep] {name} k={k}: oracle on the host")
            r["cpu_oracle"] = cpu_config_baseline(cfg, k, cache[key])
            log(f"[sweep] {json.dumps(r)}")
            results.append(r)
            torch.cuda.empty_cache()
    lines = ["# Decode throughput on every workload (one MI355X)", "",
             "Command: `python3 bench.py --config-sweep " + out_md + "` (repository root, library built by",
             "`__graft_entry__.build()`). Random-init weights (seed 0), uniform-random prompts (seed 1),",
             "ragged batch lengths (seed 2); rounds replayed from HIP graphs. `measured` = real drafts",
             "(acceptance ~0 with random weights); `forced a` = drafts overridden after the draft kernels",
             "ran so that exactly a are accepted each round; `model` = the cost model B(a+1)/(k t_draft +",
             "t_verify) with the step latencies measured in the same run; greedy = plain greedy decoding",
             "(k = 0). Bytes are algorithmic (weights + KV read at the mean context). Step latencies are",
             "medians over the rounds of the measured-acceptance run, stamped by the kernels inside the",
             "replayed rounds. CPU oracle = the fp32 NumPy oracle on this host's cores, the same workload",
             "(notes in the raw results: bounded rounds; batch sequences one after another; the 16k",
             "workload on a random cache of its length instead of its 20-minute prefill).", "",
             "| workload | B | k | greedy tok/s | measured tok/s (accept) | verify ms (TB/s, frac) | draft step ms "
             "(TB/s, frac) | forced a: tok/s (model) | spec == greedy | CPU oracle tok/s (cores) |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for r in results:
        fa = "; ".join(f"{a}: {v['tokens_per_s']:.0f} ({v['model_tokens_per_s']:.0f})"
                       for a, v in r["forced_acceptance"].items())
        ok = r["measured"]["output_equals_greedy"] and all(v["output_equals_greedy"]
                                                            for v in r["forced_acceptance"].values())
        dr = (f"{r['draft_step_ms']:.3f} ({r['draft_gbps'] / 1e3:.2f}, {r['draft_frac']:.2f})"
              if r["k"] else "-")
        lines.append(f"| {r['workload']} | {r['batch']} | {r['k']} | {r['greedy_tokens_per_s']:.0f} | "
                     f"{r['measured']['tokens_per_s']:.0f} ({r['measured']['mean_accept']:.2f}) | "
                     f"{r['verify_ms']:.3f} ({r['verify_gbps'] / 1e3:.2f}, {r['verify_frac']:.2f}) | {dr} | "
                     f"{fa} | {ok} | {r['cpu_oracle']['tokens_per_s']:.2f} ({r['cpu_oracle']['cores']}) |")
    lines += ["", "Raw results:", "", "```json"] + [json.dumps(r) for r in results] + ["```"]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    log(f"[sweep] done in {time.perf_counter() - t0:.1f}s")
    print(json.dumps({"config_sweep": out_md, "workloads": len(results)}), flush=True)


# ------------------------------------------------------------------------------------------
# decoder size sweep (Fig. 6 / Table 4): draft-step cost vs the number of decoder layers
# ------------------------------------------------------------------------------------------
SPLITS = (1, 2, 4, 6, 8, 10, 12, 14)


def split_sweep(torch, out_md):
    base = synth.CONFIGS["28L-h2048"]
    k, gen = base.k, base.gen_len
    log(f"[split] weights for {base.name} (the same tensors serve every split)")
    weights = synth.make_weights(base)
    prompt = synth.make_prompts(base)[0]
    Lm = len(prompt) + gen // 2
    rows = []
    t0 = time.perf_counter()
    for n in SPLITS:
        cfg = base.replace(name=f"{base.name}-dec{n}", n_dec_layers=n)
        log(f"[split] n_dec={n}")
        dec = binding.Decoder(cfg, max_batch=1, max_ctx=len(prompt) + gen + 2 * 7 + 2, max_draft=k)
        dec.load_weights(weights)
        out0, _, st0 = dec.generate([prompt], 0, gen, use_graph=True)
        out, cnt, st = dec.generate([prompt], k, gen, use_graph=True)
        dec.prefill([prompt])
        t_ver, t_dr = step_latency(dec, k, torch)
        db = step_bytes(cfg, 1, Lm, n)
        vb = step_bytes(cfg, k + 1, Lm, cfg.n_layers)
        r = {"n_dec": n, "draft_step_ms": round(t_dr, 4), "verify_ms": round(t_ver, 4),
             "draft_gbps": round(db / (t_dr * 1e-3) / 1e9, 1), "draft_frac": round(db / (t_dr * 1e-3) / PEAK_HBM, 4),
             "draft_over_verify": round(t_dr / t_ver, 4),
             # the byte model of the cost appendix: a draft step reads n decoder layers + the head,
             # a verification the whole model
             "byte_model_ratio": round(db / vb, 4),
             "greedy_tokens_per_s": round(gen / (st0["decode_ms"] * 1e-3), 2),
             "measured": {"tokens_per_s": round(int(cnt.sum()) / (st["decode_ms"] * 1e-3), 2),
                          "mean_accept": round(st["accepted"] / max(1, st["rounds"]), 4),
                          "output_equals_greedy": bool(np.array_equal(out, out0))}}
        forced = {}
        for a in (0, k):
            o, c, sa = dec.generate([prompt], k, gen, sim_accept=a, forced_trace=out0, use_graph=True)
            forced[str(a)] = {"tokens_per_s": round(int(c.sum()) / (sa["decode_ms"] * 1e-3), 2),
                              "model_tokens_per_s": round((a + 1) / ((k * t_dr + t_ver) * 1e-3), 2),
                              "output_equals_greedy": bool(np.array_equal(o, out0))}
        r["forced_acceptance"] = forced
        log(f"[split] {json.dumps(r)}")
        rows.append(r)
        dec.close()
        torch.cuda.empty_cache()
    lines = ["# Draft-step cost vs decoder size (one MI355X)", "",
             f"Command: `python3 bench.py --split-sweep {out_md}` (repository root, library built by",
             "`__graft_entry__.build()`). Model: " + base.name + f" (28 layers, hidden 2048), k={k}, "
             f"{len(prompt)}-token prompt, {gen} generated tokens; the split n_dec = l - l' only changes",
             "which layers the drafter runs (same random-init weights, seed 0). Step latencies are HIP-event",
             "medians; bytes are algorithmic (weights + KV at the mean context). `byte model` = draft-step",
             "bytes / verification bytes (the cost appendix's c_draft in bytes), against the measured",
             "latency ratio. `forced a` = drafts overridden after the draft kernels ran so that exactly a",
             "are accepted per round (model = (a+1)/(k t_draft + t_verify)).", "",
             "| n_dec | draft step ms (TB/s, frac) | t_draft / t_verify | byte model | verify ms | "
             "forced a=0 tok/s (model) | forced a=k tok/s (model) | spec == greedy |",
             "|---|---|---|---|---|---|---|---|"]
    for r in rows:
        f0, fk = r["forced_acceptance"]["0"], r["forced_acceptance"][str(k)]
        ok = r["measured"]["output_equals_greedy"] and f0["output_equals_greedy"] and fk["output_equals_greedy"]
        lines.append(f"| {r['n_dec']} | {r['draft_step_ms']:.3f} ({r['draft_gbps'] / 1e3:.2f}, "
                     f"{r['draft_frac']:.2f}) | {r['draft_over_verify']:.3f} | {r['byte_model_ratio']:.3f} | "
                     f"{r['verify_ms']:.3f} | {f0['tokens_per_s']:.0f} ({f0['model_tokens_per_s']:.0f}) | "
                     f"{fk['tokens_per_s']:.0f} ({fk['model_tokens_per_s']:.0f}) | {ok} |")
    lines += ["", "Raw results:", "", "```json"] + [json.dumps(r) for r in rows] + ["```"]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    log(f"[split] done in {time.perf_counter() - t0:.1f}s")
    print(json.dumps({"split_sweep": out_md, "splits": len(rows)}), flush=True)


# ------------------------------------------------------------------------------------------
# forward pass of the speculative drafting objective (Algorithm 1) on the 4B model
# ------------------------------------------------------------------------------------------
SPEC_ROWS = 1024   # rows per pass of the GPU path (its prefill chunk, tiled MFMA GEMMs)


def spec_sweep(torch, out_md, reps=5):
    cfg = synth.C3_4B
    n = cfg.prompt_len
    log(f"[spec] weights for {cfg.name}")
    weights = synth.make_weights(cfg)
    x = synth.make_prompts(cfg)[0]
    dec = binding.Decoder(cfg, max_batch=1, max_ctx=n + 8, max_draft=4)
    dec.load_weights(weights)
    es = 2
    dec_layer = sum(kernel_bytes(cfg, op, 0, 0) for op in (binding.OP_QKV, binding.OP_O, binding.OP_GATEUP,
                                                           binding.OP_DOWN))
    head = cfg.vocab * cfg.hidden * es
    passes = (n - 1 + SPEC_ROWS - 1) // SPEC_ROWS
    # weights are streamed once per pass of SPEC_ROWS rows; keys/values: each row reads the deep cache
    # below its block start and the pass's own cache of its block (decoder layers)
    kv_row = 2 * cfg.kv_dim * es
    rows = []
    for b in (4, 16):
        # prefill alone, then prefill + the drafter pass: the difference is the pass itself
        tp, ts = [], []
        for _ in range(reps):
            t0 = time.perf_counter()
            dec.prefill([x])
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            _, _, loss = dec.spec_forward(x, b, logits=False)
            t2 = time.perf_counter()
            tp.append(t1 - t0)
            ts.append(t2 - t1)
        t_pf, t_all = statistics.median(tp), statistics.median(ts)
        t_spec = t_all - t_pf
        # the method's own work: every row through the decoder layers and the head once (weights
        # read once: 1.18 GB), attention over the q+1 positions a row sees (its block's own rows
        # and the deep cache below the block); at 1023 rows that is ~1000 FLOP per weight byte,
        # far past the bf16 ridge (2.5 PFLOP/s / 8 TB/s = 312), so the bound is the matrix cores
        kv_bytes = sum((q // b * b + (q - q // b * b + 1)) for q in range(n - 1)) * kv_row * cfg.n_dec_layers
        wbytes_once = cfg.n_dec_layers * dec_layer + head
        streamed = passes * wbytes_once + kv_bytes   # what the passes read at least once
        attn = sum(4 * (q + 1) * cfg.n_heads * cfg.head_dim for q in range(n - 1)) * cfg.n_dec_layers
        flops = 2 * (n - 1) * (cfg.n_dec_layers * dec_layer / es + head / es) + attn
        pf_flops = 2 * n * cfg.n_layers * dec_layer / es + sum(
            4 * (q + 1) * cfg.n_heads * cfg.head_dim for q in range(n)) * cfg.n_layers
        r = {"block": b, "n": n, "rows": n - 1, "passes": passes, "prefill_ms": round(t_pf * 1e3, 3),
             "spec_ms": round(t_spec * 1e3, 3), "rows_per_s": round((n - 1) / t_spec, 1),
             "flops": int(flops), "tflops": round(flops / t_spec / 1e12, 2),
             "frac_mfma_bf16": round(flops / t_spec / PEAK_BF16, 4),
             "alg_bytes": int(wbytes_once + kv_bytes), "streamed_bytes": int(streamed),
             "streamed_gbps": round(streamed / t_spec / 1e9, 1),
             "prefill_flops": int(pf_flops), "prefill_tflops": round(pf_flops / t_pf / 1e12, 2),
             "prefill_frac_mfma_bf16": round(pf_flops / t_pf / PEAK_BF16, 4), "L_spec": round(loss, 4)}
        log(f"[spec] {json.dumps(r)}")
        rows.append(r)
    dec.close()
    lines = ["# Forward pass of the speculative drafting objective (one MI355X)", "",
             f"Command: `python3 bench.py --spec-forward {out_md}` (repository root, library built by",
             "`__graft_entry__.build()`). Model " + cfg.name + f", one {n}-token sequence of uniform-random",
             "tokens (seed 1), random-init weights (seed 0). `seed_spec_forward` runs the full model over",
             "the sequence (prefill) and then the decoder layers over the raw embeddings of every block",
             "at once with the block-causal mask; the pass time is the median of prefill + pass minus the",
             f"median of the prefill alone ({reps} repetitions, host clock around synchronous calls). The",
             "method's work is FLOPs = 2 x rows x (decoder-layer + head parameters) + attention (4 x",
             "visible positions x heads x head_dim per row and layer); at 1023 rows it is ~1000 FLOP per",
             "weight byte, past the bf16 ridge (2.5 PFLOP/s / 8 TB/s = 312 FLOP/B), so its roofline is",
             "the dense bf16 MFMA peak (2.5 PFLOP/s). The prefill (36 layers over 1024 rows, same rule)",
             f"likewise. The GPU path takes {SPEC_ROWS} rows per pass (tiled MFMA GEMMs; each n-group's",
             "weights come from HBM once per pass and are shared by its row tiles through the XCD's L2),",
             "so the decoder layers and the head are streamed once per pass (`streamed` bytes below: the",
             "weights once, 1.18 GB per pass, plus the keys/values each row reads).", "",
             "| block | rows | pass ms | rows/s | TFLOP/s (frac of 2.5 PFLOP/s bf16) | streamed GB (GB/s) | "
             "prefill ms | prefill TFLOP/s (frac) | L_spec |",
             "|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['block']} | {r['rows']} | {r['spec_ms']:.3f} | {r['rows_per_s']:.0f} | "
                     f"{r['tflops']:.1f} ({r['frac_mfma_bf16']:.3f}) | {r['streamed_bytes'] / 1e9:.1f} "
                     f"({r['streamed_gbps']:.0f}) | {r['prefill_ms']:.2f} | {r['prefill_tflops']:.1f} "
                     f"({r['prefill_frac_mfma_bf16']:.3f}) | {r['L_spec']:.2f} |")
    lines += ["", "Raw results:", "", "```json"] + [json.dumps(r) for r in rows] + ["```"]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps({"spec_forward": out_md, "blocks": [r["block"] for r in rows]}), flush=True)


# ------------------------------------------------------------------------------------------
# dynamic drafting + tree verification
# ------------------------------------------------------------------------------------------
# emulated tree shapes (label, top-p table, fan-out below it, depth, forced accepted lengths): tau
# = 0 keeps drafting to the depth, the table fixes the fan-out of every step
TREE_SHAPES = [("chain, depth 4", ((-1.0, 1),), 1, 4, (0, 2, 4)),
               ("fan-out 3, depth 4", ((-1.0, 3),), 3, 4, (0, 2, 4)),
               ("chain, depth 8", ((-1.0, 1),), 1, 8, (4, 8)),
               ("fan-out 3, depth 6", ((-1.0, 3),), 3, 6, (4, 6))]
TREE_OPS = (binding.OP_SETUP, binding.OP_QKV, binding.OP_ATTN, binding.OP_COMBINE, binding.OP_O, binding.OP_GATEUP,
            binding.OP_DOWN, binding.OP_HEAD, binding.OP_HEAD_ARGMAX, binding.OP_ACCEPT, binding.OP_TOPK)
OP_NAMES = {binding.OP_SETUP: "setup", binding.OP_QKV: "qkv", binding.OP_ATTN: "attn", binding.OP_COMBINE: "combine",
            binding.OP_O: "o", binding.OP_GATEUP: "gateup", binding.OP_DOWN: "down", binding.OP_HEAD: "head",
            binding.OP_ACCEPT: "accept", binding.OP_HEAD_ARGMAX: "argmax", binding.OP_TOPK: "topk"}


def tree_bench(torch, out_md):
    cfg = synth.C3_4B
    gen = cfg.gen_len
    log(f"[tree] weights for {cfg.name}")
    weights = synth.make_weights(cfg)
    prompt = synth.make_prompts(cfg)[0]
    P = len(prompt)
    max_depth = max(s[3] for s in TREE_SHAPES)
    dec = binding.Decoder(cfg, max_batch=1, max_ctx=P + gen + 2 * 65 + 8, max_draft=max_depth)
    dec.load_weights(weights)
    out0, _, st0 = dec.generate([prompt], 0, gen, use_graph=True)
    trace = out0[0]
    res = {"workload": cfg.name, "prompt_len": P, "gen": gen, "ar_tokens_per_s": round(gen / (st0["decode_ms"] * 1e-3), 2)}
    # the paper's options, acceptance as random weights give it
    rows = []
    for depth in (4, 8):
        opts = binding.tree_opts(depth)
        toks, st = dec.generate_tree(prompt, opts, gen, use_graph=True)   # warm-up (graph capture)
        toks, st = dec.generate_tree(prompt, opts, gen, use_graph=True)
        r = {"shape": f"paper table, tau 0.7, depth <= {depth}", "forced": None,
             "tokens_per_s": round(gen / (st["decode_ms"] * 1e-3), 2), "rounds": st["rounds"],
             "nodes_per_round": round(1 + st["drafted"] / st["rounds"], 2),
             "accepted_per_round": round(st["accepted"] / st["rounds"], 3),
             "output_equals_greedy": bool(np.array_equal(toks, trace))}
        log(f"[tree] {json.dumps(r)}")
        rows.append(r)
    for label, table, rest, depth, accepts in TREE_SHAPES:
        opts = binding.tree_opts(depth, tau=0.0, table=table, rest=rest)
        for a in accepts:
            kw = dict(use_graph=True, sim_accept=a, forced_trace=trace, log_cap=gen + 8)
            dec.generate_tree(prompt, opts, gen, **kw)
            toks, st = dec.generate_tree(prompt, opts, gen, **kw)
            r = {"shape": label, "forced": a, "tokens_per_s": round(gen / (st["decode_ms"] * 1e-3), 2),
                 "rounds": st["rounds"], "nodes_per_round": round(1 + st["drafted"] / st["rounds"], 2),
                 "accepted_per_round": round(st["accepted"] / st["rounds"], 3),
                 "output_equals_greedy": bool(np.array_equal(toks, trace))}
            log(f"[tree] {json.dumps(r)}")
            rows.append(r)
    res["runs"] = rows
    # per-kernel time of one emulated shape (eager launches with HIP events around each operation)
    label, table, rest, depth, _ = TREE_SHAPES[1]
    a = 4
    opts = binding.tree_opts(depth, tau=0.0, table=table, rest=rest)
    n_nodes = 1 + depth * rest
    kw = dict(use_graph=False, sim_accept=a, forced_trace=trace, log_cap=gen + 8)
    _, st = dec.generate_tree(prompt, opts, gen, **kw)
    rounds = st["rounds"]
    L = P + gen // 2
    per_kernel = {}
    for phase, M, layers in ((binding.PHASE_VERIFY, n_nodes, cfg.n_layers), (binding.PHASE_DRAFT, 1, cfg.n_dec_layers)):
        for op in TREE_OPS:
            binding.seed_kernel_timing(dec.ctx, binding.kernel_id(phase, op), True)
            dec.generate_tree(prompt, opts, gen, **kw)
            n, ms = binding.seed_kernel_timing_read(dec.ctx)
            binding.seed_kernel_timing(dec.ctx, 0, False)
            if n == 0:
                continue
            name = ("verify_" if phase == binding.PHASE_VERIFY else "draft_") + OP_NAMES[op]
            b = kernel_bytes(cfg, op, M, L)
            per_kernel[name] = {"launches_per_round": round(n / rounds, 2), "avg_us": round(ms / n * 1e3, 3),
                                "us_per_round": round(ms * 1e3 / rounds, 2),
                                "gbps": round(b / (ms / n * 1e-3) / 1e9, 1) if b else None}
    dom = max(per_kernel, key=lambda kk: per_kernel[kk]["us_per_round"])
    res["per_kernel_shape"] = f"{label}, forced {a}, {n_nodes} nodes"
    res["per_kernel"] = per_kernel
    res["dominant"] = dom
    dec.close()
    lines = ["# Dynamic drafting + tree verification (one MI355X)", "",
             f"Command: `python3 bench.py --tree {out_md}` (repository root, library built by",
             "`__graft_entry__.build()`). Model " + cfg.name + f", bf16, one {P}-token prompt, {gen} generated",
             "tokens, random-init weights (seed 0). `seed_generate_tree` runs confidence-aware dynamic drafting",
             "(per step: decoder layers, LM head, top-k/p0 kernels) and tree verification (one full-model pass",
             "over the packed tree, acceptance, leaf cache move), each drafting step and each tree size's",
             "verification replayed from a HIP graph; decode time from HIP events. Random weights put p0 near",
             "1/vocab, so the paper's options stop after one step with 10 candidates and accept nothing; the",
             "emulated shapes set tau = 0 and a one-level table (fixed fan-out per step) and force the",
             "accepted chain length with the greedy trace (chain nodes 1..a take it, node a+1 does not).",
             f"Plain greedy decoding (AR): {res['ar_tokens_per_s']:.1f} tok/s.", "",
             "| shape | forced accept | nodes/round | accepted/round | tok/s | x AR | output = greedy |",
             "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['shape']} | {r['forced'] if r['forced'] is not None else 'measured'} | {r['nodes_per_round']} | "
                     f"{r['accepted_per_round']} | {r['tokens_per_s']:.1f} | {r['tokens_per_s'] / res['ar_tokens_per_s']:.2f} | "
                     f"{r['output_equals_greedy']} |")
    lines += ["", f"Per-operation time, {res['per_kernel_shape']} (eager launches, HIP events around each",
              f"operation, mean over the run; GB/s = algorithmic bytes at {L} cached positions / time):", "",
              "| operation | launches/round | avg us | us/round | GB/s |", "|---|---|---|---|---|"]
    for kk, v in sorted(per_kernel.items(), key=lambda x: -x[1]["us_per_round"]):
        lines.append(f"| {kk} | {v['launches_per_round']} | {v['avg_us']:.2f} | {v['us_per_round']:.1f} | "
                     f"{v['gbps'] if v['gbps'] is not None else '-'} |")
    lines += ["", "Raw results:", "", "```json", json.dumps(res), "```"]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps({"tree": out_md, "runs": len(rows), "dominant": dom}), flush=True)


def copy_ceiling(torch, n=1 << 30, reps=5):
    """Bytes read + written per second by a plain device-to-device copy of n bytes (median)."""
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b.copy_(a)
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e-3)
    del a, b
    return 2 * n / statistics.median(ts)


# ------------------------------------------------------------------------------------------
# CPU oracle baseline
# ------------------------------------------------------------------------------------------
def cpu_baseline(cfg, weights, prompt, k, rounds):
    from oracle import model as om
    from oracle import seed as os_

    cores = len(os.sched_getaffinity(0))
    log(f"[cpu] widening weights to fp32 ({cores} host cores)")
    model = om.Model(cfg, synth.weights_as_f32(cfg, weights), np.float32)
    log("[cpu] oracle prefill")
    t0 = time.perf_counter()
    st = os_.prefill(model, prompt, len(prompt) + (k + 1) * rounds + 2)
    t_prefill = time.perf_counter() - t0
    log(f"[cpu] timing {rounds} oracle rounds")
    before = st.t
    t_draft, t_verify = [], []
    t0 = time.perf_counter()
    for _ in range(rounds):
        a = time.perf_counter()
        d, _ = os_.draft(st, k)
        b = time.perf_counter()
        n, bonus = os_.accept(d, os_.verify(st, d))
        os_.commit(st, d, n, bonus)
        c = time.perf_counter()
        t_draft.append((b - a) / max(k, 1))
        t_verify.append(c - b)
    dt = time.perf_counter() - t0
    return {"value": (st.t - before) / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "verify_ms": round(statistics.median(t_verify) * 1e3, 1),
            "draft_step_ms": round(statistics.median(t_draft) * 1e3, 1),
            "prefill_s": round(t_prefill, 2),
            "sample": f"{rounds} rounds of Algorithm 2 (k={k}) on the same model and 1024-token prompt "
                      f"after the oracle prefill (timed apart); {dt:.1f} s, {st.t - before} tokens, "
                      f"{dt / rounds * 1e3:.0f} ms per round; fp32 NumPy with BLAS on {cores} host threads"}


# ------------------------------------------------------------------------------------------
REPS = 5   # timed repetitions of the K rounds; value is their median



def profile_workload(torch, cfg, k, args):
    """--profile-run (prefill, eager rounds, optional eager draft calls: the runs the rocprofv3
    counter passes are taken over) and --kernel-breakdown (per-kernel HIP-event times of the
    verification and draft step against algorithmic bytes) for any workload, batched ones
    included: every sequence of the workload is decoded."""
    lens = synth.make_prompt_lengths(cfg)
    prompts = synth.make_prompts(cfg, lengths=lens)
    B = len(prompts)
    rounds = args.warmup + args.steps + 8
    gen_probe = min(cfg.gen_len, 64)
    max_ctx = max(lens) + max(rounds, gen_probe) * (k + 1) + 2 * k + 2
    weights = synth.make_weights(cfg)
    dec = binding.Decoder(cfg, max_batch=B, max_ctx=max_ctx, max_draft=max(k, 1))
    dec.load_weights(weights)
    ctx, stream = dec.ctx, dec.stream
    if args.profile_run:
        dec.prefill(prompts)
        binding.seed_rounds(ctx, k, args.warmup, False)
        stream.synchronize()
        t0 = time.perf_counter()
        binding.seed_rounds(ctx, k, args.steps, False)
        for _ in range(args.profile_drafts):
            dec.draft(k)
        stream.synchronize()
        log(f"[bench] profile run ({cfg.name}, batch {B}): {args.steps} eager rounds and {args.profile_drafts} "
            f"draft calls in {(time.perf_counter() - t0) * 1e3:.1f} ms")
        print(json.dumps({"profile_run": cfg.name, "batch": B, "k": k, "rounds": args.steps,
                          "draft_calls": args.profile_drafts, "t_end": [int(len(dec.tokens(b))) for b in range(B)]}),
              flush=True)
        dec.close()
        return
    # --kernel-breakdown: HIP events around every launch of one operation over a few eager rounds
    probe_rounds = 4
    M_ver, M_dr = B * (k + 1), B
    table = []
    for phase, M in ((binding.PHASE_VERIFY, M_ver), (binding.PHASE_DRAFT, M_dr)):
        for op in (binding.OP_SETUP, binding.OP_QKV, binding.OP_ATTN, binding.OP_COMBINE, binding.OP_O,
                   binding.OP_GATEUP, binding.OP_DOWN, binding.OP_HEAD, binding.OP_HEAD_ARGMAX, binding.OP_ACCEPT):
            dec.prefill(prompts)
            binding.seed_rounds(ctx, k, 2, False)
            binding.seed_kernel_timing(ctx, binding.kernel_id(phase, op), True)
            binding.seed_rounds(ctx, k, probe_rounds, False)
            n, ms = binding.seed_kernel_timing_read(ctx)
            binding.seed_kernel_timing(ctx, 0, False)
            if n == 0:
                continue
            Ls = [len(dec.tokens(b)) - probe_rounds // 2 for b in range(B)]
            if op == binding.OP_ATTN:   # every sequence's keys/values at its own context
                b_op = sum(kernel_bytes(cfg, op, 0, L) for L in Ls) + M * cfg.q_dim * 4
            elif op == binding.OP_COMBINE:
                b_op = sum(combine_bytes(cfg, M // B, L, attention_span(max_ctx, B)) for L in Ls)
            else:
                b_op = kernel_bytes(cfg, op, M, int(np.mean(Ls)))
            name = ("verify_" if phase == binding.PHASE_VERIFY else "draft_") + OP_NAMES[op]
            avg_us = ms / n * 1e3
            table.append({"kernel": name, "rows": M, "launches_per_round": n / probe_rounds, "avg_us": avg_us,
                          "us_per_round": avg_us * n / probe_rounds, "alg_bytes": b_op,
                          "gbps": b_op / (avg_us * 1e-6) / 1e9 if b_op else None})
    # step latencies inside graph-replayed rounds (kernel-stamped clock), for the sum check
    _, _, st = dec.generate(prompts, k, gen_probe, use_graph=True)
    dec.close()
    Lm = int(np.mean(lens)) + gen_probe // 2
    vb = step_bytes(cfg, M_ver, Lm, cfg.n_layers) + (B - 1) * cfg.n_layers * kernel_bytes(cfg, binding.OP_ATTN, 0, Lm)
    db = step_bytes(cfg, M_dr, Lm, cfg.n_dec_layers) + (B - 1) * cfg.n_dec_layers * kernel_bytes(cfg, binding.OP_ATTN, 0, Lm)
    out = args.kernel_breakdown
    lines = [f"# Per-kernel breakdown: {cfg.name}, batch {B}, k = {k}", "",
             f"Prompt lengths {lens}; verification passes of {M_ver} rows (every sequence's pending token and "
             f"{k} drafts), draft steps of {M_dr} rows. Eager rounds, HIP events around every launch of one "
             "operation at a time (the events add about 1-3 us per launch against the graph-replayed rounds); "
             "algorithmic bytes per launch as in bench.py (weights once, activations in and out, every "
             "sequence's keys/values at its own context). `frac` is against the 8 TB/s HBM peak.", "",
             "| kernel | rows | launches / round | mean us | us / round | alg. MB / launch | GB/s | frac |",
             "|---|---|---|---|---|---|---|---|"]
    for r in sorted(table, key=lambda x: (not x["kernel"].startswith("verify"), -x["us_per_round"])):
        g = f"{r['gbps']:.0f}" if r["gbps"] else "-"
        fr = f"{r['gbps'] * 1e9 / PEAK_HBM:.3f}" if r["gbps"] else "-"
        lines.append(f"| {r['kernel']} | {r['rows']} | {r['launches_per_round']:.2f} | {r['avg_us']:.2f} | "
                     f"{r['us_per_round']:.1f} | {r['alg_bytes'] / 1e6:.2f} | {g} | {fr} |")
    ver_sum = sum(r["us_per_round"] for r in table if r["kernel"].startswith("verify"))
    dr_sum = sum(r["us_per_round"] for r in table if r["kernel"].startswith("draft")) / max(k, 1)
    lines += ["", f"Sum of the event-timed kernels: verification {ver_sum / 1e3:.3f} ms, draft step "
                  f"{dr_sum / 1e3:.4f} ms. Graph-replayed rounds (kernel-stamped device clock, medians over "
                  f"{st['rounds']} rounds of a {gen_probe}-token generate): verification "
                  f"{st['verify_ms']:.3f} ms ({vb / (st['verify_ms'] * 1e-3) / 1e9:.0f} GB/s, "
                  f"{vb / (st['verify_ms'] * 1e-3) / PEAK_HBM:.3f} of 8 TB/s for {vb / 1e9:.3f} GB), draft step "
                  f"{st['draft_ms']:.4f} ms ({db / (st['draft_ms'] * 1e-3) / 1e9:.0f} GB/s, "
                  f"{db / (st['draft_ms'] * 1e-3) / PEAK_HBM:.3f} for {db / 1e9:.3f} GB).", "",
              "Command (one MI355X, library built by `__graft_entry__.build()`):", "", "```",
              f"python3 bench.py --config {cfg.name} --k {k} --kernel-breakdown {out}", "```", ""]
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps({"kernel_breakdown": cfg.name, "verify_ms": st["verify_ms"], "draft_ms": st["draft_ms"],
                      "verify_event_sum_ms": ver_sum / 1e3, "draft_event_sum_ms": dr_sum / 1e3}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200, help="timed draft-verify rounds")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--k", type=int, default=4)
    ap.add_argument("--config", default=synth.C3_4B.name, choices=sorted(synth.CONFIGS))
    ap.add_argument("--cpu-rounds", type=int, default=40, help="oracle rounds timed on the host (about 13 s)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--profile-run", action="store_true",
                    help="only prefill + eager rounds (for rocprofv3 counter passes)")
    ap.add_argument("--kernel-breakdown", metavar="OUT_MD",
                    help="per-kernel HIP-event times, algorithmic bytes and rates of the verification and "
                         "draft step of --config (every sequence of a batched workload), written to OUT_MD")
    ap.add_argument("--profile-drafts", type=int, default=0,
                    help="with --profile-run: this many eager seed_draft calls (k steps each) after the rounds")
    ap.add_argument("--copy-calib", action="store_true",
                    help="only a plain 1 GiB device-to-device copy (counter calibration)")
    ap.add_argument("--config-sweep", metavar="OUT_MD",
                    help="measure every workload (tiny, 28L, 4B k=2/4/6, 4B batch 8, 4B 16k) at the "
                         "measured and forced acceptance lengths and write a summary to OUT_MD")
    ap.add_argument("--split-sweep", metavar="OUT_MD",
                    help="draft-step cost of the 28-layer model for n_dec in 1..14 decoder layers "
                         "(measured and forced acceptance); write a summary to OUT_MD")
    ap.add_argument("--tree", metavar="OUT_MD",
                    help="dynamic drafting + tree verification on the 4B-scale model: measured and "
                         "forced-acceptance tree shapes, per-operation time; writes OUT_MD")
    ap.add_argument("--spec-forward", metavar="OUT_MD",
                    help="time the forward pass of the speculative drafting objective (4B model, "
                         "1024 tokens, block sizes 4 and 16) and write a summary to OUT_MD")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch

    if args.copy_calib:
        copy_calibration(torch)
        return
    if args.config_sweep:
        config_sweep(torch, args.config_sweep)
        return
    if args.split_sweep:
        split_sweep(torch, args.split_sweep)
        return
    if args.tree:
        tree_bench(torch, args.tree)
        return
    if args.spec_forward:
        spec_sweep(torch, args.spec_forward)
        return

    cfg = synth.CONFIGS[args.config]
    k = args.k
    if args.profile_run or args.kernel_breakdown:
        profile_workload(torch, cfg, k, args)
        return
    t_start = time.perf_counter()
    log(f"[bench] generating weights for {cfg.name}")
    weights = synth.make_weights(cfg)
    prompt = synth.make_prompts(cfg)[0]
    P = len(prompt)
    gen = cfg.gen_len
    max_ctx = P + max(gen + 2 * 6 + 2, (args.warmup + args.steps) * (k + 1) + k + 2)
    log(f"[bench] weights ready in {time.perf_counter() - t_start:.1f}s; creating decoder (max_ctx={max_ctx})")
    dec = binding.Decoder(cfg, max_batch=1, max_ctx=max_ctx, max_draft=6)
    dec.load_weights(weights)
    log(f"[bench] weights on device: {dec.bytes['weights'] / 1e9:.2f} GB")
    ctx = dec.ctx
    stream = dec.stream

    def sync():
        stream.synchronize()

    # ---------------- timed rounds (graph replay): 5 repetitions, median ----------------
    # each repetition starts from the prompt (so the context stays at the workload's length), runs
    # W untimed rounds, then times exactly K rounds between two synchronisations; the first
    # repetition is a warm-up and is discarded
    samples = []
    for rep in range(REPS + 1):
        dec.prefill([prompt])
        binding.seed_rounds(ctx, k, args.warmup, True)
        sync()
        tb = len(dec.tokens(0))
        sync()
        t0 = time.perf_counter()
        binding.seed_rounds(ctx, k, args.steps, True)
        sync()
        t1 = time.perf_counter()
        ta = len(dec.tokens(0))
        if rep > 0:
            samples.append({"tokens": ta - tb, "s": t1 - t0, "kv_positions": [tb, ta]})
        log(f"[bench] graph repetition {rep}{' (warm-up)' if rep == 0 else ''}: {args.steps} rounds, {ta - tb} tokens "
            f"in {(t1 - t0) * 1e3:.1f} ms -> {(ta - tb) / (t1 - t0):.1f} tok/s")
    rates = [x["tokens"] / x["s"] for x in samples]
    med = sorted(range(len(samples)), key=lambda i: rates[i])[len(samples) // 2]
    value = rates[med]
    elapsed, tokens = samples[med]["s"], samples[med]["tokens"]
    t_before, t_after = samples[med]["kv_positions"]

    # ---------------- same rounds, eager, with per-kernel HIP events ----------------
    dec.prefill([prompt])
    binding.seed_rounds(ctx, k, args.warmup, False)
    sync()
    kinds = []
    for phase, M, layers in ((binding.PHASE_VERIFY, k + 1, cfg.n_layers), (binding.PHASE_DRAFT, 1, cfg.n_dec_layers)):
        for op in (binding.OP_QKV, binding.OP_ATTN, binding.OP_COMBINE, binding.OP_O, binding.OP_GATEUP,
                   binding.OP_DOWN, binding.OP_HEAD, binding.OP_HEAD_ARGMAX, binding.OP_SETUP, binding.OP_ACCEPT):
            if phase == binding.PHASE_DRAFT and op == binding.OP_ACCEPT:
                continue
            kinds.append((phase, op, M, layers))
    names = {binding.OP_SETUP: "setup", binding.OP_QKV: "qkv", binding.OP_ATTN: "attn", binding.OP_COMBINE: "combine",
             binding.OP_O: "o", binding.OP_GATEUP: "gateup", binding.OP_DOWN: "down", binding.OP_HEAD: "head",
             binding.OP_ACCEPT: "accept", binding.OP_HEAD_ARGMAX: "argmax"}
    per_kernel = {}
    probe_rounds = 4
    for phase, op, M, layers in kinds:
        dec.prefill([prompt])
        binding.seed_rounds(ctx, k, 2, False)
        binding.seed_kernel_timing(ctx, binding.kernel_id(phase, op), True)
        binding.seed_rounds(ctx, k, probe_rounds, False)
        n, ms = binding.seed_kernel_timing_read(ctx)
        binding.seed_kernel_timing(ctx, 0, False)
        if n == 0:
            continue
        L_here = len(dec.tokens(0)) - probe_rounds // 2
        name = ("verify_" if phase == binding.PHASE_VERIFY else "draft_") + names[op]
        avg = ms / n
        b = (combine_bytes(cfg, M, L_here, attention_span(max_ctx, 1)) if op == binding.OP_COMBINE
             else kernel_bytes(cfg, op, M, L_here))
        per_kernel[name] = {"launches_per_round": n / probe_rounds, "avg_us": avg * 1e3,
                            "us_per_round": avg * 1e3 * n / probe_rounds,
                            "alg_bytes": b, "gbps": (b / (avg * 1e-3) / 1e9) if b else None}
    dominant = max(per_kernel, key=lambda kk: per_kernel[kk]["us_per_round"])
    dom_phase = binding.PHASE_VERIFY if dominant.startswith("verify_") else binding.PHASE_DRAFT
    dom_op = {v: kk for kk, v in names.items()}[dominant.split("_", 1)[1]]
    dom_M = k + 1 if dom_phase == binding.PHASE_VERIFY else 1
    log(f"[bench] dominant kernel: {dominant} ({per_kernel[dominant]['us_per_round']:.0f} us/round)")

    # timed region of K eager rounds with HIP events around every launch of the dominant kernel
    dec.prefill([prompt])
    binding.seed_rounds(ctx, k, args.warmup, False)
    sync()
    binding.seed_kernel_timing(ctx, binding.kernel_id(dom_phase, dom_op), True)
    tb = len(dec.tokens(0))
    sync()
    e0 = time.perf_counter()
    binding.seed_rounds(ctx, k, args.steps, False)
    sync()
    e1 = time.perf_counter()
    n_dom, ms_dom = binding.seed_kernel_timing_read(ctx)
    binding.seed_kernel_timing(ctx, 0, False)
    t_end = len(dec.tokens(0))
    eager_value = (t_end - tb) / (e1 - e0)
    L_mean = (tb + t_end) // 2
    dom_avg_s = ms_dom / n_dom * 1e-3
    dom_bytes = kernel_bytes(cfg, dom_op, dom_M, L_mean)
    achieved = dom_bytes / dom_avg_s
    roofline = {"bound": "hbm", "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                "frac": achieved / PEAK_HBM, "traffic": measured_traffic(dominant), "kernel": dominant,
                "launches": n_dom, "avg_us": dom_avg_s * 1e6, "alg_bytes_per_launch": dom_bytes}

    # ---------------- verify / draft step latency ----------------
    # inside the replayed rounds: the kernels that open and close each phase stamp the device's
    # constant-rate clock (seed_stats); medians over the rounds of one generate call of the
    # workload (prompt -> gen tokens), so the context runs from P to P + gen
    _, _, stg = dec.generate([prompt], k, gen, use_graph=True)
    verify_ms, draft_ms = stg["verify_ms"], stg["draft_ms"]
    L_gen = P + gen // 2
    verify_bytes = step_bytes(cfg, k + 1, L_gen, cfg.n_layers)
    draft_bytes = step_bytes(cfg, 1, L_gen, cfg.n_dec_layers)
    # the same steps called one at a time from the host (eager launches, host synchronisation
    # inside the interval), for comparison
    dec.prefill([prompt])
    ver_ms, dr_ms = [], []
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    for _ in range(10):
        ev[0].record(stream)
        d, _ = dec.draft(k)
        ev[1].record(stream)
        dec.verify(k)
        ev[2].record(stream)
        sync()
        dr_ms.append(ev[0].elapsed_time(ev[1]) / k)
        ver_ms.append(ev[1].elapsed_time(ev[2]))

    result = {
        "metric": METRIC, "value": round(value, 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed / args.steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.n_layers} layers ({cfg.n_enc_layers} encoder + {cfg.n_dec_layers} "
                               f"decoder), hidden {cfg.hidden}, GQA {cfg.n_heads}/{cfg.n_kv_heads}x{cfg.head_dim}, "
                               f"SwiGLU {cfg.ffn}, vocab {cfg.vocab}, random-init N(0,0.02)",
                   "prompt_len": P, "k": k, "batch": 1, "step": "one draft-verify round",
                   "kv_positions": [t_before, t_after], "graph_replay": True},
        "repetitions": REPS, "value_samples": [round(r, 2) for r in rates],
        "tokens_per_round": round(tokens / args.steps, 4),
        "eager_value": round(eager_value, 2),
        "verify_ms": round(verify_ms, 4), "draft_step_ms": round(draft_ms, 4),
        "step_timing": f"medians over the {stg['rounds']} rounds of one graph-replayed generate "
                       f"({P} -> {gen} tokens), kernel-stamped device clock; bytes at the mean context {L_gen}",
        "eager_verify_ms": round(statistics.median(ver_ms), 4),
        "eager_draft_step_ms": round(statistics.median(dr_ms), 4),
        "verify_gbps": round(verify_bytes / (verify_ms * 1e-3) / 1e9, 1),
        "draft_gbps": round(draft_bytes / (draft_ms * 1e-3) / 1e9, 1),
        "verify_frac": round(verify_bytes / (verify_ms * 1e-3) / PEAK_HBM, 4),
        "draft_frac": round(draft_bytes / (draft_ms * 1e-3) / PEAK_HBM, 4),
        "verify_alg_bytes": verify_bytes, "draft_alg_bytes": draft_bytes,
        "per_kernel": {kk: {a: (round(b, 3) if isinstance(b, float) else b) for a, b in v.items()}
                       for kk, v in per_kernel.items()},
        "roofline": roofline,
    }

    # ---------------- forced acceptance sweep and plain greedy ----------------
    if not args.no_sweep:
        out0, _, st0 = dec.generate([prompt], 0, gen, use_graph=True)
        trace = out0[0]
        result["ar_tokens_per_s"] = round(gen / (st0["decode_ms"] * 1e-3), 2)
        forced = {}
        for a in range(k + 1):
            out, cnt, st = dec.generate([prompt], k, gen, sim_accept=a, forced_trace=trace[None], use_graph=True,
                                        log_cap=gen + 8)
            ok = bool(np.array_equal(out[0], trace))
            full = st["n_accept_log"][:, 0]
            full_rounds = full[:max(0, len(full) - 2)]
            forced[str(a)] = {"tokens_per_s": round(gen / (st["decode_ms"] * 1e-3), 2), "rounds": st["rounds"],
                              "output_equals_greedy": ok, "n_accept_all_equal_a": bool(np.all(full_rounds == a))}
            log(f"[bench] forced a={a}: {forced[str(a)]}")
        result["forced_acceptance"] = forced
        out4, _, st4 = dec.generate([prompt], k, gen, use_graph=True)
        result["measured_acceptance"] = {"tokens_per_s": round(gen / (st4["decode_ms"] * 1e-3), 2),
                                         "mean_accept": round(st4["accepted"] / max(1, st4["rounds"]), 4),
                                         "output_equals_greedy": bool(np.array_equal(out4[0], trace))}
        # end to end through the C ABI with host buffers: the prompt goes in from host memory and the
        # tokens come back to it; prefill, every round and both PCIe copies inside the wall clock
        sync()
        w0 = time.perf_counter()
        out5, _, st5 = dec.generate([prompt], k, gen, use_graph=True)
        w1 = time.perf_counter()
        result["end_to_end"] = {"tokens_per_s": round(gen / (w1 - w0), 2), "wall_s": round(w1 - w0, 4),
                                "prefill_ms": round(st5["prefill_ms"], 2), "decode_ms": round(st5["decode_ms"], 2),
                                "what": f"seed_generate, {P}-token host prompt -> {gen} tokens to host, graph replay"}

    dec.close()
    del dec
    torch.cuda.empty_cache()
    result["copy_ceiling_gbps"] = round(copy_ceiling(torch) / 1e9, 1)
    torch.cuda.empty_cache()
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(cfg, weights, prompt, k, args.cpu_rounds)
    log(f"[bench] total wall {time.perf_counter() - t_start:.1f}s")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
