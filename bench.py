#!/usr/bin/env python3
"""PIPO pair-in/pair-out throughput on one MI355X.

One timed step is one whole request of the workload: the compressed-prompt
prefill (pair gather, compressor, backbone over ceil(n/2) latents, heads)
followed by every pair-decode step (compressor, backbone over one latent, LM
head, MTP head, LM head, confidence gate), with the prompt already resident
in HBM.  ``value`` = emitted output tokens (1 + accept per sequence per pair
step, the prefill's pair included) / wall time of the timed steps.

Also reported on the same JSON line:
  roofline      the weight-streaming GEMM kernel (k_gemv, the dominant
                kernel of decode): algorithmic bytes of its launches in one
                pair step / their summed duration, from start / stop HIP
                events each launch records itself on the library's stream
                (hipExtLaunchKernelGGL, eager profiling pass);
  cpu_baseline  the float64 oracle timed on this host on a bounded sample;
  regular       regular one-token decoding on the same kernels and weights
                (Sec. 4.3's baseline): the n prompt tokens prefilled as n
                positions, then token steps; TTFT and per-token ratios
                against the pair decoder on the same prompt.
Diagnostics go to stderr; stdout carries the one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
from synth.configs import HEADS_MLP_COMPRESSOR, HEADS_MTP_LAYER, HEADS_MLP_CONFIDENCE, HEADS_PAPER  # noqa: E402

METRIC = "output tokens/s per step at bs=1/32 (4B-class); HBM GB/s and % roofline"
HBM_PEAK_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemv_step_bytes(m, B):
    """Algorithmic HBM bytes of the k_gemv launches of one pair step.

    Every weight matrix once (bf16), except the tied embedding / LM head, which
    is streamed twice (backbone token, then the draft token that depends on
    it); plus each launch's activations read once and outputs written once.
    """
    h, f, v, L = m.hidden, m.ffn, m.vocab, m.n_layers
    nqkv = m.q_dim + 2 * m.kv_dim
    w = 2 * (L * (nqkv * h + h * m.q_dim + 2 * f * h + h * f) + 2 * (h * 2 * h) + 2 * v * h)
    act = B * 4 * (L * (h + m.q_dim // 2 + h + f // 2) + 2 * h + 2 * h)        # inputs
    act += B * 4 * (L * (nqkv // 2 + h + f // 2 + h) + h + h + 2 * v)         # outputs
    heads = getattr(m, "heads", 0)
    if heads & HEADS_MLP_COMPRESSOR:       # W1 2H->H replaces W_c, plus W2 H->H
        w += 2 * h * h
        act += B * 4 * (h + h + h)
    if heads & HEADS_MTP_LAYER:            # one more decoder layer
        w += 2 * (nqkv * h + h * m.q_dim + 2 * f * h + h * f)
        act += B * 4 * ((h + m.q_dim // 2 + h + f // 2) + (nqkv // 2 + h + f // 2 + h))
    if heads & HEADS_MLP_CONFIDENCE:       # W1 2H->H
        w += 2 * 2 * h * h
        act += B * 4 * (2 * h + h)
    return w + act


def kv_step_bytes(m, B, length):
    """KV-cache bytes one pair step reads at a context of ``length`` latents
    (the App. B MTP layer's cache included when the model has one)."""
    layers = m.n_layers + (1 if getattr(m, "heads", 0) & HEADS_MTP_LAYER else 0)
    return 2 * layers * B * m.n_kv_heads * (length + 1) * m.head_dim * 2


def measured_traffic(workload):
    """HBM bytes per k_gemv launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary, or None when that summary is missing, covers another
    workload, or was taken on a different version of the kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "k_gemv_4b_bs1_traffic.txt")
    if workload != "4b-bs1-ctx2048" or not os.path.exists(path):
        return None
    kv = dict(line.split("=", 1) for line in open(path).read().splitlines() if "=" in line and " " not in line)
    src = os.path.join(ROOT, "paper_2605_27255_amd", "csrc", "gemv.hip")
    if kv.get("gemv_source_sha256") != hashlib.sha256(open(src, "rb").read()).hexdigest():
        return None
    return int(kv["traffic_bytes_per_launch"])


def cpu_baseline(wl, accept_rate, budget_s=12.0):
    """The oracle (float64, NumPy) on a bounded sample of one pair step.

    Sample: the per-layer step (two decoder layers of the workload's shape over
    synthetic KV caches at the workload's prompt length) and the heads (LM
    head, MTP head, LM head, confidence) for one sequence; one pair step is
    heads + layers/2 * (two-layer time); scaled to output tokens/s with the
    acceptance the GPU run measured.
    """
    import numpy as np
    from oracle import pipo_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    m2 = wl.model.with_layers(2)
    W = O.OracleWeights.generate(m2, seed=wl.seed, precision="bf16")
    rng = np.random.default_rng(0)
    T = wl.latents
    caches0 = [[rng.standard_normal((m2.n_kv_heads, T, m2.head_dim)),
                rng.standard_normal((m2.n_kv_heads, T, m2.head_dim))] for _ in range(2)]
    orc = O.PipoOracle(W)
    orc.sampling = O.Sampling(tau=wl.tau, temperature=wl.temperature, top_p=wl.top_p,
                              seeds=(wl.sample_seed_base,), top_k=wl.top_k, rep_penalty=wl.rep_penalty)
    from synth import rspec
    orc.seen = [set(int(t) for t in rspec.prompt_tokens(1, wl.prompt_tokens, m2.vocab, wl.prompt_seed)[0])]
    mtp0 = [rng.standard_normal((m2.n_kv_heads, T, m2.head_dim)), rng.standard_normal((m2.n_kv_heads, T, m2.head_dim))]
    z = rng.standard_normal(m2.hidden)
    t_layers, t_heads, reps = [], [], 0
    t_start = time.perf_counter()
    while reps < 2 or (time.perf_counter() - t_start < budget_s and reps < 200):
        caches = [[c[0], c[1]] for c in caches0]
        orc.mtp_caches = [[mtp0[0], mtp0[1]]]       # the App. B MTP layer's cache, when the model has one
        t0 = time.perf_counter()
        h = O.backbone_step(W, z, T, caches)
        t1 = time.perf_counter()
        orc.heads(h, 0, 1, T)
        t2 = time.perf_counter()
        t_layers.append(t1 - t0)
        t_heads.append(t2 - t1)
        reps += 1
    step_s = min(t_heads) + wl.model.n_layers / 2 * min(t_layers)
    # the oracle runs the batch's sequences one after another: (1 + acceptance) tokens per step_s
    return {"value": (1.0 + accept_rate) / step_s,
            "unit": "output tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"float64 oracle, one sequence: {reps} repetitions (best taken) of 2 decoder layers at "
                       f"{T} cached latents plus the heads; pair step = heads + {wl.model.n_layers}/2 x "
                       f"(2-layer time) = {step_s * 1e3:.1f} ms; batch sequences run one after another; "
                       f"tokens per pair step 1 + {accept_rate:.3f} (GPU-measured acceptance)")}


def opd_leg(T=2048, V=151936, reps=20):
    """The OPD target kernel (App. C) on one chunk of the paper's size: T
    positions of student and teacher logits over V tokens, already in HBM.
    Algorithmic bytes: both fp32 logit rows of every position, plus labels,
    rows and the two fp32 outputs."""
    import torch
    from paper_2605_27255_amd import opd_targets
    g = torch.Generator(device="cuda").manual_seed(0)
    ls = torch.randn((T, V), generator=g, device="cuda", dtype=torch.float32) * 3.0
    lt = ls + torch.randn((T, V), generator=g, device="cuda", dtype=torch.float32) * 0.5
    labels = torch.randint(0, V, (T,), generator=g, device="cuda", dtype=torch.int32)
    for _ in range(3):
        opd_targets(ls, lt, labels, None, sums=False)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        opd_targets(ls, lt, labels, None, sums=False)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = 2 * T * V * 4 + T * 4 * 3
    gbs = nbytes / (ms * 1e-3) / 1e9
    # the same chunk with bf16 logit rows
    ls, lt = ls.to(torch.bfloat16), lt.to(torch.bfloat16)
    for _ in range(3):
        opd_targets(ls, lt, labels, None, sums=False)
    e0.record(stream)
    for _ in range(reps):
        opd_targets(ls, lt, labels, None, sums=False)
    e1.record(stream)
    torch.cuda.synchronize()
    ms16 = e0.elapsed_time(e1) / reps
    gbs16 = (2 * T * V * 2 + T * 4 * 3) / (ms16 * 1e-3) / 1e9
    del ls, lt
    torch.cuda.empty_cache()
    log(f"OPD targets: {T} x {V}: {ms * 1e3:.1f} us per chunk, {gbs:.0f} GB/s (bf16 rows {ms16 * 1e3:.1f} us)")
    return {"kernel": "k_opd", "positions": T, "vocab": V, "us_per_chunk": round(ms * 1e3, 2),
            "algorithmic_bytes": nbytes, "achieved_gbs": round(gbs, 1), "bound": "hbm",
            "frac_of_8tbs": round(gbs / HBM_PEAK_GBS, 4),
            "bf16_rows": {"us_per_chunk": round(ms16 * 1e3, 2), "achieved_gbs": round(gbs16, 1)},
            "timing": "torch events on the launching stream around 20 launches (the kernel is the only work)"}


def ceilings_leg(m, reps=20):
    """Attainable ceilings on this GPU, from the library's measurement kernels.

    stream: the decode GEMV's weight-stream pattern (1 KB tiles per wave load,
    nontemporal, two batches of five in flight, 256 x 8 waves) reading each
    matrix size of one pair step once, each launch from other bytes of a
    2 GiB buffer (from HBM, as the step's matrices are); ``step_ms`` is the sum over a pair
    step's matrices (layers, the embedding twice, compressor and MTP), the
    time a pure weight stream of the step would take launch by launch.
    mfma: v_mfma_f32_16x16x32_bf16 issue rate with register operands (4 x 4
    independent accumulators per wave) on random and on zero bf16 data, at
    1, 2 and 4 waves per SIMD."""
    import torch
    from paper_2605_27255_amd import calibrate_stream, calibrate_mfma
    h, f, v, L = m.hidden, m.ffn, m.vocab, m.n_layers
    mats = {"qkv": ((m.q_dim + 2 * m.kv_dim) * h * 2, L), "o": (h * m.q_dim * 2, L), "gate_up": (2 * f * h * 2, L),
            "down": (h * f * 2, L), "lm_head": (v * h * 2, 2), "compressor_mtp": (2 * h * h * 2, 2)}
    # 2 GiB: each launch reads another window, so nothing is served from L2 or the memory-side cache
    buf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
    stream, step_us = {}, 0.0
    for name, (nbytes, count) in mats.items():
        nb = nbytes // 1024 * 1024
        us = calibrate_stream(buf, nb, reps)
        stream[name] = {"bytes": nb, "us": round(us, 2), "gbs": round(nb / (us * 1e3), 1), "per_step": count}
        step_us += us * count
    del buf
    g = torch.Generator(device="cuda").manual_seed(0)
    rnd = (torch.randn(8192, generator=g, device="cuda") * 0.5).to(torch.bfloat16)
    zer = torch.zeros(8192, dtype=torch.bfloat16, device="cuda")
    mfma = {}
    for w in (1, 2, 4):
        mfma[f"random_{w}w"] = round(calibrate_mfma(rnd, w, iters=4096 // w), 1)
        mfma[f"zero_{w}w"] = round(calibrate_mfma(zer, w, iters=4096 // w), 1)
    torch.cuda.empty_cache()
    res = {"stream": stream, "stream_step_ms": round(step_us / 1e3, 4), "mfma_bf16_tflops": mfma,
           "kernels": "k_cal_stream, k_cal_mfma (csrc/calibrate.hip)"}
    log(f"ceilings: weight stream of a pair step {step_us / 1e3:.3f} ms; "
        + ", ".join(f"{k} {x['gbs']:.0f} GB/s" for k, x in stream.items()) + f"; MFMA bf16 TF/s {mfma}")
    return res


def regular_leg(wl, prompts, seeds, pipo_ttft, pipo_ms_step, acc_rate, pipo_job_s, lens, emitted, reps):
    """Regular decoding of the same prompt on the same kernels: one timed job is
    the n-position prefill plus as many token steps as the pair decoder ran
    pair steps; ``reps`` timed jobs after one warm-up."""
    import numpy as np
    import torch
    from paper_2605_27255_amd import PipoModel

    m, B, steps = wl.model, wl.batch, wl.decode_steps
    n = wl.prompt_tokens
    t0 = time.perf_counter()
    model = PipoModel(m, seed=wl.seed, max_batch=B, max_latent=n + steps + 1, prefill_chunk=wl.prefill_chunk)
    toks = torch.empty((steps, B), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    log(f"regular decoding: init {time.perf_counter() - t0:.1f} s, prompt {n} positions + {steps} token steps")

    def job(ev=None):
        if ev:
            ev[0].record(stream)
        model.regular_prefill(prompts, wl.temperature, wl.top_p, seeds, top_k=wl.top_k, rep_penalty=wl.rep_penalty,
                              lens=lens)
        if ev:
            ev[1].record(stream)
        for s in range(steps):
            model.regular_into(toks[s])
        if ev:
            ev[2].record(stream)

    job()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
    t_start = time.perf_counter()
    for k in range(reps):
        job(evs[k])
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t_start) / reps
    model.close()
    del model
    torch.cuda.empty_cache()
    ttft = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    ms_tok = float(np.mean([e[1].elapsed_time(e[2]) for e in evs])) / max(steps, 1)
    # the same number of output tokens as one pair-decoder job emitted
    reg_same_out_s = (ttft + (emitted / B - 1) * ms_tok) * 1e-3
    res = {"ttft_ms": round(ttft, 3), "ms_per_token_step": round(ms_tok, 4),
           "output_tokens_per_s": round(B * 1e3 / ms_tok, 2), "job_s": round(wall, 4),
           "ttft_speedup": round(ttft / pipo_ttft, 3),
           "pair_step_cost_over_token_step": round(pipo_ms_step / ms_tok, 3),
           "per_token_speedup_at_measured_acceptance": round(ms_tok * (1 + acc_rate) / pipo_ms_step, 3),
           "per_token_speedup_two_slots_per_pair": round(ms_tok * 2 / pipo_ms_step, 3),
           "end_to_end_speedup_same_output": round(reg_same_out_s / pipo_job_s, 3),
           "paper_context": "Sec. 4.3 / Fig. 4 (4B model, HF backend; the paper names H20-141G GPUs): "
                            "up to 2.64x TTFT, 2.07x TPOT counting both slots of a pair"}
    log(f"regular decoding: TTFT {ttft:.2f} ms, {ms_tok:.3f} ms/token step; TTFT speedup "
        f"{res['ttft_speedup']}x, pair step / token step {res['pair_step_cost_over_token_step']}")
    return res


def measure(wl, n_steps, n_warmup, profile=True, ragged=False):
    """Time ``n_steps`` whole requests of workload ``wl`` after ``n_warmup``
    untimed ones (prompts resident in HBM), then, with ``profile``, one eager
    pass with per-kernel-class HIP events.  Returns the JSON fields of the
    workload and the figures the other legs reuse."""
    import numpy as np
    import torch
    from paper_2605_27255_amd import PipoModel, unpack_pairs
    from synth import rspec

    m = wl.model
    B, steps = wl.batch, wl.decode_steps
    torch.cuda.set_device(0)
    log(f"workload {wl.name}: {m.n_layers}L h{m.hidden} B{B} prompt {wl.prompt_tokens} "
        f"({wl.latents} latents) + {steps} pair steps")
    t0 = time.perf_counter()
    model = PipoModel(m, seed=wl.seed, max_batch=B, max_latent=wl.latents + steps + 1,
                      prefill_chunk=wl.prefill_chunk)
    prompts = torch.from_numpy(rspec.prompt_tokens(B, wl.prompt_tokens, m.vocab, wl.prompt_seed)).cuda()
    n_tok = wl.prompt_tokens
    lens = [n_tok - (7919 * b) % max(1, n_tok // 2) for b in range(B)] if ragged else None
    lat = [(n + 1) // 2 for n in lens] if lens else [wl.latents] * B
    seeds = [wl.sample_seed_base + b for b in range(B)] if wl.temperature > 0 else None
    outs = torch.empty((steps, B, 4), dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    log(f"init (device weight generation) {time.perf_counter() - t0:.1f} s")

    stream = torch.cuda.current_stream()

    def job(ev=None):
        if ev:
            ev[0].record(stream)
        first, _, _ = model.prefill(prompts, wl.tau, wl.temperature, wl.top_p, seeds, top_k=wl.top_k,
                                    rep_penalty=wl.rep_penalty, lens=lens)
        if ev:
            ev[1].record(stream)
        for s in range(steps):
            model.decode_into(outs[s])
        if ev:
            ev[2].record(stream)
        return first

    for _ in range(n_warmup):
        job()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_steps)]
    firsts = []
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(n_steps):
        firsts.append(job(evs[k]))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    # emitted tokens: the last timed request's records (all requests are identical)
    fb = unpack_pairs(firsts[-1])
    acc_all = outs[:, :, 3].cpu().numpy()
    accepts = int(acc_all.sum()) + int(fb[3].sum())
    pairs = steps * B + B
    emitted_per_job = pairs + accepts
    value = emitted_per_job * n_steps / wall
    ttft = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    dec_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    ms_step = dec_ms / max(steps, 1)
    acc_rate = accepts / pairs
    kv_mean = float(np.mean([sum(kv_step_bytes(m, 1, L + s) for L in lat) for s in range(max(steps, 1))]))
    step_bytes = gemv_step_bytes(m, B) + kv_mean
    log(f"timed {n_steps} requests in {wall:.3f} s: TTFT {ttft:.2f} ms, decode {ms_step:.3f} ms/pair step, "
        f"acceptance {acc_rate:.3f}, {value:.1f} output tokens/s")
    res = {
        "value": round(value, 3), "ms_per_step": round(wall / n_steps * 1e3, 3),
        "config": {"workload": wl.name, "layers": m.n_layers, "hidden": m.hidden, "ffn": m.ffn,
                   "heads_q_kv": [m.n_q_heads, m.n_kv_heads], "head_dim": m.head_dim, "vocab": m.vocab,
                   "batch": B, "prompt_tokens": wl.prompt_tokens, "latents": wl.latents,
                   "prompt_lengths": ("ragged, mean %.0f" % np.mean(lens)) if lens else "uniform",
                   "decode_steps": steps, "tau": wl.tau,
                   "sampling": ("greedy" if wl.temperature <= 0 else f"T{wl.temperature} top-p{wl.top_p}"
                                + (f" top-k{wl.top_k} rep-penalty{wl.rep_penalty}"
                                   if wl.top_k or wl.rep_penalty != 1.0 else "")),
                   "parallelism": "none (1 GPU)"},
        "ttft_ms": round(ttft, 3),
        "decode": {"ms_per_pair_step": round(ms_step, 4), "pair_steps_per_s": round(B * 1e3 / ms_step, 2),
                   "output_tokens_per_s": round(B * (1 + acc_rate) * 1e3 / ms_step, 2),
                   "acceptance": round(acc_rate, 4),
                   "algorithmic_gb_per_step": round(step_bytes / 1e9, 4),
                   "hbm_gbs": round(step_bytes / ms_step / 1e6, 1),
                   "hbm_frac": round(step_bytes / ms_step / 1e6 / HBM_PEAK_GBS, 4)},
    }

    if profile:
        settle = min(4, steps // 4)          # eager steps before the counted ones
        psteps = max(1, min(steps - settle, 32))
        model.profile(True)
        model.prefill(prompts, wl.tau, wl.temperature, wl.top_p, seeds, top_k=wl.top_k, rep_penalty=wl.rep_penalty,
                      lens=lens)
        torch.cuda.synchronize()
        pre = model.profile_read()
        model.profile(True)
        for s in range(settle):              # settle the eager path first; not counted
            model.decode_into(outs[s])
        torch.cuda.synchronize()
        model.profile_read()
        model.profile(True)
        for s in range(psteps):
            model.decode_into(outs[settle + s])
        torch.cuda.synchronize()
        prof = model.profile_read()
        model.profile(False)
        gemv_ms = sum(prof[k][0] for k in ("gemv_layer", "gemv_lmhead", "gemv_small")) / psteps
        gemv_n = sum(prof[k][1] for k in ("gemv_layer", "gemv_lmhead", "gemv_small")) / psteps
        gb = gemv_step_bytes(m, B)
        achieved = gb / (gemv_ms * 1e-3) / 1e9
        per_class = {k: {"ms_per_step": round(v[0] / psteps, 4), "launches_per_step": v[1] / psteps}
                     for k, v in prof.items() if v[1]}
        res["roofline"] = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                           "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                           "traffic": measured_traffic(wl.name),
                           "kernel": "k_gemv (decode weight-streaming GEMM, all launches of a pair step)",
                           "bytes_per_launch": round(gb / gemv_n), "launches_per_step": gemv_n,
                           "avg_launch_us": round(gemv_ms / gemv_n * 1e3, 3),
                           "timing": "HIP events recorded by each k_gemv launch itself "
                                     "(hipExtLaunchKernelGGL start/stop) on the library stream, in an "
                                     "eager profiling pass after the timed region"}
        if prof.get("attn_decode", (0, 0))[1]:
            att_ms = prof["attn_decode"][0] / psteps
            res["attn_decode"] = {"ms_per_pair_step": round(att_ms, 4), "kv_gb_per_step": round(kv_mean / 1e9, 4),
                                  "hbm_gbs": round(kv_mean / att_ms / 1e6, 1),
                                  "hbm_frac": round(kv_mean / att_ms / 1e6 / HBM_PEAK_GBS, 4)}
        res["kernel_ms_per_pair_step"] = per_class
        res["prefill_kernel_ms"] = {k: round(v[0], 3) for k, v in pre.items() if v[1]}
        if pre.get("prefill_gemm", (0, 0))[1]:
            # the prefill GEMMs (k_gemm_wd): 2 flops per weight per latent row; every
            # layer GEMM also multiplies the activations' lo plane (a second MFMA)
            h, f, L = m.hidden, m.ffn, m.n_layers
            layer_w = (m.q_dim + 2 * m.kv_dim) * h + h * m.q_dim + 2 * f * h + h * f
            rows = B * wl.latents
            useful = 2.0 * rows * (L * layer_w + 2 * h * h)
            issued = 2.0 * rows * (2 * L * layer_w + 2 * h * h)
            sec = pre["prefill_gemm"][0] * 1e-3
            res["prefill_gemm"] = {
                "kernel": "k_gemm_wd", "bound": "mfma", "peak_tflops": 2500.0,
                "useful_tflops": round(useful / sec / 1e12, 1), "issued_tflops": round(issued / sec / 1e12, 1),
                "issued_frac": round(issued / sec / 1e12 / 2500.0, 4),
                "note": "issued counts the lo-plane MFMAs (activations carried as bf16 hi + lo); times are the "
                        "profiling pass's HIP events around every prefill GEMM launch"}
        log("per-class decode ms/step:", {k: v["ms_per_step"] for k, v in per_class.items()})
        log("prefill kernel ms:", res["prefill_kernel_ms"])

    model.close()
    del model
    torch.cuda.empty_cache()
    info = dict(prompts=prompts, seeds=seeds, ttft=ttft, ms_step=ms_step, acc_rate=acc_rate, wall=wall, lens=lens,
                emitted_per_job=emitted_per_job)
    return res, info


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="4b-bs1-ctx2048")
    ap.add_argument("--decode-steps", type=int, default=None, help="override the workload's step count")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true")
    ap.add_argument("--no-regular", action="store_true", help="skip the regular-decoding baseline leg")
    ap.add_argument("--no-opd", action="store_true", help="skip the OPD target kernel leg")
    ap.add_argument("--no-ceilings", action="store_true", help="skip the stream / MFMA ceiling measurements")
    ap.add_argument("--no-bs32", action="store_true",
                    help="skip the 4B batch-32 leg that the default (4B batch-1) run adds as the bs32 object")
    ap.add_argument("--heads", choices=("linear", "paper"), default="linear",
                    help="linear: the workloads' one-linear heads; paper: the App. B forms of all three heads")
    ap.add_argument("--batch", type=int, default=None, help="override the workload's batch (up to 64)")
    ap.add_argument("--ragged", action="store_true",
                    help="a ragged batch: sequence b's prompt is the first n - (7919 b mod n/2) tokens of its row")
    ap.add_argument("--sampler", choices=("workload", "eval"), default="workload",
                    help="workload: the workload's own selection; eval: the paper's evaluation sampler "
                         "(T 1.0, top-p 0.95, top-k 20, repetition penalty 1.5)")
    ap.add_argument("--calibrate", action="store_true",
                    help="only measure the attainable ceilings (weight stream per matrix size, MFMA issue rate)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (counter calibration) and exit")
    args = ap.parse_args()
    if args.calibrate:
        import torch
        from synth.configs import WORKLOADS
        torch.cuda.set_device(0)
        print(json.dumps({"ceilings": ceilings_leg(WORKLOADS[args.workload].model)}), flush=True)
        return
    if args.calibrate_copy:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")      # 1 GiB
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copied 1073741824 bytes")
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the PIPO decode path shards "
              "as independent data-parallel replicas, one per GPU, with no inter-GPU traffic, so the "
              "one-GPU figure is the per-GPU figure.", file=sys.stderr)
        sys.exit(2)

    from dataclasses import replace
    from synth.configs import WORKLOADS

    wl = WORKLOADS[args.workload]
    if args.decode_steps is not None:
        wl = replace(wl, decode_steps=args.decode_steps)
    if args.heads == "paper":
        wl = replace(wl, name=wl.name + "+appB-heads", model=replace(wl.model, heads=HEADS_PAPER))
    if args.batch is not None:
        wl = replace(wl, name=f"{wl.name}@bs{args.batch}", batch=args.batch)
    if args.ragged:
        wl = replace(wl, name=wl.name + "+ragged")
    if args.sampler == "eval":
        wl = replace(wl, name=wl.name + "+eval-sampler", temperature=1.0, top_p=0.95, top_k=20, rep_penalty=1.5)
    res, info = measure(wl, args.steps, args.warmup, profile=not args.no_profile, ragged=args.ragged)
    result = {"metric": METRIC, "value": res.pop("value"), "unit": "output tokens/s", "n_gpus": 1,
              "steps": args.steps, "warmup": args.warmup, "ms_per_step": res.pop("ms_per_step"),
              "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
              "data": "synthetic (R-spec random-init weights and uniform random prompts)"}
    result.update(res)
    prompts, seeds, lens = info["prompts"], info["seeds"], info["lens"]
    ttft, ms_step, acc_rate, wall = info["ttft"], info["ms_step"], info["acc_rate"], info["wall"]
    emitted_per_job = info["emitted_per_job"]
    if not args.no_bs32 and wl.name == "4b-bs1-ctx2048":
        # the batch-32 half of the metric: the 4B batch-32 workload, one timed request
        wl32 = WORKLOADS["4b-bs32-ctx8192-topp"]
        r32, _ = measure(wl32, 1, 1, profile=not args.no_profile)
        result["bs32"] = {"workload": wl32.name, "output_tokens_per_s": r32["value"],
                          "ms_per_request": r32["ms_per_step"], "ttft_ms": r32["ttft_ms"], **r32["decode"]}
        for k in ("roofline", "attn_decode", "kernel_ms_per_pair_step"):
            if k in r32:
                result["bs32"][k] = r32[k]
    if not args.no_regular:
        result["regular"] = regular_leg(wl, prompts, seeds, ttft, ms_step, acc_rate, wall / args.steps, lens,
                                        emitted_per_job, max(1, min(args.steps, 2)))
    if not args.no_opd:
        result["opd"] = opd_leg()
    if not args.no_ceilings:
        cl = ceilings_leg(wl.model)
        kc = result.get("kernel_ms_per_pair_step", {})
        gm = sum(kc.get(k, {}).get("ms_per_step", 0.0) for k in ("gemv_layer", "gemv_lmhead", "gemv_small"))
        if gm:
            # the step's GEMV time against a pure weight stream of the same matrices
            cl["gemv_ms_per_step"] = round(gm, 4)
            cl["gemv_over_stream_ceiling"] = round(gm / cl["stream_step_ms"], 3)
        result["ceilings"] = cl
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        result["cpu_baseline"] = cpu_baseline(wl, acc_rate)
        log(f"cpu baseline {time.perf_counter() - t0:.1f} s: {result['cpu_baseline']['value']:.3f} tokens/s")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
