"""Teacher-forced parity protocol between the HIP path and the oracle.

The GPU runs free (each step's input pair is the pair its previous step
produced on the device); the oracle, with the workloads' bf16 KV cache,
replays exactly those input pairs and,
inside each step, the GPU's backbone token as the MTP head's input, and every
output is compared:

* logits: max |d| <= 2e-2 and sum|d| / sum|ref| <= 5e-3 per row;
* confidence: |c_gpu - c_ref| <= 1e-3;
* accept flags: equal wherever |c_ref - tau| > 1e-3;
* greedy tokens: equal, unless the oracle's margin between its choice and
  the GPU's choice is within twice that row's max logit error (a near-tie
  either answer is correct for); then the step is counted as ambiguous, and
  the GPU token must still be the argmax of the GPU's own logits;
* sampled tokens: equal, or else (a draw at a boundary that the logit error
  or the sampler's own fp32 arithmetic moves) the selection rule applied to
  the GPU's logits must give the GPU token, taken either in float64 or in
  the kernel's precision (fp32 probabilities, 2^-40 fixed-point masses; see
  ``_kernel_precision_rule``); the evaluation sampler's rule takes the
  oracle's penalised set of that step.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from oracle import pipo_oracle as O
from synth import rspec

LOGIT_MAX_ABS = 2e-2
LOGIT_MEAN_REL = 5e-3
CONF_TOL = 1e-3


@dataclass
class ParityReport:
    steps: int = 0
    rows: int = 0
    max_abs: float = 0.0
    max_mean_rel: float = 0.0
    max_conf_err: float = 0.0
    ambiguous_tokens: int = 0
    ambiguous_accepts: int = 0
    penalty_decisive: int = 0   # rows whose oracle token the repetition penalty changed
    failures: list = field(default_factory=list)

    def check(self):
        assert not self.failures, "\n".join(self.failures[:20])


def _row_err(gpu_row, ref_row):
    d = np.abs(gpu_row.astype(np.float64) - ref_row)
    return float(d.max()), float(d.sum() / np.abs(ref_row).sum())


def _rule(smp, u, seen):
    """The oracle's selection rule for one row (sampling only)."""
    if smp.top_k or smp.rep_penalty != 1.0:
        return lambda row: O.select_eval(row, seen, smp.temperature, smp.top_k, smp.top_p, smp.rep_penalty, u)
    return lambda row: O.select_top_p(row, smp.temperature, smp.top_p, u)


def _check_token(rep, tag, gpu_tok, ref_tok, gpu_row, ref_row, max_abs, smp, u, seen=()):
    if smp.temperature > 0 and smp.rep_penalty != 1.0:
        plain = O.select_eval(ref_row, (), smp.temperature, smp.top_k, smp.top_p, 1.0, u)
        rep.penalty_decisive += int(plain != ref_tok)
    if gpu_tok == ref_tok:
        return
    if smp.temperature <= 0:
        margin = ref_row[ref_tok] - ref_row[gpu_tok]
        if margin <= 2 * max_abs + 1e-12 and gpu_tok == int(np.argmax(gpu_row)):
            rep.ambiguous_tokens += 1
            return
        rep.failures.append(f"{tag}: token {gpu_tok} != oracle {ref_tok} (margin {margin:.3g}, "
                            f"max_abs {max_abs:.3g})")
    else:
        again = _rule(smp, u, seen)(gpu_row.astype(np.float64))
        again32 = _kernel_precision_rule(gpu_row, smp, u, seen)
        if gpu_tok in (again, again32):
            rep.ambiguous_tokens += 1
            return
        rep.failures.append(f"{tag}: sampled {gpu_tok}, oracle {ref_tok}, rule on GPU logits {again} "
                            f"(in the kernel's precision {again32})")


def _kernel_precision_rule(row, smp, u, seen):
    """The selection rule of the oracle (penalty, temperature, top-k, top-p
    threshold, inverse CDF in id order) taken in the sampler kernel's
    precision instead of float64: penalised logits and
    p_j = exp2((l_j - max) * (log2(e) / T)) in fp32 (exp2 rounded from
    float64 here; results below fp32's normal range are 0), each mass
    rint(p_j 2^40) as an integer, theta* the largest p value whose upper
    integer mass reaches top_p * total, t = floor(u * M) for the nucleus mass
    M, and the first nucleus id whose running integer mass exceeds t."""
    v = np.asarray(row, dtype=np.float32).copy()
    f32 = np.float32
    eval_smp = bool(smp.top_k) or smp.rep_penalty != 1.0
    if eval_smp and seen:
        idx = np.fromiter(sorted(set(int(t) for t in seen)), dtype=np.int64)
        pen = f32(smp.rep_penalty)
        x = v[idx]
        v[idx] = np.where(x > 0, x / pen, x * pen).astype(np.float32)
    mx = v.max()
    kT = f32(f32(1.4426950408889634) / f32(smp.temperature))
    arg = ((v - mx).astype(np.float32) * kT).astype(np.float32)
    ev = np.exp2(arg.astype(np.float64)).astype(np.float32)
    ev[ev < np.finfo(np.float32).tiny] = 0.0
    mass = np.rint(ev.astype(np.float64) * 2.0 ** 40).astype(np.int64)
    kept = np.ones(v.size, dtype=bool)
    if eval_smp and 0 < smp.top_k < v.size:
        kept = v >= np.sort(v)[::-1][smp.top_k - 1]
    total = int(mass[kept].sum())
    target = float(f32(smp.top_p)) * float(total)
    ids = np.nonzero(kept)[0]
    order = ids[np.argsort(-ev[ids], kind="stable")]
    vals = ev[order]
    upper = np.cumsum(mass[order])
    # a tie group of equal values enters whole: its upper mass is the group's last
    last = np.searchsorted(-vals, -vals, side="right") - 1
    ok = upper[last].astype(np.float64) >= target
    nucleus = kept & (ev >= vals[np.argmax(ok)]) if ok.any() else kept
    M = int(mass[nucleus].sum())
    r24 = int(round(u * 2 ** 24))
    tsel = (r24 * M) >> 24
    nid = np.nonzero(nucleus)[0]
    run = np.cumsum(mass[nid])
    hit = np.nonzero(run > tsel)[0]
    return int(nid[hit[0]] if hit.size else nid[-1])


def compare_step(rep, tag, out_np, lb, ld, recs, smp, seeds, step, mean_rel_tol=LOGIT_MEAN_REL, conf_tol=CONF_TOL,
                 max_abs_tol=LOGIT_MAX_ABS, seen=None, seq_ids=None):
    tok_b, tok_d, conf, acc = out_np
    rep.steps += 1
    for i, r in enumerate(recs):
        rep.rows += 1
        t = f"{tag} seq {i if seq_ids is None else seq_ids[i]}"
        for name, g, ref in (("logits_b", lb[i], r["logits_b"]), ("logits_d", ld[i], r["logits_d"])):
            ma, mr = _row_err(g, ref)
            rep.max_abs = max(rep.max_abs, ma)
            rep.max_mean_rel = max(rep.max_mean_rel, mr)
            if ma > max_abs_tol or mr > mean_rel_tol:
                rep.failures.append(f"{t} {name}: max_abs {ma:.3g} mean_rel {mr:.3g}")
        u_b = rspec.uniform_draw(seeds[i], step, 0) if smp.temperature > 0 else None
        u_d = rspec.uniform_draw(seeds[i], step, 1) if smp.temperature > 0 else None
        ma_b, _ = _row_err(lb[i], r["logits_b"])
        ma_d, _ = _row_err(ld[i], r["logits_d"])
        sb = seen[i] if seen is not None else set()
        _check_token(rep, t + " backbone", int(tok_b[i]), r["tok_b"], lb[i], r["logits_b"], ma_b, smp, u_b, sb)
        # the draft penalises its pair's backbone token too (the GPU's, which the oracle was forced to)
        _check_token(rep, t + " draft", int(tok_d[i]), r["tok_d"], ld[i], r["logits_d"], ma_d, smp, u_d,
                     sb | {int(tok_b[i])})
        ce = abs(float(conf[i]) - r["conf"])
        rep.max_conf_err = max(rep.max_conf_err, ce)
        if ce > conf_tol:
            rep.failures.append(f"{t}: conf {conf[i]:.6f} vs {r['conf']:.6f}")
        if bool(acc[i]) != r["accept"]:
            if abs(r["conf"] - smp.tau) <= conf_tol:
                rep.ambiguous_accepts += 1
            else:
                rep.failures.append(f"{t}: accept {acc[i]} vs {r['accept']} (c_ref {r['conf']:.6f})")
        # the accept flag the GPU reports must follow its own confidence exactly
        if bool(acc[i]) != (float(conf[i]) >= np.float32(smp.tau)):
            rep.failures.append(f"{t}: accept flag inconsistent with conf {conf[i]} and tau {smp.tau}")


def run_parity(gpu_model, W, prompts, steps, smp, log=print, mean_rel_tol=LOGIT_MEAN_REL, conf_tol=CONF_TOL,
               max_abs_tol=LOGIT_MAX_ABS, lens=None, seqs=None, check_steps=None):
    """Run the GPU free for ``steps`` pair steps after prefill; replay on the
    oracle.  ``lens``: a ragged batch, sequence i's prompt being the first
    lens[i] tokens of row i of ``prompts``.  ``seqs``: the sequences the
    oracle replays (default all; the GPU always runs the whole batch);
    ``check_steps``: the step indices compared (0 is the prefill's pair;
    default all).  The oracle reaches a step that does not follow the last
    compared one by one prefill over the prompt's and the GPU's input pairs
    up to that step (the forced-pair prefill, equal to the step-by-step
    replay by causality)."""
    import torch
    from paper_2605_27255_amd import unpack_pairs

    B = prompts.shape[0]
    seeds = list(smp.seeds) if smp.seeds else [0] * B
    seqs = list(range(B)) if seqs is None else [int(i) for i in seqs]
    check = sorted(set(range(steps + 1)) if check_steps is None else {int(v) for v in check_steps})
    assert check and 0 <= check[0] and check[-1] <= steps, check
    tokens = torch.from_numpy(np.ascontiguousarray(prompts, dtype=np.int32)).cuda()
    sel = torch.tensor(seqs, dtype=torch.long, device="cuda")
    outs = [gpu_model.prefill(tokens, smp.tau, smp.temperature, smp.top_p,
                              seeds if smp.temperature > 0 else None, logits=0 in check, top_k=smp.top_k,
                              rep_penalty=smp.rep_penalty, lens=lens)]
    for s in range(1, steps + 1):
        outs.append(gpu_model.decode_step(logits=s in check))
    torch.cuda.synchronize()
    host = []
    for s, (o, lb, ld) in enumerate(outs):
        lg = (lb.index_select(0, sel).cpu().numpy(), ld.index_select(0, sel).cpu().numpy()) if s in check else None
        host.append((unpack_pairs(o), lg))
    del outs
    log(f"gpu done: {B} sequences, {steps} steps; oracle replays sequences {seqs if len(seqs) < B else 'all'}, "
        f"steps {check if len(check) <= steps else 'all'}")
    pad = W.cfg.pad_id

    def in_pair(s, i):   # the input pair of decode step s >= 1 for sequence i: step s-1's output
        o = host[s - 1][0]
        return int(o[0][i]), int(o[1][i]) if o[3][i] else pad

    own = _own_prompts(prompts, lens)
    sub_prompts = [own[i] for i in seqs]
    sub_seeds = [seeds[i] for i in seqs]
    sub_smp = smp if smp.temperature <= 0 else O.Sampling(
        tau=smp.tau, temperature=smp.temperature, top_p=smp.top_p, seeds=tuple(sub_seeds), top_k=smp.top_k,
        rep_penalty=smp.rep_penalty)
    orc = O.PipoOracle(W, kv_bf16=True)      # the device's KV cache is bf16, as the workloads state
    rep = ParityReport()
    last = None
    for s in check:
        o, (lb, ld) = host[s]
        force = [int(o[0][i]) for i in seqs]
        if last is not None and s == last + 1:
            recs = orc.decode_step(in_pairs=[in_pair(s, i) for i in seqs], force_b=force)
        else:
            forced = [[in_pair(t, i) for t in range(1, s + 1)] for i in seqs] if s else None
            recs = orc.prefill(sub_prompts, sub_smp, force_b=force, forced_pairs=forced)
        last = s
        o_sub = tuple(np.asarray(a)[seqs] for a in o)
        compare_step(rep, f"step {s}", o_sub, lb, ld, recs, sub_smp, sub_seeds, s, mean_rel_tol, conf_tol,
                     max_abs_tol, seen=[set(x) for x in orc.seen], seq_ids=seqs)
    log(f"parity: steps {rep.steps} rows {rep.rows} max_abs {rep.max_abs:.3g} "
        f"max_mean_rel {rep.max_mean_rel:.3g} conf_err {rep.max_conf_err:.3g} "
        f"ambiguous tokens {rep.ambiguous_tokens} accepts {rep.ambiguous_accepts} "
        f"penalty-decisive {rep.penalty_decisive}")
    return rep, [(h[0], h[1][0] if h[1] else None, h[1][1] if h[1] else None) for h in host]


def _own_prompts(prompts, lens):
    return prompts if lens is None else [prompts[i][:int(n)] for i, n in enumerate(lens)]


def run_regular_parity(gpu_model, W, prompts, steps, smp, log=print, mean_rel_tol=LOGIT_MEAN_REL, lens=None):
    """Regular decoding: the GPU runs free for ``steps`` token steps after its
    prefill; the oracle replays the GPU's tokens as inputs.  Logits and tokens
    are held to the bounds of the pair path."""
    import torch

    B = prompts.shape[0]
    seeds = list(smp.seeds) if smp.seeds else [0] * B
    tokens = torch.from_numpy(np.ascontiguousarray(prompts, dtype=np.int32)).cuda()
    outs = [gpu_model.regular_prefill(tokens, smp.temperature, smp.top_p,
                                      seeds if smp.temperature > 0 else None, logits=True, top_k=smp.top_k,
                                      rep_penalty=smp.rep_penalty, lens=lens)]
    for _ in range(steps):
        outs.append(gpu_model.regular_step(logits=True))
    torch.cuda.synchronize()
    host = [(t.cpu().numpy(), lg.cpu().numpy()) for t, lg in outs]
    log(f"gpu done (regular): {B} sequences, {steps} steps")
    orc = O.RegularOracle(W, kv_bf16=True)
    rep = ParityReport()
    for s, (tok, lg) in enumerate(host):
        recs = orc.prefill(_own_prompts(prompts, lens), smp) if s == 0 else \
            orc.step(in_tok=[int(v) for v in host[s - 1][0]])
        rep.steps += 1
        for i, r in enumerate(recs):
            rep.rows += 1
            t = f"step {s} seq {i}"
            ma, mr = _row_err(lg[i], r["logits"])
            rep.max_abs = max(rep.max_abs, ma)
            rep.max_mean_rel = max(rep.max_mean_rel, mr)
            if ma > LOGIT_MAX_ABS or mr > mean_rel_tol:
                rep.failures.append(f"{t} logits: max_abs {ma:.3g} mean_rel {mr:.3g}")
            u = rspec.uniform_draw(seeds[i], s, 0) if smp.temperature > 0 else None
            _check_token(rep, t, int(tok[i]), r["tok"], lg[i], r["logits"], ma, smp, u, set(orc.seen[i]))
    log(f"regular parity: steps {rep.steps} rows {rep.rows} max_abs {rep.max_abs:.3g} "
        f"max_mean_rel {rep.max_mean_rel:.3g} ambiguous tokens {rep.ambiguous_tokens} "
        f"penalty-decisive {rep.penalty_decisive}")
    return rep, host
