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
* sampled tokens: equal, or else the oracle's selection rule applied to the
  GPU's logits must give the GPU token (a boundary case moved by logit error);
  the evaluation sampler's rule takes the oracle's penalised set of that step.
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
        if again == gpu_tok:
            rep.ambiguous_tokens += 1
            return
        rep.failures.append(f"{tag}: sampled {gpu_tok}, oracle {ref_tok}, rule on GPU logits {again}")


def compare_step(rep, tag, out_np, lb, ld, recs, smp, seeds, step, mean_rel_tol=LOGIT_MEAN_REL, conf_tol=CONF_TOL,
                 max_abs_tol=LOGIT_MAX_ABS, seen=None):
    tok_b, tok_d, conf, acc = out_np
    rep.steps += 1
    for i, r in enumerate(recs):
        rep.rows += 1
        t = f"{tag} seq {i}"
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
               max_abs_tol=LOGIT_MAX_ABS, lens=None):
    """Run the GPU free for ``steps`` pair steps after prefill; replay on the
    oracle.  ``lens``: a ragged batch, sequence i's prompt being the first
    lens[i] tokens of row i of ``prompts``."""
    import torch
    from paper_2605_27255_amd import unpack_pairs

    B = prompts.shape[0]
    seeds = list(smp.seeds) if smp.seeds else [0] * B
    tokens = torch.from_numpy(np.ascontiguousarray(prompts, dtype=np.int32)).cuda()
    outs = [gpu_model.prefill(tokens, smp.tau, smp.temperature, smp.top_p,
                              seeds if smp.temperature > 0 else None, logits=True, top_k=smp.top_k,
                              rep_penalty=smp.rep_penalty, lens=lens)]
    for _ in range(steps):
        outs.append(gpu_model.decode_step(logits=True))
    torch.cuda.synchronize()
    host = [(unpack_pairs(o), lb.cpu().numpy(), ld.cpu().numpy()) for o, lb, ld in outs]
    log(f"gpu done: {B} sequences, {steps} steps")
    orc = O.PipoOracle(W, kv_bf16=True)      # the device's KV cache is bf16, as the workloads state
    rep = ParityReport()
    for s, (o, lb, ld) in enumerate(host):
        force = [int(v) for v in o[0]]
        if s == 0:
            recs = orc.prefill(_own_prompts(prompts, lens), smp, force_b=force)
        else:
            prev = host[s - 1][0]
            pairs = [(int(prev[0][i]), int(prev[1][i]) if prev[3][i] else W.cfg.pad_id) for i in range(B)]
            recs = orc.decode_step(in_pairs=pairs, force_b=force)
        compare_step(rep, f"step {s}", o, lb, ld, recs, smp, seeds, s, mean_rel_tol, conf_tol, max_abs_tol,
                     seen=[set(x) for x in orc.seen])
    log(f"parity: steps {rep.steps} rows {rep.rows} max_abs {rep.max_abs:.3g} "
        f"max_mean_rel {rep.max_mean_rel:.3g} conf_err {rep.max_conf_err:.3g} "
        f"ambiguous tokens {rep.ambiguous_tokens} accepts {rep.ambiguous_accepts} "
        f"penalty-decisive {rep.penalty_decisive}")
    return rep, host


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
