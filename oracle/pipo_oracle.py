"""Float64 reference of the PIPO pair-in/pair-out path: TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may use this module.  It is deliberately plain: every function follows one
definition of the paper, with NumPy matrix products as the only library steps,
and there is no blocking or fusion beyond looping over independent heads and
query rows.

What the paper fixes (Sec. 3.1-3.2, App. B) and the readings taken where it is
silent:

* Pair-in (eq. 1, App. B.1 Table 4 "Linear"): ``z = W_c [x_a; x_b] + b_c``.
  The configurations fix the Linear variant.  A prompt of odd length gets the
  PAD token appended so that PAD sits at the odd slot of the last pair
  (App. C.1, random PAD injection); a prompt of n tokens gives ceil(n/2)
  latents.  PAD is the reserved last vocabulary row.
* Backbone (eq. 2): a dense pre-norm decoder over latent positions:
  ``x += W_o Attn(RoPE(W_q n), RoPE(W_k n), W_v n)`` with ``n = RMSNorm(x)``,
  grouped-query attention with query head ``h`` reading KV group
  ``h * n_kv // n_q``, scale ``1/sqrt(d)``, causal over latent positions;
  then ``x += W_down(SiLU(W_gate n) * W_up n)``.  RoPE uses the latent index
  as position, rotate-half pairs ``(j, j + d/2)`` and frequencies
  ``base**(-2j/d)``.  No biases, no QK norm.
* Pair-out (eqs. 3-5, App. B.2): ``h_b`` is the last residual state before the
  final norm; ``logits_b = E RMSNorm(h_b; g_f)`` with the LM head tied to the
  embedding E.  The MTP head is ``h_d = W_fc [RMSNorm(h_b; g_mh);
  RMSNorm(E[b]; g_me)]`` with W_fc: 2H -> H; the decoder layer App. B.2
  places after W_fc is omitted because the configurations fix a one-linear
  MTP head; ``logits_d = E RMSNorm(h_d; g_mo)``.
* Confidence (eq. 6, App. B.3): ``c = sigmoid(w_c . RMSNorm([h_b; h_d]; g_c))``;
  a single linear replaces App. B.3's two-layer MLP, as the configurations
  fix it.  The draft is accepted iff ``c >= tau`` (equality accepts), and the
  next input pair is ``(b, d)`` if accepted else ``(b, PAD)`` (Sec. 3.2).
* Paper-default heads (``ModelConfig.heads`` flags; the workloads use none):
  the MLP compressor of Table 4, read as ``E[a] + E[b] + W2 SiLU(W1 [E[a];
  E[b]])`` with an inner width of H: the paper initialises it to a + b by
  zeroing "the residual branch", so the printed W2 SiLU(W1 .) is that branch
  and a + b its skip path; the MTP head of App. B.2, W_fc followed by one
  decoder layer shaped like the backbone's, with its own KV cache over latent
  positions (RoPE at the latent index); during prefill, latent i < L-1 gets
  the prompt token that follows its pair (x^{2i+2}) as the MTP input token,
  the last latent the selected backbone token; the confidence head of App.
  B.3, ``sigmoid(W2 SiLU(W1 RMSNorm([h_b; h_d]; g_c)))`` without biases.
* KV cache storage: the workloads fix a bf16 KV cache (like the bf16
  weights, a storage format), so with ``kv_bf16`` the keys (after RoPE) and
  values are rounded to bf16 (nearest even) as they enter the cache; every
  other value stays float64.
* Token selection: greedy argmax with ties to the lowest id; or temperature
  plus nucleus (top-p): ``p = softmax(logits / T)``; the threshold
  ``theta*`` is the largest value among the ``p_j`` whose upper mass
  ``sum_{p_j >= theta} p_j`` reaches ``top_p`` (all tokens if none does);
  the nucleus is ``{j : p_j >= theta*}``, of mass ``M``; with ``t = u M`` the
  token is the first id, scanning ids upwards through the nucleus, at which
  the running mass exceeds ``t`` (the last nucleus id if rounding leaves
  none).  ``u`` is an input.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np
from threadpoolctl import threadpool_limits

from synth import rspec
from synth.configs import (ModelConfig, model_tensor_shapes, HEADS_MLP_COMPRESSOR, HEADS_MTP_LAYER,
                           HEADS_MLP_CONFIDENCE)

F64 = np.float64


# ---------------------------------------------------------------- primitives

def rms_norm(x, g, eps):
    """RMSNorm over the last axis: ``x / sqrt(mean(x^2) + eps) * g``."""
    x = np.asarray(x, dtype=F64)
    g = np.asarray(g, dtype=F64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(g, F64)


def rope_cos_sin(pos, head_dim, base):
    """cos/sin of the angles ``p * base**(-2j/d)``, j < d/2, for positions ``pos``."""
    half = head_dim // 2
    j = np.arange(half, dtype=F64)
    inv_freq = np.power(F64(base), -2.0 * j / head_dim)
    ang = np.asarray(pos, dtype=F64)[..., None] * inv_freq
    return np.cos(ang), np.sin(ang)


def apply_rope(x, cos, sin):
    """Rotate-half RoPE on the last axis of ``x`` (pairs ``j`` and ``j + d/2``).

    ``cos``/``sin`` broadcast against ``x[..., :d/2]``.
    """
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(u):
    """SiLU(u) = u / (1 + exp(-u))."""
    return u / (1.0 + np.exp(-u))


def to_bf16(x):
    """Nearest bf16 value (ties to even) of each element, via float32."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(F64)


def softmax(s, axis=-1):
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def prompt_pairs(tokens, pad_id):
    """Eq. 1's pairing of a prompt: PAD appended at the odd slot if n is odd."""
    t = [int(v) for v in tokens]
    if len(t) % 2:
        t.append(int(pad_id))
    return np.asarray(t, dtype=np.int64).reshape(-1, 2)


def compress(E, W_c, b_c, pairs):
    """Pair-in compressor (eq. 1, Linear variant): ``W_c [E[a]; E[b]] + b_c``."""
    pairs = np.asarray(pairs).reshape(-1, 2)
    cat = np.concatenate([E[pairs[:, 0]], E[pairs[:, 1]]], axis=-1)
    return cat @ np.asarray(W_c, F64).T + np.asarray(b_c, F64)


def compress_mlp(E, W1, W2, pairs):
    """Pair-in compressor, MLP variant (Table 4, with its a + b skip path):
    ``E[a] + E[b] + W2 SiLU(W1 [E[a]; E[b]])``."""
    pairs = np.asarray(pairs).reshape(-1, 2)
    a, b = E[pairs[:, 0]].astype(F64), E[pairs[:, 1]].astype(F64)
    cat = np.concatenate([a, b], axis=-1)
    return a + b + silu(cat @ np.asarray(W1, F64).T) @ np.asarray(W2, F64).T


def attention_decode(q, K, V):
    """One query position against a causal prefix, grouped-query.

    ``q``: [n_q, d]; ``K``, ``V``: [n_kv, T, d] holding positions 0..T-1 (the
    query's own position last).  Returns ``o`` [n_q, d] and the probability
    rows [n_q, T].
    """
    n_q, d = q.shape
    n_kv = K.shape[0]
    out = np.empty((n_q, d), dtype=F64)
    probs = np.empty((n_q, K.shape[1]), dtype=F64)
    for h in range(n_q):
        g = h * n_kv // n_q
        a = softmax(K[g] @ q[h] / np.sqrt(d))
        probs[h] = a
        out[h] = a @ V[g]
    return out, probs


def attention_causal(Q, K, V, block=256):
    """Causal grouped-query attention over a whole sequence.

    ``Q``: [n_q, T, d]; ``K``, ``V``: [n_kv, T, d].  Query row ``i`` attends to
    keys ``0..i``.  Rows are independent; they are processed ``block`` at a
    time only to bound memory.  Heads are independent too: they run
    concurrently on a thread pool, each head's arithmetic in one thread (its
    matrix products single-threaded), so the values do not depend on the
    number of threads.
    """
    n_q, T, d = Q.shape
    n_kv = K.shape[0]
    out = np.empty_like(Q, dtype=F64)

    def one_head(h):
        g = h * n_kv // n_q
        for r0 in range(0, T, block):
            r1 = min(T, r0 + block)
            s = Q[h, r0:r1] @ K[g, :r1].T / np.sqrt(d)
            rows = np.arange(r0, r1)[:, None]
            cols = np.arange(r1)[None, :]
            s = np.where(cols <= rows, s, -np.inf)
            out[h, r0:r1] = softmax(s) @ V[g, :r1]

    workers = max(1, min(n_q, 16, len(os.sched_getaffinity(0))))
    with threadpool_limits(1), ThreadPoolExecutor(workers) as ex:
        list(ex.map(one_head, range(n_q)))
    return out


def lm_logits(E, g, h, eps):
    """Tied LM head (eq. 3): ``E RMSNorm(h; g)``."""
    return rms_norm(h, g, eps) @ E.T


def mtp_hidden(W_fc, g_h, g_e, h_b, e_tok, eps):
    """MTP head (eq. 4, App. B.2, one linear): ``W_fc [RMSNorm(h_b); RMSNorm(x)]``."""
    u = np.concatenate([rms_norm(h_b, g_h, eps), rms_norm(e_tok, g_e, eps)], axis=-1)
    return u @ np.asarray(W_fc, F64).T


def confidence(w_c, g_c, h_b, h_d, eps):
    """Confidence head (eq. 6, App. B.3 as one linear): returns (s, sigmoid(s))."""
    s = rms_norm(np.concatenate([h_b, h_d], axis=-1), g_c, eps) @ np.asarray(w_c, F64)
    return s, 1.0 / (1.0 + np.exp(-s))


def confidence_mlp(W1, w2, g_c, h_b, h_d, eps):
    """Confidence head, App. B.3 form: s = w2 . SiLU(W1 RMSNorm([h_b; h_d]; g_c));
    returns (s, sigmoid(s))."""
    n = rms_norm(np.concatenate([h_b, h_d], axis=-1), g_c, eps)
    s = silu(n @ np.asarray(W1, F64).T) @ np.asarray(w2, F64)
    return s, 1.0 / (1.0 + np.exp(-s))


def gate(c, tau):
    """Accept the draft iff ``c >= tau`` (Sec. 3.2)."""
    return bool(c >= tau)


def select_greedy(logits):
    """argmax; exact ties go to the lowest id."""
    return int(np.argmax(logits))


def top_p_nucleus(logits, temperature, top_p):
    """``p = softmax(logits / T)`` and the nucleus threshold ``theta*`` (see
    header): the largest ``p_j`` whose upper mass reaches ``top_p``."""
    y = np.asarray(logits, F64) / F64(temperature)
    e = np.exp(y - np.max(y))
    p = e / np.sum(e)
    desc = np.sort(p)[::-1]
    upper = np.cumsum(desc)
    # mass(theta) counts every p_j >= theta, so a tie group contributes whole:
    # evaluate the cumulative sum at the last member of each value's group.
    last_of_group = np.searchsorted(-desc, -desc, side="right") - 1
    ok = upper[last_of_group] >= top_p
    theta = desc[np.argmax(ok)] if ok.any() else desc[-1]
    return p, theta


def select_top_p(logits, temperature, top_p, u):
    """Temperature + nucleus sampling by inverse CDF in id order (see header)."""
    p, theta = top_p_nucleus(logits, temperature, top_p)
    nucleus = np.nonzero(p >= theta)[0]
    mass = np.sum(p[nucleus])
    t = u * mass
    run = np.cumsum(p[nucleus])
    hit = np.nonzero(run > t)[0]
    return int(nucleus[hit[0]] if hit.size else nucleus[-1])


def repetition_penalty(logits, seen, theta):
    """CTRL-style repetition penalty: the logit of every token in ``seen`` is
    divided by ``theta`` when positive and multiplied by it otherwise."""
    y = np.asarray(logits, F64).copy()
    idx = np.fromiter(sorted(set(int(t) for t in seen)), dtype=np.int64)
    if idx.size and theta != 1.0:
        v = y[idx]
        y[idx] = np.where(v > 0, v / theta, v * theta)
    return y


def select_eval(logits, seen, temperature, top_k, top_p, theta, u):
    """The paper's evaluation sampler (Sec. 4, after Qwen3.5): repetition
    penalty, temperature, top-k (every value at least the k-th largest, ties
    kept), then top-p over the kept tokens and the inverse-CDF draw of
    ``select_top_p`` (ids of the kept set scanned upwards)."""
    return select_top_p(eval_scores(logits, seen, temperature, top_k, theta), 1.0, top_p, u)


def eval_scores(logits, seen, temperature, top_k, theta):
    """The evaluation sampler's scores before its top-p draw: penalised logits
    over the temperature, with every token below the k-th largest at -inf."""
    y = repetition_penalty(logits, seen, theta) / F64(temperature)
    if 0 < top_k < y.size:
        kth = np.sort(y)[::-1][top_k - 1]
        y = np.where(y >= kth, y, -np.inf)
    return y


# ------------------------------------------------------- OPD targets (App. C)

def opd_teacher_rows(tokens, pad_id):
    """PAD compaction of the OPD teacher pass (App. C, OPD training): the
    teacher runs on the trajectory with every PAD removed, and position t of
    the PAD-augmented trajectory takes the teacher row of the last non-PAD
    position at or before t (the row index is the count of non-PAD tokens in
    tokens[0..t], minus one; -1 where there is none yet)."""
    keep = np.asarray(tokens) != pad_id
    return np.cumsum(keep) - 1


def log_softmax_at(logits, y):
    """log p(y) for p = softmax(logits): logits[y] - log sum_j exp(logits[j])."""
    l = np.asarray(logits, F64)
    m = np.max(l)
    return float(l[y] - (m + np.log(np.sum(np.exp(l - m)))))


def opd_targets(logits_s, logits_t, rows, labels):
    """Per-position sampled reverse-KL term and confidence target (App. C):
    d_t = log p_s(y_t) - log p_t(y_t) with the teacher row rows[t], and
    alpha_t = exp(-max(d_t, 0)) = min(p_t(y_t) / p_s(y_t), 1).  Positions with
    a negative label are not scored (d = 0, alpha = 1).  Returns (d, alpha)."""
    T = len(labels)
    d = np.zeros(T)
    alpha = np.ones(T)
    for t in range(T):
        y = int(labels[t])
        if y < 0:
            continue
        d[t] = log_softmax_at(logits_s[t], y) - log_softmax_at(logits_t[int(rows[t])], y)
        alpha[t] = np.exp(-max(d[t], 0.0))
    return d, alpha


def opd_loss_sums(d, labels):
    """The sampled-KL loss's sums, kept apart for even positions (backbone
    head) and odd positions (MTP head): [sum_even, n_even, sum_odd, n_odd]
    over the scored positions."""
    d = np.asarray(d, F64)
    lab = np.asarray(labels)
    out = []
    for par in (0, 1):
        sel = (np.arange(len(lab)) % 2 == par) & (lab >= 0)
        out += [float(np.sum(d[sel])), float(np.count_nonzero(sel))]
    return out


# ------------------------------------------------------------------- weights

class OracleWeights:
    """All tensors of one model in logical ``[out][in]`` order.

    Values are held as float64, or as float32 when every value is exactly
    representable in it (bf16-valued weights of large models, to halve the
    memory); arithmetic is float64 either way (NumPy promotes the operands).
    """

    def __init__(self, cfg: ModelConfig, tensors: dict, storage=F64):
        self.cfg = cfg
        self.t = {k: np.asarray(v, dtype=storage) for k, v in tensors.items()}   # no copy if already

    @classmethod
    def generate(cls, cfg: ModelConfig, seed: int = 0, precision: str = "bf16", storage=F64):
        """R-spec weights; ``precision`` 'bf16' rounds every tensor to bf16 first."""
        tensors = {}
        for name, shape in model_tensor_shapes(cfg).items():
            tid = rspec.tensor_id(name)
            base = name.split(".")[-1]
            if base.startswith("g_"):
                v = rspec.gain_values(seed, tid, shape[0], cfg.gain_mode)
                if precision == "bf16":
                    v = rspec.bf16_round(v)
            else:
                v = rspec.weight_tensor(seed, tid, shape, bf16=precision == "bf16", dtype=storage)
            tensors[name] = v
        return cls(cfg, tensors, storage)

    def __getitem__(self, k):
        return self.t[k]

    def layer(self, li):
        return {k.split(".", 1)[1]: v for k, v in self.t.items() if k.startswith(f"l{li}.")}


# ------------------------------------------------------------------ backbone

def _layer_qkv(cfg, L, x, pos, kv_bf16=False):
    n = rms_norm(x, L["g_attn"], cfg.rms_eps)
    T = n.shape[0]
    q = (n @ L["wq"].T).reshape(T, cfg.n_q_heads, cfg.head_dim).transpose(1, 0, 2)
    k = (n @ L["wk"].T).reshape(T, cfg.n_kv_heads, cfg.head_dim).transpose(1, 0, 2)
    v = (n @ L["wv"].T).reshape(T, cfg.n_kv_heads, cfg.head_dim).transpose(1, 0, 2)
    cos, sin = rope_cos_sin(pos, cfg.head_dim, cfg.rope_base)
    q, k = apply_rope(q, cos, sin), apply_rope(k, cos, sin)
    if kv_bf16:
        k, v = to_bf16(k), to_bf16(v)
    return q, k, v


def _layer_ffn(cfg, L, x):
    n = rms_norm(x, L["g_ffn"], cfg.rms_eps)
    return x + (silu(n @ L["wgate"].T) * (n @ L["wup"].T)) @ L["wdown"].T


def backbone_full(W: OracleWeights, Z, kv_bf16=False, last_only=False):
    """Eq. 2 by brute force: all latent positions 0..T-1 from scratch.

    Returns the final residual states [T, H] (before the final norm) and the
    per-layer caches ``[(K, V)]`` with K, V of shape [n_kv, T, d].  With
    ``last_only`` the states returned are the last position's alone ([1, H]):
    the last layer then forms its keys and values at every position (the
    cache) but attends and runs its FFN for the last query only, which is
    all that position's state depends on.
    """
    cfg = W.cfg
    x = np.asarray(Z, F64).copy()
    T = x.shape[0]
    caches = []
    for li in range(cfg.n_layers):
        L = W.layer(li)
        q, k, v = _layer_qkv(cfg, L, x, np.arange(T), kv_bf16)
        if last_only and li == cfg.n_layers - 1:
            o, _ = attention_decode(q[:, -1], k, v)
            x = x[-1:] + o.reshape(1, cfg.q_dim) @ L["wo"].T
        else:
            o = attention_causal(q, k, v)
            x = x + o.transpose(1, 0, 2).reshape(T, cfg.q_dim) @ L["wo"].T
        x = _layer_ffn(cfg, L, x)
        caches.append((k, v))
    if last_only and cfg.n_layers == 0:
        x = x[-1:]
    return x, caches


def mtp_layer(W: OracleWeights):
    """Weights of the MTP head's decoder layer (App. B.2) as a layer dict."""
    return {k.split(".", 1)[1]: v for k, v in W.t.items() if k.startswith("mtp.")}


def layer_full(cfg, L, X, kv_bf16=False):
    """One decoder layer over positions 0..T-1 from scratch: (output, (K, V))."""
    x = np.asarray(X, F64).copy()
    T = x.shape[0]
    q, k, v = _layer_qkv(cfg, L, x, np.arange(T), kv_bf16)
    o = attention_causal(q, k, v)
    x = x + o.transpose(1, 0, 2).reshape(T, cfg.q_dim) @ L["wo"].T
    return _layer_ffn(cfg, L, x), (k, v)


def layer_step(cfg, L, x, pos, cache, kv_bf16=False):
    """One decoder layer for one position against ``cache`` = [K, V] (appended)."""
    x = np.asarray(x, F64).reshape(1, -1).copy()
    q, k, v = _layer_qkv(cfg, L, x, np.array([pos]), kv_bf16)
    cache[0] = np.concatenate([cache[0], k], axis=1)
    cache[1] = np.concatenate([cache[1], v], axis=1)
    o, _ = attention_decode(q[:, 0], cache[0], cache[1])
    x = x + o.reshape(1, cfg.q_dim) @ L["wo"].T
    return _layer_ffn(cfg, L, x)[0]


def backbone_step(W: OracleWeights, z, pos, caches, kv_bf16=False):
    """Eq. 2 incrementally: one latent at position ``pos`` against the cache.

    ``caches`` is a list per layer of ``[K, V]`` arrays [n_kv, pos, d]; the new
    key/value are appended in place.  Returns the final residual state [H].
    """
    cfg = W.cfg
    x = np.asarray(z, F64).reshape(1, -1).copy()
    for li in range(cfg.n_layers):
        L = W.layer(li)
        q, k, v = _layer_qkv(cfg, L, x, np.array([pos]), kv_bf16)
        K = np.concatenate([caches[li][0], k], axis=1)
        V = np.concatenate([caches[li][1], v], axis=1)
        caches[li][0], caches[li][1] = K, V
        o, _ = attention_decode(q[:, 0], K, V)
        x = x + o.reshape(1, cfg.q_dim) @ L["wo"].T
        x = _layer_ffn(cfg, L, x)
    return x[0]


# ------------------------------------------------------------------- session

@dataclass
class Sampling:
    tau: float
    temperature: float = 0.0       # <= 0: greedy
    top_p: float = 1.0
    seeds: tuple = ()              # one per sequence (sampling only)
    top_k: int = 0                 # 0: no top-k (sampling only)
    rep_penalty: float = 1.0       # 1: none (sampling only)


class PipoOracle:
    """A batch of independent PIPO sequences: prefill, then pair-decode steps.

    ``kv_bf16``: store keys and values in bf16 (the workloads' KV format)."""

    def __init__(self, W: OracleWeights, kv_bf16: bool = False):
        self.W = W
        self.cfg = W.cfg
        self.kv_bf16 = kv_bf16

    def _compress(self, pairs):
        W = self.W
        if self.cfg.heads & HEADS_MLP_COMPRESSOR:
            return compress_mlp(W["embed"], W["comp_w1"], W["comp_w2"], pairs)
        return compress(W["embed"], W["w_comp"], W["b_comp"], pairs)

    # heads: eqs. 3-6 and the gate, for one sequence; ``pos`` is h_b's latent index
    def heads(self, h_b, seq, step, pos, force_b=None):
        cfg, W, smp = self.cfg, self.W, self.sampling
        eps = cfg.rms_eps
        logits_b = lm_logits(W["embed"], W["g_final"], h_b, eps)
        b = self._select(logits_b, seq, step, 0)
        b_used = b if force_b is None else int(force_b)
        h_d = mtp_hidden(W["w_fc"], W["g_mtp_h"], W["g_mtp_e"], h_b, W["embed"][b_used], eps)
        if cfg.heads & HEADS_MTP_LAYER:
            h_d = layer_step(cfg, mtp_layer(W), h_d, pos, self.mtp_caches[seq], self.kv_bf16)
        logits_d = lm_logits(W["embed"], W["g_mtp_o"], h_d, eps)
        d = self._select(logits_d, seq, step, 1, extra=(b_used,))   # b precedes d in the output
        if cfg.heads & HEADS_MLP_CONFIDENCE:
            s, c = confidence_mlp(W["conf_w1"], W["conf_w2"], W["g_conf"], h_b, h_d, eps)
        else:
            s, c = confidence(W["w_conf"], W["g_conf"], h_b, h_d, eps)
        return dict(tok_b=b, tok_d=d, s=float(s), conf=float(c), accept=gate(c, smp.tau),
                    logits_b=logits_b, logits_d=logits_d, h_b=h_b, h_d=h_d)

    def _select(self, logits, seq, step, slot, extra=()):
        smp = self.sampling
        if smp.temperature <= 0:
            return select_greedy(logits)
        u = rspec.uniform_draw(smp.seeds[seq], step, slot)
        if smp.top_k or smp.rep_penalty != 1.0:
            return select_eval(logits, self.seen[seq] | set(extra), smp.temperature, smp.top_k, smp.top_p,
                               smp.rep_penalty, u)
        return select_top_p(logits, smp.temperature, smp.top_p, u)

    def prefill(self, prompts, sampling: Sampling, force_b=None, forced_pairs=None):
        """Compressed-prompt prefill of every sequence; returns the first pair.

        ``forced_pairs`` (one list per sequence, all of the same length k):
        the input pairs of the first k decode steps after the prefill,
        teacher-forced.  Their latents follow the prompt's, and eq. 2 is
        causal, so running the backbone over all of them at once gives the
        same states as the prefill followed by k steps; the records returned
        are then those of step k (sampler step index k), and the session
        continues from there."""
        self.sampling = sampling
        W, cfg = self.W, self.cfg
        self.caches, self.length, self.step_idx, self.next_pairs, self.mtp_caches = [], [], [], [], []
        prompts = [np.asarray(p) for p in prompts]   # a ragged batch: prompts of their own lengths
        self.seen = [set(int(t) for t in p) for p in prompts]   # tokens the penalty applies to
        nforced = 0 if forced_pairs is None else len(forced_pairs[0])
        out = []
        for i, prompt in enumerate(prompts):
            pairs = prompt_pairs(prompt, cfg.pad_id)
            if nforced:
                fp = np.asarray(forced_pairs[i], dtype=np.int64).reshape(nforced, 2)
                for pair in fp:
                    self._emitted(i, pair)
                pairs = np.concatenate([pairs, fp])
            Z = self._compress(pairs)
            # the heads read the last latent only; the MTP layer of App. B reads every latent's state
            X, caches = backbone_full(W, Z, self.kv_bf16, last_only=not cfg.heads & HEADS_MTP_LAYER)
            self.caches.append([[k, v] for k, v in caches])
            self.length.append(len(pairs))
            if cfg.heads & HEADS_MTP_LAYER:
                # latents 0..L-2 take the prompt token after their pair as the MTP token
                L = len(pairs)
                U = np.stack([mtp_hidden(W["w_fc"], W["g_mtp_h"], W["g_mtp_e"], X[j], W["embed"][pairs[j + 1, 0]],
                                         cfg.rms_eps) for j in range(L - 1)]) if L > 1 else np.zeros((0, cfg.hidden))
                if L > 1:
                    _, (k, v) = layer_full(cfg, mtp_layer(W), U, self.kv_bf16)
                else:
                    k = np.zeros((cfg.n_kv_heads, 0, cfg.head_dim))
                    v = np.zeros((cfg.n_kv_heads, 0, cfg.head_dim))
                self.mtp_caches.append([k, v])
            rec = self.heads(X[-1], i, nforced, len(pairs) - 1, None if force_b is None else force_b[i])
            out.append(rec)
            self.step_idx.append(nforced + 1)
            self.next_pairs.append(self._next_pair(rec))
        return out

    def _next_pair(self, rec):
        return (rec["tok_b"], rec["tok_d"] if rec["accept"] else self.cfg.pad_id)

    def _emitted(self, seq, pair):
        """The tokens a pair step emitted, (b, d) or (b, PAD), join the penalised
        set when they come back as the next input pair (PAD never does)."""
        self.seen[seq].add(int(pair[0]))
        if int(pair[1]) != self.cfg.pad_id:
            self.seen[seq].add(int(pair[1]))

    def decode_step(self, in_pairs=None, force_b=None):
        """One pair step for every sequence; ``in_pairs`` teacher-forces the input."""
        W = self.W
        out = []
        for i in range(len(self.caches)):
            pair = self.next_pairs[i] if in_pairs is None else tuple(int(v) for v in in_pairs[i])
            self._emitted(i, pair)
            z = self._compress(np.array([pair]))[0]
            pos = self.length[i]
            h_b = backbone_step(W, z, pos, self.caches[i], self.kv_bf16)
            self.length[i] += 1
            rec = self.heads(h_b, i, self.step_idx[i], pos, None if force_b is None else force_b[i])
            out.append(rec)
            self.step_idx[i] += 1
            self.next_pairs[i] = self._next_pair(rec)
        return out


class RegularOracle:
    """Regular decoding on the same backbone, the baseline of Sec. 4.3 (Fig. 4).

    Every token is one position: the backbone input is ``E[t]`` itself (no
    compressor), the next token is selected from ``E RMSNorm(h; g_f)`` (eq. 3
    on the last position) and fed back; neither the MTP nor the confidence
    head runs.  Top-p draws use slot 0 of each step, step 0 being the prefill.
    """

    def __init__(self, W: OracleWeights, kv_bf16: bool = False):
        self.W = W
        self.cfg = W.cfg
        self.kv_bf16 = kv_bf16

    def _select(self, logits, seq, step):
        smp = self.sampling
        if smp.temperature <= 0:
            return select_greedy(logits)
        u = rspec.uniform_draw(smp.seeds[seq], step, 0)
        if smp.top_k or smp.rep_penalty != 1.0:
            return select_eval(logits, self.seen[seq], smp.temperature, smp.top_k, smp.top_p, smp.rep_penalty, u)
        return select_top_p(logits, smp.temperature, smp.top_p, u)

    def _head(self, h, seq, step):
        logits = lm_logits(self.W["embed"], self.W["g_final"], h, self.cfg.rms_eps)
        return dict(tok=self._select(logits, seq, step), logits=logits, h=h)

    def prefill(self, prompts, sampling: Sampling):
        """The prompt's n tokens as n positions; returns the first generated token."""
        self.sampling = sampling
        W = self.W
        self.caches, self.length, self.step_idx, self.next_tok = [], [], [], []
        prompts = [np.asarray(p) for p in prompts]
        self.seen = [set(int(t) for t in p) for p in prompts]
        out = []
        for i, prompt in enumerate(prompts):
            X, caches = backbone_full(W, W["embed"][np.asarray(prompt)], self.kv_bf16, last_only=True)
            self.caches.append([[k, v] for k, v in caches])
            self.length.append(len(prompt))
            rec = self._head(X[-1], i, 0)
            out.append(rec)
            self.step_idx.append(1)
            self.next_tok.append(rec["tok"])
        return out

    def step(self, in_tok=None):
        """One token per sequence; ``in_tok`` teacher-forces the input."""
        W = self.W
        out = []
        for i in range(len(self.caches)):
            t = self.next_tok[i] if in_tok is None else int(in_tok[i])
            self.seen[i].add(t)
            h = backbone_step(W, W["embed"][t], self.length[i], self.caches[i], self.kv_bf16)
            self.length[i] += 1
            rec = self._head(h, i, self.step_idx[i])
            out.append(rec)
            self.step_idx[i] += 1
            self.next_tok[i] = rec["tok"]
        return out
