"""Pins of the oracle against facts the paper and the mathematics fix.

Each test checks one part of the oracle against something other than itself:
published generator outputs, library routines that implement a textbook
definition (PyTorch CPU float64), closed forms, invariants, brute force, and
the paper's stated rules (latent length, PAD slot, gate at equality, tau
extremes).  None of these tests needs a GPU.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from synth import rspec
from synth.configs import ModelConfig, TINY
from oracle import pipo_oracle as O

SMALL = ModelConfig(n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                    ffn=96, vocab=64, rope_base=1e4, rms_eps=1e-6, gain_mode=1)


@pytest.fixture(scope="module")
def small_w():
    return O.OracleWeights.generate(SMALL, seed=3, precision="bf16")


# ------------------------------------------------------------ input generator

def test_splitmix64_published_outputs():
    # SplitMix64 seeded with 0 returns these three words first (published
    # reference outputs of the generator).
    g = 0x9E3779B97F4A7C15
    outs = [rspec.splitmix64((k * g) & ((1 << 64) - 1)) for k in range(3)]
    assert outs == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_weight_distribution_moments():
    w = rspec.weight_values(0, 0, 0, 1 << 21).astype(np.float64)
    assert abs(w.mean()) < 1e-4
    assert abs(w.std() - 0.02) < 0.0002                        # sd within 1%
    kurt = ((w - w.mean()) ** 4).mean() / w.var() ** 2 - 3.0
    assert abs(kurt - (-0.3)) < 0.03                            # Irwin-Hall(4)
    assert np.abs(w).max() <= 2 * 0.02 * np.sqrt(3) + 1e-7


def test_weight_values_are_position_addressable():
    a = rspec.weight_values(5, 7, 0, 1000)
    b = rspec.weight_values(5, 7, 400, 100)
    np.testing.assert_array_equal(a[400:500], b)
    assert not np.array_equal(rspec.weight_values(5, 8, 0, 100), a[:100])


def test_bf16_rounding_matches_torch():
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -3.14159,
                  1e-30, 65504.0, 0.02], dtype=np.float32)
    x = np.concatenate([x, rspec.weight_values(1, 2, 0, 4096)])
    ours = rspec.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    assert rspec.bf16_round(np.float32([1.0 + 2 ** -8]))[0] == 1.0          # tie to even
    assert rspec.bf16_round(np.float32([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6


def test_prompt_tokens_never_pad_and_roughly_uniform():
    t = rspec.prompt_tokens(2, 200000, 64)
    assert t.min() >= 0 and t.max() <= 62                      # PAD id 63 never drawn
    counts = np.bincount(t.ravel(), minlength=63)
    exp = t.size / 63
    chi2 = ((counts - exp) ** 2 / exp).sum()
    assert chi2 < 150                                          # 62 dof
    assert not np.array_equal(t[0], t[1])


# ---------------------------------------------------------------- primitives

def test_rms_norm_matches_torch_and_is_scale_invariant():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 64))
    g = rng.standard_normal(64)
    ref = F.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(O.rms_norm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.rms_norm(7.5 * x, g, 0.0), O.rms_norm(x, g, 0.0), rtol=1e-12)


def test_oracle_bf16_rounding_matches_torch():
    x = np.random.default_rng(15).standard_normal(10000) * np.exp(np.random.default_rng(16).uniform(-20, 20, 10000))
    x = np.concatenate([x, [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, 0.0]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.to_bf16(x), ref)


def test_kv_bf16_rounds_exactly_the_cached_keys_and_values(small_w):
    """With the bf16 KV cache, the cached K and V are the bf16 roundings of the
    float64 ones, and the rounding changes the outputs only slightly."""
    Z = np.random.default_rng(17).standard_normal((7, SMALL.hidden))
    X, c64 = O.backbone_full(small_w, Z)
    Xb, cb = O.backbone_full(small_w, Z, kv_bf16=True)
    np.testing.assert_array_equal(cb[0][0], O.to_bf16(c64[0][0]))   # layer 0 sees identical inputs
    np.testing.assert_array_equal(cb[0][1], O.to_bf16(c64[0][1]))
    assert 0 < np.abs(Xb - X).max() < 1e-2 * np.abs(X).max()
    # incremental decode with the bf16 cache equals brute force with it
    caches = [[np.zeros((SMALL.n_kv_heads, 0, SMALL.head_dim))] * 2 for _ in range(SMALL.n_layers)]
    for p in range(7):
        h = O.backbone_step(small_w, Z[p], p, caches, kv_bf16=True)
    np.testing.assert_allclose(h, Xb[-1], rtol=1e-10, atol=1e-12)


def test_silu_matches_torch():
    u = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(O.silu(u), F.silu(torch.from_numpy(u)).numpy(), rtol=1e-13, atol=1e-300)


def test_rope_identities():
    rng = np.random.default_rng(1)
    d = 16
    x = rng.standard_normal(d)
    c0, s0 = O.rope_cos_sin(np.array([0]), d, 1e4)
    np.testing.assert_array_equal(O.apply_rope(x[None], c0, s0)[0], x)      # p = 0
    c, s = O.rope_cos_sin(np.array([37]), d, 1e4)
    y = O.apply_rope(x[None], c, s)[0]
    assert abs(np.linalg.norm(y) - np.linalg.norm(x)) < 1e-12                # rotation
    # complex form: (x_j + i x_{j+d/2}) * exp(i p w_j)
    zc = (x[:d // 2] + 1j * x[d // 2:]) * np.exp(1j * 37 * 1e4 ** (-2 * np.arange(d // 2) / d))
    np.testing.assert_allclose(y, np.concatenate([zc.real, zc.imag]), atol=1e-12)
    # q_m . k_n depends only on m - n
    q, k = rng.standard_normal(d), rng.standard_normal(d)

    def dot(m, n):
        cm, sm_ = O.rope_cos_sin(np.array([m]), d, 1e4)
        cn, sn = O.rope_cos_sin(np.array([n]), d, 1e4)
        return O.apply_rope(q[None], cm, sm_)[0] @ O.apply_rope(k[None], cn, sn)[0]
    assert abs(dot(10, 3) - dot(107, 100)) < 1e-10
    assert abs(dot(10, 3) - dot(3, 10)) > 1e-6                               # not symmetric


def test_attention_matches_torch_sdpa_gqa():
    rng = np.random.default_rng(2)
    n_q, n_kv, T, d = 8, 2, 23, 16
    Q = rng.standard_normal((n_q, T, d))
    K = rng.standard_normal((n_kv, T, d))
    V = rng.standard_normal((n_kv, T, d))
    rep = n_q // n_kv
    ref = F.scaled_dot_product_attention(
        torch.from_numpy(Q)[None], torch.from_numpy(K).repeat_interleave(rep, 0)[None],
        torch.from_numpy(V).repeat_interleave(rep, 0)[None], is_causal=True)[0].numpy()
    np.testing.assert_allclose(O.attention_causal(Q, K, V, block=7), ref, rtol=1e-11, atol=1e-12)
    # the decode form at the last position agrees with the causal form
    o, probs = O.attention_decode(Q[:, -1], K, V)
    np.testing.assert_allclose(o, ref[:, -1], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(probs.sum(axis=1), 1.0, atol=1e-12)          # normalised


def test_attention_single_key_and_zero_query():
    rng = np.random.default_rng(3)
    K = rng.standard_normal((2, 1, 8))
    V = rng.standard_normal((2, 1, 8))
    o, _ = O.attention_decode(rng.standard_normal((4, 8)), K, V)
    np.testing.assert_array_equal(o[:2], np.repeat(V[0], 2, axis=0))       # exactly v_0
    np.testing.assert_array_equal(o[2:], np.repeat(V[1], 2, axis=0))
    K = rng.standard_normal((2, 9, 8))
    V = rng.standard_normal((2, 9, 8))
    o, _ = O.attention_decode(np.zeros((4, 8)), K, V)                        # W_q = 0
    np.testing.assert_allclose(o[0], V[0].mean(axis=0), rtol=1e-12)
    np.testing.assert_allclose(o[3], V[1].mean(axis=0), rtol=1e-12)


def test_gqa_group_mapping():
    # value rows of group g are constant g: head h must return h * n_kv // n_q
    n_q, n_kv, T, d = 12, 3, 5, 4
    V = np.stack([np.full((T, d), float(g)) for g in range(n_kv)])
    K = np.random.default_rng(4).standard_normal((n_kv, T, d))
    o, _ = O.attention_decode(np.ones((n_q, d)), K, V)
    np.testing.assert_allclose(o[:, 0], [h // 4 for h in range(n_q)], atol=1e-12)


# ------------------------------------------------------- pairs and compressor

def test_prompt_pairs_pad_at_odd_slot_and_latent_length():
    for n in (1, 2, 7, 8, 63, 64):
        p = O.prompt_pairs(list(range(10, 10 + n)), pad_id=99)
        assert p.shape == (-(-n // 2), 2)                                   # ceil(n/2)
        assert p[0, 0] == 10
        if n % 2:
            assert p[-1, 1] == 99 and p[-1, 0] == 10 + n - 1
        assert (p[:, 0] != 99).all()


def test_compressor_closed_forms():
    rng = np.random.default_rng(5)
    H, V = 6, 10
    E = rng.standard_normal((V, H))
    W = np.concatenate([np.eye(H), np.eye(H)], axis=1)                      # f([a;b]) = a + b
    pairs = np.array([[1, 2], [3, 9]])
    np.testing.assert_allclose(O.compress(E, W, np.zeros(H), pairs), E[[1, 3]] + E[[2, 9]], rtol=1e-15)
    b = rng.standard_normal(H)
    np.testing.assert_allclose(O.compress(E, W, b, pairs), E[[1, 3]] + E[[2, 9]] + b, rtol=1e-14)
    E[9] = 0.0                                                              # PAD row zero
    np.testing.assert_allclose(O.compress(E, W, np.zeros(H), [[3, 9]])[0], E[3], rtol=1e-15)
    # the two halves of W_c act on the first and second token respectively
    W2 = np.concatenate([np.eye(H), 2 * np.eye(H)], axis=1)
    np.testing.assert_allclose(O.compress(E, W2, np.zeros(H), [[1, 2]])[0], E[1] + 2 * E[2], rtol=1e-14)


# ------------------------------------------------------------------- backbone

def test_brute_force_equals_incremental(small_w):
    rng = np.random.default_rng(6)
    Z = rng.standard_normal((13, SMALL.hidden))
    X_full, caches_full = O.backbone_full(small_w, Z)
    caches = [[np.zeros((SMALL.n_kv_heads, 0, SMALL.head_dim))] * 2 for _ in range(SMALL.n_layers)]
    for p in range(13):
        h = O.backbone_step(small_w, Z[p], p, caches)
        np.testing.assert_allclose(h, X_full[p], rtol=1e-10, atol=1e-12)
    for li in range(SMALL.n_layers):
        np.testing.assert_allclose(caches[li][0], caches_full[li][0], rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(caches[li][1], caches_full[li][1], rtol=1e-12, atol=1e-14)


def test_last_only_backbone_is_the_full_pass_at_the_last_position(small_w):
    """The last-position form of the brute-force pass: the same state at the
    last latent and the same caches, for one, several and zero layers."""
    rng = np.random.default_rng(5)
    Z = rng.standard_normal((13, SMALL.hidden))
    X, caches = O.backbone_full(small_w, Z, kv_bf16=True)
    Xl, caches_l = O.backbone_full(small_w, Z, kv_bf16=True, last_only=True)
    assert Xl.shape == (1, SMALL.hidden)
    np.testing.assert_allclose(Xl[0], X[-1], rtol=1e-12, atol=1e-13)
    for (k, v), (kl, vl) in zip(caches, caches_l):
        np.testing.assert_array_equal(k, kl)
        np.testing.assert_array_equal(v, vl)
    W1 = O.OracleWeights.generate(SMALL.with_layers(1), seed=3, precision="bf16")
    X, _ = O.backbone_full(W1, Z)
    np.testing.assert_allclose(O.backbone_full(W1, Z, last_only=True)[0][0], X[-1], rtol=1e-12, atol=1e-13)
    W0 = O.OracleWeights.generate(SMALL.with_layers(0), seed=3, precision="bf16")
    np.testing.assert_array_equal(O.backbone_full(W0, Z, last_only=True)[0][0], Z[-1])


def test_attention_threads_do_not_change_values():
    """Heads run concurrently; each head's values are those of a plain
    single-head evaluation."""
    rng = np.random.default_rng(6)
    Q, K, V = rng.standard_normal((6, 300, 16)), rng.standard_normal((2, 300, 16)), rng.standard_normal((2, 300, 16))
    out = O.attention_causal(Q, K, V)
    for h in range(6):
        np.testing.assert_array_equal(out[h:h + 1], O.attention_causal(Q[h:h + 1], K[h // 3:h // 3 + 1],
                                                                       V[h // 3:h // 3 + 1]))


def test_causality(small_w):
    rng = np.random.default_rng(7)
    Z = rng.standard_normal((9, SMALL.hidden))
    X, _ = O.backbone_full(small_w, Z)
    Z2 = Z.copy()
    Z2[6:] += rng.standard_normal((3, SMALL.hidden))
    X2, _ = O.backbone_full(small_w, Z2)
    np.testing.assert_array_equal(X2[:6], X[:6])                            # bit-unchanged
    assert np.abs(X2[6:] - X[6:]).max() > 1e-3


def test_zero_layers_is_identity():
    cfg = SMALL.with_layers(0)
    W = O.OracleWeights.generate(cfg, seed=1)
    Z = np.random.default_rng(8).standard_normal((4, cfg.hidden))
    X, _ = O.backbone_full(W, Z)
    np.testing.assert_array_equal(X, Z)


def test_layer_matches_torch_modules(small_w):
    """One decoder layer, rebuilt from torch library modules in float64."""
    cfg = SMALL
    L = small_w.layer(0)
    T = 11
    x = np.random.default_rng(9).standard_normal((T, cfg.hidden))
    X1, _ = O.backbone_full(O.OracleWeights(cfg.with_layers(1), {**{k: v for k, v in small_w.t.items() if not k.startswith("l1.")}}), x)
    t = {k: torch.from_numpy(v) for k, v in L.items()}
    xt = torch.from_numpy(x)
    n = F.rms_norm(xt, (cfg.hidden,), t["g_attn"], eps=cfg.rms_eps)
    q = F.linear(n, t["wq"]).view(T, cfg.n_q_heads, cfg.head_dim).transpose(0, 1)
    k = F.linear(n, t["wk"]).view(T, cfg.n_kv_heads, cfg.head_dim).transpose(0, 1)
    v = F.linear(n, t["wv"]).view(T, cfg.n_kv_heads, cfg.head_dim).transpose(0, 1)
    half = cfg.head_dim // 2
    inv = cfg.rope_base ** (-torch.arange(half, dtype=torch.float64) * 2 / cfg.head_dim)
    ang = torch.arange(T, dtype=torch.float64)[:, None] * inv
    cos, sin = torch.cat([ang.cos(), ang.cos()], -1), torch.cat([ang.sin(), ang.sin()], -1)

    def rot(u):
        return torch.cat([-u[..., half:], u[..., :half]], -1)
    q, k = q * cos + rot(q) * sin, k * cos + rot(k) * sin
    rep = cfg.n_q_heads // cfg.n_kv_heads
    o = F.scaled_dot_product_attention(q[None], k.repeat_interleave(rep, 0)[None],
                                       v.repeat_interleave(rep, 0)[None], is_causal=True)[0]
    xt = xt + F.linear(o.transpose(0, 1).reshape(T, -1), t["wo"])
    n = F.rms_norm(xt, (cfg.hidden,), t["g_ffn"], eps=cfg.rms_eps)
    xt = xt + F.linear(F.silu(F.linear(n, t["wgate"])) * F.linear(n, t["wup"]), t["wdown"])
    np.testing.assert_allclose(X1, xt.numpy(), rtol=1e-10, atol=1e-12)


# ---------------------------------------------------------------------- heads

def test_tied_head_closed_form():
    H = 8
    E = 0.5 * np.eye(H)
    h = np.random.default_rng(10).standard_normal(H)
    logits = O.lm_logits(E, np.ones(H), h, 0.0)
    np.testing.assert_allclose(logits, 0.5 * h / np.sqrt(np.mean(h * h)), rtol=1e-14)
    assert O.select_greedy(logits) == int(np.argmax(h))


def test_mtp_closed_forms_and_dependence_on_backbone_token():
    rng = np.random.default_rng(11)
    H, V = 8, 12
    E = rng.standard_normal((V, H))
    h_b = rng.standard_normal(H)
    g = rng.standard_normal(H)
    I, Z = np.eye(H), np.zeros((H, H))
    np.testing.assert_allclose(O.mtp_hidden(np.hstack([I, Z]), g, g, h_b, E[3], 1e-6),
                               O.rms_norm(h_b, g, 1e-6), rtol=1e-14)
    np.testing.assert_allclose(O.mtp_hidden(np.hstack([Z, I]), g, g, h_b, E[3], 1e-6),
                               O.rms_norm(E[3], g, 1e-6), rtol=1e-14)


def test_session_mtp_reads_the_backbone_token(small_w):
    cfg = SMALL
    prompt = rspec.prompt_tokens(1, 10, cfg.vocab)
    smp = O.Sampling(tau=0.5)
    a = O.PipoOracle(small_w).prefill(prompt, smp)[0]
    W2 = O.OracleWeights(cfg, dict(small_w.t))
    W2.t["embed"] = small_w["embed"].copy()
    W2.t["embed"][a["tok_b"]] *= -1.0            # only E[b]'s row changes ...
    b = O.PipoOracle(W2).prefill(prompt, smp)[0]
    # ... the backbone logits move only at that row of the tied head
    diff = np.abs(b["logits_b"] - a["logits_b"])
    assert diff[a["tok_b"]] > 0
    np.testing.assert_allclose(np.delete(diff, a["tok_b"]), 0.0, atol=1e-9)
    assert np.abs(b["logits_d"] - a["logits_d"]).max() > 1e-3


def test_confidence_closed_form_and_gate_rule():
    rng = np.random.default_rng(12)
    H = 6
    h_b, h_d = rng.standard_normal(H), rng.standard_normal(H)
    w = np.zeros(2 * H)
    w[H + 2] = 1.0
    s, c = O.confidence(w, np.ones(2 * H), h_b, h_d, 0.0)
    cat = np.concatenate([h_b, h_d])
    assert abs(s - cat[H + 2] / np.sqrt(np.mean(cat * cat))) < 1e-14
    assert abs(c - 1 / (1 + np.exp(-s))) < 1e-15
    assert O.gate(c, c)                            # equality accepts
    assert O.gate(c, 0.0)                          # tau = 0: always accept
    assert not O.gate(c, 1.0 + 1e-9)               # tau > 1: never accept
    assert not O.gate(c, np.nextafter(c, 2.0))


# -------------------------------------------------------------------- sampler

def test_top_p_worked_example():
    p = np.array([0.5, 0.3, 0.15, 0.05])
    logits = np.log(p)
    # top_p 0.8 -> nucleus {0, 1}, mass 0.8; u 0.7 -> t 0.56 -> running 0.5, 0.8.
    # The mass of {0, 1} equals top_p exactly, so the example is posed with
    # top_p a hair below 0.8: exp/log rounding must not decide the nucleus.
    tp = 0.8 - 1e-9
    assert O.select_top_p(logits, 1.0, tp, 0.7) == 1
    assert O.select_top_p(logits, 1.0, tp, 0.6) == 0           # t = 0.48 < 0.5
    assert O.select_top_p(logits, 1.0, 0.81, 0.999) == 2       # nucleus grows to {0,1,2}
    assert O.select_top_p(logits, 1.0, 1.0, 0.999) == 3


def test_top_p_limits_reduce_to_greedy():
    logits = np.random.default_rng(13).standard_normal(50)
    g = O.select_greedy(logits)
    for u in (0.0, 0.3, 0.9999):
        assert O.select_top_p(logits, 1.0, 1e-9, u) == g
        assert O.select_top_p(logits, 1e-4, 0.95, u) == g


def test_top_p_tie_group_is_whole():
    logits = np.log(np.array([0.3, 0.3, 0.3, 0.1]))
    # top_p 0.35 is reached inside the tie group: all three tied ids are in N
    picks = {O.select_top_p(logits, 1.0, 0.35, u) for u in np.linspace(0, 0.999, 30)}
    assert picks == {0, 1, 2}


def test_top_p_inverse_cdf_distribution():
    rng = np.random.default_rng(14)
    logits = rng.standard_normal(8) * 1.5
    T, top_p = 0.7, 0.9
    p = np.exp(logits / T - np.max(logits / T))
    p /= p.sum()
    order = np.argsort(-p)
    keep = order[: np.argmax(np.cumsum(p[order]) >= top_p) + 1]
    target = np.zeros(8)
    target[keep] = p[keep] / p[keep].sum()
    N = 20000
    draws = [O.select_top_p(logits, T, top_p, (i + 0.5) / N) for i in range(N)]
    freq = np.bincount(draws, minlength=8) / N
    np.testing.assert_allclose(freq, target, atol=2.0 / N)


def test_greedy_ties_lowest_id():
    assert O.select_greedy(np.array([0.1, 0.7, 0.2, 0.7])) == 1


# --------------------------------------------------------------- the session

def test_session_latent_length_and_pair_feedback(small_w):
    cfg = SMALL
    for tau in (0.0, 2.0):
        orc = O.PipoOracle(small_w)
        out = orc.prefill(rspec.prompt_tokens(2, 11, cfg.vocab), O.Sampling(tau=tau))
        assert orc.length == [6, 6]                                         # ceil(11/2)
        for k in range(3):
            prev = orc.next_pairs[0]
            rec = out[0]
            expect = (rec["tok_b"], rec["tok_d"] if tau <= rec["conf"] else cfg.pad_id)
            assert prev == expect
            assert rec["accept"] == (tau == 0.0)
            out = orc.decode_step()
            assert orc.length == [6 + k + 1] * 2                           # +1 per step


def test_session_decode_equals_brute_force(small_w):
    """Prefill + decode steps reproduce a from-scratch pass over all latents."""
    cfg = SMALL
    prompt = rspec.prompt_tokens(1, 9, cfg.vocab)
    orc = O.PipoOracle(small_w)
    recs = [orc.prefill(prompt, O.Sampling(tau=0.5))[0]]
    pairs = [tuple(p) for p in O.prompt_pairs(prompt[0], cfg.pad_id)]
    for _ in range(4):
        pairs.append(orc.next_pairs[0])
        recs.append(orc.decode_step()[0])
    Z = O.compress(small_w["embed"], small_w["w_comp"], small_w["b_comp"], np.array(pairs))
    X, _ = O.backbone_full(small_w, Z)
    for k, rec in enumerate(recs):
        np.testing.assert_allclose(rec["h_b"], X[len(pairs) - len(recs) + k], rtol=1e-10, atol=1e-12)


def test_teacher_forcing_reproduces_free_run(small_w):
    cfg = SMALL
    prompt = rspec.prompt_tokens(2, 8, cfg.vocab)
    smp = O.Sampling(tau=0.4, temperature=0.8, top_p=0.9, seeds=(1000, 1001))
    a = O.PipoOracle(small_w)
    a.prefill(prompt, smp)
    b = O.PipoOracle(small_w)
    b.prefill(prompt, smp)
    for _ in range(3):
        forced = [a.next_pairs[i] for i in range(2)]
        ra, rb = a.decode_step(), b.decode_step(in_pairs=forced)
        for x, y in zip(ra, rb):
            assert (x["tok_b"], x["tok_d"], x["accept"]) == (y["tok_b"], y["tok_d"], y["accept"])


def _forced_prefill_matches_steps(W, cfg, prompts, smp, k_list):
    """Prefill + k teacher-forced steps, step by step, against one prefill over
    the prompt's and the forced pairs' latents together (eq. 2 is causal):
    the records of step k, the sampler's step index and penalised sets, and
    the step after it."""
    B = len(prompts)
    run = O.PipoOracle(W)
    recs = [run.prefill(prompts, smp)]
    history = []
    for _ in range(max(k_list) + 1):
        history.append([run.next_pairs[i] for i in range(B)])
        recs.append(run.decode_step(in_pairs=history[-1]))
    for k in k_list:
        jump = O.PipoOracle(W)
        forced = [[history[s][i] for s in range(k)] for i in range(B)]
        got = jump.prefill(prompts, smp, force_b=[r["tok_b"] for r in recs[k]], forced_pairs=forced)
        for x, y in zip(got, recs[k]):
            for key in ("logits_b", "logits_d", "h_b", "h_d"):
                np.testing.assert_allclose(x[key], y[key], rtol=1e-9, atol=1e-12, err_msg=f"{key} step {k}")
            assert (x["tok_b"], x["tok_d"], x["accept"]) == (y["tok_b"], y["tok_d"], y["accept"])
            assert abs(x["conf"] - y["conf"]) < 1e-12
        assert jump.length == [run.length[i] - (len(history) - k) for i in range(B)]
        assert jump.step_idx == [k + 1] * B
        # the session continues from the jump exactly as from the steps
        nxt = jump.decode_step(in_pairs=history[k])
        for x, y in zip(nxt, recs[k + 1]):
            np.testing.assert_allclose(x["logits_d"], y["logits_d"], rtol=1e-9, atol=1e-12)
            assert (x["tok_b"], x["tok_d"]) == (y["tok_b"], y["tok_d"])


def test_forced_prefill_equals_forced_steps(small_w):
    """Greedy, and the evaluation sampler (penalised sets and draws follow the
    step index), over a ragged pair of prompts."""
    cfg = SMALL
    prompts = [rspec.prompt_tokens(1, 9, cfg.vocab, seed=31)[0], rspec.prompt_tokens(1, 14, cfg.vocab, seed=32)[0]]
    _forced_prefill_matches_steps(small_w, cfg, prompts, O.Sampling(tau=0.5), [1, 3])
    smp = O.Sampling(tau=0.3, temperature=1.0, top_p=0.9, seeds=(7, 8), top_k=10, rep_penalty=1.5)
    _forced_prefill_matches_steps(small_w, cfg, prompts, smp, [2, 4])


def test_tiny_workload_shapes_run():
    """The tiny workload's model runs end to end in the oracle (smoke)."""
    W = O.OracleWeights.generate(TINY, seed=0, precision="fp32")
    orc = O.PipoOracle(W)
    out = orc.prefill(rspec.prompt_tokens(1, 64, TINY.vocab), O.Sampling(tau=0.5))
    assert orc.length == [32]
    assert 0 <= out[0]["tok_b"] < TINY.vocab and 0 < out[0]["conf"] < 1
    orc.decode_step()
    assert orc.length == [33]


# ------------------------------------------------- regular decoding baseline

def test_regular_session_equals_brute_force(small_w):
    """Regular prefill + steps reproduce a from-scratch pass over E[tokens]."""
    cfg = SMALL
    prompt = rspec.prompt_tokens(1, 7, cfg.vocab)
    orc = O.RegularOracle(small_w)
    recs = [orc.prefill(prompt, O.Sampling(tau=0.0))[0]]
    toks = list(prompt[0])
    assert orc.length == [7]
    for k in range(4):
        toks.append(orc.next_tok[0])
        recs.append(orc.step()[0])
        assert orc.length == [8 + k]
    X, _ = O.backbone_full(small_w, small_w["embed"][np.array(toks)])
    for k, rec in enumerate(recs):
        np.testing.assert_allclose(rec["h"], X[6 + k], rtol=1e-10, atol=1e-12)
        # the fed-back token is the greedy choice of the tied head on that position
        logits = (F.rms_norm(torch.from_numpy(X[6 + k]), (cfg.hidden,), torch.from_numpy(small_w["g_final"]),
                             cfg.rms_eps) @ torch.from_numpy(small_w["embed"]).T).numpy()
        assert rec["tok"] == int(np.argmax(logits))


def test_regular_zero_layers_is_the_tied_head_of_the_embedding():
    cfg = ModelConfig(n_layers=0, hidden=32, n_q_heads=2, n_kv_heads=1, head_dim=16, ffn=48, vocab=40,
                      rope_base=1e4, rms_eps=1e-6, gain_mode=1)
    W = O.OracleWeights.generate(cfg, seed=5, precision="bf16")
    orc = O.RegularOracle(W)
    prompt = rspec.prompt_tokens(1, 3, cfg.vocab)
    rec = orc.prefill(prompt, O.Sampling(tau=0.0))[0]
    e = torch.from_numpy(W["embed"])
    expect = F.rms_norm(e[int(prompt[0, -1])], (cfg.hidden,), torch.from_numpy(W["g_final"]), cfg.rms_eps) @ e.T
    np.testing.assert_allclose(rec["logits"], expect.numpy(), rtol=1e-12, atol=1e-12)


def test_pipo_with_first_slot_compressor_is_regular_decoding_on_odd_tokens(small_w):
    """With W_c = [I 0] and b_c = 0, eq. 1 passes E[a] through, so the pair
    decoder over a prompt's pairs equals the regular decoder over its tokens
    at even indices: the two sessions share one backbone."""
    cfg = SMALL
    t = dict(small_w.t)
    t["w_comp"] = np.concatenate([np.eye(cfg.hidden), np.zeros((cfg.hidden, cfg.hidden))], axis=1)
    t["b_comp"] = np.zeros(cfg.hidden)
    W = O.OracleWeights(cfg, t)
    prompt = rspec.prompt_tokens(2, 10, cfg.vocab)
    p = O.PipoOracle(W)
    rp = p.prefill(prompt, O.Sampling(tau=0.5))
    r = O.RegularOracle(W)
    rr = r.prefill(prompt[:, 0::2], O.Sampling(tau=0.0))
    for a, b in zip(rp, rr):
        np.testing.assert_allclose(a["h_b"], b["h"], rtol=1e-12, atol=1e-12)
        assert a["tok_b"] == b["tok"]
    forced = [[a["tok_b"], 5] for a in rp]
    sp = p.decode_step(in_pairs=forced)
    sr = r.step(in_tok=[f[0] for f in forced])
    for a, b in zip(sp, sr):
        np.testing.assert_allclose(a["h_b"], b["h"], rtol=1e-12, atol=1e-12)


# ------------------------------------------- paper-default heads (App. B)

from synth.configs import HEADS_PAPER, HEADS_MTP_LAYER  # noqa: E402

SMALL_P = ModelConfig(**{**SMALL.__dict__, "heads": HEADS_PAPER})


@pytest.fixture(scope="module")
def paper_w():
    return O.OracleWeights.generate(SMALL_P, seed=4, precision="bf16")


def test_mlp_compressor_zeroed_branch_is_the_sum(paper_w):
    """The paper initialises the MLP compressor to a + b by zeroing its
    residual branch: W2 = 0 (or W1 = 0, since SiLU(0) = 0) gives exactly a + b."""
    E = paper_w["embed"]
    pairs = np.array([[3, 7], [11, 2], [5, 5]])
    for w1, w2 in ((paper_w["comp_w1"], np.zeros_like(paper_w["comp_w2"])),
                   (np.zeros_like(paper_w["comp_w1"]), paper_w["comp_w2"])):
        np.testing.assert_array_equal(O.compress_mlp(E, w1, w2, pairs), E[pairs[:, 0]] + E[pairs[:, 1]])


def test_mlp_compressor_branch_is_linear_in_w2_and_symmetric_when_w1_is(paper_w):
    E = paper_w["embed"]
    pairs = np.array([[3, 7], [11, 2]])
    base = E[pairs[:, 0]] + E[pairs[:, 1]]
    f1 = O.compress_mlp(E, paper_w["comp_w1"], paper_w["comp_w2"], pairs) - base
    f2 = O.compress_mlp(E, paper_w["comp_w1"], 2 * paper_w["comp_w2"], pairs) - base
    np.testing.assert_allclose(f2, 2 * f1, rtol=1e-12, atol=1e-15)
    assert np.abs(f1).max() > 0
    # W1 = [M M] sees a + b only, so swapping the pair leaves z unchanged; a generic W1 does not
    M = paper_w["comp_w1"][:, :SMALL.hidden]
    w1s = np.concatenate([M, M], axis=1)
    np.testing.assert_allclose(O.compress_mlp(E, w1s, paper_w["comp_w2"], pairs),
                               O.compress_mlp(E, w1s, paper_w["comp_w2"], pairs[:, ::-1]), rtol=1e-12, atol=1e-15)
    assert not np.allclose(O.compress_mlp(E, paper_w["comp_w1"], paper_w["comp_w2"], pairs),
                           O.compress_mlp(E, paper_w["comp_w1"], paper_w["comp_w2"], pairs[:, ::-1]))


def test_confidence_mlp_closed_forms(paper_w):
    h_b = np.linspace(-1, 1, SMALL.hidden)
    h_d = np.cos(np.arange(SMALL.hidden))
    g = paper_w["g_conf"]
    for w1, w2 in ((np.zeros_like(paper_w["conf_w1"]), paper_w["conf_w2"]),
                   (paper_w["conf_w1"], np.zeros_like(paper_w["conf_w2"]))):
        s, c = O.confidence_mlp(w1, w2, g, h_b, h_d, 1e-6)
        assert s == 0.0 and c == 0.5
    # worked example, H = 1: RMSNorm([3; 4]) = [3, 4] / sqrt(12.5 + eps), W1 = [[1, 0]], w2 = [2]
    n0 = 3 / np.sqrt(12.5 + 1e-6)
    s, c = O.confidence_mlp(np.array([[1.0, 0.0]]), np.array([2.0]), np.ones(2), np.array([3.0]), np.array([4.0]), 1e-6)
    assert abs(s - 2 * n0 / (1 + np.exp(-n0))) < 1e-14 and abs(c - 1 / (1 + np.exp(-s))) < 1e-15


def test_mtp_layer_with_zero_output_projections_is_the_linear_head():
    """With the MTP layer's W_o and W_down zero the layer is the identity, so
    the paper-default MTP head reduces to the one-linear form."""
    cfg = ModelConfig(**{**SMALL.__dict__, "heads": HEADS_MTP_LAYER})
    W = O.OracleWeights.generate(cfg, seed=6, precision="bf16")
    W.t["mtp.wo"] = np.zeros_like(W.t["mtp.wo"])
    W.t["mtp.wdown"] = np.zeros_like(W.t["mtp.wdown"])
    W0 = O.OracleWeights(SMALL, {k: v for k, v in W.t.items() if not k.startswith("mtp.")})
    prompt = rspec.prompt_tokens(1, 9, cfg.vocab, seed=8)
    a, b = O.PipoOracle(W), O.PipoOracle(W0)
    ra, rb = a.prefill(prompt, O.Sampling(tau=0.5)), b.prefill(prompt, O.Sampling(tau=0.5))
    for _ in range(3):
        np.testing.assert_allclose(ra[0]["h_d"], rb[0]["h_d"], rtol=1e-12, atol=1e-14)
        assert (ra[0]["tok_b"], ra[0]["tok_d"]) == (rb[0]["tok_b"], rb[0]["tok_d"])
        ra, rb = a.decode_step(), b.decode_step()


def test_paper_heads_session_equals_brute_force(paper_w):
    """Prefill + pair steps with all three App. B heads: the backbone states
    equal a from-scratch pass over the compressed inputs, and the MTP states
    equal a from-scratch pass of the MTP layer over its inputs (the prompt
    token after each pair for the prompt's latents, the selected backbone
    token afterwards)."""
    cfg, W = SMALL_P, paper_w
    prompt = rspec.prompt_tokens(1, 11, cfg.vocab, seed=9)
    orc = O.PipoOracle(W)
    recs = [orc.prefill(prompt, O.Sampling(tau=0.5))[0]]
    pairs = [tuple(p) for p in O.prompt_pairs(prompt[0], cfg.pad_id)]
    L0 = len(pairs)
    for _ in range(4):
        pairs.append(orc.next_pairs[0])
        recs.append(orc.decode_step()[0])
    Z = O.compress_mlp(W["embed"], W["comp_w1"], W["comp_w2"], np.array(pairs))
    X, _ = O.backbone_full(W, Z)
    for k, rec in enumerate(recs):
        np.testing.assert_allclose(rec["h_b"], X[L0 - 1 + k], rtol=1e-10, atol=1e-12)
    toks = [pairs[j + 1][0] for j in range(L0 - 1)] + [r["tok_b"] for r in recs]
    U = np.stack([O.mtp_hidden(W["w_fc"], W["g_mtp_h"], W["g_mtp_e"], X[j], W["embed"][t], cfg.rms_eps)
                  for j, t in enumerate(toks)])
    Hd, _ = O.layer_full(cfg, O.mtp_layer(W), U)
    for k, rec in enumerate(recs):
        np.testing.assert_allclose(rec["h_d"], Hd[L0 - 1 + k], rtol=1e-10, atol=1e-12)
        s, c = O.confidence_mlp(W["conf_w1"], W["conf_w2"], W["g_conf"], rec["h_b"], rec["h_d"], cfg.rms_eps)
        assert abs(c - rec["conf"]) < 1e-15


def test_paper_heads_forced_prefill_equals_forced_steps(paper_w):
    """With the App. B MTP layer, the forced latents' MTP inputs take the next
    pair's first token, which is the backbone token each step selected."""
    prompts = rspec.prompt_tokens(2, 10, SMALL_P.vocab, seed=12)
    _forced_prefill_matches_steps(paper_w, SMALL_P, list(prompts), O.Sampling(tau=0.5), [1, 3])


# --------------------------------------------- evaluation sampler (Sec. 4)

def test_repetition_penalty_closed_form():
    l = np.array([2.0, -1.0, 0.5, 3.0, -4.0])
    y = O.repetition_penalty(l, {0, 1, 4}, 1.5)
    np.testing.assert_array_equal(y, [2.0 / 1.5, -1.5, 0.5, 3.0, -6.0])
    np.testing.assert_array_equal(O.repetition_penalty(l, {0, 1}, 1.0), l)


def test_eval_sampler_limits():
    rng = np.random.default_rng(0)
    l = rng.standard_normal(200)
    # top_k = 1: the argmax of the penalised logits, for any draw
    seen = {int(np.argmax(l))}
    pen = O.repetition_penalty(l, seen, 1.5)
    for u in (0.0, 0.3, 0.999):
        assert O.select_eval(l, seen, 1.0, 1, 0.95, 1.5, u) == int(np.argmax(pen))
    # top_k >= V and no penalty: the plain top-p rule
    for u in (0.1, 0.5, 0.9):
        assert O.select_eval(l, set(), 0.8, 500, 0.9, 1.0, u) == O.select_top_p(l, 0.8, 0.9, u)
    # top_k keeps ties at the k-th value whole
    t = np.array([1.0, 3.0, 2.0, 2.0, 0.5])
    kept = {O.select_eval(t, set(), 1.0, 2, 1.0, 1.0, u) for u in np.linspace(0, 0.999, 200)}
    assert kept == {1, 2, 3}


def test_eval_sampler_worked_example():
    # logits [ln 4, ln 2, ln 1, ln 8] with token 3 penalised by 1.5 (positive: divided),
    # T = 1, top-k 3 keeps ids {0, 1, 3}: p ~ (4, 2, 8^(1/1.5) = 4) / 10; top-p 0.7:
    # masses sorted 0.4, 0.4, 0.2 -> theta* = 0.4 (upper mass 0.8 >= 0.7), nucleus {0, 3},
    # mass 0.8; u = 0.6 -> t = 0.48 -> running mass 0.4 (id 0), 0.8 (id 3) -> id 3
    l = np.log(np.array([4.0, 2.0, 1.0, 8.0]))
    assert O.select_eval(l, {3}, 1.0, 3, 0.7, 1.5, 0.6) == 3
    assert O.select_eval(l, {3}, 1.0, 3, 0.7, 1.5, 0.3) == 0


# ------------------------------------------------- OPD targets (App. C)

def test_opd_teacher_rows_worked_example():
    P = 99
    # non-PAD prefix counts minus one; a PAD inherits the row before it
    assert list(O.opd_teacher_rows([5, P, 7, 8, P, P, 9], P)) == [0, 0, 1, 2, 2, 2, 3]
    assert list(O.opd_teacher_rows([P, 4], P)) == [-1, 0]


def test_opd_targets_closed_forms():
    rng = np.random.default_rng(3)
    V, T = 50, 12
    ls = rng.standard_normal((T, V)) * 2
    lt = rng.standard_normal((T, V)) * 2
    y = rng.integers(0, V, T)
    y[3] = -1
    rows = np.arange(T)
    d, a = O.opd_targets(ls, lt, rows, y)
    # alpha = min(p_t / p_s, 1) from the probabilities themselves
    ps = np.exp(ls) / np.exp(ls).sum(1, keepdims=True)
    pt = np.exp(lt) / np.exp(lt).sum(1, keepdims=True)
    for t in range(T):
        if y[t] < 0:
            assert d[t] == 0 and a[t] == 1
            continue
        np.testing.assert_allclose(a[t], min(pt[t, y[t]] / ps[t, y[t]], 1.0), rtol=1e-12)
        np.testing.assert_allclose(d[t], np.log(ps[t, y[t]]) - np.log(pt[t, y[t]]), rtol=1e-10, atol=1e-12)
    # a student equal to its teacher: d = 0, alpha = 1
    d0, a0 = O.opd_targets(ls, ls, rows, np.abs(y))
    np.testing.assert_allclose(d0, 0, atol=1e-12)
    np.testing.assert_allclose(a0, 1, atol=1e-12)
    # shifting a whole logit row changes nothing
    d1, _ = O.opd_targets(ls + 7.5, lt - 3.0, rows, y)
    np.testing.assert_allclose(d1, d, atol=1e-10)
    # the teacher row map is honoured
    rows2 = np.maximum(np.arange(T) - 1, 0)
    d2, _ = O.opd_targets(ls, lt, rows2, y)
    t = 5
    np.testing.assert_allclose(d2[t], np.log(ps[t, y[t]]) - np.log(pt[t - 1, y[t]]), rtol=1e-10)


def test_opd_sampled_kl_is_unbiased():
    # E_{y ~ p_s}[log p_s(y) - log p_t(y)] = KL(p_s || p_t): the mean of d over
    # draws from the student converges to the full-sum divergence
    rng = np.random.default_rng(4)
    V, N = 20, 40000
    ls, lt = rng.standard_normal(V), rng.standard_normal(V)
    ps = np.exp(ls) / np.exp(ls).sum()
    pt = np.exp(lt) / np.exp(lt).sum()
    kl = float(np.sum(ps * np.log(ps / pt)))
    y = rng.choice(V, size=N, p=ps)
    d, _ = O.opd_targets(np.tile(ls, (N, 1)), lt[None, :], np.zeros(N, int), y)
    sd = np.std(d) / np.sqrt(N)
    assert abs(d.mean() - kl) < 4 * sd


def test_opd_loss_sums_by_parity():
    d = np.array([1.0, 2.0, 3.0, 4.0, 5.0])
    lab = np.array([1, 1, -1, 1, 1])
    assert O.opd_loss_sums(d, lab) == [6.0, 2.0, 6.0, 2.0]
