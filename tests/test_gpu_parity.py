"""GPU parity of the HIP path (through the C ABI) against the float64 oracle."""
import os
import sys

import numpy as np
import pytest

from synth import rspec
from synth.configs import TINY, DENSE_4B, DENSE_9B, ModelConfig, model_tensor_shapes
from oracle import pipo_oracle as O

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from parity import run_parity, run_regular_parity  # noqa: E402

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


def _model(cfg, **kw):
    from paper_2605_27255_amd import PipoModel
    return PipoModel(cfg, **kw)


def _expected_bits(cfg, name, seed, start, count):
    shapes = model_tensor_shapes(cfg)
    base = name.split(".")[-1]
    tid = rspec.tensor_id(name)
    if base.startswith("g_"):
        v = rspec.gain_values(seed, tid, shapes[name][0], cfg.gain_mode)[start:start + count]
    else:
        v = rspec.weight_values(seed, tid, start, count)
    return rspec.bf16_bits(v)


def test_device_weights_bit_identical_tiny(torch):
    for gm in (0, 1):
        cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": gm})
        m = _model(cfg, seed=5, max_batch=1, max_latent=40, prefill_chunk=16)
        for name, shape in model_tensor_shapes(cfg).items():
            n = int(np.prod(shape))
            got = m.read_weight(name, 0, n)
            np.testing.assert_array_equal(got, _expected_bits(cfg, name, 5, 0, n), err_msg=name)
        m.close()


def test_device_weights_bit_identical_4b_slices(torch):
    cfg = DENSE_4B.with_layers(1)
    m = _model(cfg, seed=0, max_batch=1, max_latent=64, prefill_chunk=64)
    shapes = model_tensor_shapes(cfg)
    rng = np.random.default_rng(0)
    for name in ("embed", "w_comp", "w_fc", "b_comp", "w_conf", "l0.wq", "l0.wk", "l0.wv", "l0.wo",
                 "l0.wgate", "l0.wup", "l0.wdown", "l0.g_attn"):
        n = int(np.prod(shapes[name]))
        cnt = min(4096, n)
        for start in sorted({0, n - cnt, int(rng.integers(0, n - cnt + 1))}):
            got = m.read_weight(name, start, cnt)
            np.testing.assert_array_equal(got, _expected_bits(cfg, name, 0, start, cnt), err_msg=f"{name}@{start}")
    m.close()


def test_tiny_workload_parity_greedy(torch):
    """Tiny model: 64-token prompt (32 latents, 2 chunks), 16 greedy pair steps,
    against the oracle on the bf16-valued weights the device holds."""
    n, steps, tau = 64, 16, 0.5
    prompts = rspec.prompt_tokens(1, n, TINY.vocab)
    m = _model(TINY, seed=0, max_batch=1, max_latent=32 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(TINY, seed=0, precision="bf16")
    rep, host = run_parity(m, W, prompts, steps, O.Sampling(tau=tau), log)
    rep.check()
    # the workload's tokens and accept flags match bit for bit: no near-tie waivers
    assert rep.ambiguous_tokens == 0 and rep.ambiguous_accepts == 0
    m.close()


def test_tiny_workload_against_fp32_weights(torch):
    """The same run against the oracle on the unrounded float32 weights the
    workload names (bf16 weights against the fp32 oracle), at the same bounds;
    storing the weights in bf16 alone moves these logits by 4.5e-3
    mean-relative (oracle against oracle)."""
    n, steps, tau = 64, 16, 0.5
    prompts = rspec.prompt_tokens(1, n, TINY.vocab)
    m = _model(TINY, seed=0, max_batch=1, max_latent=32 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(TINY, seed=0, precision="fp32")
    rep, host = run_parity(m, W, prompts, steps, O.Sampling(tau=tau), log)
    rep.check()
    assert rep.ambiguous_tokens == 0 and rep.ambiguous_accepts == 0
    m.close()


def test_tiny_parity_odd_prompt_ragged_chunks_gains(torch):
    """Odd prompt (PAD at the odd slot), ragged chunks, non-unit RMSNorm gains."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    n, steps, tau = 61, 6, 0.5
    prompts = rspec.prompt_tokens(1, n, cfg.vocab, seed=3)
    m = _model(cfg, seed=11, max_batch=1, max_latent=31 + steps + 1, prefill_chunk=8)
    W = O.OracleWeights.generate(cfg, seed=11, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=tau), log)
    rep.check()
    m.close()


def test_tiny_parity_batch_top_p(torch):
    """Batch 3, temperature 0.6, top-p 0.95, tau 0.7, per-sequence seeds."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    B, n, steps = 3, 40, 5
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=4)
    smp = O.Sampling(tau=0.7, temperature=0.6, top_p=0.95, seeds=tuple(1000 + b for b in range(B)))
    m = _model(cfg, seed=2, max_batch=4, max_latent=20 + steps + 1, prefill_chunk=32)
    W = O.OracleWeights.generate(cfg, seed=2, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, smp, log)
    rep.check()
    m.close()


def test_tiny_parity_batch_greedy_tau_extremes(torch):
    """tau = 0 accepts every draft, tau > 1 none (pair-in single-token decoding)."""
    B, n, steps = 2, 30, 4
    prompts = rspec.prompt_tokens(B, n, TINY.vocab, seed=6)
    W = O.OracleWeights.generate(TINY, seed=1, precision="bf16")
    for tau, expect in ((0.0, 1), (1.5, 0)):
        m = _model(TINY, seed=1, max_batch=2, max_latent=15 + steps + 1, prefill_chunk=64)
        rep, host = run_parity(m, W, prompts, steps, O.Sampling(tau=tau), log)
        rep.check()
        assert all((h[0][3] == expect).all() for h in host)
        m.close()


def test_tiny_parity_gemv_workgroups_run_several_strip_groups(torch, monkeypatch):
    """Decode GEMV workgroups capped at 3 (batch 1, greedy) and 7 (batch 3,
    top-p): every workgroup streams several strip groups in a row, with the
    reduction and epilogue of each in between, including the residual rows
    that later groups read in their epilogue."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    W = O.OracleWeights.generate(cfg, seed=9, precision="bf16")
    for cap, B, smp in ((3, 1, O.Sampling(tau=0.5)),
                        (7, 3, O.Sampling(tau=0.7, temperature=0.6, top_p=0.95, seeds=(7, 8, 9)))):
        monkeypatch.setenv("PIPO_GEMV_WG_CAP", str(cap))
        n, steps = 36, 5
        prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=cap)
        m = _model(cfg, seed=9, max_batch=B, max_latent=18 + steps + 1, prefill_chunk=16)
        log(f"wg_cap={cap} B={B}")
        rep, _ = run_parity(m, W, prompts, steps, smp, log)
        rep.check()
        m.close()


def test_4b_width_two_layers_2048_latents(torch):
    """Full 4B-class width (hidden 2560, 32/8 heads of 128, FFN 9728, vocab 151936)
    with two layers: 4096-token prompt (2048 latents, one chunk), 3 greedy steps."""
    cfg = DENSE_4B.with_layers(2)
    n, steps = 4096, 3
    prompts = rspec.prompt_tokens(1, n, cfg.vocab)
    m = _model(cfg, seed=0, max_batch=1, max_latent=2048 + steps + 1, prefill_chunk=4096)
    log("generating oracle weights")
    W = O.OracleWeights.generate(cfg, seed=0, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.95), log)
    rep.check()
    m.close()


def test_4b_full_depth_36_layers(torch):
    """The whole 4B-class model (36 layers, bench launch configuration at batch 1):
    a 40-token prompt (20 latents) and 3 greedy pair steps."""
    n, steps = 40, 3
    prompts = rspec.prompt_tokens(1, n, DENSE_4B.vocab)
    m = _model(DENSE_4B, seed=0, max_batch=1, max_latent=2048 + 257, prefill_chunk=4096)
    log("generating oracle weights (36 layers)")
    W = O.OracleWeights.generate(DENSE_4B, seed=0, precision="bf16")
    log("oracle weights ready")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.95), log)
    rep.check()
    m.close()


@pytest.mark.parametrize("hidden,nq,nkv", [(2048, 32, 16), (1536, 64, 16)])
def test_head_dim_64_attention_finishes_qkv(torch, hidden, nq, nkv):
    """Head dim 64 at batch 32 (hidden 2048 with two query heads per KV group,
    hidden 1536 with four): the QKV GEMV cuts K into four (three) ranges, so
    the decode attention sums them, rotates q and k and appends the new key
    and value itself (the d = 64 form of that path); the steps cross a 32-key
    block."""
    cfg = ModelConfig(n_layers=2, hidden=hidden, n_q_heads=nq, n_kv_heads=nkv, head_dim=64, ffn=2048, vocab=4096,
                      rope_base=1e4)
    B, n, steps = 32, 64, 3
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=21)
    m = _model(cfg, seed=8, max_batch=32, max_latent=32 + steps + 1, prefill_chunk=4096)
    W = O.OracleWeights.generate(cfg, seed=8, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.95), log)
    rep.check()
    m.close()


@pytest.mark.parametrize("hidden,nq,nkv,d,B", [(2560, 32, 8, 128, 64), (2048, 32, 8, 64, 32)])
def test_workgroup_merged_attention_unfused(torch, hidden, nq, nkv, d, B):
    """Batch x KV groups >= 256, so the decode attention runs one workgroup per
    (sequence, KV group) and merges its splits (one per wave) in LDS, with the QKV
    GEMV finishing its own k-ranges (five ranges at 4B width and batch 64,
    eight at head dim 64 and batch 32): the unfused form of that kernel, at
    d = 128 and 64.  The oracle replays the first and the last sequence."""
    cfg = ModelConfig(n_layers=1, hidden=hidden, n_q_heads=nq, n_kv_heads=nkv, head_dim=d, ffn=2048, vocab=4096,
                      rope_base=1e4)
    n, steps = 96, 3
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=23)
    m = _model(cfg, seed=12, max_batch=B, max_latent=48 + steps + 1, prefill_chunk=4096)
    W = O.OracleWeights.generate(cfg, seed=12, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.95), log, seqs=[0, B - 1])
    rep.check()
    m.close()


@pytest.mark.parametrize("max_latent,n,xcd", [(26 * 32, 40, "1"), (48 * 32, 300, "1"), (90 * 32, 5000, "1"),
                                              (90 * 32, 5000, "0"), (100 * 32, 300, "1")])
def test_attention_split_merges(torch, monkeypatch, max_latent, n, xcd):
    """4B width, batch 2: the decode attention's key splits and their merges.
    13 splits (a 40-token prompt leaves every split of the first round of
    twelve empty) and 24 (two rounds) merge on their XCD; at 90 blocks two
    per split would make 45, so 24 splits of three or four blocks, every one
    holding keys of the 2500-latent prompt, merge on their XCD, or, with
    PIPO_NO_XCD_MERGE=1, 45 splits and the merge launch; at 100 blocks, 48
    splits (the three-waves-per-CU cap) and the merge launch."""
    monkeypatch.setenv("PIPO_NO_XCD_MERGE", "0" if xcd == "1" else "1")
    cfg = DENSE_4B.with_layers(1)
    B, steps = 2, 3
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=25)
    m = _model(cfg, seed=13, max_batch=B, max_latent=max_latent, prefill_chunk=4096)
    W = O.OracleWeights.generate(cfg, seed=13, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.95), log)
    rep.check()
    m.close()


@pytest.mark.parametrize("B,max_latent", [(3, 300), (5, 1200)])
def test_attention_xcd_merge_ragged_pair_grid(torch, B, max_latent):
    """Head dim 128 with four KV groups: 3 x 4 = 12 and 5 x 4 = 20 (sequence,
    KV group) pairs, not a multiple of eight, so the XCD-merged grid has
    workgroups past the last pair that leave at once; 5 and 19 splits of one
    or two blocks each over prompts of 400 and 2000 tokens, T 0.6, top-p
    0.9."""
    cfg = ModelConfig(n_layers=1, hidden=1024, n_q_heads=16, n_kv_heads=4, head_dim=128, ffn=2048, vocab=4096,
                      rope_base=1e4)
    n = 400 if B == 3 else 2000
    steps = 3
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=27)
    smp = O.Sampling(tau=0.8, temperature=0.6, top_p=0.9, seeds=tuple(300 + b for b in range(B)))
    m = _model(cfg, seed=14, max_batch=B, max_latent=max_latent, prefill_chunk=4096)
    W = O.OracleWeights.generate(cfg, seed=14, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, smp, log)
    rep.check()
    m.close()


def test_4b_width_batch20_top_p(torch):
    """4B width, two layers, 20 sequences (two 16-column MFMA tiles), T 0.6,
    top-p 0.95, tau 0.7, per-sequence seeds."""
    cfg = DENSE_4B.with_layers(2)
    B, n, steps = 20, 64, 3
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=9)
    smp = O.Sampling(tau=0.7, temperature=0.6, top_p=0.95, seeds=tuple(1000 + b for b in range(B)))
    m = _model(cfg, seed=4, max_batch=32, max_latent=32 + steps + 1, prefill_chunk=4096)
    W = O.OracleWeights.generate(cfg, seed=4, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, smp, log)
    rep.check()
    m.close()


def test_9b_width_chunked_prefill(torch):
    """9B-class width (hidden 4096, FFN 12288), one layer, batch 2, a 517-token
    prompt (259 latents, odd) prefilled in chunks of 100 latents, 3 steps."""
    cfg = DENSE_9B.with_layers(1)
    B, n, steps = 2, 517, 3
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=5)
    m = _model(cfg, seed=7, max_batch=2, max_latent=259 + steps + 1, prefill_chunk=100)
    W = O.OracleWeights.generate(cfg, seed=7, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.95), log)
    rep.check()
    m.close()


def test_4b_width_long_prompt_four_chunks(torch):
    """One 4B-width layer, 8192-token prompt (4096 latents) prefilled in four
    1024-latent chunks (causal attention across chunks), then 3 steps."""
    cfg = DENSE_4B.with_layers(1)
    n, steps = 8192, 3
    prompts = rspec.prompt_tokens(1, n, cfg.vocab, seed=2)
    m = _model(cfg, seed=3, max_batch=1, max_latent=4096 + steps + 1, prefill_chunk=1024)
    W = O.OracleWeights.generate(cfg, seed=3, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log)
    rep.check()
    m.close()


def test_tiny_batch20_greedy_and_graph_replay(torch):
    """Batch 20 on the tiny model, 6 steps: the decode graph replayed with the
    device-side pair feedback."""
    B, n, steps = 20, 24, 6
    prompts = rspec.prompt_tokens(B, n, TINY.vocab, seed=8)
    m = _model(TINY, seed=0, max_batch=20, max_latent=12 + steps + 1, prefill_chunk=8)
    W = O.OracleWeights.generate(TINY, seed=0, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log)
    rep.check()
    m.close()


def test_deterministic_repeat(torch):
    prompts = torch.from_numpy(rspec.prompt_tokens(2, 50, TINY.vocab)).cuda()
    res = []
    for _ in range(2):
        m = _model(TINY, seed=0, max_batch=2, max_latent=40, prefill_chunk=16)
        outs = [m.prefill(prompts, 0.5, logits=True)]
        for _ in range(4):
            outs.append(m.decode_step(logits=True))
        torch.cuda.synchronize()
        res.append([(o.cpu().numpy(), lb.cpu().numpy(), ld.cpu().numpy()) for o, lb, ld in outs])
        m.close()
    for a, b in zip(*res):
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)


def test_abi_state_and_capacity_errors(torch):
    from paper_2605_27255_amd import PipoError, PIPO_ESTATE, PIPO_ECAPACITY
    m = _model(TINY, seed=0, max_batch=2, max_latent=12, prefill_chunk=16)
    with pytest.raises(PipoError) as e:
        m.batch = 1
        m.decode_step()
    assert e.value.code == PIPO_ESTATE
    toks = torch.from_numpy(rspec.prompt_tokens(3, 8, TINY.vocab)).cuda()
    with pytest.raises(PipoError) as e:
        m.prefill(toks, 0.5)
    assert e.value.code == PIPO_ECAPACITY                       # batch 3 > 2
    with pytest.raises(PipoError) as e:
        m.prefill(torch.from_numpy(rspec.prompt_tokens(1, 23, TINY.vocab)).cuda(), 0.5)
    assert e.value.code == PIPO_ECAPACITY                       # 12 latents + 1 > 12
    m.prefill(torch.from_numpy(rspec.prompt_tokens(1, 20, TINY.vocab)).cuda(), 0.5)   # 10 latents
    m.decode_step()                                              # 11 latents
    m.decode_step()                                              # 12 latents: full
    with pytest.raises(PipoError) as e:
        m.decode_step()
    torch.cuda.synchronize()
    assert e.value.code == PIPO_ECAPACITY
    m.close()


# ------------------------------------------------- regular decoding baseline

def test_tiny_regular_parity_greedy_ragged_chunks(torch):
    """Regular decoding on the tiny model: 37-token prompt (3 ragged chunks of
    16), 10 greedy token steps, the decode graph replayed."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    n, steps = 37, 10
    prompts = rspec.prompt_tokens(1, n, cfg.vocab, seed=12)
    m = _model(cfg, seed=7, max_batch=1, max_latent=n + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(cfg, seed=7, precision="bf16")
    rep, _ = run_regular_parity(m, W, prompts, steps, O.Sampling(tau=0.0), log)
    rep.check()
    m.close()


def test_tiny_regular_parity_batch_top_p(torch):
    B, n, steps = 3, 20, 6
    prompts = rspec.prompt_tokens(B, n, TINY.vocab, seed=13)
    smp = O.Sampling(tau=0.0, temperature=0.7, top_p=0.9, seeds=tuple(77 + b for b in range(B)))
    m = _model(TINY, seed=3, max_batch=4, max_latent=n + steps + 1, prefill_chunk=64)
    W = O.OracleWeights.generate(TINY, seed=3, precision="bf16")
    rep, _ = run_regular_parity(m, W, prompts, steps, smp, log)
    rep.check()
    m.close()


def test_4b_width_regular_two_layers_1024_tokens(torch):
    """4B widths (2 layers), a 1024-token prompt in two chunks, 4 greedy steps."""
    cfg = DENSE_4B.with_layers(2)
    n, steps = 1024, 4
    prompts = rspec.prompt_tokens(1, n, cfg.vocab, seed=14)
    m = _model(cfg, seed=0, max_batch=1, max_latent=n + steps + 1, prefill_chunk=512)
    W = O.OracleWeights.generate(cfg, seed=0, precision="bf16")
    rep, _ = run_regular_parity(m, W, prompts, steps, O.Sampling(tau=0.0), log)
    rep.check()
    m.close()


def test_regular_and_pair_sessions_share_one_context(torch):
    """One context serves both decoders in turn; a step of the other kind is
    refused until its own prefill."""
    from paper_2605_27255_amd import PipoError, PIPO_ESTATE, PIPO_ECAPACITY
    W = O.OracleWeights.generate(TINY, seed=0, precision="bf16")
    m = _model(TINY, seed=0, max_batch=2, max_latent=24, prefill_chunk=16)
    prompts = rspec.prompt_tokens(2, 16, TINY.vocab, seed=15)
    rep, _ = run_regular_parity(m, W, prompts, 3, O.Sampling(tau=0.0), log)
    rep.check()
    with pytest.raises(PipoError) as e:
        m.decode_step()
    assert e.value.code == PIPO_ESTATE
    rep, _ = run_parity(m, W, prompts, 3, O.Sampling(tau=0.5), log)
    rep.check()
    with pytest.raises(PipoError) as e:
        m.regular_step()
    assert e.value.code == PIPO_ESTATE
    with pytest.raises(PipoError) as e:
        m.regular_prefill(torch.from_numpy(rspec.prompt_tokens(1, 24, TINY.vocab)).cuda())
    assert e.value.code == PIPO_ECAPACITY                       # 24 positions + 1 > 24
    rep, _ = run_regular_parity(m, W, prompts[:1], 2, O.Sampling(tau=0.0), log)
    rep.check()
    m.close()


# ------------------------------------- each workload at its own shape
#
# The bench's launch configuration (max_latent = latents + steps + 1, chunks
# of 4096 latents, the workload's batch), so the decode attention splits the
# keys as the timed runs do (C3: one workgroup per sequence and KV group,
# eight splits of 32 blocks merged in LDS; C4: 16 one-wave splits of about 32
# blocks and the merge kernel) and the prefill attention reaches its later
# chunks; the layer count is cut where the float64 oracle needs it, every
# other dimension is the workload's.

from synth.configs import WORKLOADS  # noqa: E402


def _workload_model(wl, layers=None):
    model = wl.model if layers is None else wl.model.with_layers(layers)
    return model, _model(model, seed=wl.seed, max_batch=wl.batch, max_latent=wl.max_latent + 1,
                         prefill_chunk=wl.prefill_chunk)


def test_c2_full_depth_2048_latents_256_steps(torch):
    """The 4B batch-1 workload as timed: 36 layers, a 4096-token prompt (2048
    latents), 256 greedy pair steps run free; the oracle checks the prefill's
    pair, steps 1-7 and the last two."""
    wl = WORKLOADS["4b-bs1-ctx2048"]
    model, m = _workload_model(wl)
    prompts = rspec.prompt_tokens(1, wl.prompt_tokens, model.vocab, seed=wl.prompt_seed)
    W = O.OracleWeights.generate(model, seed=wl.seed, precision="bf16")
    steps = wl.decode_steps
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=wl.tau), log,
                        check_steps=list(range(8)) + [steps - 1, steps])
    rep.check()
    m.close()


def test_c3_shape_batch32_8192_latents_top_p(torch):
    """The 4B batch-32 workload's shape (two layers): 32 prompts of 16384
    tokens (8192 latents each, two 4096-latent chunks), T 0.6, top-p 0.95,
    tau 0.7, per-sequence seeds; 6 steps; the oracle replays sequences 0 and
    31.  Each decode-attention split (a wave of the sequence's workgroup)
    covers 32 key blocks."""
    wl = WORKLOADS["4b-bs32-ctx8192-topp"]
    model, m = _workload_model(wl, layers=2)
    B = wl.batch
    prompts = rspec.prompt_tokens(B, wl.prompt_tokens, model.vocab, seed=wl.prompt_seed)
    smp = O.Sampling(tau=wl.tau, temperature=wl.temperature, top_p=wl.top_p,
                     seeds=tuple(wl.sample_seed_base + b for b in range(B)))
    W = O.OracleWeights.generate(model, seed=wl.seed, precision="bf16")
    rep, _ = run_parity(m, W, prompts, 6, smp, log, seqs=[0, B - 1])
    rep.check()
    m.close()


def test_c4_shape_9b_batch8_16384_latents(torch):
    """The 9B batch-8 workload's shape (two layers): 8 prompts of 32768 tokens
    (16384 latents, four chunks), greedy, tau 0.95; 4 steps; the oracle
    replays sequences 0 and 7."""
    wl = WORKLOADS["9b-bs8-ctx16384"]
    model, m = _workload_model(wl, layers=2)
    B = wl.batch
    prompts = rspec.prompt_tokens(B, wl.prompt_tokens, model.vocab, seed=wl.prompt_seed)
    W = O.OracleWeights.generate(model, seed=wl.seed, precision="bf16")
    rep, _ = run_parity(m, W, prompts, 4, O.Sampling(tau=wl.tau), log, seqs=[0, B - 1])
    rep.check()
    m.close()


def test_c5_shape_32768_latent_prefill(torch):
    """The prefill workload's shape (two layers): a 65536-token prompt
    compressed to 32768 latents and prefilled in eight 4096-latent chunks
    (the last chunk's queries attend 32768 keys; the second layer's keys and
    values carry every first-layer attention row into the steps), then 3
    pair steps at tau 0.5."""
    wl = WORKLOADS["4b-prefill-ctx32768"]
    model, m = _workload_model(wl, layers=2)
    prompts = rspec.prompt_tokens(1, wl.prompt_tokens, model.vocab, seed=wl.prompt_seed)
    W = O.OracleWeights.generate(model, seed=wl.seed, precision="bf16")
    rep, _ = run_parity(m, W, prompts, 3, O.Sampling(tau=wl.tau), log)
    rep.check()
    m.close()


# ------------------------------------------- paper-default heads (App. B)

from synth.configs import HEADS_PAPER  # noqa: E402

# The App. B heads are held to the workloads' bounds (max-abs 2e-2,
# mean-relative 5e-3, confidence 1e-3), like every other path.


def test_device_weights_bit_identical_paper_heads(torch):
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1, "heads": HEADS_PAPER})
    m = _model(cfg, seed=9, max_batch=1, max_latent=40, prefill_chunk=16)
    for name, shape in model_tensor_shapes(cfg).items():
        if not (name.startswith("mtp.") or name in ("comp_w1", "comp_w2", "conf_w1", "conf_w2")):
            continue
        n = int(np.prod(shape))
        np.testing.assert_array_equal(m.read_weight(name, 0, n), _expected_bits(cfg, name, 9, 0, n), err_msg=name)
    m.close()


def test_tiny_paper_heads_parity_odd_prompt_ragged_chunks(torch):
    """All three App. B heads on the tiny model: odd prompt, three ragged
    chunks (the MTP layer's prefill runs per chunk), 8 greedy pair steps."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1, "heads": HEADS_PAPER})
    n, steps = 45, 8
    prompts = rspec.prompt_tokens(1, n, cfg.vocab, seed=21)
    m = _model(cfg, seed=13, max_batch=1, max_latent=23 + steps + 1, prefill_chunk=8)
    W = O.OracleWeights.generate(cfg, seed=13, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log)
    rep.check()
    m.close()


def test_tiny_paper_heads_batch_top_p(torch):
    cfg = ModelConfig(**{**TINY.__dict__, "heads": HEADS_PAPER})
    B, n, steps = 3, 40, 5
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=22)
    smp = O.Sampling(tau=0.5, temperature=0.7, top_p=0.9, seeds=tuple(300 + b for b in range(B)))
    m = _model(cfg, seed=14, max_batch=4, max_latent=20 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(cfg, seed=14, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, smp, log)
    rep.check()
    m.close()


def test_4b_width_paper_heads(torch):
    """4B widths (2 layers) with the App. B heads, 512-token prompt in two
    chunks, batch 1 (weight-streaming GEMVs) then batch 8 (k-range GEMVs)."""
    cfg = ModelConfig(**{**DENSE_4B.with_layers(2).__dict__, "heads": HEADS_PAPER})
    W = O.OracleWeights.generate(cfg, seed=2, precision="bf16")
    for B, steps in ((1, 4), (8, 2)):
        prompts = rspec.prompt_tokens(B, 512, cfg.vocab, seed=23 + B)
        m = _model(cfg, seed=2, max_batch=B, max_latent=256 + steps + 1, prefill_chunk=128)
        rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log)
        rep.check()
        m.close()


# ------------------------------------------------------------ edge cases

def test_tiny_degenerate_and_tile_boundary_prompts(torch):
    """Prompts of 1, 2 and 3 tokens (a single latent, PAD at the odd slot for
    odd n) and latent counts on both sides of the 32-key decode tile and the
    64-key prefill stage, each followed by pair steps that cross the next
    boundary; one context, re-prefilled per prompt."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    W = O.OracleWeights.generate(cfg, seed=17, precision="bf16")
    m = _model(cfg, seed=17, max_batch=1, max_latent=70, prefill_chunk=32)
    for n, steps in ((1, 3), (2, 3), (3, 2), (62, 3), (64, 2), (66, 1), (126, 3), (128, 2), (130, 2)):
        log(f"prompt of {n} tokens, {steps} steps")
        prompts = rspec.prompt_tokens(1, n, cfg.vocab, seed=100 + n)
        rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log)
        rep.check()
    m.close()


def test_tiny_top_p_floor_is_greedy(torch):
    """A nucleus mass far below any single token's probability keeps only the
    most probable token, so top-p sampling must return the greedy choice."""
    from paper_2605_27255_amd import unpack_pairs
    prompts = rspec.prompt_tokens(2, 30, TINY.vocab, seed=31)
    m = _model(TINY, seed=4, max_batch=2, max_latent=24, prefill_chunk=16)
    t = torch.from_numpy(prompts).cuda()
    greedy = [m.prefill(t, 0.5)[0]] + [m.decode_step()[0] for _ in range(4)]
    sampled = [m.prefill(t, 0.5, temperature=0.7, top_p=1e-6, seeds=[5, 6])[0]] + \
              [m.decode_step()[0] for _ in range(4)]
    torch.cuda.synchronize()
    for g, s_ in zip(greedy, sampled):
        gb, gd, _, _ = unpack_pairs(g)
        sb, sd, _, _ = unpack_pairs(s_)
        np.testing.assert_array_equal(gb, sb)
        np.testing.assert_array_equal(gd, sd)
    m.close()


# ------------------------------------------- the evaluation sampler (Sec. 4)

def _eval_smp(B, tau=0.5, base=500):
    """The paper's evaluation settings: T 1.0, top-p 0.95, top-k 20, repetition penalty 1.5."""
    return O.Sampling(tau=tau, temperature=1.0, top_p=0.95, seeds=tuple(base + b for b in range(B)), top_k=20,
                      rep_penalty=1.5)


def test_tiny_eval_sampler_parity(torch):
    """Pair path, batch 3, odd prompt, 8 steps: penalised set = prompt + input
    pairs (+ the pair's backbone token for the draft), top-k 20 over 4096."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    B, n, steps = 3, 41, 8
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=40)
    m = _model(cfg, seed=5, max_batch=4, max_latent=21 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(cfg, seed=5, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, _eval_smp(B), log)
    rep.check()
    assert rep.penalty_decisive > 0      # the penalty changed some draws: the test can see it
    assert rep.ambiguous_tokens <= rep.rows // 10
    m.close()


def test_tiny_regular_eval_sampler_parity(torch):
    B, n, steps = 2, 25, 8
    prompts = rspec.prompt_tokens(B, n, TINY.vocab, seed=41)
    m = _model(TINY, seed=6, max_batch=2, max_latent=n + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(TINY, seed=6, precision="bf16")
    rep, _ = run_regular_parity(m, W, prompts, steps, _eval_smp(B, tau=0.0), log)
    rep.check()
    assert rep.penalty_decisive > 0
    assert rep.ambiguous_tokens <= rep.rows // 10
    m.close()


def test_4b_width_eval_sampler_parity(torch):
    """Full 151936-token vocabulary, two layers, batch 4: the radix top-k and
    the bitmap over every vocabulary tile."""
    cfg = DENSE_4B.with_layers(2)
    B, n, steps = 4, 64, 3
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=42)
    m = _model(cfg, seed=4, max_batch=4, max_latent=32 + steps + 1, prefill_chunk=4096)
    W = O.OracleWeights.generate(cfg, seed=4, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, _eval_smp(B, tau=0.7), log)
    rep.check()
    m.close()


def test_tiny_eval_sampler_top1_is_greedy_and_bad_settings(torch):
    """top-k 1 without a penalty keeps only the argmax, so it must return the
    greedy tokens (pair and regular paths); invalid settings are refused."""
    from paper_2605_27255_amd import unpack_pairs, PipoError, PIPO_EINVAL
    prompts = rspec.prompt_tokens(2, 30, TINY.vocab, seed=43)
    m = _model(TINY, seed=4, max_batch=2, max_latent=40, prefill_chunk=16)
    t = torch.from_numpy(prompts).cuda()
    greedy = [m.prefill(t, 0.5)[0]] + [m.decode_step()[0] for _ in range(4)]
    top1 = [m.prefill(t, 0.5, temperature=1.0, seeds=[5, 6], top_k=1)[0]] + [m.decode_step()[0] for _ in range(4)]
    rg = [m.regular_prefill(t)[0]] + [m.regular_step()[0] for _ in range(4)]
    r1 = [m.regular_prefill(t, temperature=1.0, seeds=[5, 6], top_k=1)[0]] + [m.regular_step()[0] for _ in range(4)]
    torch.cuda.synchronize()
    for g, s_ in zip(greedy, top1):
        gb, gd, _, _ = unpack_pairs(g)
        sb, sd, _, _ = unpack_pairs(s_)
        np.testing.assert_array_equal(gb, sb)
        np.testing.assert_array_equal(gd, sd)
    for g, s_ in zip(rg, r1):
        np.testing.assert_array_equal(g.cpu().numpy(), s_.cpu().numpy())
    for kw in (dict(temperature=1.0, seeds=[1, 2], top_k=-1), dict(temperature=1.0, seeds=[1, 2], rep_penalty=0.0),
               dict(top_k=5), dict(rep_penalty=1.5)):
        with pytest.raises(PipoError) as e:
            m.prefill(t, 0.5, **kw)
        assert e.value.code == PIPO_EINVAL
    m.close()


# ------------------------------------------------------------- ragged batches

def _ragged(B, lens, vocab, seed):
    """Prompts of their own lengths in one [B][max] array; the tail of each
    row holds other random tokens, which must never be read."""
    stride = max(lens)
    full = rspec.prompt_tokens(B, stride, vocab, seed=seed)
    junk = rspec.prompt_tokens(B, stride, vocab, seed=seed + 1000)
    for i, n in enumerate(lens):
        full[i, n:] = junk[i, n:]
    return full


def test_tiny_ragged_pair_parity(torch):
    """Five prompts of 1, 2, 37, 64 and 17 tokens (1 to 32 latents) in chunks
    of 16: sequences end in different chunks and step at their own positions."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    lens = [1, 2, 37, 64, 17]
    B, steps = len(lens), 6
    prompts = _ragged(B, lens, cfg.vocab, 50)
    m = _model(cfg, seed=5, max_batch=8, max_latent=32 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(cfg, seed=5, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log, lens=lens)
    rep.check()
    rep, _ = run_parity(m, W, prompts, steps, _eval_smp(B, base=700), log, lens=lens)
    rep.check()
    m.close()


def test_tiny_ragged_equal_lengths_match_uniform(torch):
    """A ragged prefill whose lengths are all equal is the uniform prefill, bit for bit."""
    from paper_2605_27255_amd import unpack_pairs
    prompts = rspec.prompt_tokens(3, 33, TINY.vocab, seed=51)
    m = _model(TINY, seed=2, max_batch=3, max_latent=30, prefill_chunk=8)
    t = torch.from_numpy(prompts).cuda()
    a = [m.prefill(t, 0.5, logits=True)] + [m.decode_step(logits=True) for _ in range(3)]
    b = [m.prefill(t, 0.5, logits=True, lens=[33, 33, 33])] + [m.decode_step(logits=True) for _ in range(3)]
    torch.cuda.synchronize()
    for (oa, la, da), (ob, lb, db) in zip(a, b):
        for x, y in zip(unpack_pairs(oa), unpack_pairs(ob)):
            np.testing.assert_array_equal(x, y)
        assert torch.equal(la, lb) and torch.equal(da, db)
    m.close()


def test_tiny_ragged_regular_parity(torch):
    lens = [5, 33, 20]
    B, steps = len(lens), 6
    prompts = _ragged(B, lens, TINY.vocab, 52)
    m = _model(TINY, seed=3, max_batch=4, max_latent=33 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(TINY, seed=3, precision="bf16")
    rep, _ = run_regular_parity(m, W, prompts, steps, O.Sampling(tau=0.0), log, lens=lens)
    rep.check()
    smp = O.Sampling(tau=0.0, temperature=0.7, top_p=0.9, seeds=tuple(90 + b for b in range(B)))
    rep, _ = run_regular_parity(m, W, prompts, steps, smp, log, lens=lens)
    rep.check()
    m.close()


def test_tiny_ragged_paper_heads_parity(torch):
    """App. B heads: the MTP layer's prompt rows stop at each sequence's own end."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1, "heads": HEADS_PAPER})
    lens = [3, 30, 15]
    B, steps = len(lens), 5
    prompts = _ragged(B, lens, cfg.vocab, 53)
    m = _model(cfg, seed=13, max_batch=3, max_latent=15 + steps + 1, prefill_chunk=8)
    W = O.OracleWeights.generate(cfg, seed=13, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log, lens=lens)
    rep.check()
    m.close()


def test_4b_width_ragged_pair_parity(torch):
    """4B width, two layers: prompts of 100, 513 and 257 tokens over chunks of 128 latents."""
    cfg = DENSE_4B.with_layers(2)
    lens = [100, 513, 257]
    B, steps = len(lens), 3
    prompts = _ragged(B, lens, cfg.vocab, 54)
    m = _model(cfg, seed=4, max_batch=4, max_latent=257 + steps + 1, prefill_chunk=128)
    W = O.OracleWeights.generate(cfg, seed=4, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.95), log, lens=lens)
    rep.check()
    m.close()


def test_ragged_bad_lengths(torch):
    from paper_2605_27255_amd import PipoError, PIPO_EINVAL, PIPO_ECAPACITY
    m = _model(TINY, seed=0, max_batch=2, max_latent=12, prefill_chunk=16)
    t = torch.from_numpy(rspec.prompt_tokens(2, 30, TINY.vocab)).cuda()
    for lens, code in (([0, 5], PIPO_EINVAL), ([5, 31], PIPO_EINVAL), ([4, 30], PIPO_ECAPACITY)):
        with pytest.raises(PipoError) as e:
            m.prefill(t, 0.5, lens=lens)
        assert e.value.code == code
    m.prefill(t, 0.5, lens=[4, 22])      # 11 latents + 1 fits
    m.decode_step()
    torch.cuda.synchronize()
    m.close()


def test_tiny_batch64_ragged_eval_sampler(torch):
    """64 sequences (four 16-column tiles), ragged prompts of 1..64 tokens,
    the evaluation sampler; then greedy."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    B, steps = 64, 4
    lens = [1 + (7 * i) % 64 for i in range(B)]
    prompts = _ragged(B, lens, cfg.vocab, 60)
    m = _model(cfg, seed=8, max_batch=64, max_latent=32 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(cfg, seed=8, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, _eval_smp(B, base=900), log, lens=lens)
    rep.check()
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log, lens=lens)
    rep.check()
    m.close()


def test_4b_width_batch64_top_p(torch):
    """4B width, two layers, 64 sequences: the k-range and wide GEMV forms at
    four column tiles, T 0.6, top-p 0.95, tau 0.7."""
    cfg = DENSE_4B.with_layers(2)
    B, n, steps = 64, 48, 2
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=61)
    smp = O.Sampling(tau=0.7, temperature=0.6, top_p=0.95, seeds=tuple(2000 + b for b in range(B)))
    m = _model(cfg, seed=4, max_batch=64, max_latent=24 + steps + 1, prefill_chunk=4096)
    W = O.OracleWeights.generate(cfg, seed=4, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, smp, log)
    rep.check()
    m.close()


def test_tiny_paper_heads_ragged_eval_sampler(torch):
    """All three App. B heads, a ragged batch and the evaluation sampler
    together: the draft penalises its pair's backbone token, which is also the
    MTP layer's input."""
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1, "heads": HEADS_PAPER})
    lens = [2, 27, 40, 9]
    B, steps = len(lens), 5
    prompts = _ragged(B, lens, cfg.vocab, 70)
    m = _model(cfg, seed=13, max_batch=4, max_latent=20 + steps + 1, prefill_chunk=8)
    W = O.OracleWeights.generate(cfg, seed=13, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, _eval_smp(B, base=1100), log, lens=lens)
    rep.check()
    m.close()


def test_tiny_regular_ragged_eval_sampler(torch):
    lens = [3, 31, 18]
    B, steps = len(lens), 6
    prompts = _ragged(B, lens, TINY.vocab, 71)
    m = _model(TINY, seed=6, max_batch=3, max_latent=31 + steps + 1, prefill_chunk=16)
    W = O.OracleWeights.generate(TINY, seed=6, precision="bf16")
    rep, _ = run_regular_parity(m, W, prompts, steps, _eval_smp(B, tau=0.0, base=1200), log, lens=lens)
    rep.check()
    m.close()


def test_empty_inputs_are_refused(torch):
    """An empty prompt or an empty batch is refused with PIPO_EINVAL before any device work."""
    from paper_2605_27255_amd import PipoError, PIPO_EINVAL
    m = _model(TINY, seed=0, max_batch=2, max_latent=16, prefill_chunk=16)
    for shape in ((1, 0), (0, 8)):
        t = torch.zeros(shape, dtype=torch.int32, device="cuda")
        for call in (lambda: m.prefill(t, 0.5), lambda: m.regular_prefill(t)):
            with pytest.raises(PipoError) as e:
                call()
            assert e.value.code == PIPO_EINVAL
    # the context still works afterwards
    m.prefill(torch.from_numpy(rspec.prompt_tokens(2, 6, TINY.vocab)).cuda(), 0.5)
    m.decode_step()
    torch.cuda.synchronize()
    m.close()


def test_refused_prefill_leaves_sequences_running(torch):
    """A prefill refused by its host-side checks (empty prompt, too many
    sequences, a prompt past the capacity) leaves the context as it was: the
    next decode steps continue the old sequences, bit-identical to a run
    without the refused calls."""
    from paper_2605_27255_amd import PipoError, PIPO_EINVAL, PIPO_ECAPACITY
    prompts = torch.from_numpy(rspec.prompt_tokens(2, 20, TINY.vocab, seed=33)).cuda()
    runs = []
    for refuse in (False, True):
        m = _model(TINY, seed=0, max_batch=2, max_latent=20, prefill_chunk=16)
        outs = [m.prefill(prompts, 0.5, logits=True), m.decode_step(logits=True)]
        if refuse:
            for bad, code in ((torch.zeros((2, 0), dtype=torch.int32, device="cuda"), PIPO_EINVAL),
                              (torch.from_numpy(rspec.prompt_tokens(3, 8, TINY.vocab)).cuda(), PIPO_ECAPACITY),
                              (torch.from_numpy(rspec.prompt_tokens(1, 40, TINY.vocab)).cuda(), PIPO_ECAPACITY)):
                with pytest.raises(PipoError) as e:
                    m.prefill(bad, 0.5)
                assert e.value.code == code
            with pytest.raises(PipoError) as e:
                m.regular_prefill(torch.zeros((2, 0), dtype=torch.int32, device="cuda"))
            assert e.value.code == PIPO_EINVAL
        outs += [m.decode_step(logits=True) for _ in range(3)]
        torch.cuda.synchronize()
        runs.append([[t.cpu().numpy() for t in o] for o in outs])
        m.close()
    for a, b in zip(*runs):
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)


def test_check_mode_tiny_parity(torch, monkeypatch):
    """PIPO_CHECK=1: every kernel is launched eagerly and waited for, with its
    error checked; the tiny workload still matches the oracle."""
    monkeypatch.setenv("PIPO_CHECK", "1")
    cfg = ModelConfig(**{**TINY.__dict__, "gain_mode": 1})
    B, n, steps = 2, 37, 4
    prompts = rspec.prompt_tokens(B, n, cfg.vocab, seed=34)
    m = _model(cfg, seed=3, max_batch=B, max_latent=n + steps + 1, prefill_chunk=8)   # regular: n positions
    W = O.OracleWeights.generate(cfg, seed=3, precision="bf16")
    rep, _ = run_parity(m, W, prompts, steps, O.Sampling(tau=0.5), log)
    rep.check()
    rep, _ = run_regular_parity(m, W, prompts, steps, O.Sampling(tau=0.0), log)
    rep.check()
    m.close()
