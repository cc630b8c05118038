"""pipo_decode_step_noalloc (scratch in the library's static device array, no
allocation, eager launches) against pipo_decode_step on the same inputs:
two calls in a row on one context, the second with a smaller batch, each
held to the parity bounds (tokens and accept flags equal, logits within
max-abs 2e-2 and mean-relative 5e-3, confidence within 1e-3)."""
import numpy as np
import pytest

from synth import rspec
from synth.configs import DENSE_4B, ModelConfig

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


def _models(cfg, B, max_latent, chunk):
    from paper_2605_27255_amd import PipoModel
    return [PipoModel(cfg, seed=0, max_batch=B, max_latent=max_latent, prefill_chunk=chunk) for _ in range(2)]


def _step_pair(torch, ref, new, steps):
    """`steps` auto-fed pair steps on both contexts: the existing entry point
    on `ref`, the no-allocation one on `new`; every step compared."""
    B, V = ref.batch, ref.model.vocab
    for k in range(steps):
        o1, lb1, ld1 = ref.decode_step(logits=True)
        o2 = torch.empty((B, 4), dtype=torch.int32, device="cuda")
        lb2 = torch.empty((B, V), dtype=torch.float32, device="cuda")
        ld2 = torch.empty((B, V), dtype=torch.float32, device="cuda")
        new.decode_step_noalloc(o2, logits_b=lb2, logits_d=ld2)
        torch.cuda.synchronize()
        a, b = o1.cpu().numpy(), o2.cpu().numpy()
        np.testing.assert_array_equal(a[:, [0, 1, 3]], b[:, [0, 1, 3]], err_msg=f"step {k}: tokens / accept")
        conf_err = np.abs(a[:, 2].view(np.float32) - b[:, 2].view(np.float32)).max()
        assert conf_err <= 1e-3, conf_err
        for x, y in ((lb1, lb2), (ld1, ld2)):
            x, y = x.cpu().numpy().astype(np.float64), y.cpu().numpy().astype(np.float64)
            d = np.abs(x - y)
            assert d.max() <= 2e-2, d.max()
            assert (d.sum(1) / np.abs(x).sum(1)).max() <= 5e-3


def test_noalloc_step_matches_decode_step_two_calls(torch):
    """4B widths, one layer: batch 8 (the k-range GEMVs, their partials in the
    scratch), then a new prefill at batch 4 (the batch-1 style GEMVs) on the
    same contexts; the scratch keeps the first call's contents."""
    cfg = DENSE_4B.with_layers(1)
    ref, new = _models(cfg, 8, 300, 128)
    for B, n in ((8, 400), (4, 150)):
        t = torch.from_numpy(rspec.prompt_tokens(B, n, cfg.vocab, seed=90 + B)).cuda()
        for m in (ref, new):
            m.prefill(t, 0.7)
        _step_pair(torch, ref, new, 3)
    ref.close()
    new.close()


def test_noalloc_step_refuses_attention_partials_past_the_scratch(torch):
    """Attention partials of 64 x 1024 heads x (64 + 2) floats (17.3 MB) do not
    fit the 16 MiB scratch: PIPO_ECAPACITY, and the context still steps
    through pipo_decode_step."""
    from paper_2605_27255_amd import PipoError, PIPO_ECAPACITY
    cfg = ModelConfig(n_layers=1, hidden=256, n_q_heads=1024, n_kv_heads=64, head_dim=64, ffn=256, vocab=4096,
                      rope_base=1e4)
    from paper_2605_27255_amd import PipoModel
    m = PipoModel(cfg, seed=0, max_batch=64, max_latent=8, prefill_chunk=64)
    m.prefill(torch.from_numpy(rspec.prompt_tokens(64, 6, cfg.vocab)).cuda(), 0.5)
    out = torch.empty((64, 4), dtype=torch.int32, device="cuda")
    with pytest.raises(PipoError) as e:
        m.decode_step_noalloc(out)
    assert e.value.code == PIPO_ECAPACITY
    m.decode_step()
    torch.cuda.synchronize()
    m.close()
