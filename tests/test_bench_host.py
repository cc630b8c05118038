"""Host-side checks of bench.py's contract (no GPU needed)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_algorithmic_bytes_of_the_4b_step():
    import bench
    from synth.configs import WORKLOADS
    m = WORKLOADS["4b-bs1-ctx2048"].model
    # layers 7.267 GB + the embedding twice 1.556 GB + W_c and W_fc 0.052 GB (bf16), plus activations
    w = bench.gemv_step_bytes(m, 1)
    assert 8.87e9 < w < 8.89e9
    # batch 1, 2048 cached latents, 36 layers of 8 KV heads x 128 dims, K and V in bf16
    assert bench.kv_step_bytes(m, 1, 2048) >= 36 * 2 * 8 * 128 * 2 * 2048


@pytest.mark.parametrize("name", ["tiny-bs1", "4b-bs1-ctx2048", "4b-bs32-ctx8192-topp", "9b-bs8-ctx16384",
                                  "4b-prefill-ctx32768"])
def test_workloads_have_the_stated_shapes(name):
    from synth.configs import WORKLOADS
    wl = WORKLOADS[name]
    assert wl.latents == (wl.prompt_tokens + 1) // 2
    assert wl.model.vocab % 16 == 0 and wl.model.hidden % 32 == 0
