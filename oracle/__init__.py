"""Oracle for the PIPO pair-in/pair-out path: TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 CPU implementation of what the PIPO decode step and the
compressed-prompt prefill compute, written from the paper's method section
(Sec. 3.2, eqs. 1-6) and its architecture appendix (App. B).  Only the tests,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with the HIP library: it depends on NumPy and on
the seeded-input package ``synth`` only.
"""
from .pipo_oracle import (  # noqa: F401
    OracleWeights, PipoOracle, rms_norm, rope_cos_sin, apply_rope, silu,
    compress, attention_decode, attention_causal, backbone_full, lm_logits,
    mtp_hidden, confidence, gate, select_greedy, select_top_p, prompt_pairs,
    Sampling, to_bf16,
)
