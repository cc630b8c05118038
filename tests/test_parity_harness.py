"""The parity harness's kernel-precision selection rule (CPU): away from a
cumulative-mass boundary it takes the float64 oracle rule's decision."""
import os
import sys

import numpy as np

from oracle import pipo_oracle as O

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from parity import _kernel_precision_rule  # noqa: E402


def test_kernel_precision_rule_agrees_with_the_oracle_rule():
    rng = np.random.default_rng(0)
    for _ in range(200):
        row = (rng.standard_normal(4096) * 2).astype(np.float32)
        u = int(rng.integers(0, 2 ** 24)) / 2 ** 24
        seen = set(rng.integers(0, 4096, 50).tolist())
        plain = O.Sampling(tau=0.5, temperature=0.6, top_p=0.95, seeds=(1,))
        assert _kernel_precision_rule(row, plain, u, seen) == O.select_top_p(row.astype(np.float64), 0.6, 0.95, u)
        ev = O.Sampling(tau=0.5, temperature=1.0, top_p=0.95, seeds=(1,), top_k=20, rep_penalty=1.5)
        assert _kernel_precision_rule(row, ev, u, seen) == O.select_eval(row.astype(np.float64), seen, 1.0, 20, 0.95,
                                                                         1.5, u)


def test_kernel_precision_rule_floor_and_greedy_limit():
    """A nucleus mass far below the top probability keeps the argmax alone."""
    rng = np.random.default_rng(1)
    row = (rng.standard_normal(1000) * 3).astype(np.float32)
    smp = O.Sampling(tau=0.5, temperature=0.7, top_p=1e-6, seeds=(1,))
    for u in (0.0, 0.5, 1 - 2 ** -24):
        assert _kernel_precision_rule(row, smp, u, set()) == int(np.argmax(row))
