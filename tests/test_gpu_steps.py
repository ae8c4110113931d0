"""Fresh step measurements on the GPU against the committed step-latency
model (fitted to earlier MI355X measurements; section 4.3.1, Eq. 4)."""
import numpy as np
import pytest

from paper_2607_02043_amd import deflect as D

pytestmark = pytest.mark.gpu


def test_committed_model_predicts_fresh_steps():
    from paper_2607_02043_amd import steps as S
    configs = [(4, 842, 0, 0), (32, 3569, 0, 0), (128, 13968, 0, 0), (16, 998, 496, 0), (32, 3569, 992, 992),
               (64, 14013, 1984, 3968), (8, 13968, 2040, 8160), (128, 842, 384, 768), (0, 0, 2048, 4096),
               (0, 0, 1024, 0)]
    bench = S.StepBench(configs, seed=3)
    rows = [(B, K, c, p, bench.time_config(B, K, c, p, steps=5)) for B, K, c, p in configs]
    print("fresh steps (B, K, c, p, us):", rows, flush=True)
    err = D.mape(D.StepModel.load(), rows)
    assert err < 0.15, (err, rows)
