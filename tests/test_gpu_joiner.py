"""HIP decoder + joiner + log-softmax (tbs_joiner_logp) against the oracle."""
import numpy as np
import pytest

import oracle
from gpu_util import say
from paper_2211_00484_amd import synth

pytestmark = pytest.mark.gpu

SHAPES = [  # (V, C, sigma, R)
    (16, 32, 0.1, 37),        # Tiny shapes, ragged row count
    (500, 512, 0.05, 70),     # Standard / Graph / Throughput shapes
    (5000, 512, 0.05, 20),    # Large shapes
    (129, 100, 0.3, 33),      # ragged V and C (padding paths)
    # enough rows for the 128 x 128 GEMM tiles (at least one per compute unit):
    (5000, 512, 0.05, 2100),  # Large shapes, ragged row tile
    (129, 100, 0.3, 16500),   # odd number of 64-column tiles, ragged K and rows
]


@pytest.mark.parametrize("V,C,sigma,R", SHAPES)
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_joiner_matches_oracle(V, C, sigma, R, dtype):
    import torch
    from paper_2211_00484_amd import tbs
    say(f"joiner V={V} C={C} R={R} {dtype}")
    rng = np.random.default_rng(V + C)
    model_np = synth.make_model(rng, V, C, sigma)
    enc = rng.standard_normal((R, C), dtype=np.float32)
    a = rng.integers(0, V, R).astype(np.int32)
    b = rng.integers(0, V, R).astype(np.int32)
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    ctx = torch.from_numpy((a.astype(np.int64) * V + b).astype(np.int32))
    got = tbs.joiner_logp(model, torch.from_numpy(enc).cuda(), ctx).cpu().numpy()
    want = oracle.logp(model_np, enc, a, b, bf16=(dtype == "bf16"))
    err = np.abs(got - want).max()
    say(f"  max |dlogp| = {err:.3g}")
    tol = 1e-4 if dtype == "fp32" else 2e-2
    assert err <= tol
    if dtype == "bf16":  # distance to the exact fp32-operand joiner, for the record
        exact = oracle.logp(model_np, enc, a, b, bf16=False)
        say(f"  bf16 vs fp32-operand oracle: {np.abs(got - exact).max():.3g}")


def test_joiner_empty_batch():
    import torch
    from paper_2211_00484_amd import tbs
    model = tbs.Model.from_synth(synth.make_model(np.random.default_rng(0), 8, 16, 0.1))
    out = tbs.joiner_logp(model, torch.zeros((0, 16), device="cuda"), torch.zeros(0, dtype=torch.int32))
    assert out.shape == (0, 8)


# Batches large enough for the 256 x 256 bf16 tiles (at least four per compute unit),
# checked on sampled rows (every row is independent): the first and last row tiles,
# the ragged tail and random rows in between.
WIDE = [  # (V, C, sigma, R)
    (5000, 512, 0.05, 256 * 53 + 77),   # Large shapes: 54 x 20 tiles, ragged rows
    (999, 300, 0.3, 256 * 256 + 5),     # partial last vocabulary tile, ragged K
]


@pytest.mark.parametrize("V,C,sigma,R", WIDE)
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_joiner_large_batches_sampled_rows(V, C, sigma, R, dtype):
    import torch
    from paper_2211_00484_amd import tbs
    say(f"joiner (large batch) V={V} C={C} R={R} {dtype}")
    rng = np.random.default_rng(V + C + R)
    model_np = synth.make_model(rng, V, C, sigma)
    enc = rng.standard_normal((R, C), dtype=np.float32)
    a = rng.integers(0, V, R).astype(np.int32)
    b = rng.integers(0, V, R).astype(np.int32)
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    ctx = torch.from_numpy((a.astype(np.int64) * V + b).astype(np.int32))
    got = tbs.joiner_logp(model, torch.from_numpy(enc).cuda(), ctx).cpu().numpy()
    idx = np.unique(np.concatenate([np.arange(300), np.arange(R - 300, R),
                                    rng.integers(0, R, 400)]))
    want = oracle.logp(model_np, enc[idx], a[idx], b[idx], bf16=(dtype == "bf16"))
    err = np.abs(got[idx] - want).max()
    say(f"  max |dlogp| over {len(idx)} rows = {err:.3g}")
    assert err <= (1e-4 if dtype == "fp32" else 2e-2)
    assert np.isfinite(got).all()
