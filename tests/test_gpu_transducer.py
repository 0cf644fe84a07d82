"""HIP transducer forward recursions (tbs_transducer_forward; Sec. 3, eq. 1-3) against the
CPU oracle: totals within 1e-9 relative (both accumulate in fp64 from the same fp32
log-probabilities) and every visited alpha cell within fp32 rounding."""
import math

import numpy as np
import pytest

import oracle
from gpu_util import say

pytestmark = pytest.mark.gpu

KINDS = ["standard", "modified", "constrained"]


def _inputs(seed, B, T, U, ragged=True):
    rng = np.random.default_rng(seed)
    blank = np.log(rng.uniform(0.01, 1.0, size=(B, T, U + 1))).astype(np.float32)
    label = np.log(rng.uniform(0.01, 1.0, size=(B, T, U))).astype(np.float32)
    if ragged:
        frames = rng.integers(1, T + 1, size=B).astype(np.int32)
        labels = rng.integers(0, U + 1, size=B).astype(np.int32)
        frames[0], labels[0] = T, U
    else:
        frames = np.full(B, T, dtype=np.int32)
        labels = np.full(B, U, dtype=np.int32)
    return blank, label, frames, labels


def _check(kind, blank, label, frames, labels):
    import torch
    from paper_2211_00484_amd import tbs
    B, T, U1 = blank.shape
    say(f"transducer {kind} B={B} T={T} U={U1 - 1}")
    lens = np.stack([frames, labels], axis=1)
    total, alpha, status = tbs.transducer_forward(kind, torch.from_numpy(blank).cuda(),
                                                  torch.from_numpy(label).cuda(), lens,
                                                  want_alpha=True)
    torch.cuda.synchronize()
    total, alpha, status = total.cpu().numpy(), alpha.cpu().numpy(), status.cpu().numpy()
    want, walpha = oracle.transducer_forward(kind, blank, label, frames, labels)
    assert (status == 0).all()
    for b in range(B):
        if math.isinf(want[b]):
            assert total[b] == want[b]
        else:
            assert total[b] == pytest.approx(want[b], rel=1e-9, abs=1e-9), b
        rows = frames[b] + (0 if kind == "standard" else 1)
        g = alpha[b, :rows, :labels[b] + 1].astype(np.float64)
        w = walpha[b, :rows, :labels[b] + 1]
        fin = np.isfinite(w)
        assert np.array_equal(np.isfinite(g), fin), b
        assert np.allclose(g[fin], w[fin], rtol=2e-7, atol=1e-5), b


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("U", [0, 1, 5, 63, 64, 130, 300])
def test_against_oracle(kind, U):
    T = 40 if U < 64 else 160
    blank, label, frames, labels = _inputs(U * 7 + len(kind), 7, T, U)
    if kind != "standard":  # one label per frame at most: keep most utterances feasible
        labels = np.minimum(labels, frames)
    _check(kind, blank, label, frames, labels)


@pytest.mark.parametrize("kind", KINDS)
def test_training_shapes(kind):
    """B = 32, T = 250 frames (10 s at 25 frames/s), U = 80 labels."""
    blank, label, frames, labels = _inputs(11, 32, 250, 80)
    _check(kind, blank, label, frames, np.minimum(labels, frames))


@pytest.mark.parametrize("kind", KINDS)
def test_widest_rows(kind):
    blank, label, frames, labels = _inputs(3, 3, 1100, 1023, ragged=False)
    _check(kind, blank, label, frames, labels)


def test_constant_logprobs_and_invalid_lengths():
    import torch
    from paper_2211_00484_amd import tbs
    T, U, c = 30, 12, math.log(0.25)
    blank = torch.full((3, T, U + 1), c, dtype=torch.float32, device="cuda")
    label = torch.full((3, T, U), c, dtype=torch.float32, device="cuda")
    cf = float(np.float32(c))
    lens = [[T, U], [0, 3], [T, U + 1]]
    for kind, want in (("standard", math.log(math.comb(T - 1 + U, U)) + (T + U) * cf),
                       ("modified", math.log(math.comb(T, U)) + T * cf),
                       ("constrained", math.log(math.comb(T, U)) + (T + U) * cf)):
        total, _, status = tbs.transducer_forward(kind, blank, label, lens)
        torch.cuda.synchronize()
        total, status = total.cpu().numpy(), status.cpu().numpy()
        assert total[0] == pytest.approx(want, rel=1e-12)
        assert status.tolist() == [0, 1, 1] and np.isnan(total[1:]).all()
    with pytest.raises(tbs.TbsError):
        tbs.transducer_forward("standard", torch.zeros((1, 2, 1025), device="cuda"),
                               torch.zeros((1, 2, 1024), device="cuda"), [[2, 3]])
