"""Pins of the oracle's transducer forward recursions (Sec. 3, eq. 1-3)."""
import itertools
import math

import numpy as np
import pytest

import oracle


def _lse(xs):
    m = max(xs)
    return m + math.log(sum(math.exp(x - m) for x in xs))


def _enumerate(kind, bl, lb, T, U):
    """log of the summed weight of every alignment of U labels to T frames."""
    terms = []
    if kind == "standard":
        moves = T - 1 + U
        for lab_pos in itertools.combinations(range(moves), U):
            t = u = 0
            w = 0.0
            for k in range(moves):
                if k in lab_pos:
                    w += lb[t, u]
                    u += 1
                else:
                    w += bl[t, u]
                    t += 1
            terms.append(w + bl[T - 1, U])
    else:
        for lab_frames in itertools.combinations(range(T), U):
            u = 0
            w = 0.0
            for t in range(T):
                if t in lab_frames:
                    w += lb[t, u] + (bl[t, u + 1] if kind == "constrained" else 0.0)
                    u += 1
                else:
                    w += bl[t, u]
            terms.append(w)
    return _lse(terms)


@pytest.mark.parametrize("kind", ["standard", "modified", "constrained"])
@pytest.mark.parametrize("seed", range(10))
def test_equals_enumeration(kind, seed):
    rng = np.random.default_rng(seed)
    T = int(rng.integers(1, 7))
    U = int(rng.integers(0, min(T, 4) + 1)) if kind != "standard" else int(rng.integers(0, 4))
    bl = np.log(rng.uniform(0.05, 1.0, size=(1, T, U + 1))).astype(np.float32)
    lb = np.log(rng.uniform(0.05, 1.0, size=(1, T, U))).astype(np.float32)
    total, alpha = oracle.transducer_forward(kind, bl, lb, [T], [U])
    want = _enumerate(kind, bl[0].astype(np.float64), lb[0].astype(np.float64), T, U)
    assert total[0] == pytest.approx(want, abs=1e-9)


@pytest.mark.parametrize("kind", ["standard", "modified", "constrained"])
def test_constant_logprobs_count_paths(kind):
    T, U, c = 9, 4, math.log(0.3)
    bl = np.full((1, T, U + 1), c, dtype=np.float32)
    lb = np.full((1, T, U), c, dtype=np.float32)
    total, _ = oracle.transducer_forward(kind, bl, lb, [T], [U])
    cf = float(np.float32(c))
    if kind == "standard":
        want = math.log(math.comb(T - 1 + U, U)) + (T + U) * cf
    elif kind == "modified":
        want = math.log(math.comb(T, U)) + T * cf
    else:
        want = math.log(math.comb(T, U)) + (T + U) * cf
    assert total[0] == pytest.approx(want, abs=1e-9)


@pytest.mark.parametrize("kind", ["standard", "modified", "constrained"])
def test_ragged_lengths_equal_cropped_problems(kind):
    rng = np.random.default_rng(5)
    B, T, U = 4, 12, 6
    bl = np.log(rng.uniform(0.05, 1.0, size=(B, T, U + 1))).astype(np.float32)
    lb = np.log(rng.uniform(0.05, 1.0, size=(B, T, U))).astype(np.float32)
    frames = [12, 7, 1, 9]
    labels = [6, 3, 0, 5]
    total, _ = oracle.transducer_forward(kind, bl, lb, frames, labels)
    for b in range(B):
        Tb, Ub = frames[b], labels[b]
        t1, _ = oracle.transducer_forward(kind, np.ascontiguousarray(bl[b:b + 1, :Tb, :Ub + 1]),
                                          np.ascontiguousarray(lb[b:b + 1, :Tb, :Ub]), [Tb], [Ub])
        assert total[b] == pytest.approx(t1[0], abs=1e-12)


def test_more_labels_than_frames_is_impossible_for_one_label_per_frame():
    bl = np.zeros((1, 3, 5), dtype=np.float32)
    lb = np.zeros((1, 3, 4), dtype=np.float32)
    for kind in ("modified", "constrained"):
        total, _ = oracle.transducer_forward(kind, bl, lb, [3], [4])
        assert total[0] == -math.inf
    total, _ = oracle.transducer_forward("standard", bl, lb, [3], [4])
    assert total[0] == pytest.approx(math.log(math.comb(2 + 4, 4)))
