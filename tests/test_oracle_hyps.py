"""Pins of the oracle's full-sequence beam search (Table 5's comparison search)."""
import math

import numpy as np
import pytest

import oracle
from paper_2211_00484_amd import synth
from ref_search import LayerJoiner, brute_force, greedy, hyp_beam_search, sequence_totals

BIG = 100000


def _case(seed, T, V, C=5, sigma=0.8, B=1):
    rng = np.random.default_rng(seed)
    model = synth.make_model(rng, V, C, sigma)
    inputs = synth.make_inputs(rng, B, T, C)
    return model, inputs


@pytest.mark.parametrize("seed", range(16))
def test_unpruned_max_is_the_best_path(seed):
    rng = np.random.default_rng(3000 + seed)
    T, V = int(rng.integers(1, 6)), int(rng.integers(2, 5))
    model, inputs = _case(seed, T, V)
    r = oracle.hyp_search(model, inputs.encoder_out, inputs.lengths, BIG, logadd=False)
    score, tokens, _, _ = brute_force(LayerJoiner(model), synth.trivial_graph(V),
                                      inputs.encoder_out[0], T)
    assert r.scores[0] == pytest.approx(score, abs=1e-9)
    if r.frame_margins[0, T] > 1e-9:
        assert r.token_lists()[0] == tokens


@pytest.mark.parametrize("seed", range(16))
def test_unpruned_logadd_is_the_most_probable_sequence(seed):
    rng = np.random.default_rng(4000 + seed)
    T, V = int(rng.integers(1, 6)), int(rng.integers(2, 5))
    model, inputs = _case(seed, T, V)
    totals, _ = sequence_totals(LayerJoiner(model), synth.trivial_graph(V),
                                inputs.encoder_out[0], T)
    ranked = sorted(totals.values(), reverse=True)
    if len(ranked) > 1 and ranked[0] - ranked[1] < 1e-9:
        pytest.skip("two sequences tie")
    r = oracle.hyp_search(model, inputs.encoder_out, inputs.lengths, BIG, logadd=True)
    want = max(totals, key=totals.get)
    assert tuple(r.token_lists()[0]) == want
    assert r.scores[0] == pytest.approx(totals[want], abs=1e-9)


@pytest.mark.parametrize("logadd", [False, True])
@pytest.mark.parametrize("seed", range(6))
def test_single_hypothesis_is_greedy(seed, logadd):
    model, inputs = _case(seed, 30, 7, C=8, sigma=0.5)
    r = oracle.hyp_search(model, inputs.encoder_out, inputs.lengths, 1, logadd=logadd)
    score, tokens = greedy(LayerJoiner(model), inputs.encoder_out[0], 30)
    assert r.token_lists()[0] == tokens
    assert r.scores[0] == pytest.approx(score, abs=1e-9)


@pytest.mark.parametrize("N", [2, 4, 7])
@pytest.mark.parametrize("logadd", [False, True])
@pytest.mark.parametrize("seed", range(4))
def test_pruned_equals_independent_reference(seed, logadd, N):
    model, inputs = _case(100 + seed, 12, 6, C=7, sigma=0.7)
    r = oracle.hyp_search(model, inputs.encoder_out, inputs.lengths, N, logadd=logadd)
    tokens, score = hyp_beam_search(LayerJoiner(model), inputs.encoder_out[0], 12, N, logadd)
    if np.min(r.frame_margins[0]) > 1e-9:
        assert r.token_lists()[0] == tokens
        assert r.scores[0] == pytest.approx(score, abs=1e-9)


def test_trace_reconstructs_the_result():
    model, inputs = _case(7, 15, 9, C=6, sigma=0.6, B=3)
    inputs.lengths[:] = [15, 0, 9]
    for b in range(3):
        inputs.encoder_out[b, inputs.lengths[b]:] = 0.0
    r = oracle.hyp_search(model, inputs.encoder_out, inputs.lengths, 4, logadd=True)
    for b in range(3):
        L = int(inputs.lengths[b])
        k, labels = 0, []
        for f in range(L, 0, -1):
            parent, lab = r.trace[f, b, k]
            if lab > 0:
                labels.append(int(lab))
            k = int(parent)
        assert k == 0 and labels[::-1] == r.token_lists()[b]
        assert (r.trace[L + 1:, b] == -1).all()
    assert r.ntok[1] == 0 and r.scores[1] == 0.0
