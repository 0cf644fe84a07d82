"""Exact-tie pins for the oracle's merge / prune ordering (Sec. 2.5 readings).

With a zero joiner weight and zero bias every label has the same log-probability
-log V, so candidate scores tie exactly and only the ordering rules decide:

* merge: max score, then smaller (parent index, arc position), blank counting as -1;
* beam + max-states: score descending, then (graph state, context) ascending;
  a tuple exactly at best - beam is kept;
* max-contexts: context score descending, then context id ascending;
* survivors stored in (context, state) ascending order; final pick: first in that order.

The hand-derived traces below are the expected results of those rules.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2211_00484_amd import synth
from ref_search import LayerJoiner, beam_search_sorted


def _flat_model(V, C=4):
    return synth.Model(V, C, embed=np.zeros((V, C), np.float32), conv=np.zeros((C, 2), np.float32),
                       w_out=np.zeros((V, C), np.float32), b_out=np.zeros(V, np.float32))


def _graph(S, start, arcs, V, final=None):
    arcs = sorted(arcs, key=lambda a: a[0])
    rp = np.zeros(S + 1, np.int32)
    for s, _, _, _ in arcs:
        rp[s + 1] += 1
    rp = np.cumsum(rp).astype(np.int32)
    return synth.Graph(S, start, V, rp, np.array([a[1] for a in arcs], np.int32),
                       np.array([a[2] for a in arcs], np.int32),
                       np.array([a[3] for a in arcs], np.float32), final)


def _run(model, graph, T, beam, Ns, Nc, lengths=None):
    enc = np.zeros((1, T, model.dim), np.float32)
    lens = np.array([T] if lengths is None else lengths, np.int32)
    return oracle.decode(model, graph, enc, lens, beam, Ns, Nc)


def _surv(res, f):
    return [tuple(int(v) for v in x) for x in res.trace[f, 0] if x[0] >= 0]


def test_trivial_graph_all_ties():
    # V = 3, one state, T = 2, Ns = Nc = 2.  Frame 0: blank -> ctx 0, labels 1, 2 -> ctx 1, 2,
    # all scored -log 3; (state, ctx) order keeps ctx 0 and ctx 1.  Frame 1: key (0, ctx 1)
    # is reached by label 1 from parent 0 and by blank from parent 1: parent 0 wins.
    V = 3
    res = _run(_flat_model(V), synth.trivial_graph(V), 2, math.inf, 2, 2)
    assert _surv(res, 1) == [(0, 0, 0, 0), (1, 0, 0, 1)]
    assert _surv(res, 2) == [(0, 0, 0, 0), (1, 0, 0, 1)]
    assert res.token_lists()[0] == []
    assert res.scores[0] == pytest.approx(-2 * math.log(3), abs=1e-12)


def test_state_before_context_in_prune_order():
    # Two states; from start 1: label 1 -> state 0, label 2 -> state 1 (both q = 0).  Candidates
    # after frame 0: (s1, ctx 0) blank, (s0, ctx 1), (s1, ctx 2).  Ns = 1 keeps the smallest
    # (state, context) = (s0, ctx 1), not the smallest context.
    V = 3
    g = _graph(2, 1, [(1, 0, 1, 0.0), (1, 1, 2, 0.0)], V)
    res = _run(_flat_model(V), g, 1, math.inf, 1, 1)
    assert _surv(res, 1) == [(1, 0, 0, 1)]
    assert res.token_lists()[0] == [1]


def test_blank_beats_arc_on_tie_of_same_parent():
    # s0 --1 (+1)--> s1 --1 (+1)--> s2, and s2 has a self-loop labelled 1 (q = 0).  With
    # max_states = 1 the positive arc scores steer the path to (ctx (1,1), s2) after two
    # frames.  On frame 2 blank and the loop reach the same (s2, ctx (1,1)) from the same
    # parent with equal score; blank counts as arc position -1 and wins.
    V = 2
    g = _graph(3, 0, [(0, 1, 1, 1.0), (1, 2, 1, 1.0), (2, 2, 1, 0.0)], V)
    res = _run(_flat_model(V), g, 3, math.inf, 1, 1)
    assert _surv(res, 1) == [(1, 1, 0, 1)]
    assert _surv(res, 2) == [(3, 2, 0, 1)]
    assert _surv(res, 3) == [(3, 2, 0, 0)]
    assert res.token_lists()[0] == [1, 1]


def test_tuple_exactly_at_beam_edge_is_kept():
    # First frame: blank and label 1 (q = 0) score -log 3; label 2 (q = -1) scores -1 - log 3,
    # exactly best - beam for beam = 1.  The comparison is inclusive, so all three survive.
    V = 3
    g = _graph(1, 0, [(0, 0, 1, 0.0), (0, 0, 2, -1.0)], V)
    res = _run(_flat_model(V), g, 1, 1.0, 8, 8)
    assert _surv(res, 1) == [(0, 0, 0, 0), (1, 0, 0, 1), (2, 0, 0, 2)]
    res = _run(_flat_model(V), g, 1, 0.999, 8, 8)
    assert _surv(res, 1) == [(0, 0, 0, 0), (1, 0, 0, 1)]


def test_context_ties_broken_by_context_id():
    # Three contexts tie; max_contexts = 2 keeps the two smallest context ids, and the
    # final pick among equal scores is the first survivor in canonical order.
    V = 4
    g = _graph(1, 0, [(0, 0, 3, 0.0), (0, 0, 2, 0.0), (0, 0, 1, 0.0)], V)
    res = _run(_flat_model(V), g, 1, math.inf, 4, 2)
    assert _surv(res, 1) == [(0, 0, 0, 0), (1, 0, 0, 1)]
    assert res.token_lists()[0] == []


def test_final_weights_and_nonfinal_fallback():
    V = 3
    fin = np.array([-np.inf, -0.5], np.float32)
    g = _graph(2, 0, [(0, 1, 1, 0.0), (0, 0, 2, 0.0)], V, final=fin)
    res = _run(_flat_model(V), g, 1, math.inf, 4, 4)
    # survivors: (ctx 0, s0) blank, (ctx 1, s1), (ctx 2, s0); only s1 is final
    assert res.status[0] == 0 and res.token_lists()[0] == [1]
    assert res.scores[0] == pytest.approx(-math.log(3) - 0.5, abs=1e-6)
    g.final = np.array([-np.inf, -np.inf], np.float32)
    res = _run(_flat_model(V), g, 1, math.inf, 4, 4)
    assert res.status[0] == 1 and res.token_lists()[0] == []


@pytest.mark.parametrize("seed", range(24))
def test_tie_heavy_random_graphs_match_sorted_reference(seed):
    # Flat joiner, arc scores from {0, -1, -2}, duplicate arcs: ties everywhere.
    rng = np.random.default_rng(500 + seed)
    V = int(rng.integers(2, 6))
    S = int(rng.integers(1, 6))
    T = int(rng.integers(1, 8))
    arcs = []
    for s in range(S):
        for _ in range(int(rng.integers(0, 5))):
            arcs.append((s, int(rng.integers(0, S)), int(rng.integers(1, V)),
                         float(-int(rng.integers(0, 3)))))
    if not arcs:
        arcs.append((0, 0, 1, 0.0))
    g = _graph(S, int(rng.integers(0, S)), arcs, V)
    beam = [math.inf, 1.0, 2.0][seed % 3]
    Ns = int(rng.integers(1, 7))
    Nc = int(rng.integers(1, Ns + 1))
    model = _flat_model(V)
    res = _run(model, g, T, beam, Ns, Nc)
    score, tokens, trace = beam_search_sorted(LayerJoiner(model), g, np.zeros((T, model.dim), np.float32),
                                              T, beam, Ns, Nc)
    assert res.token_lists()[0] == tokens
    for f, surv in enumerate(trace):
        assert _surv(res, f) == [tuple(int(v) for v in x) for x in surv]
