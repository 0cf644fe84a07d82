"""Pins of the oracle's lattice and label-sequence (LogAdd) search, Sec. 2.5.

Independent references: exhaustive enumeration of alignments (``ref_search``), the
library-layer joiner, and path posteriors enumerated here from the lattice arrays.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2211_00484_amd import synth
from ref_search import LayerJoiner, sequence_totals

BIG = 100000


def _case(seed, T, V, C, S, max_degree, with_final, sigma=0.8):
    rng = np.random.default_rng(seed)
    model = synth.make_model(rng, V, C, sigma)
    inputs = synth.make_inputs(rng, 1, T, C)
    if S == 0:
        graph = synth.trivial_graph(V)
    else:
        graph = synth.random_small_graph(rng, S, V, max_degree=max_degree, with_final=with_final)
    return model, inputs, graph


def _tiny(seed):
    rng = np.random.default_rng(2000 + seed)
    T = int(rng.integers(1, 6))
    V = int(rng.integers(2, 5))
    S = int(rng.integers(0, 4))
    return _case(seed, T, V, 5, S, max_degree=3, with_final=bool(seed % 2)), T


@pytest.mark.parametrize("seed", range(24))
def test_unpruned_lattice_total_and_sequences_equal_enumeration(seed):
    (model, inputs, graph), T = _tiny(seed)
    lat = oracle.lattice(model, graph, inputs.encoder_out, inputs.lengths, math.inf, BIG, BIG)
    s = lat.stream(0)
    totals, total = sequence_totals(LayerJoiner(model), graph, inputs.encoder_out[0], T)
    assert s.total == pytest.approx(total, abs=1e-9)
    for y, v in totals.items():
        assert lat.sequence_score(0, y) == pytest.approx(v, abs=1e-9), y
    # a sequence no alignment produces has probability zero
    assert lat.sequence_score(0, [1] * (T + 1)) == -math.inf


@pytest.mark.parametrize("seed", range(16))
def test_logadd_best_equals_enumeration(seed):
    (model, inputs, graph), T = _tiny(seed)
    totals, _ = sequence_totals(LayerJoiner(model), graph, inputs.encoder_out[0], T)
    ranked = sorted(totals.values(), reverse=True)
    if len(ranked) > 1 and ranked[0] - ranked[1] < 1e-9:
        pytest.skip("two label sequences tie")
    lat = oracle.lattice(model, graph, inputs.encoder_out, inputs.lengths, math.inf, BIG, BIG)
    u = np.random.default_rng(seed).uniform(size=(3000, T + 1))
    nb = lat.nbest(0, u)
    want = max(totals, key=totals.get)
    assert tuple(nb.tokens) == want
    assert nb.score == pytest.approx(totals[want], abs=1e-9)
    # every sampled distinct sequence is scored with its exact total
    for y, v in zip(nb.seqs, nb.scores):
        assert v == pytest.approx(totals[tuple(y)], abs=1e-9)
    assert len({tuple(y) for y in nb.seqs}) == len(nb.seqs)


def _lattice_paths(s):
    """All complete paths of a stream lattice by enumeration: {(arc index per frame...,
    final node): log weight}."""
    out = {}

    def rec(f, node, arcs, w):
        if f == 0:
            out[tuple(reversed(arcs))] = w
            return
        for k, a in enumerate(s.arcs[f - 1]):
            if a[1] == node:
                rec(f - 1, int(a[0]), arcs + [k], w + float(s.w[f - 1][k]))

    for j, fwj in enumerate(s.fw):
        if fwj != -math.inf:
            before = len(out)
            rec(s.len, j, [], float(fwj))
            # key the paths of node j with the final node appended
            new = list(out.items())[before:]
            for key, val in new:
                del out[key]
                out[key + (j,)] = val
    return out


@pytest.mark.parametrize("seed", range(4))
def test_sampling_follows_path_posteriors(seed):
    model, inputs, graph = _case(50 + seed, 4, 3, 5, 0 if seed % 2 else 2, 2, bool(seed // 2),
                                 sigma=0.5)
    lat = oracle.lattice(model, graph, inputs.encoder_out, inputs.lengths, math.inf, BIG, BIG)
    s = lat.stream(0)
    paths = _lattice_paths(s)
    logs = np.array(list(paths.values()))
    m = logs.max()
    tot = m + math.log(np.exp(logs - m).sum())
    assert tot == pytest.approx(s.total, abs=1e-9)
    N = 20000
    u = np.random.default_rng(seed).uniform(size=(N, s.len + 1))
    nb = lat.nbest(0, u)
    counts = {}
    for p in range(N):
        key = tuple(int(x) for x in nb.paths[p])
        assert key in paths, "sampled a sequence of arcs that is not a lattice path"
        counts[key] = counts.get(key, 0) + 1
    for key, lw in paths.items():
        pr = math.exp(lw - tot)
        freq = counts.get(key, 0) / N
        assert abs(freq - pr) <= 5 * math.sqrt(pr * (1 - pr) / N) + 2e-3, (key, freq, pr)


def test_sampling_single_path_lattice():
    # Ns = Nc = 1: one node per frame, so every sampled path is the search's best path
    rng = np.random.default_rng(3)
    model = synth.make_model(rng, 4, 6, 0.5)
    inputs = synth.make_inputs(rng, 1, 6, 6)
    lat = oracle.lattice(model, synth.trivial_graph(4), inputs.encoder_out, inputs.lengths,
                         math.inf, 1, 1)
    s = lat.stream(0)
    nb = lat.nbest(0, np.random.default_rng(0).uniform(size=(20, 7)))
    assert len(nb.seqs) == 1
    r = oracle.decode(model, synth.trivial_graph(4), inputs.encoder_out, inputs.lengths,
                      math.inf, 1, 1)
    assert nb.tokens == [int(x) for x in r.token_lists()[0]]
    # one node per frame: the only choices are among parallel arcs into it
    for f in range(s.len):
        if len(s.arcs[f]) == 1:
            assert (nb.margins[:, f] == np.inf).all()


@pytest.mark.parametrize("beam,Ns,Nc", [(2.0, 4, 3), (math.inf, 3, 2), (0.7, 8, 8), (math.inf, 1, 1)])
@pytest.mark.parametrize("seed", range(3))
def test_pruned_lattice_structure(seed, beam, Ns, Nc):
    """Nodes are the search's survivors; arcs are exactly the expansions of frame-f
    survivors whose (state, context) survived, with weight q + log P; the best lattice
    path is the search's best path."""
    rng = np.random.default_rng(70 + seed)
    V, C = 7, 9
    model = synth.make_model(rng, V, C, 0.8)
    inputs = synth.make_inputs(rng, 2, 12, C, length_range=(0, 12))
    graph = synth.random_small_graph(rng, 5, V, max_degree=4, with_final=bool(seed % 2))
    lat = oracle.lattice(model, graph, inputs.encoder_out, inputs.lengths, beam, Ns, Nc)
    dec = oracle.decode(model, graph, inputs.encoder_out, inputs.lengths, beam, Ns, Nc)
    J = LayerJoiner(model)
    rp, dest, lab, q = graph.row_ptr, graph.dest, graph.label, graph.score
    for b in range(inputs.B):
        s = lat.stream(b)
        L = int(inputs.lengths[b])
        assert s.len == L
        for f in range(L + 1):
            n = len(s.nodes[f])
            assert np.array_equal(s.nodes[f], dec.trace[f, b, :n])
            assert (dec.trace[f, b, n:] == -1).all()
        vit = [np.array([0.0])]
        for f in range(L):
            nxt = {(int(x[0]), int(x[1])): j for j, x in enumerate(s.nodes[f + 1])}
            want = []
            for i, x in enumerate(s.nodes[f]):
                ctx, st = int(x[0]), int(x[1])
                lp = J(inputs.encoder_out[b, f], ctx // V, ctx % V)
                if (ctx, st) in nxt:
                    want.append((nxt[(ctx, st)], i, -1, 0, -1, lp[0]))
                for k in range(rp[st], rp[st + 1]):
                    key = ((ctx % V) * V + int(lab[k]), int(dest[k]))
                    if key in nxt:
                        want.append((nxt[key], i, k - rp[st], int(lab[k]), k,
                                     float(q[k]) + lp[int(lab[k])]))
            want.sort(key=lambda a: (a[0], a[1], a[2]))
            got = s.arcs[f]
            assert len(got) == len(want)
            for g_, w_ in zip(got, want):
                assert (int(g_[1]), int(g_[0]), int(g_[2]), int(g_[3])) == (w_[0], w_[1], w_[3], w_[4])
            assert np.allclose(s.w[f], [w_[5] for w_ in want], atol=1e-9, rtol=0)
            # Viterbi over the lattice
            v = np.full(len(s.nodes[f + 1]), -math.inf)
            for k, a in enumerate(got):
                v[a[1]] = max(v[a[1]], vit[f][a[0]] + s.w[f][k])
            vit.append(v)
        best = max(vit[L][j] + s.fw[j] for j in range(len(s.fw)))
        assert best == pytest.approx(dec.scores[b], abs=1e-9)
        assert s.status == dec.status[b]


def test_nbest_paths_are_valid_and_sequences_distinct():
    w, inputs, model, graph = synth.make_workload("tiny")
    lat = oracle.lattice(model, graph, inputs.encoder_out, inputs.lengths, math.inf, 4, 4)
    for b in range(inputs.B):
        s = lat.stream(b)
        u = np.random.default_rng(b).uniform(size=(64, s.len + 1))
        nb = lat.nbest(b, u)
        for p in range(64):
            node = int(nb.paths[p, s.len])
            assert s.fw[node] != -math.inf
            for f in range(s.len - 1, -1, -1):
                a = s.arcs[f][nb.paths[p, f]]
                assert a[1] == node
                node = int(a[0])
            assert node == 0
        assert len({tuple(y) for y in nb.seqs}) == len(nb.seqs)
        assert nb.score == max(nb.scores)
        assert nb.score <= s.total + 1e-12
        assert (nb.margins >= 0).all()
