"""Pins for the oracle's decision margins (Sec. 2.5 pruning; the margins decide which
frames the GPU parity rule compares bit for bit).

A frame's margin is the smallest gap at any decision the frame takes: the max-states
cut, each tuple's distance to the beam threshold, the max-contexts cut and, for every
kept tuple, the gap between its merge winner and the best candidate with another
(parent, label); the final margin is the gap between the two best final values.
Three checks pin the oracle's value on random pruned cases, walking the oracle's own
trajectory with an independent stage-by-stage selection (``ref_search.frame_decisions``):

* it equals the minimum of the gaps that selection derives;
* soundness: random perturbations of every candidate's score by less than half the
  margin never change any decision of the frame;
* tightness: shifting the two sides of the binding decision by just over half the
  margin changes the frame's decisions, so the margin is not under-reported.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2211_00484_amd import synth
from ref_search import LayerJoiner, frame_candidates, frame_decisions


def _outcome(d):
    return (tuple(sorted(d["winners"].items())), d["pre"], d["ctx"], tuple(d["kept"]))


def _cases():
    out = []
    for seed in range(14):
        rng = np.random.default_rng(500 + seed)
        V = int(rng.integers(3, 9))
        C = int(rng.integers(4, 12))
        S = int(rng.integers(1, 6))
        trivial = seed % 4 == 0
        beam = [math.inf, 2.0, 0.7, 0.0][seed % 4]
        Ns = int(rng.integers(1, 9))
        Nc = int(rng.integers(1, Ns + 1))
        out.append((seed, V, C, S, trivial, beam, Ns, Nc))
    return out


@pytest.mark.parametrize("seed,V,C,S,trivial,beam,Ns,Nc", _cases())
def test_frame_margins_pinned(seed, V, C, S, trivial, beam, Ns, Nc):
    rng = np.random.default_rng(seed)
    model = synth.make_model(rng, V, C, 0.8)
    inputs = synth.make_inputs(rng, 2, 12, C)
    graph = synth.trivial_graph(V) if trivial else synth.random_small_graph(
        rng, S, V, max_degree=4, with_final=bool(seed % 2))
    res = oracle.decode(model, graph, inputs.encoder_out, inputs.lengths, beam, Ns, Nc)
    j = LayerJoiner(model)
    checked = tight = 0
    for b in range(inputs.B):
        enc = inputs.encoder_out[b]
        hyps = [(0, graph.start, 0.0)]
        L = int(inputs.lengths[b])
        for t in range(L):
            cands = frame_candidates(lambda ctx: j(enc[t], ctx // V, ctx % V), graph, hyps, V)
            d = frame_decisions(cands, beam, Ns, Nc)
            got = [[k[1], k[0], *d["winners"][k]] for k in d["kept"]]
            n = len(got)
            assert res.trace[t + 1, b, :n].tolist() == got, (b, t)
            m = min((g for g, _, _ in d["terms"]), default=math.inf)
            fm = float(res.frame_margins[b, t])
            assert fm == pytest.approx(m, abs=1e-9), (b, t)
            base = _outcome(d)
            if math.isfinite(m) and m > 1e-9:
                for _ in range(6):
                    delta = rng.uniform(-0.49 * m, 0.49 * m, len(cands))
                    assert _outcome(frame_decisions(cands, beam, Ns, Nc, delta)) == base, (b, t)
            if math.isfinite(m):
                g, lower, rise = min(d["terms"], key=lambda x: x[0])
                shift = 0.51 * g + 1e-9
                delta = np.zeros(len(cands))
                lo = set(lower) if lower is not None else set(range(len(cands))) - set(rise)
                hi = set(rise) if rise is not None else set(range(len(cands))) - set(lower)
                delta[list(lo)] -= shift
                delta[list(hi)] += shift
                assert _outcome(frame_decisions(cands, beam, Ns, Nc, delta)) != base, (b, t)
                tight += 1
            checked += 1
            hyps = [(k[1], k[0], d["scores"][k]) for k in d["kept"]]
        # final margin: gap between the two best final values of the last survivors
        fin = graph.final
        vals = []
        for ctx, s, v in hyps:
            f = 0.0 if fin is None else float(fin[s])
            vals.append(v + f if math.isfinite(f) else -math.inf)
        if not any(math.isfinite(x) for x in vals):
            vals = [v for _, _, v in hyps]
        vals = sorted(vals, reverse=True)
        want = vals[0] - vals[1] if len(vals) > 1 and math.isfinite(vals[1]) else math.inf
        assert float(res.frame_margins[b, inputs.T]) == pytest.approx(want, abs=1e-9)
    assert checked > 0


def test_zero_beam_margins_are_not_all_zero():
    # beam 0 keeps only tuples tied with the best; the best itself is not a contested
    # decision, so a frame without ties has a positive margin
    rng = np.random.default_rng(3)
    model = synth.make_model(rng, 6, 8, 0.8)
    inputs = synth.make_inputs(rng, 1, 10, 8)
    res = oracle.decode(model, synth.trivial_graph(6), inputs.encoder_out, inputs.lengths,
                        0.0, 4, 4)
    assert (res.frame_margins[0, :10] > 1e-3).all()
