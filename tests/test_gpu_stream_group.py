"""Grouped per-stream kernel (several workgroups share one stream) against the oracle.

Trivial graph, fp32 joiner: G workgroups per stream (8, 4 or 2, each with 64 or 128
vocabulary columns) exchange per-row normaliser terms and best labels every frame.
Each case states the grouping the shape must take (G = 1: the single-workgroup
kernel); the profile counters confirm which kernel ran.  Parity as in
test_gpu_decode.py.
"""
import math

import numpy as np
import pytest

import oracle
from gpu_util import say
from parity import check_trace_invariants, compare, replay_check
from paper_2211_00484_amd import synth

pytestmark = pytest.mark.gpu

# V, C, B, Ns, Nc, beam, grouped
CASES = [
    (128, 64, 5, 4, 4, math.inf, True),      # 2 column groups: G = 2, one each
    (256, 512, 40, 8, 8, math.inf, True),    # G = 4, 8 rows (2 row groups)
    (256, 96, 100, 4, 3, 2.0, True),         # B x 4 > 256 CUs: G = 2, two column groups each
    (500, 300, 48, 16, 12, 6.0, True),       # G = 4, two column groups each, 12 rows
    (500, 700, 7, 4, 2, 3.0, True),          # K = 1024, G = 8
    (448, 512, 20, 16, 16, math.inf, False),  # 7 column groups: no grouping
    # B x G = 256, one workgroup on every CU: a stream's members share one XCD and pass
    # their words through its L2
    (256, 512, 64, 8, 8, math.inf, True),    # G = 4, 8 rows
    (128, 64, 128, 4, 4, 2.0, True),         # G = 2, the per-wave fast path
]


@pytest.mark.parametrize("V,C,B,Ns,Nc,beam,grouped", CASES)
def test_grouped_trivial(V, C, B, Ns, Nc, beam, grouped):
    import torch
    from paper_2211_00484_amd import tbs
    rng = np.random.default_rng(1000 + V + B)
    model_np = synth.make_model(rng, V, C, 0.05)
    inputs = synth.make_inputs(rng, B, 30, C, length_range=(0, 30))
    graph_np = synth.trivial_graph(V)
    say(f"grouped decode V={V} C={C} B={B} Ns={Ns} Nc={Nc} beam={beam}")
    model = tbs.Model.from_synth(model_np)
    graph = tbs.Graph.from_synth(graph_np)
    model.set_schedule("stream")
    model.set_profiling(True)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    out = tbs.decode(model, graph, enc, inputs.lengths, beam=beam, max_states=Ns,
                     max_contexts=Nc, want_arcs=True, want_trace=True)
    torch.cuda.synchronize()
    prof = model.read_profile()
    model.set_profiling(False)
    assert (prof["stream_group"][0] > 0) == grouped, prof
    assert (prof["stream"][0] > 0) == (not grouped), prof
    g = {"tokens": out.tokens.cpu().numpy(), "ntok": out.num_tokens.cpu().numpy(),
         "scores": out.scores.cpu().numpy(), "status": out.status.cpu().numpy(),
         "arcs": out.arcs.cpu().numpy(), "trace": out.trace.cpu().numpy()}
    assert (g["status"] != 2).all(), "exchange wait timed out"
    streams = list(range(B))
    o = oracle.decode(model_np, graph_np, inputs.encoder_out, inputs.lengths, beam, Ns, Nc,
                      streams=streams)
    rep = compare(g, o, model_np, graph_np, inputs.encoder_out, inputs.lengths, streams,
                  margin=1e-4, score_tol=1e-4)
    check_trace_invariants(g["trace"], inputs.lengths, graph_np, V, Ns, min(Nc, Ns), streams)
    say(f"  {rep}")
    rrep = replay_check(g, model_np, graph_np, inputs.encoder_out, inputs.lengths, streams, beam,
                        Ns, min(Nc, Ns), margin=1e-4, tol=1e-4)
    say(f"  {rrep}")
    assert rrep.exact >= 0.9 * rrep.frames


def test_grouped_repeated_decodes_agree():
    # Successive decodes reuse the exchange buffer under new epochs: identical results.
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("standard")
    model = tbs.Model.from_synth(model_np)
    graph = tbs.Graph.from_synth(graph_np)
    model.set_schedule("stream")
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    outs = []
    for _ in range(3):
        out = tbs.decode(model, graph, enc, inputs.lengths, beam=math.inf, max_states=4,
                         max_contexts=4, want_trace=True)
        torch.cuda.synchronize()
        outs.append((out.tokens.cpu().numpy(), out.scores.cpu().numpy(), out.trace.cpu().numpy()))
    for a in outs[1:]:
        for x, y in zip(outs[0], a):
            assert np.array_equal(x, y)


def test_grouped_timeout_path_reports_and_recovers():
    # A one-poll budget makes exchange waits give up while other members are still
    # working (every kernel still finishes: waits are bounded and a timed-out wait takes
    # a neutral payload).  Streams that gave up report status 2 and a NaN score; with
    # the default budget restored the next decode is the normal one again.
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("standard")
    model = tbs.Model.from_synth(model_np)
    graph = tbs.Graph.from_synth(graph_np)
    model.set_schedule("stream")
    enc = torch.from_numpy(inputs.encoder_out).cuda()

    def run():
        out = tbs.decode(model, graph, enc, inputs.lengths, beam=math.inf, max_states=4,
                         max_contexts=4, want_trace=True)
        torch.cuda.synchronize()
        return (out.status.cpu().numpy(), out.scores.cpu().numpy(), out.tokens.cpu().numpy(),
                out.trace.cpu().numpy())

    ref = run()
    assert (ref[0] == 0).all()
    model.set_exchange_spin_limit(1)
    st, sc, _, _ = run()
    say(f"  one-poll budget: {int((st == 2).sum())} of {inputs.B} streams timed out")
    assert set(np.unique(st).tolist()) <= {0, 2}
    assert np.array_equal(st == 2, np.isnan(sc))
    model.set_exchange_spin_limit(0)
    again = run()
    for x, y in zip(ref, again):
        assert np.array_equal(x, y)
    with pytest.raises(tbs.TbsError, match="EINVAL"):
        model.set_exchange_spin_limit(-1)
