"""Streaming decode (tbs_state_create / tbs_decode_chunk / tbs_state_finish).

A stream's frames split into chunks in any way must give exactly what one
tbs_decode over all of them gives on the same schedule: the same kernels run the
same arithmetic on the same survivors, so tokens, arcs, status, fp64 scores and
the survivor trace are compared bit for bit.  (The one-shot decode itself is
checked against the CPU oracle in test_gpu_decode.py and test_gpu_stream_group.py.)
"""
import math

import numpy as np
import pytest

from gpu_util import say
from paper_2211_00484_amd import synth

pytestmark = pytest.mark.gpu


def _one_shot(model, graph, inputs, beam, Ns, Nc):
    import torch
    from paper_2211_00484_amd import tbs
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    out = tbs.decode(model, graph, enc, inputs.lengths, beam=beam, max_states=Ns,
                     max_contexts=Nc, want_arcs=True, want_trace=True)
    torch.cuda.synchronize()
    return out


def _chunked(model, graph, inputs, beam, Ns, Nc, rng, max_chunk, finish_midway=False):
    import torch
    from paper_2211_00484_amd import tbs
    B, T, C = inputs.encoder_out.shape
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    state = tbs.DecodeState(model, graph, B, max(T, 1), beam=beam, max_states=Ns,
                            max_contexts=Nc)
    trace = torch.full((max(T, 1) + 1, B, Ns, 4), -1, dtype=torch.int32, device="cuda")
    pos = np.zeros(B, dtype=np.int64)
    calls = 0
    while (pos < inputs.lengths).any():
        # each stream takes a random piece (possibly none) of what it has left
        left = inputs.lengths - pos
        piece = np.array([rng.integers(0, min(max_chunk, l) + 1) if l > 0 else 0 for l in left],
                         dtype=np.int32)
        if piece.max() == 0:
            continue
        Tc = int(piece.max())
        chunk = torch.zeros((B, Tc, C), dtype=torch.float32, device="cuda")
        for b in range(B):
            if piece[b]:
                chunk[b, :piece[b]] = enc[b, pos[b]:pos[b] + piece[b]]
        state.chunk(chunk, piece, trace=trace)
        pos += piece
        calls += 1
        if finish_midway and calls == 2:
            state.finish()  # an intermediate result; decoding continues afterwards
    out = state.finish(want_arcs=True)
    torch.cuda.synchronize()
    return out, trace, calls


def _compare(a, b_out, b_trace, lengths, T):
    assert np.array_equal(a.num_tokens.cpu().numpy(), b_out.num_tokens.cpu().numpy())
    assert np.array_equal(a.tokens.cpu().numpy(), b_out.tokens.cpu().numpy()[:, :T])
    assert np.array_equal(a.scores.cpu().numpy(), b_out.scores.cpu().numpy())
    assert np.array_equal(a.status.cpu().numpy(), b_out.status.cpu().numpy())
    assert np.array_equal(a.arcs.cpu().numpy(), b_out.arcs.cpu().numpy()[:, :T])
    # the chunked trace has frame 0 of a stream only once a chunk of it ran, so a
    # stream with no frames keeps its -1 fill there
    want = a.trace.cpu().numpy().copy()
    want[0, lengths == 0] = -1
    assert np.array_equal(want, b_trace.cpu().numpy()[:T + 1])


def _case(name):
    rng = np.random.default_rng(7)
    if name == "standard":
        w, inputs, model, graph = synth.make_workload("standard")
        return inputs, model, graph, math.inf, 4, 4, "fp32"
    if name == "standard-ns8":
        w, inputs, model, graph = synth.make_workload("standard", B=24)
        return inputs, model, graph, 5.0, 8, 6, "fp32"
    if name == "graph":
        w, inputs, model, graph = synth.make_workload("graph", B=16)
        return inputs, model, graph, 4.0, 32, 8, "fp32"
    if name == "tiny-bf16":
        w, inputs, model, graph = synth.make_workload("tiny")
        return inputs, model, graph, math.inf, 4, 4, "bf16"
    if name == "small-graph-final":
        model = synth.make_model(rng, 12, 48, 0.3)
        graph = synth.random_small_graph(rng, 6, 12, max_degree=4, with_final=True)
        inputs = synth.make_inputs(rng, 9, 17, 48, length_range=(0, 17))
        return inputs, model, graph, 6.0, 8, 5, "fp32"
    raise ValueError(name)


CASES = [("standard", "stream"), ("standard", "stream1"), ("standard", "frame"),
         ("standard-ns8", "stream"), ("standard-ns8", "frame"),
         ("graph", "frame"), ("graph", "stream"),
         ("tiny-bf16", "stream"), ("tiny-bf16", "frame"),
         ("small-graph-final", "frame"), ("small-graph-final", "stream")]


@pytest.mark.parametrize("name,schedule", CASES)
def test_chunked_equals_one_shot(name, schedule):
    from paper_2211_00484_amd import tbs
    inputs, model_np, graph_np, beam, Ns, Nc, dtype = _case(name)
    say(f"streaming {name} {schedule} B={inputs.B} T={inputs.T}")
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    model.set_schedule(schedule)
    graph = tbs.Graph.from_synth(graph_np)
    try:
        ref = _one_shot(model, graph, inputs, beam, Ns, Nc)
    except tbs.TbsError as e:
        if e.status == -5:
            pytest.skip(f"shape not supported by the {schedule} schedule")
        raise
    rng = np.random.default_rng(11)
    for max_chunk, midway in ((5, False), (64, True)):
        out, trace, calls = _chunked(model, graph, inputs, beam, Ns, Nc, rng, max_chunk, midway)
        say(f"  {calls} chunks of at most {max_chunk} frames")
        _compare(ref, out, trace, inputs.lengths, inputs.T)


def test_chunk_capacity_and_arguments():
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("tiny")
    model = tbs.Model.from_synth(model_np)
    graph = tbs.Graph.from_synth(graph_np)
    state = tbs.DecodeState(model, graph, 2, 10)
    enc = torch.zeros((2, 8, model_np.dim), device="cuda")
    state.chunk(enc, [8, 3])
    with pytest.raises(tbs.TbsError) as e:
        state.chunk(enc, [3, 0])  # stream 0 would reach 11 > 10 frames
    assert e.value.status == -4
    with pytest.raises(tbs.TbsError) as e:
        state.chunk(enc, [9, 0])  # longer than the chunk
    assert e.value.status == -1
    state.chunk(enc, [2, 7])      # still usable after the refusals
    out = state.finish()
    torch.cuda.synchronize()
    n = out.num_tokens.cpu().numpy()
    assert (n >= 0).all() and n[0] <= 10 and n[1] <= 10
    with pytest.raises(tbs.TbsError) as e:
        tbs.DecodeState(model, graph, 0, 10)
    assert e.value.status == -1
