"""tbs_decode_noalloc (the decode whose workspace lives in the library's fixed device
array) against tbs_decode on the same inputs: identical outputs, on two calls in a
row with the second smaller than the first (the array keeps the first call's contents),
for the grouped per-stream kernel (Standard, trivial graph) and the frame kernels
(Graph, a 5,000-state graph); and a workspace larger than the array is refused."""
import ctypes
import math

import numpy as np
import pytest

from gpu_util import say
from paper_2211_00484_amd import synth

pytestmark = pytest.mark.gpu


def _both(model, graph, enc_np, lengths, beam, Ns, Nc):
    import torch
    from paper_2211_00484_amd import tbs
    enc = torch.from_numpy(np.ascontiguousarray(enc_np)).cuda()
    B, T = enc.shape[0], enc.shape[1]
    ref = tbs.allocate_outputs(B, T, Ns, status=True, arcs=True, trace=True)
    got = tbs.allocate_outputs(B, T, Ns, status=True, arcs=True, trace=True)
    for o in (got.tokens, got.num_tokens, got.status, got.arcs, got.trace):
        o.fill_(12345)
    got.scores.fill_(-7.0)
    tbs.decode_into(model, graph, enc, lengths, beam, Ns, Nc, ref)
    lens_dev = torch.from_numpy(np.ascontiguousarray(lengths, dtype=np.int32)).cuda()
    tbs.decode_noalloc_into(model, graph, enc, lens_dev, beam, Ns, Nc, got)
    torch.cuda.synchronize()
    for name in ("tokens", "num_tokens", "status", "arcs", "trace", "scores"):
        a, b = getattr(ref, name).cpu().numpy(), getattr(got, name).cpu().numpy()
        assert np.array_equal(a, b), f"{name} differs (B={B}, T={T})"
    say(f"  B={B} T={T}: identical to tbs_decode")


@pytest.mark.parametrize("workload,beam,Ns,Nc,small", [
    ("standard", math.inf, 4, 4, (9, 100)),
    ("graph", 4.0, 32, 8, (7, 80)),
])
def test_noalloc_matches_decode_twice(workload, beam, Ns, Nc, small):
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload(workload, seed=0)
    model = tbs.Model.from_synth(model_np)
    graph = tbs.Graph.from_synth(graph_np)
    say(f"no-alloc decode, {workload}: full batch, then {small}")
    _both(model, graph, inputs.encoder_out, inputs.lengths, beam, Ns, Nc)
    B2, T2 = small
    lens2 = np.minimum(inputs.lengths[:B2], T2).astype(np.int32)
    enc2 = inputs.encoder_out[:B2, :T2].copy()
    for b in range(B2):
        enc2[b, lens2[b]:] = 0.0
    _both(model, graph, enc2, lens2, beam, Ns, Nc)


def test_noalloc_refuses_a_workspace_beyond_the_array():
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("standard", seed=0)
    model = tbs.Model.from_synth(model_np)
    graph = tbs.Graph.from_synth(graph_np)
    B, T = 32, 100_000   # the history alone needs 32 x 4 x 100,000 x 8 bytes
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    p = ctypes.c_void_p(dummy.data_ptr())
    params = tbs.BeamParams(math.inf, 4, 4)
    st = tbs.lib().tbs_decode_noalloc(model._h, graph._h, ctypes.byref(params), p, p, B, T,
                                      p, p, p, None, None, None, None)
    assert st == -4, tbs.lib().tbs_last_error()
    assert b"scratch array" in tbs.lib().tbs_last_error()
