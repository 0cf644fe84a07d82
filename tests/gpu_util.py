"""Helpers shared by the GPU tests: run the HIP decode and fetch results as numpy."""
from __future__ import annotations

import math
import sys

import numpy as np


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_decode(model_np, graph_np, inputs, beam, Ns, Nc, dtype="fp32", trace=True, arcs=True,
               model=None, graph=None, repeat=1, schedule="auto"):
    """Decode on the GPU with the given frame-loop schedule ("auto", "frame", "stream")."""
    import torch
    from paper_2211_00484_amd import tbs
    if model is None:
        model = tbs.Model.from_synth(model_np, dtype=dtype)
    model.set_schedule(schedule)
    if graph is None:
        graph = tbs.Graph.from_synth(graph_np)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    out = None
    for _ in range(repeat):
        out = tbs.decode(model, graph, enc, inputs.lengths, beam=beam, max_states=Ns,
                         max_contexts=Nc, want_arcs=arcs, want_trace=trace)
    torch.cuda.synchronize()
    res = {"tokens": out.tokens.cpu().numpy(), "ntok": out.num_tokens.cpu().numpy(),
           "scores": out.scores.cpu().numpy(), "status": out.status.cpu().numpy(),
           "arcs": out.arcs.cpu().numpy() if arcs else None,
           "trace": out.trace.cpu().numpy() if trace else None}
    return res


def inf_or(x):
    return math.inf if x is None else x
