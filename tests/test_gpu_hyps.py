"""HIP full-sequence beam search (tbs_hyp_search, Table 5's comparison search) against
the CPU oracle.

Parity rule: the kept hypotheses' back-pointers (parent rank, label) are identical up to
the first frame with an oracle decision margin (a gap between neighbouring ranks up to the
N-best cut, or between the two best members of a merged sequence) of at most MARGIN; on streams with no such frame and a clear final
pick the tokens are identical and the scores agree within TOL.  fp32 joiner: MARGIN 1e-4,
TOL 1e-4; bf16 against the bf16-operand oracle: 2e-3 and 2e-2.
"""
import math

import numpy as np
import pytest

import oracle
from gpu_util import say
from paper_2211_00484_amd import synth

pytestmark = pytest.mark.gpu

TOL = {"fp32": (1e-4, 1e-4), "bf16": (2e-3, 2e-2)}


def _run(inputs, model_np, N, merge, dtype="fp32", streams=None):
    import torch
    from paper_2211_00484_amd import tbs
    say(f"hyps B={inputs.B} T={inputs.T} V={model_np.vocab_size} N={N} {merge} {dtype}")
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    out = tbs.hyp_search(model, enc, inputs.lengths, beam_size=N, merge=merge, want_trace=True)
    torch.cuda.synchronize()
    tok, nt, sc = out.tokens.cpu().numpy(), out.num_tokens.cpu().numpy(), out.scores.cpu().numpy()
    tr = out.trace.cpu().numpy()
    streams = list(range(inputs.B)) if streams is None else list(streams)
    o = oracle.hyp_search(model_np, inputs.encoder_out, inputs.lengths, N, merge == "logadd",
                          bf16=(dtype == "bf16"), streams=streams)
    margin, tol = TOL[dtype]
    T = inputs.T
    clean = 0
    for k, b in enumerate(streams):
        L = int(inputs.lengths[b])
        fm = o.frame_margins[k]
        bad = [t for t in range(L) if fm[t] <= margin]
        t_star = bad[0] if bad else L
        # frame f of the trace holds the decisions of frame f - 1
        assert np.array_equal(tr[1:t_star + 1, b], o.trace[1:t_star + 1, k]), \
            f"stream {b}: back-pointers differ before frame {t_star}"
        assert (tr[L + 1:, b] == -1).all()
        n = int(nt[b])
        assert 0 <= n <= L and (tok[b, n:] == -1).all() and (tok[b, :n] > 0).all()
        if not bad and fm[T] > margin:
            clean += 1
            assert tok[b, :n].tolist() == o.tokens[k, :o.ntok[k]].tolist(), f"stream {b}"
            assert sc[b] == pytest.approx(o.scores[k], abs=tol), f"stream {b}"
    say(f"  {clean} of {len(streams)} streams clean")
    return clean


@pytest.mark.parametrize("merge", ["max", "logadd"])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_tiny(dtype, merge):
    w, inputs, model, graph = synth.make_workload("tiny")
    _run(inputs, model, 4, merge, dtype)


@pytest.mark.parametrize("N", [1, 2, 3, 8, 16])
@pytest.mark.parametrize("merge", ["max", "logadd"])
def test_beam_sizes(N, merge):
    rng = np.random.default_rng(50 + N)
    model = synth.make_model(rng, 11, 24, 0.6)
    inputs = synth.make_inputs(rng, 6, 30, 24, length_range=(0, 30))
    assert _run(inputs, model, N, merge) >= 1


def test_ragged_and_empty_streams():
    rng = np.random.default_rng(9)
    model = synth.make_model(rng, 16, 32, 0.3)
    inputs = synth.make_inputs(rng, 5, 25, 32)
    inputs.lengths[:] = [0, 25, 1, 13, 0]
    for b in range(inputs.B):
        inputs.encoder_out[b, inputs.lengths[b]:] = 0.0
    _run(inputs, model, 4, "logadd")


@pytest.mark.parametrize("merge", ["max", "logadd"])
def test_standard_workload(merge):
    """Standard shapes: B = 32, T up to 250, V = 500, beam 4."""
    w, inputs, model, graph = synth.make_workload("standard")
    assert _run(inputs, model, 4, merge) >= 1


def test_arguments():
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("tiny")
    model = tbs.Model.from_synth(model_np)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    for N, st in ((0, -1), (17, -4)):
        with pytest.raises(tbs.TbsError) as e:
            tbs.hyp_search(model, enc, inputs.lengths, beam_size=N)
        assert e.value.status == st
    out = tbs.hyp_search(model, enc, inputs.lengths, beam_size=2, merge="max")
    torch.cuda.synchronize()
    assert out.num_tokens.shape == (2,)
