"""Element-by-element comparison of the HIP decode against the CPU oracle.

Rule (spec tolerance): where every decision margin of a stream exceeds
``margin`` (1e-3 by default), the HIP path must reproduce the oracle's survivor
trace (context, state, parent, label) bit for bit, the same tokens and arcs, and
the score within ``score_tol``.  Where a frame has a closer decision, the traces
must agree up to and including that frame (later survivors may legitimately
differ), and the returned path must be valid: the oracle rescoring of the HIP
alignment reproduces the HIP score within ``score_tol``, it has at most one
symbol per frame, and the trace keeps the search invariants.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

import oracle


@dataclass
class ParityReport:
    streams: int = 0
    clean: int = 0
    max_score_err_clean: float = 0.0
    max_rescore_err: float = 0.0
    notes: list = field(default_factory=list)

    def __str__(self):
        return (f"streams={self.streams} clean={self.clean} "
                f"max|dscore|(clean)={self.max_score_err_clean:.3g} "
                f"max|rescore-gpu|={self.max_rescore_err:.3g}")


def compare(gpu, orc, model, graph, enc, lengths, streams, *, margin=1e-3, score_tol=1e-4,
            bf16=False, check_rescore=True) -> ParityReport:
    """gpu: dict of numpy arrays (tokens, ntok, scores, status, arcs, trace) for the full
    batch; orc: oracle result for ``streams`` (same order)."""
    rep = ParityReport()
    T = enc.shape[1]
    for k, b in enumerate(streams):
        L = int(lengths[b])
        rep.streams += 1
        fm = orc.frame_margins[k]
        bad = [t for t in range(L) if fm[t] <= margin]
        t_star = bad[0] if bad else L
        # survivor trace up to the first contested frame (inclusive)
        if gpu.get("trace") is not None:
            g_tr = gpu["trace"][: t_star + 1, b]
            o_tr = orc.trace[: t_star + 1, k]
            if not np.array_equal(g_tr, o_tr):
                f = int(np.argmax([not np.array_equal(g_tr[i], o_tr[i]) for i in range(len(g_tr))]))
                raise AssertionError(f"stream {b}: trace differs at frame {f} (first contested "
                                     f"frame {t_star}):\n gpu {g_tr[f].tolist()}\n orc {o_tr[f].tolist()}")
            assert (gpu["trace"][L + 1:, b] == -1).all(), f"stream {b}: trace not padded"
        n = int(gpu["ntok"][b])
        assert 0 <= n <= L, f"stream {b}: {n} tokens for {L} frames"
        assert (gpu["tokens"][b, n:] == -1).all(), f"stream {b}: tokens not -1 padded"
        assert (gpu["tokens"][b, :n] > 0).all(), f"stream {b}: blank or negative token"
        if gpu.get("arcs") is not None:
            assert (gpu["arcs"][b, L:] == -2).all(), f"stream {b}: arcs not -2 padded"
        clean = not bad and fm[T] > margin
        if clean:
            rep.clean += 1
            assert gpu["tokens"][b, :n].tolist() == orc.tokens[k, : orc.ntok[k]].tolist(), \
                f"stream {b}: tokens differ on a clean stream"
            assert int(gpu["status"][b]) == int(orc.status[k])
            if gpu.get("arcs") is not None:
                assert np.array_equal(gpu["arcs"][b, :L], orc.arcs[k, :L]), f"stream {b}: arcs differ"
            err = abs(float(gpu["scores"][b]) - float(orc.scores[k]))
            rep.max_score_err_clean = max(rep.max_score_err_clean, err)
            assert err <= score_tol, f"stream {b}: |score diff| {err} > {score_tol}"
        if check_rescore and gpu.get("arcs") is not None:
            arcs = gpu["arcs"][b, :L]
            lab = np.where(arcs >= 0, graph.label[np.maximum(arcs, 0)], 0)
            assert lab[lab > 0].tolist() == gpu["tokens"][b, :n].tolist(), \
                f"stream {b}: tokens are not the labels of the returned arcs"
            code, s = oracle.rescore(model, graph, enc[b, :L], arcs, bf16=bf16)
            assert code >= 0, f"stream {b}: returned alignment is not a graph path"
            assert code == int(gpu["status"][b])
            err = abs(s - float(gpu["scores"][b]))
            rep.max_rescore_err = max(rep.max_rescore_err, err)
            assert err <= score_tol, f"stream {b}: rescoring differs by {err}"
    return rep


def check_trace_invariants(trace, lengths, graph, V, Ns, Nc, streams):
    """Search invariants on the HIP trace (independent of the oracle)."""
    rp, dest, lab = graph.row_ptr, graph.dest, graph.label
    for b in streams:
        L = int(lengths[b])
        for f in range(1, L + 1):
            cur, prev = trace[f, b], trace[f - 1, b]
            n = int((cur[:, 0] >= 0).sum())
            assert 1 <= n <= Ns
            keys = [(int(x[0]), int(x[1])) for x in cur[:n]]
            assert keys == sorted(keys) and len(set(keys)) == n
            assert len({k[0] for k in keys}) <= Nc
            for ctx, s, par, c in cur[:n]:
                pctx, ps = int(prev[par, 0]), int(prev[par, 1])
                if c == 0:
                    assert (ctx, s) == (pctx, ps)
                else:
                    assert ctx == (pctx % V) * V + c
                    assert any(lab[j] == c and dest[j] == s for j in range(rp[ps], rp[ps + 1]))
