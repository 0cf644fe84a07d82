"""Element-by-element comparison of the HIP decode against the CPU oracle.

Rule (spec tolerance): where every decision margin of a stream exceeds
``margin`` (1e-3 by default), the HIP path must reproduce the oracle's survivor
trace (context, state, parent, label) bit for bit, the same tokens and arcs, and
the score within ``score_tol``.  Where a frame has a closer decision, the traces
must agree up to and including that frame (later survivors may legitimately
differ), and the returned path must be valid: the oracle rescoring of the HIP
alignment reproduces the HIP score within ``score_tol``, it has at most one
symbol per frame, and the trace keeps the search invariants.

``replay_check`` then checks every frame of every stream, not only those before the
first contested one: the oracle decides each frame again from the HIP path's own
survivors of the previous frame (scored in fp64 along their (state, context)).  Where
that frame's decision margin exceeds ``margin`` the HIP survivors must equal the
oracle's bit for bit; where it does not, they must be a valid selection: real
candidates, merged parents within ``tol`` of the best, inside the beam, and every
tuple the two sides keep differently explained by a score within ``tol`` of a pruning
boundary of that frame.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

import oracle


@dataclass
class ParityReport:
    streams: int = 0
    clean: int = 0
    frames: int = 0          # frames of the checked streams
    frames_prefix: int = 0   # frames before each stream's first contested frame
    max_score_err_clean: float = 0.0
    max_rescore_err: float = 0.0
    notes: list = field(default_factory=list)

    def __str__(self):
        return (f"streams={self.streams} clean={self.clean} "
                f"prefix frames={self.frames_prefix}/{self.frames} "
                f"max|dscore|(clean)={self.max_score_err_clean:.3g} "
                f"max|rescore-gpu|={self.max_rescore_err:.3g}")


@dataclass
class ReplayReport:
    streams: int = 0
    frames: int = 0      # frames replayed
    exact: int = 0       # frames whose margin exceeds the threshold: compared bit for bit
    contested: int = 0   # frames checked for validity only
    max_final_err: float = 0.0  # |HIP score - best fp64 final value of its survivors|

    def __str__(self):
        return (f"replay: streams={self.streams} frames={self.frames} exact={self.exact} "
                f"contested={self.contested} max|final-gpu|={self.max_final_err:.3g}")


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
        rep.frames += L
        rep.frames_prefix += t_star
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


def _explained(diff, seeds, tol):
    """Whether every (score, context score) pair in ``diff`` is linked to a pruning
    boundary in ``seeds`` by a chain of values within ``tol`` of each other."""
    zs = [z for z in seeds if np.isfinite(z)]
    todo = list(diff)
    grew = True
    while todo and grew:
        grew = False
        rest = []
        for sc, cs in todo:
            if any(abs(sc - z) <= tol or abs(cs - z) <= tol for z in zs):
                zs += [sc, cs]
                grew = True
            else:
                rest.append((sc, cs))
        todo = rest
    return not todo


def replay_check(gpu, model, graph, enc, lengths, streams, beam, Ns, Nc, *, margin, tol,
                 bf16=False, nthreads=0) -> ReplayReport:
    """Every frame of the listed streams, decided again by the oracle from the HIP
    path's survivors of the previous frame (see the module docstring)."""
    tr = gpu["trace"]
    streams = list(streams)
    R = oracle.replay(model, graph, enc, lengths, tr, beam, Ns, Nc, bf16=bf16,
                      nthreads=nthreads, streams=streams)
    rep = ReplayReport()
    fin = graph.final
    for k, b in enumerate(streams):
        L = int(lengths[b])
        rep.streams += 1
        g = tr[:, b]
        assert g[0, 0].tolist() == [0, graph.start, -1, -1] and (g[0, 1:] == -1).all(), \
            f"stream {b}: frame 0 is not the initial tuple"
        for t in range(L):
            rep.frames += 1
            nxt = g[t + 1]
            n = int((nxt[:, 0] >= 0).sum())
            ks, cs = R.key_score[t + 1, k, :n], R.cand_score[t + 1, k, :n]
            where = f"stream {b} frame {t}"
            assert n >= 1 and (nxt[:n, 0] >= 0).all() and (nxt[n:] == -1).all(), \
                f"{where}: survivors not packed"
            assert np.isfinite(ks).all(), f"{where}: a survivor is not a candidate"
            m = R.margins[k, t]
            if m > margin:
                rep.exact += 1
                if not np.array_equal(nxt, R.ref[t + 1, k]):
                    raise AssertionError(
                        f"{where}: survivors differ (margin {m:.3g}):\n gpu {nxt[:n].tolist()}"
                        f"\n orc {R.ref[t + 1, k][R.ref[t + 1, k][:, 0] >= 0].tolist()}")
                continue
            rep.contested += 1
            assert np.isfinite(cs).all() and (cs >= ks - tol).all(), \
                f"{where}: a survivor's parent/label is not its best candidate"
            thr, s_in, s_out, c_in, c_out = R.bounds[k, t]
            assert (ks >= thr - tol).all(), f"{where}: a survivor is outside the beam"
            gk = {(int(x[0]), int(x[1])): float(v) for x, v in zip(nxt[:n], ks)}
            gctx = {}
            for (c, _), v in gk.items():
                gctx[c] = max(gctx.get(c, -np.inf), v)
            ref = R.ref[t + 1, k]
            no = int((ref[:, 0] >= 0).sum())
            ok = {(int(x[0]), int(x[1])): (float(R.ref_score[t + 1, k, i]),
                                           float(R.ref_cscore[t + 1, k, i]))
                  for i, x in enumerate(ref[:no])}
            diff = [(v, gctx[key[0]]) for key, v in gk.items() if key not in ok]
            diff += [v for key, v in ok.items() if key not in gk]
            assert _explained(diff, [thr, s_in, s_out, c_in, c_out], tol), \
                f"{where}: kept sets differ beyond the contested boundaries"
        # the final pick: the best fp64 value (score + final weight) of the last survivors
        last = g[L]
        n = int((last[:, 0] >= 0).sum())
        ks = R.key_score[L, k, :n]
        if fin is not None:
            fw = fin[last[:n, 1]].astype(np.float64)
            vals = np.where(np.isfinite(fw), ks + fw, -np.inf)
            if not np.isfinite(vals).any():
                vals = ks
        else:
            vals = ks
        err = abs(float(gpu["scores"][b]) - float(vals.max())) if L > 0 else \
            abs(float(gpu["scores"][b]))
        rep.max_final_err = max(rep.max_final_err, err)
        assert err <= tol, f"stream {b}: score {gpu['scores'][b]} is not the best final " \
                           f"value {vals.max()} of its survivors"
    return rep
