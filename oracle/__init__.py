"""TEST INFRASTRUCTURE ONLY: the fp64 CPU oracle for FSA-based one-symbol-per-frame
transducer beam search (Sec. 2.2-2.5, Algorithm 1 of Kang et al., arXiv 2211.00484).

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may
import this package.  It wraps ``tbs_oracle.cpp`` (plain C++17, double precision, built
with g++ by :func:`build`) through ctypes and shares no code with the HIP library.

Parity status: the decoder/joiner/log-softmax is pinned against library layers; the
unpruned search against exhaustive enumeration and a Viterbi recursion; Ns = Nc = 1 on the
trivial graph against per-frame argmax greedy search.  The exact tie-breaking of the
finite beam / max-states / max-contexts selection is this implementation's reading of
Sec. 2.5 and is pinned only by invariants ("parity unpinned" for those tie rules).

Lattice and label-sequence search (Sec. 2.5, the "LogAdd" rows of Tables 3 and 6): the
unpruned lattice's total probability, the total probability of a label sequence and the
best label sequence are pinned against exhaustive enumeration of alignments; path
sampling against the exact path posteriors of small lattices.  Which expansions a pruned
lattice keeps (every arc into a surviving tuple) is this implementation's reading and is
pinned by invariants only.

Transducer forward recursions (Sec. 3, eq. 1-3): pinned against exhaustive enumeration
of the alignments of small grids and against path-count closed forms.

Full-sequence beam search (Table 5's comparison search): with a beam wide enough to keep
every sequence it is pinned against exhaustive enumeration (max merge: the best path;
log-add merge: the sequence with the highest total probability); with one hypothesis
against per-frame argmax greedy search; pruned, against an independent Python
implementation over tuples.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tbs_oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_I = ctypes.c_int
_D = ctypes.c_double
_P = ctypes.c_void_p


def build(force: bool = True) -> str:
    """Compiles the oracle with g++ (no GPU code involved)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-pthread",
               "-ffp-contract=off", "-fno-fast-math", _SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_logp.argtypes = [_I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _I, _P]
        lib.oracle_logp.restype = _I
        lib.oracle_decode.argtypes = ([_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I,
                                       _I, _I, _P, _P, _P, _P, _P, _D, _I, _I, _I] + [_P] * 8)
        lib.oracle_decode.restype = _I
        lib.oracle_replay.argtypes = ([_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I,
                                       _I, _I, _P, _P, _P, _P, _P, _D, _I, _I, _I] + [_P] * 8)
        lib.oracle_replay.restype = _I
        lib.oracle_rescore.argtypes = [_I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _I, _I,
                                       _P, _P, _P, _P, _P, _P]
        lib.oracle_rescore.restype = _I
        lib.oracle_transducer_forward.argtypes = [_I, _I, _I, _I, _P, _P, _P, _P, _P, _P]
        lib.oracle_transducer_forward.restype = _I
        lib.oracle_hyps.argtypes = ([_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I]
                                    + [_P] * 5)
        lib.oracle_hyps.restype = _I
        lib.oracle_lattice.argtypes = ([_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I,
                                        _I, _I, _P, _P, _P, _P, _P, _D, _I, _I, _I, _P])
        lib.oracle_lattice.restype = _P
        lib.oracle_lattice_free.argtypes = [_P]
        lib.oracle_lattice_free.restype = None
        lib.oracle_lattice_sizes.argtypes = [_P, _I, _P, _P, _P]
        lib.oracle_lattice_sizes.restype = _I
        lib.oracle_lattice_get.argtypes = [_P, _I, _P, _P, _P, _P, _P, _P, _P]
        lib.oracle_lattice_get.restype = _I
        lib.oracle_lattice_nbest.argtypes = [_P, _I, _I, _P, _P, _P, _P, _P, _P]
        lib.oracle_lattice_nbest.restype = _I
        lib.oracle_lattice_seqscore.argtypes = [_P, _I, _P, _I]
        lib.oracle_lattice_seqscore.restype = _D
        _lib = lib
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def logp(model, enc_rows: np.ndarray, ctx_a: np.ndarray, ctx_b: np.ndarray,
         bf16: bool = False) -> np.ndarray:
    """Joiner log-probabilities [R, V] (fp64) for R (encoder row, (a, b) context) pairs."""
    lib = _load()
    enc_rows = _f32(enc_rows)
    R = int(enc_rows.shape[0])
    a, b = _i32(ctx_a), _i32(ctx_b)
    E, conv, W = _f32(model.embed), _f32(model.conv), _f32(model.w_out)
    bias = None if model.b_out is None else _f32(model.b_out)
    out = np.empty((R, model.vocab_size), dtype=np.float64)
    lib.oracle_logp(model.dim, model.vocab_size, R, _ptr(enc_rows), _ptr(a), _ptr(b),
                    _ptr(E), _ptr(conv), _ptr(W), _ptr(bias), int(bf16), _ptr(out))
    return out


class OracleResult:
    def __init__(self, tokens, ntok, scores, status, arcs, trace, margins, frame_margins):
        self.tokens, self.ntok, self.scores, self.status = tokens, ntok, scores, status
        self.arcs, self.trace, self.margins = arcs, trace, margins
        self.frame_margins = frame_margins

    def token_lists(self):
        return [list(self.tokens[b, : self.ntok[b]]) for b in range(self.tokens.shape[0])]


def decode(model, graph, encoder_out: np.ndarray, lengths: np.ndarray, beam: float,
           max_states: int, max_contexts: int, bf16: bool = False, nthreads: int = 0,
           want_trace: bool = True, want_arcs: bool = True, streams=None) -> OracleResult:
    """Decodes every stream (or the listed ``streams``) of a batch; see tbs_oracle.cpp."""
    lib = _load()
    enc = _f32(encoder_out)
    lens = _i32(lengths)
    if streams is not None:
        idx = np.asarray(streams, dtype=np.int64)
        enc = np.ascontiguousarray(enc[idx])
        lens = np.ascontiguousarray(lens[idx])
    B, T, C = enc.shape
    V = model.vocab_size
    if max_states < 1 or max_contexts < 1:
        raise ValueError("max_states and max_contexts must be >= 1")
    E, conv, W = _f32(model.embed), _f32(model.conv), _f32(model.w_out)
    bias = None if model.b_out is None else _f32(model.b_out)
    rp, dest, lab, q = _i32(graph.row_ptr), _i32(graph.dest), _i32(graph.label), _f32(graph.score)
    fin = None if graph.final is None else _f32(graph.final)
    tokens = np.empty((B, T), dtype=np.int32)
    ntok = np.empty(B, dtype=np.int32)
    scores = np.empty(B, dtype=np.float64)
    status = np.empty(B, dtype=np.int32)
    arcs = np.empty((B, T), dtype=np.int32) if want_arcs else None
    trace = np.empty((T + 1, B, max_states, 4), dtype=np.int32) if want_trace else None
    margins = np.empty(B, dtype=np.float64)
    frame_margins = np.empty((B, T + 1), dtype=np.float64)
    beam_v = float(beam) if beam is not None else math.inf
    lib.oracle_decode(B, T, C, V, _ptr(enc), _ptr(lens), _ptr(E), _ptr(conv), _ptr(W),
                      _ptr(bias), int(bf16), graph.num_states, graph.start, _ptr(rp), _ptr(dest),
                      _ptr(lab), _ptr(q), _ptr(fin), beam_v, int(max_states), int(max_contexts),
                      int(nthreads), _ptr(tokens), _ptr(ntok), _ptr(scores), _ptr(status),
                      _ptr(arcs), _ptr(trace), _ptr(margins), _ptr(frame_margins))
    return OracleResult(tokens, ntok, scores, status, arcs, trace, margins, frame_margins)


class ReplayResult:
    """Frame-by-frame replay of a given survivor trace (see ``replay``)."""

    def __init__(self, ref, ref_score, ref_cscore, key_score, cand_score, margins, bounds):
        self.ref, self.ref_score, self.ref_cscore = ref, ref_score, ref_cscore
        self.key_score, self.cand_score = key_score, cand_score
        self.margins, self.bounds = margins, bounds


def replay(model, graph, encoder_out: np.ndarray, lengths: np.ndarray, given_trace: np.ndarray,
           beam: float, max_states: int, max_contexts: int, bf16: bool = False,
           nthreads: int = 0, streams=None) -> ReplayResult:
    """Decides every frame again from the survivors of the previous frame as given in
    ``given_trace`` ([T+1, B, Ns, 4], the layout of ``decode``'s trace), each scored in
    fp64 along its (state, context); see ``oracle_replay`` in tbs_oracle.cpp.  With
    ``streams``, the given trace and the outputs hold those streams only."""
    lib = _load()
    enc = _f32(encoder_out)
    lens = _i32(lengths)
    given = _i32(given_trace)
    if streams is not None:
        idx = np.asarray(streams, dtype=np.int64)
        enc = np.ascontiguousarray(enc[idx])
        lens = np.ascontiguousarray(lens[idx])
        given = np.ascontiguousarray(given[:, idx])
    B, T, C = enc.shape
    Ns = int(max_states)
    if given.shape != (T + 1, B, Ns, 4):
        raise ValueError(f"given trace has shape {given.shape}, expected {(T + 1, B, Ns, 4)}")
    E, conv, W = _f32(model.embed), _f32(model.conv), _f32(model.w_out)
    bias = None if model.b_out is None else _f32(model.b_out)
    rp, dest, lab, q = _i32(graph.row_ptr), _i32(graph.dest), _i32(graph.label), _f32(graph.score)
    fin = None if graph.final is None else _f32(graph.final)
    ref = np.empty((T + 1, B, Ns, 4), dtype=np.int32)
    ref_score = np.empty((T + 1, B, Ns), dtype=np.float64)
    ref_cscore = np.empty_like(ref_score)
    key_score = np.empty_like(ref_score)
    cand_score = np.empty_like(ref_score)
    margins = np.empty((B, T + 1), dtype=np.float64)
    bounds = np.empty((B, T, 5), dtype=np.float64)
    beam_v = float(beam) if beam is not None else math.inf
    lib.oracle_replay(B, T, C, model.vocab_size, _ptr(enc), _ptr(lens), _ptr(E), _ptr(conv),
                      _ptr(W), _ptr(bias), int(bf16), graph.num_states, graph.start, _ptr(rp),
                      _ptr(dest), _ptr(lab), _ptr(q), _ptr(fin), beam_v, Ns, int(max_contexts),
                      int(nthreads), _ptr(given), _ptr(ref), _ptr(ref_score), _ptr(ref_cscore),
                      _ptr(key_score), _ptr(cand_score), _ptr(margins), _ptr(bounds))
    return ReplayResult(ref, ref_score, ref_cscore, key_score, cand_score, margins, bounds)


def rescore(model, graph, enc_stream: np.ndarray, arcs: np.ndarray, bf16: bool = False):
    """Path score (fp64) of one stream's alignment (arc id per frame, -1 = blank).

    Returns (code, score): code 0 = valid path ending in a final state, 1 = valid path
    ending in a non-final state (score then excludes any final weight), -1 = not a path."""
    lib = _load()
    enc = _f32(enc_stream)
    arcs = _i32(arcs)
    E, conv, W = _f32(model.embed), _f32(model.conv), _f32(model.w_out)
    bias = None if model.b_out is None else _f32(model.b_out)
    rp, dest, lab, q = _i32(graph.row_ptr), _i32(graph.dest), _i32(graph.label), _f32(graph.score)
    fin = None if graph.final is None else _f32(graph.final)
    out = ctypes.c_double(0.0)
    code = lib.oracle_rescore(model.dim, model.vocab_size, int(arcs.shape[0]), _ptr(enc),
                              _ptr(arcs), _ptr(E), _ptr(conv), _ptr(W), _ptr(bias), int(bf16),
                              graph.num_states, graph.start, _ptr(rp), _ptr(dest), _ptr(lab),
                              _ptr(q), _ptr(fin), ctypes.byref(out))
    return int(code), float(out.value)


class StreamLattice:
    """One stream's lattice: nodes[f] [n_f, 4] (ctx, state, parent, label) for f = 0..len;
    arcs[f] [a_f, 4] (src, dst, label, graph arc) with weights w[f] [a_f] (fp64), ordered by
    (dst, src, arc position) with blank first; fw: final weights of the last frame's nodes;
    alpha[f]: forward log scores; total: log of the sum over complete paths; status as in
    decode."""

    def __init__(self, len_, nodes, arcs, w, fw, alpha, total, status):
        self.len, self.nodes, self.arcs, self.w = len_, nodes, arcs, w
        self.fw, self.alpha, self.total, self.status = fw, alpha, total, status


class NBest:
    """Result of the n-best label-sequence search on one stream (see Lattice.nbest)."""

    def __init__(self, paths, margins, first, scores, best, seqs):
        self.paths, self.margins, self.first, self.scores = paths, margins, first, scores
        self.best, self.seqs = best, seqs

    @property
    def tokens(self):
        return self.seqs[self.best]

    @property
    def score(self):
        return float(self.scores[self.best])


class Lattice:
    """Lattices of a batch from the oracle search (Sec. 2.5); see tbs_oracle.cpp."""

    def __init__(self, handle, B, T, frame_margins, streams):
        self._h, self.B, self.T = handle, B, T
        self.frame_margins, self.streams = frame_margins, streams

    def __del__(self):
        if getattr(self, "_h", None) is not None and _lib is not None:
            _lib.oracle_lattice_free(self._h)
            self._h = None

    def stream(self, k: int) -> StreamLattice:
        """Lattice of the k-th decoded stream (index into ``streams``)."""
        lib = _load()
        ln = ctypes.c_int(0)
        lib.oracle_lattice_sizes(self._h, k, ctypes.byref(ln), None, None)
        L = ln.value
        nn = np.empty(L + 1, dtype=np.int32)
        na = np.empty(max(L, 1), dtype=np.int32)
        lib.oracle_lattice_sizes(self._h, k, ctypes.byref(ln), _ptr(nn), _ptr(na))
        na = na[:L]
        nodes = np.empty((int(nn.sum()), 4), dtype=np.int32)
        arcs = np.empty((max(int(na.sum()), 1), 4), dtype=np.int32)
        w = np.empty(max(int(na.sum()), 1), dtype=np.float64)
        fw = np.empty(int(nn[L]), dtype=np.float64)
        alpha = np.empty(int(nn.sum()), dtype=np.float64)
        tot = ctypes.c_double(0.0)
        st = ctypes.c_int(0)
        lib.oracle_lattice_get(self._h, k, _ptr(nodes), _ptr(arcs), _ptr(w), _ptr(fw),
                               _ptr(alpha), ctypes.byref(tot), ctypes.byref(st))
        no = np.concatenate([[0], np.cumsum(nn)])
        ao = np.concatenate([[0], np.cumsum(na)]).astype(np.int64)
        return StreamLattice(L, [nodes[no[f]:no[f + 1]] for f in range(L + 1)],
                             [arcs[ao[f]:ao[f + 1]] for f in range(L)],
                             [w[ao[f]:ao[f + 1]] for f in range(L)], fw,
                             [alpha[no[f]:no[f + 1]] for f in range(L + 1)], tot.value, st.value)

    def nbest(self, k: int, uniforms: np.ndarray) -> NBest:
        """n-best label-sequence search on the k-th stream; uniforms [n, len+1] in [0, 1)."""
        lib = _load()
        ln = ctypes.c_int(0)
        lib.oracle_lattice_sizes(self._h, k, ctypes.byref(ln), None, None)
        L = ln.value
        u = np.ascontiguousarray(uniforms, dtype=np.float64)
        n = int(u.shape[0])
        if n < 1 or u.shape != (n, L + 1):
            raise ValueError(f"uniforms must be [n >= 1, {L + 1}]")
        paths = np.empty((n, L + 1), dtype=np.int32)
        margins = np.empty((n, L + 1), dtype=np.float64)
        first = np.empty(n, dtype=np.int32)
        scores = np.empty(n, dtype=np.float64)
        best = ctypes.c_int(0)
        nu = lib.oracle_lattice_nbest(self._h, k, n, _ptr(u), _ptr(paths), _ptr(margins),
                                      _ptr(first), _ptr(scores), ctypes.byref(best))
        lat = self.stream(k)
        seqs = []
        for p in first[:nu]:
            seqs.append([int(lat.arcs[f][paths[p, f], 2]) for f in range(L)
                         if lat.arcs[f][paths[p, f], 2] > 0])
        return NBest(paths, margins, first[:nu], scores[:nu], best.value, seqs)

    def sequence_score(self, k: int, y) -> float:
        """Total probability (log) of label sequence y in the k-th stream's lattice."""
        y = _i32(np.asarray(list(y), dtype=np.int64))
        return float(_load().oracle_lattice_seqscore(self._h, k, _ptr(y), int(y.shape[0])))


def lattice(model, graph, encoder_out: np.ndarray, lengths: np.ndarray, beam: float,
            max_states: int, max_contexts: int, bf16: bool = False, nthreads: int = 0,
            streams=None) -> Lattice:
    """Runs the search and keeps every stream's lattice (Sec. 2.5)."""
    lib = _load()
    enc = _f32(encoder_out)
    lens = _i32(lengths)
    if streams is not None:
        idx = np.asarray(streams, dtype=np.int64)
        enc = np.ascontiguousarray(enc[idx])
        lens = np.ascontiguousarray(lens[idx])
    B, T, C = enc.shape
    if max_states < 1 or max_contexts < 1:
        raise ValueError("max_states and max_contexts must be >= 1")
    E, conv, W = _f32(model.embed), _f32(model.conv), _f32(model.w_out)
    bias = None if model.b_out is None else _f32(model.b_out)
    rp, dest, lab, q = _i32(graph.row_ptr), _i32(graph.dest), _i32(graph.label), _f32(graph.score)
    fin = None if graph.final is None else _f32(graph.final)
    fm = np.empty((B, T + 1), dtype=np.float64)
    beam_v = float(beam) if beam is not None else math.inf
    h = lib.oracle_lattice(B, T, C, model.vocab_size, _ptr(enc), _ptr(lens), _ptr(E), _ptr(conv),
                           _ptr(W), _ptr(bias), int(bf16), graph.num_states, graph.start,
                           _ptr(rp), _ptr(dest), _ptr(lab), _ptr(q), _ptr(fin), beam_v,
                           int(max_states), int(max_contexts), int(nthreads), _ptr(fm))
    return Lattice(h, B, T, fm, list(range(B)) if streams is None else list(streams))


def hyp_search(model, encoder_out: np.ndarray, lengths: np.ndarray, beam_size: int,
               logadd: bool, bf16: bool = False, nthreads: int = 0, streams=None):
    """Full-sequence beam search (Table 5's comparison search); see tbs_oracle.cpp.
    Returns an OracleResult with trace [T+1, B, N, 2] (parent rank, label)."""
    lib = _load()
    enc = _f32(encoder_out)
    lens = _i32(lengths)
    if streams is not None:
        idx = np.asarray(streams, dtype=np.int64)
        enc = np.ascontiguousarray(enc[idx])
        lens = np.ascontiguousarray(lens[idx])
    B, T, C = enc.shape
    N = int(beam_size)
    if N < 1:
        raise ValueError("beam_size must be >= 1")
    E, conv, W = _f32(model.embed), _f32(model.conv), _f32(model.w_out)
    bias = None if model.b_out is None else _f32(model.b_out)
    tokens = np.empty((B, T), dtype=np.int32)
    ntok = np.empty(B, dtype=np.int32)
    scores = np.empty(B, dtype=np.float64)
    trace = np.empty((T + 1, B, N, 2), dtype=np.int32)
    fm = np.empty((B, T + 1), dtype=np.float64)
    lib.oracle_hyps(B, T, C, model.vocab_size, _ptr(enc), _ptr(lens), _ptr(E), _ptr(conv),
                    _ptr(W), _ptr(bias), int(bf16), N, int(bool(logadd)), int(nthreads),
                    _ptr(tokens), _ptr(ntok), _ptr(scores), _ptr(trace), _ptr(fm))
    return OracleResult(tokens, ntok, scores, np.zeros(B, dtype=np.int32), None, trace,
                        fm.min(axis=1), fm)


TRANSDUCER_KINDS = {"standard": 0, "modified": 1, "constrained": 2}


def transducer_forward(kind: str, blank: np.ndarray, label: np.ndarray, frames, labels):
    """Forward recursion of the standard (eq. 1), modified (eq. 2) or constrained (eq. 3)
    transducer on log-probabilities blank [B, T, U+1] and label [B, T, U].
    Returns (total [B], alpha [B, T+1, U+1]), fp64."""
    lib = _load()
    blank, label = _f32(blank), _f32(label)
    B, T, U1 = blank.shape
    U = U1 - 1
    if label.shape != (B, T, U):
        raise ValueError("label must be [B, T, U]")
    fr, lb = _i32(frames), _i32(labels)
    if (fr < 1).any() or (fr > T).any() or (lb < 0).any() or (lb > U).any():
        raise ValueError("frames must be in [1, T] and labels in [0, U]")
    alpha = np.empty((B, T + 1, U + 1), dtype=np.float64)
    total = np.empty(B, dtype=np.float64)
    lib.oracle_transducer_forward(TRANSDUCER_KINDS[kind], B, T, U, _ptr(blank), _ptr(label),
                                  _ptr(fr), _ptr(lb), _ptr(alpha), _ptr(total))
    return total, alpha
