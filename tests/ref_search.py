"""Independent references that pin the CPU oracle (test code only).

None of these share code with the oracle or with the HIP path:

* ``LayerJoiner`` builds the stateless decoder and joiner from library layers
  (``nn.Embedding`` + depthwise ``nn.Conv1d`` with kernel size 2, ReLU, tanh,
  ``nn.Linear``, ``log_softmax``) in float64, as Sec. 5.1 describes the model.
* ``brute_force`` enumerates every frame-label sequence and graph path (the
  one-symbol-per-frame lattice composed with the graph, Sec. 2.3 / 2.4).
* ``viterbi`` is the textbook max-product recursion over (context, state).
* ``greedy`` is per-frame argmax decoding with max-symbols = 1 (Table 5).
* ``beam_search_sorted`` re-implements the pruned search of Sec. 2.5 by
  materialising and sorting every candidate with Python's ``sorted``.
"""
from __future__ import annotations

import math
from functools import lru_cache

import numpy as np
import torch


class LayerJoiner:
    """log P(. | (a, b), t) from library layers, float64."""

    def __init__(self, model, bf16: bool = False):
        V, C = model.vocab_size, model.dim
        self.V, self.C, self.bf16 = V, C, bf16
        self.emb = torch.nn.Embedding(V, C).double()
        self.conv = torch.nn.Conv1d(C, C, kernel_size=2, groups=C, bias=False).double()
        self.lin = torch.nn.Linear(C, V, bias=True).double()
        with torch.no_grad():
            self.emb.weight.copy_(torch.from_numpy(model.embed.astype(np.float64)))
            # Conv1d weight [C, 1, 2]: position 0 of the kernel sees the older label.
            self.conv.weight.copy_(torch.from_numpy(model.conv.astype(np.float64)).unsqueeze(1))
            w = torch.from_numpy(model.w_out.astype(np.float32))
            if bf16:
                w = w.to(torch.bfloat16)
            self.lin.weight.copy_(w.double())
            b = model.b_out if model.b_out is not None else np.zeros(V, np.float32)
            self.lin.bias.copy_(torch.from_numpy(b.astype(np.float64)))

    @torch.no_grad()
    def __call__(self, enc_row: np.ndarray, a: int, b: int) -> np.ndarray:
        seq = self.emb(torch.tensor([[a, b]]))            # [1, 2, C]
        dec = torch.relu(self.conv(seq.transpose(1, 2)))  # [1, C, 1]
        h = torch.tanh(torch.from_numpy(enc_row.astype(np.float64)) + dec[0, :, 0])
        if self.bf16:
            h = h.float().to(torch.bfloat16).double()
        return torch.log_softmax(self.lin(h), dim=-1).numpy()


def _final(graph, s):
    if graph.final is None:
        return 0.0
    f = float(graph.final[s])
    return f if math.isfinite(f) else None


def _logp_fn(joiner, enc):
    @lru_cache(maxsize=None)
    def lp(t, ctx):
        a, b = divmod(ctx, joiner.V)
        return joiner(enc[t], a, b)
    return lp


def brute_force(joiner, graph, enc, length):
    """Best path by exhaustive enumeration.  Returns (score, tokens, arcs, is_final);
    ``score`` includes the final weight; paths ending in non-final states are used only
    if no path ends in a final state."""
    V = joiner.V
    lp = _logp_fn(joiner, enc)
    rp, dest, lab, q = graph.row_ptr, graph.dest, graph.label, graph.score
    best = {True: (-math.inf, None), False: (-math.inf, None)}

    def rec(t, ctx, s, score, arcs):
        if t == length:
            f = _final(graph, s)
            key = f is not None
            val = score + (f if key else 0.0)
            if val > best[key][0]:
                best[key] = (val, list(arcs))
            return
        p = lp(t, ctx)
        arcs.append(-1)
        rec(t + 1, ctx, s, score + p[0], arcs)
        arcs.pop()
        for j in range(rp[s], rp[s + 1]):
            c = int(lab[j])
            arcs.append(j)
            rec(t + 1, (ctx % V) * V + c, int(dest[j]), score + float(q[j]) + p[c], arcs)
            arcs.pop()

    rec(0, 0, graph.start, 0.0, [])
    is_final = best[True][1] is not None
    score, arcs = best[True] if is_final else best[False]
    tokens = [int(lab[j]) for j in arcs if j >= 0]
    return score, tokens, arcs, is_final


def viterbi(joiner, graph, enc, length):
    """Max-product recursion over (context, state) pairs.  Returns (score, tokens, is_final)."""
    V = joiner.V
    lp = _logp_fn(joiner, enc)
    rp, dest, lab, q = graph.row_ptr, graph.dest, graph.label, graph.score
    alpha = {(0, graph.start): (0.0, None)}
    backs = []
    for t in range(length):
        nxt = {}
        for (ctx, s), (sc, _) in alpha.items():
            p = lp(t, ctx)
            cands = [((ctx, s), sc + p[0], 0)]
            for j in range(rp[s], rp[s + 1]):
                c = int(lab[j])
                cands.append((((ctx % V) * V + c, int(dest[j])), sc + float(q[j]) + p[c], c))
            for key, v, c in cands:
                if key not in nxt or v > nxt[key][0]:
                    nxt[key] = (v, ((ctx, s), c))
        backs.append(nxt)
        alpha = nxt
    best_key, best_val, is_final = None, -math.inf, False
    for want_final in (True, False):
        for key, (v, _) in alpha.items():
            f = _final(graph, key[1])
            if want_final and f is None:
                continue
            val = v + (f if want_final else 0.0)
            if val > best_val:
                best_key, best_val = key, val
        if best_key is not None:
            is_final = want_final
            break
    tokens = []
    key = best_key
    for t in range(length - 1, -1, -1):
        _, (prev, c) = backs[t][key]
        if c:
            tokens.append(c)
        key = prev
    return best_val, tokens[::-1], is_final


def greedy(joiner, enc, length):
    """Per-frame argmax with one symbol per frame; blank keeps the context."""
    V = joiner.V
    ctx, score, tokens = 0, 0.0, []
    for t in range(length):
        p = joiner(enc[t], ctx // V, ctx % V)
        c = int(np.argmax(p))
        score += float(p[c])
        if c:
            tokens.append(c)
            ctx = (ctx % V) * V + c
    return score, tokens


def beam_search_sorted(joiner, graph, enc, length, beam, max_states, max_contexts):
    """Pruned search, candidates materialised and ordered with ``sorted``.

    Returns (score, tokens, trace) with trace[f] = list of (ctx, state, parent, label)."""
    V = joiner.V
    lp = _logp_fn(joiner, enc)
    rp, dest, lab, q = graph.row_ptr, graph.dest, graph.label, graph.score
    hyps = [(0, graph.start, 0.0)]            # (ctx, state, score)
    trace = [[(0, graph.start, -1, -1)]]
    backs = []
    for t in range(length):
        cands = []
        for i, (ctx, s, sc) in enumerate(hyps):
            p = lp(t, ctx)
            cands.append(((s, ctx), sc + p[0], (i, -1), 0))
            for pos, j in enumerate(range(rp[s], rp[s + 1])):
                c = int(lab[j])
                cands.append(((int(dest[j]), (ctx % V) * V + c), sc + float(q[j]) + p[c], (i, pos), c))
        # max-merge: order all candidates, first occurrence of a key wins
        cands = sorted(cands, key=lambda x: (-x[1], x[2]))
        merged = {}
        for key, v, tb, c in cands:
            if key not in merged:
                merged[key] = (v, tb[0], c)
        ents = sorted(merged.items(), key=lambda kv: (-kv[1][0], kv[0]))
        top = ents[0][1][0]
        ents = [e for e in ents if e[1][0] >= top - beam][:max_states]
        cbest = {}
        for (s, ctx), (v, _, _) in ents:
            cbest[ctx] = max(cbest.get(ctx, -math.inf), v)
        keep = {c for c, _ in sorted(cbest.items(), key=lambda kv: (-kv[1], kv[0]))[:max_contexts]}
        ents = sorted([e for e in ents if e[0][1] in keep], key=lambda e: (e[0][1], e[0][0]))
        hyps = [(ctx, s, v) for (s, ctx), (v, _, _) in ents]
        trace.append([(ctx, s, par, c) for (s, ctx), (v, par, c) in ents])
        backs.append([(par, c) for (_, _), (_, par, c) in ents])
    best_i, best_v = None, -math.inf
    for want_final in (True, False):
        for i, (ctx, s, v) in enumerate(hyps):
            f = _final(graph, s)
            if want_final and f is None:
                continue
            val = v + (f if want_final else 0.0)
            if val > best_v:
                best_i, best_v = i, val
        if best_i is not None:
            break
    tokens = []
    i = best_i
    for t in range(length - 1, -1, -1):
        par, c = backs[t][i]
        if c:
            tokens.append(c)
        i = par
    return best_v, tokens[::-1], trace


def all_alignments(joiner, graph, enc, length):
    """Every alignment of ``length`` frames (one label or blank per frame, the labels a
    graph path from the start state): list of (score, frame labels, arcs, final weight or
    None for a non-final end state)."""
    V = joiner.V
    lp = _logp_fn(joiner, enc)
    rp, dest, lab, q = graph.row_ptr, graph.dest, graph.label, graph.score
    out = []

    def rec(t, ctx, s, score, labels, arcs):
        if t == length:
            out.append((score, tuple(labels), tuple(arcs), _final(graph, s)))
            return
        p = lp(t, ctx)
        rec(t + 1, ctx, s, score + p[0], labels + [0], arcs + [-1])
        for j in range(rp[s], rp[s + 1]):
            c = int(lab[j])
            rec(t + 1, (ctx % V) * V + c, int(dest[j]), score + float(q[j]) + p[c],
                labels + [c], arcs + [j])

    rec(0, 0, graph.start, 0.0, [], [])
    return out


def _logsumexp(xs):
    xs = [x for x in xs if x != -math.inf]
    if not xs:
        return -math.inf
    m = max(xs)
    return m + math.log(sum(math.exp(x - m) for x in xs))


def sequence_totals(joiner, graph, enc, length):
    """Exhaustive LogAdd merge: {blank-free label sequence: log of the summed probability of
    its alignments}, final weights included; alignments ending in non-final states count
    (with weight 0) only if no alignment ends in a final state.  Also returns the total."""
    al = all_alignments(joiner, graph, enc, length)
    any_final = any(f is not None for _, _, _, f in al)
    terms = {}
    for score, labels, _, f in al:
        if any_final and f is None:
            continue
        y = tuple(c for c in labels if c)
        terms.setdefault(y, []).append(score + (f if any_final else 0.0))
    totals = {y: _logsumexp(v) for y, v in terms.items()}
    return totals, _logsumexp([v for vs in terms.values() for v in vs])


def hyp_beam_search(joiner, enc, length, beam_size, logadd):
    """Full-sequence beam search with max-symbols 1 over tuples of labels (Table 5's
    comparison search), written independently of the oracle: expand every hypothesis by
    blank and every label, merge equal tuples (max or log-add), keep the best
    ``beam_size`` by (score desc, first candidate index asc).  Returns (tokens, score)."""
    V = joiner.V
    hyps = [((), 0.0)]
    for t in range(length):
        groups = {}
        for i, (y, sc) in enumerate(hyps):
            a = y[-2] if len(y) >= 2 else 0
            b = y[-1] if len(y) >= 1 else 0
            p = joiner(enc[t], a, b)
            for c in range(V):
                z = y + (c,) if c else y
                v = sc + float(p[c])
                idx = i * V + c
                if z in groups:
                    old, first = groups[z]
                    groups[z] = (_logsumexp([old, v]) if logadd else max(old, v), min(first, idx))
                else:
                    groups[z] = (v, idx)
        ranked = sorted(groups.items(), key=lambda kv: (-kv[1][0], kv[1][1]))
        hyps = [(z, v) for z, (v, _) in ranked[:beam_size]]
    return list(hyps[0][0]), hyps[0][1]


def frame_decisions(cands, beam, max_states, max_contexts, delta=None):
    """The decisions of one frame of the pruned search (Sec. 2.5), stage by stage.

    ``cands``: list of (key, score, (parent, arc position), label) with key = (state,
    ctx); ``delta``: optional per-candidate score perturbation (same length).  Returns a
    dict with the merge winners of the kept keys, the set after the beam + max-states
    pruning, the kept contexts and the kept keys, plus ``terms``: one (gap, lower,
    raise) triple per decision, where shifting the candidates ``lower`` down and
    ``raise`` up by just over half the gap changes that decision (None stands for
    every candidate not in the other list)."""
    sc = [c[1] + (0.0 if delta is None else float(delta[i])) for i, c in enumerate(cands)]
    order = sorted(range(len(cands)), key=lambda i: (-sc[i], cands[i][2]))
    by_key = {}
    for i in order:                      # candidates of each key, best first
        by_key.setdefault(cands[i][0], []).append(i)
    merged = {k: ix[0] for k, ix in by_key.items()}
    ents = sorted(merged, key=lambda k: (-sc[merged[k]], k))
    top = sc[merged[ents[0]]]
    thr = top - beam
    in_beam = [k for k in ents if sc[merged[k]] >= thr]
    pre = in_beam[:max_states]
    terms = []
    if len(in_beam) > max_states:
        a, b = in_beam[max_states - 1], in_beam[max_states]
        terms.append((sc[merged[a]] - sc[merged[b]], by_key[a], by_key[b]))
    if math.isfinite(beam):
        # the best tuple is never outside its own beam; the others are inside or
        # outside by their distance to the threshold (None: every other candidate)
        for k in ents[1:max_states]:
            d = sc[merged[k]] - thr
            terms.append((abs(d), by_key[k], None) if d >= 0 else (abs(d), None, by_key[k]))
    cbest = {}
    for k in pre:
        cbest[k[1]] = max(cbest.get(k[1], -math.inf), sc[merged[k]])
    cl = sorted(cbest, key=lambda c: (-cbest[c], c))
    kept_ctx = set(cl[:max_contexts])
    if len(cl) > max_contexts:
        a, b = cl[max_contexts - 1], cl[max_contexts]
        terms.append((cbest[a] - cbest[b],
                      [i for k in pre if k[1] == a for i in by_key[k]],
                      [i for k in pre if k[1] == b for i in by_key[k]]))
    kept = sorted((k for k in pre if k[1] in kept_ctx), key=lambda k: (k[1], k[0]))
    winners = {}
    for k in kept:
        w = merged[k]
        winners[k] = (cands[w][2][0], cands[w][3])
        other = [i for i in by_key[k] if (cands[i][2][0], cands[i][3]) != winners[k]]
        if other:
            terms.append((sc[w] - sc[other[0]], [w], [other[0]]))
    return {"winners": winners, "pre": frozenset(pre), "ctx": frozenset(kept_ctx),
            "kept": kept, "scores": {k: sc[merged[k]] for k in kept}, "terms": terms}


def frame_candidates(lp_row, graph, hyps, V):
    """Unpruned expansion of one frame (blank keeps (ctx, state); arcs move to
    ((b, c), dest) with q + log P(c)): (key, score, (parent, arc position), label)."""
    rp, dest, lab, q = graph.row_ptr, graph.dest, graph.label, graph.score
    cands = []
    for i, (ctx, s, v) in enumerate(hyps):
        p = lp_row(ctx)
        cands.append(((s, ctx), v + p[0], (i, -1), 0))
        for pos, j in enumerate(range(rp[s], rp[s + 1])):
            c = int(lab[j])
            cands.append(((int(dest[j]), (ctx % V) * V + c), v + float(q[j]) + p[c], (i, pos), c))
    return cands
