"""HIP lattice (tbs_lattice_create) and n-best label-sequence search (tbs_lattice_nbest)
against the CPU oracle.

Lattice parity: on streams whose search decisions all have a margin above MARGIN (the rule
of test_gpu_decode.py), the nodes and the arc structure (source, destination, label,
graph arc, in order) are identical to the oracle's, arc weights agree within WTOL and the
forward scores and totals within ATOL.  On every stream the arcs are also checked against
an enumeration of the expansions between the GPU's own nodes (complete, in order).

n-best parity: both sides take the same uniforms.  A path's picks are compared from its
last pick backwards up to its first contested pick (oracle inversion margin below DELTA,
where the fp32 and fp64 weights may legitimately pick differently).  Where no pick of a
stream is contested, the distinct sequences, their order and their scores (within ATOL)
agree, and so does the best sequence unless two scores are within 2 ATOL.  Otherwise the
GPU's distinct sequences are checked to be distinct, to be the blank-free sequences of its
paths, and to carry the oracle's total probability of that sequence within ATOL.
"""
import math

import numpy as np
import pytest

import oracle
from gpu_util import say
from paper_2211_00484_amd import synth

pytestmark = pytest.mark.gpu

TOL = {"fp32": dict(margin=1e-4, wtol=1e-4, atol=1e-3, delta=1e-4),
       "bf16": dict(margin=2e-3, wtol=5e-3, atol=5e-2, delta=1e-2)}


def _np(t):
    return t.cpu().numpy()


def _gpu_lattice(model_np, graph_np, inputs, beam, Ns, Nc, dtype, schedule, graphs_np=None):
    import torch
    from paper_2211_00484_amd import tbs
    model = tbs.Model.from_synth(model_np, dtype=dtype)
    model.set_schedule(schedule)
    if graphs_np is not None:
        graph = [tbs.Graph.from_synth(g) for g in graphs_np]
    else:
        graph = tbs.Graph.from_synth(graph_np)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    lat = tbs.Lattice(model, graph, enc, inputs.lengths, beam=beam, max_states=Ns,
                      max_contexts=Nc)
    ex = {k: _np(v) for k, v in lat.export().items()}
    torch.cuda.synchronize()
    return lat, ex


def _expected_arcs(nodes_f, nodes_f1, graph, V):
    """Expansions of frame-f nodes into frame-(f+1) nodes, in lattice order."""
    rp, dest, lab = graph.row_ptr, graph.dest, graph.label
    nxt = {(int(x[0]), int(x[1])): j for j, x in enumerate(nodes_f1)}
    out = []
    for i, x in enumerate(nodes_f):
        ctx, st = int(x[0]), int(x[1])
        if (ctx, st) in nxt:
            out.append((nxt[(ctx, st)], i, -1, 0, -1))
        for k in range(rp[st], rp[st + 1]):
            key = ((ctx % V) * V + int(lab[k]), int(dest[k]))
            if key in nxt:
                out.append((nxt[key], i, k - rp[st], int(lab[k]), k))
    out.sort(key=lambda a: (a[0], a[1], a[2]))
    return [(a[1], a[0], a[3], a[4]) for a in out]


def _stream_view(ex, b, T, Ns, L):
    nodes = []
    for f in range(L + 1):
        x = ex["nodes"][f, b]
        nodes.append(x[x[:, 0] >= 0])
    off = ex["frame_off"]
    arcs = [ex["arcs"][off[b * T + f]:off[b * T + f + 1]] for f in range(L)]
    w = [ex["weights"][off[b * T + f]:off[b * T + f + 1]] for f in range(L)]
    return nodes, arcs, w


def check_lattice(ex, orc, model_np, graphs_np, inputs, Ns, dtype, streams=None):
    """Returns the list of clean streams (lattice identical to the oracle's)."""
    tol = TOL[dtype]
    B, T = inputs.B, inputs.T
    V = model_np.vocab_size
    clean = []
    streams = range(B) if streams is None else streams
    for k, b in enumerate(streams):
        L = int(inputs.lengths[b])
        nodes, arcs, w = _stream_view(ex, b, T, Ns, L)
        g = graphs_np[b]
        # structure against the GPU's own nodes, on every stream
        for f in range(L):
            want = _expected_arcs(nodes[f], nodes[f + 1], g, V)
            got = [tuple(int(v) for v in a) for a in arcs[f]]
            assert got == want, f"stream {b} frame {f}: arcs differ from the expansions"
        assert ex["status"][b] in (0, 1)
        fm = orc.frame_margins[k]
        if not all(fm[t] > tol["margin"] for t in range(L)) or fm[T] <= tol["margin"]:
            continue
        s = orc.stream(k)
        for f in range(L + 1):
            assert np.array_equal(nodes[f], s.nodes[f]), f"stream {b}: nodes of frame {f}"
        for f in range(L):
            assert np.array_equal(arcs[f], s.arcs[f]), f"stream {b}: arcs of frame {f}"
            assert np.allclose(w[f], s.w[f], atol=tol["wtol"], rtol=0), \
                f"stream {b} frame {f}: max weight error {np.abs(w[f] - s.w[f]).max()}"
        for f in range(L + 1):
            n = len(s.nodes[f])
            assert np.allclose(ex["alpha"][b, f, :n], s.alpha[f], atol=tol["atol"], rtol=0)
        n = len(s.fw)
        assert np.array_equal(ex["final_w"][b, :n], s.fw)
        assert ex["total"][b] == pytest.approx(s.total, abs=tol["atol"])
        assert ex["status"][b] == s.status
        clean.append((k, b))
    return clean


def check_nbest(lat, ex, orc, clean, inputs, n, dtype, seed=0, streams=None):
    import torch
    tol = TOL[dtype]
    B, T = inputs.B, inputs.T
    u = np.random.default_rng(seed).uniform(size=(B, n, T + 1))
    out = lat.nbest(n, torch.from_numpy(u).cuda(), want_paths=True)
    torch.cuda.synchronize()
    g_paths, g_nu = _np(out.paths), _np(out.num_unique)
    g_us, g_uf = _np(out.unique_scores), _np(out.unique_first)
    g_tok, g_nt, g_sc = _np(out.tokens), _np(out.num_tokens), _np(out.scores)
    streams = list(range(B)) if streams is None else list(streams)
    clean_k = dict((b, k) for k, b in clean)
    n_exact = 0
    for k, b in enumerate(streams):
        L = int(inputs.lengths[b])
        nodes, arcs, w = _stream_view(ex, b, T, lat.max_states, L)
        # every GPU path is a lattice path; collect its blank-free sequence
        seqs = []
        for p in range(n):
            pp = g_paths[b, p]
            assert (pp[L + 1:] == -1).all()
            node = int(pp[L])
            assert 0 <= node < len(nodes[L]) and ex["final_w"][b, node] != -math.inf
            lab = []
            for f in range(L - 1, -1, -1):
                a = arcs[f][pp[f]]
                assert a[1] == node, f"stream {b} path {p} frame {f}: arc not into the node"
                if a[2] > 0:
                    lab.append(int(a[2]))
                node = int(a[0])
            assert node == 0
            seqs.append(lab[::-1])
        nu = int(g_nu[b])
        firsts = [int(x) for x in g_uf[b, :nu]]
        assert (g_uf[b, nu:] == -1).all() and (g_us[b, nu:] == -math.inf).all()
        # distinct sequences in order of first occurrence
        want_first, seen = [], set()
        for p, y in enumerate(seqs):
            if tuple(y) not in seen:
                seen.add(tuple(y))
                want_first.append(p)
        assert firsts == want_first, f"stream {b}: distinct sequences"
        best = int(np.argmax(g_us[b, :nu]))
        assert g_sc[b] == g_us[b, best]
        assert [int(x) for x in g_tok[b, :g_nt[b]]] == seqs[firsts[best]]
        assert (g_tok[b, g_nt[b]:] == -1).all()
        if b not in clean_k:
            continue
        kk = clean_k[b]
        nb = orc.nbest(kk, u[b, :, :L + 1])
        contested = False
        for p in range(n):
            # compare from the last pick (the final node) backwards
            order = [L] + list(range(L - 1, -1, -1))
            for f in order:
                if nb.margins[p, f] <= tol["delta"]:
                    contested = True
                    break
                assert g_paths[b, p, f] == nb.paths[p, f], f"stream {b} path {p} pick {f}"
        if not contested:
            n_exact += 1
            assert firsts == [int(x) for x in nb.first]
            assert np.allclose(g_us[b, :nu], nb.scores, atol=tol["atol"], rtol=0)
            srt = sorted(nb.scores, reverse=True)
            if len(srt) == 1 or srt[0] - srt[1] > 2 * tol["atol"]:
                assert [int(x) for x in g_tok[b, :g_nt[b]]] == nb.tokens
                assert g_sc[b] == pytest.approx(nb.score, abs=tol["atol"])
        else:
            # validity: each GPU sequence carries its total probability in the lattice
            for q in range(nu):
                want = orc.sequence_score(kk, seqs[firsts[q]])
                assert g_us[b, q] == pytest.approx(want, abs=tol["atol"]), (b, q)
    say(f"  n-best: {len(clean)} clean lattices, {n_exact} streams with no contested pick")
    return n_exact


def _run(inputs, model_np, graph_np, beam, Ns, Nc, dtype, schedule, n=48, graphs_np=None,
         min_exact=1):
    from paper_2211_00484_amd import tbs
    say(f"lattice B={inputs.B} T={inputs.T} V={model_np.vocab_size} beam={beam} Ns={Ns} "
        f"Nc={Nc} {dtype} {schedule}")
    try:
        lat, ex = _gpu_lattice(model_np, graph_np, inputs, beam, Ns, Nc, dtype, schedule,
                               graphs_np)
    except tbs.TbsError as e:
        if schedule == "stream" and e.status == -5:
            pytest.skip(f"shape not supported by the per-stream kernel: {e}")
        raise
    graphs = graphs_np if graphs_np is not None else [graph_np] * inputs.B
    say(f"  {lat.num_arcs()} arcs")
    # the oracle per distinct graph
    orcs = {}
    clean = []
    for gid in sorted({id(g) for g in graphs}):
        g = next(x for x in graphs if id(x) == gid)
        streams = [b for b in range(inputs.B) if id(graphs[b]) == gid]
        o = oracle.lattice(model_np, g, inputs.encoder_out, inputs.lengths, beam, Ns, Nc,
                           bf16=(dtype == "bf16"), streams=streams)
        c = check_lattice(ex, o, model_np, graphs, inputs, Ns, dtype, streams=streams)
        orcs[gid] = (o, streams, c)
        clean += c
    say(f"  lattice: {len(clean)} of {inputs.B} streams clean")
    n_exact = 0
    for gid, (o, streams, c) in orcs.items():
        n_exact += check_nbest(lat, ex, o, c, inputs, n, dtype, streams=streams)
    assert n_exact >= min_exact
    return lat, ex


@pytest.mark.parametrize("schedule", ["frame", "stream"])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_tiny(dtype, schedule):
    w, inputs, model, graph = synth.make_workload("tiny")
    # bf16 weights differ from the oracle's by up to ~1e-3: most streams hold a pick
    # within DELTA of a boundary, and those are checked for validity only
    _run(inputs, model, graph, math.inf, 4, 4, dtype, schedule, n=64,
         min_exact=1 if dtype == "fp32" else 0)


@pytest.mark.parametrize("schedule", ["frame", "stream"])
@pytest.mark.parametrize("seed", range(6))
def test_random_small_graphs(seed, schedule):
    rng = np.random.default_rng(400 + seed)
    V = int(rng.integers(3, 30))
    C = int(rng.integers(2, 60))
    model = synth.make_model(rng, V, C, 0.5)
    inputs = synth.make_inputs(rng, 5, 30, C, length_range=(0, 30))
    graph = synth.random_small_graph(rng, int(rng.integers(1, 30)), V,
                                     max_degree=int(rng.integers(1, 8)),
                                     with_final=bool(seed % 2))
    beam = [math.inf, 3.0, 1.5][seed % 3]
    Ns = int(rng.integers(1, 17))
    Nc = int(rng.integers(1, Ns + 1))
    _run(inputs, model, graph, beam, Ns, Nc, "fp32", schedule, n=40, min_exact=0)


def test_ragged_and_empty_streams():
    rng = np.random.default_rng(9)
    model = synth.make_model(rng, 16, 32, 0.3)
    inputs = synth.make_inputs(rng, 6, 25, 32)
    inputs.lengths[:] = [0, 25, 1, 13, 0, 24]
    for b in range(inputs.B):
        inputs.encoder_out[b, inputs.lengths[b]:] = 0.0
    lat, ex = _run(inputs, model, synth.trivial_graph(16), math.inf, 4, 4, "fp32", "frame")
    for b in (0, 4):
        off = ex["frame_off"]
        assert off[b * inputs.T] == off[(b + 1) * inputs.T]  # no arcs
        assert ex["total"][b] == 0.0


@pytest.mark.parametrize("schedule", ["frame", "stream"])
def test_standard_shapes(schedule):
    """The Standard workload (B=32, T up to 250, V=500, trivial graph, top-4)."""
    w, inputs, model, graph = synth.make_workload("standard")
    _run(inputs, model, graph, w.beam, w.max_states, w.max_contexts, "fp32", schedule, n=32,
         min_exact=4)


def test_graph_shapes():
    """Graph workload shapes (5,000-state graph, beam 4, 32 states, 8 contexts), 8 streams."""
    w, inputs, model, graph = synth.make_workload("graph", B=8)
    _run(inputs, model, graph, w.beam, w.max_states, w.max_contexts, "fp32", "frame", n=32,
         min_exact=1)


def test_per_stream_graphs():
    rng = np.random.default_rng(12)
    V, C = 12, 24
    model = synth.make_model(rng, V, C, 0.5)
    inputs = synth.make_inputs(rng, 4, 20, C, length_range=(5, 20))
    g1 = synth.random_small_graph(rng, 6, V, max_degree=4, with_final=True)
    g2 = synth.random_small_graph(rng, 9, V, max_degree=5, with_final=False)
    _run(inputs, model, None, 4.0, 8, 4, "fp32", "frame", n=32, graphs_np=[g1, g2, g2, g1])


def test_single_hypothesis_lattice():
    """Ns = Nc = 1: one node per frame; the n-best result is the search's best path."""
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("tiny")
    lat, ex = _gpu_lattice(model_np, graph_np, inputs, math.inf, 1, 1, "fp32", "frame")
    u = torch.from_numpy(np.random.default_rng(1).uniform(size=(2, 8, inputs.T + 1))).cuda()
    out = lat.nbest(8, u)
    model = tbs.Model.from_synth(model_np)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    best = tbs.decode(model, tbs.Graph.from_synth(graph_np), enc, inputs.lengths,
                      max_states=1, max_contexts=1)
    assert out.token_lists() == best.token_lists()
    assert (_np(out.num_unique) == 1).all()


def test_nbest_arguments():
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("tiny")
    lat, _ = _gpu_lattice(model_np, graph_np, inputs, math.inf, 4, 4, "fp32", "frame")
    with pytest.raises(ValueError):
        lat.nbest(4, torch.zeros((2, 3, inputs.T + 1), dtype=torch.float64, device="cuda"))
    with pytest.raises(tbs.TbsError) as e:
        lat.nbest(0, torch.zeros((2, 0, inputs.T + 1), dtype=torch.float64, device="cuda"))
    assert e.value.status == -1
    # a larger n after a smaller one regrows the scratch
    for n in (4, 70, 16):
        u = torch.from_numpy(np.random.default_rng(n).uniform(size=(2, n, inputs.T + 1))).cuda()
        out = lat.nbest(n, u)
        torch.cuda.synchronize()
        assert (_np(out.num_unique) >= 1).all() and (_np(out.num_unique) <= n).all()


def test_buffer_reuse_across_sizes():
    """Lattices built one after another on one model (smaller, equal, larger than the
    last destroyed one) equal lattices built on fresh models."""
    import torch
    from paper_2211_00484_amd import tbs
    w, inputs, model_np, graph_np = synth.make_workload("graph", B=6)
    enc = torch.from_numpy(inputs.encoder_out).cuda()
    u = torch.from_numpy(np.random.default_rng(2).uniform(size=(6, 24, inputs.T + 1))).cuda()

    def build(model, B, T):
        lat = tbs.Lattice(model, tbs.Graph.from_synth(graph_np), enc[:B, :T].contiguous(),
                          np.minimum(inputs.lengths[:B], T), beam=4.0, max_states=32,
                          max_contexts=8)
        ex = {k: _np(v) for k, v in lat.export().items()}
        nb = lat.nbest(24, u[:B, :, :T + 1].contiguous(), want_paths=True)
        res = (ex, _np(nb.tokens), _np(nb.scores), _np(nb.paths))
        torch.cuda.synchronize()
        lat.close()
        return res

    shared = tbs.Model.from_synth(model_np)
    shared.set_schedule("frame")
    for B, T in ((6, inputs.T), (3, inputs.T // 2), (3, inputs.T // 2), (6, inputs.T)):
        fresh = tbs.Model.from_synth(model_np)
        fresh.set_schedule("frame")
        a, b = build(shared, B, T), build(fresh, B, T)
        for k in a[0]:
            assert np.array_equal(a[0][k], b[0][k]), (B, T, k)
        for x, y in zip(a[1:], b[1:]):
            assert np.array_equal(x, y), (B, T)
