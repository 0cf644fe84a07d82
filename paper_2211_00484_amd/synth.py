"""Seeded synthetic inputs shaped like the paper's decoding workloads.

This module only draws random numbers and lays them out; it holds none of the
decoding arithmetic, so both the HIP path and the CPU oracle may consume what it
returns.

Shapes follow the paper's model (Sec. 5.1): encoder/decoder/joiner dimension
C = 512, a 500-piece BPE vocabulary with blank = 0, a stateless decoder with a
two-label context, and 4x-subsampled 10 ms frames (25 encoder frames per second
of audio).  Random N(0, sigma) weights stand in for the trained model and
N(0, 1) encoder frames stand in for LibriSpeech audio.  A random sparse FSA
stands in for the LG decoding graph of Table 6.

Draw order (``numpy.random.default_rng(seed)``): lengths (only when they vary),
encoder output, embedding E [V, C], depthwise conv taps [C, 2], joiner weight
W [V, C], joiner bias [V].  Graphs draw from a second generator
(``default_rng(graph_seed)``): per-state weights (power-law graphs only), the
out-degrees, then arc destinations, labels and scores.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = ["Graph", "Model", "Inputs", "Workload", "WORKLOADS", "trivial_graph",
           "uniform_random_graph", "power_law_graph", "random_small_graph",
           "make_model", "make_inputs", "make_workload"]


@dataclass
class Graph:
    """An epsilon-free decoding graph in CSR form (arcs sorted by source state)."""
    num_states: int
    start: int
    vocab_size: int
    row_ptr: np.ndarray   # int32 [S+1]
    dest: np.ndarray      # int32 [A]
    label: np.ndarray     # int32 [A], in [1, V-1]
    score: np.ndarray     # float32 [A], log domain
    final: Optional[np.ndarray] = None  # float32 [S]; -inf = not final; None = all final with 0

    @property
    def num_arcs(self) -> int:
        return int(self.row_ptr[-1])

    @property
    def max_out_degree(self) -> int:
        return int(np.max(np.diff(self.row_ptr))) if self.num_states else 0


@dataclass
class Model:
    """Stateless-decoder embedding, its context-2 depthwise conv taps and the joiner."""
    vocab_size: int
    dim: int
    embed: np.ndarray   # float32 [V, C]
    conv: np.ndarray    # float32 [C, 2]; tap 0 weights the older label
    w_out: np.ndarray   # float32 [V, C]
    b_out: np.ndarray   # float32 [V]


@dataclass
class Inputs:
    encoder_out: np.ndarray  # float32 [B, T, C]; frames >= length are zero
    lengths: np.ndarray      # int32 [B]

    @property
    def B(self) -> int:
        return int(self.encoder_out.shape[0])

    @property
    def T(self) -> int:
        return int(self.encoder_out.shape[1])


@dataclass
class Workload:
    name: str
    B: int
    T: int                       # maximum frames
    length_range: Optional[tuple]  # (lo, hi) inclusive, or None for fixed T
    C: int
    V: int
    sigma: float
    graph: str                   # "trivial" | "uniform5k" | "powerlaw1m"
    beam: float
    max_states: int
    max_contexts: int
    dtype: str                   # "fp32" | "bf16" (joiner GEMM operands)
    description: str = ""
    extra: dict = field(default_factory=dict)


WORKLOADS = {
    "tiny": Workload("tiny", B=2, T=20, length_range=None, C=32, V=16, sigma=0.1,
                     graph="trivial", beam=math.inf, max_states=4, max_contexts=4,
                     dtype="fp32",
                     description="B=2, T=20, C=32, V=16, trivial graph, beam 4"),
    "standard": Workload("standard", B=32, T=250, length_range=(100, 250), C=512, V=500,
                         sigma=0.05, graph="trivial", beam=math.inf, max_states=4,
                         max_contexts=4, dtype="fp32",
                         description="B=32, T~U{100..250}, C=512, V=500, trivial graph, beam 4, fp32"),
    "graph": Workload("graph", B=32, T=250, length_range=(100, 250), C=512, V=500,
                      sigma=0.05, graph="uniform5k", beam=4.0, max_states=32,
                      max_contexts=8, dtype="fp32",
                      description="Standard shapes + 5,000-state / 100,000-arc random FSA, "
                                  "beam 4.0, max_states 32, max_contexts 8"),
    "throughput": Workload("throughput", B=256, T=250, length_range=None, C=512, V=500,
                           sigma=0.05, graph="trivial", beam=math.inf, max_states=4,
                           max_contexts=4, dtype="bf16",
                           description="B=256, T=250, C=512, V=500, bf16 joiner, trivial graph, beam 4"),
    "large": Workload("large", B=128, T=500, length_range=(300, 500), C=512, V=5000,
                      sigma=0.05, graph="powerlaw1m", beam=8.0, max_states=64,
                      max_contexts=16, dtype="fp32",
                      description="B=128, T~U{300..500}, V=5,000, 1M-state / 5M-arc power-law FSA, "
                                  "beam 8.0, max_states 64, max_contexts 16"),
}


def trivial_graph(vocab_size: int) -> Graph:
    """One state with a 0-score self-loop for every non-blank label (Table 6 'trivial graph')."""
    V = int(vocab_size)
    row_ptr = np.array([0, V - 1], dtype=np.int32)
    dest = np.zeros(V - 1, dtype=np.int32)
    label = np.arange(1, V, dtype=np.int32)
    score = np.zeros(V - 1, dtype=np.float32)
    return Graph(1, 0, V, row_ptr, dest, label, score, None)


def _csr_from_degrees(rng: np.random.Generator, deg: np.ndarray, V: int, start: int = 0) -> Graph:
    S = int(deg.shape[0])
    row_ptr = np.zeros(S + 1, dtype=np.int64)
    np.cumsum(deg, out=row_ptr[1:])
    A = int(row_ptr[-1])
    if A >= 2 ** 31:
        raise ValueError("too many arcs for int32 CSR")
    dest = rng.integers(0, S, size=A, dtype=np.int64).astype(np.int32)
    label = rng.integers(1, V, size=A, dtype=np.int64).astype(np.int32)
    score = np.log(rng.uniform(0.01, 1.0, size=A)).astype(np.float32)
    return Graph(S, start, V, row_ptr.astype(np.int32), dest, label, score, None)


def uniform_random_graph(num_states: int = 5000, num_arcs: int = 100_000, vocab_size: int = 500,
                         seed: int = 1) -> Graph:
    """Random sparse FSA: out-degree 1 + multinomial(A - S, uniform); uniform dest and labels;
    arc scores log U(0.01, 1)."""
    rng = np.random.default_rng(seed)
    S = int(num_states)
    deg = 1 + rng.multinomial(int(num_arcs) - S, np.full(S, 1.0 / S))
    return _csr_from_degrees(rng, deg, vocab_size)


def power_law_graph(num_states: int = 1_000_000, num_arcs: int = 5_000_000,
                    vocab_size: int = 5000, seed: int = 1, alpha: float = 1.5,
                    cap: float = 3750.0) -> Graph:
    """LG-like FSA with a heavy-tailed out-degree: w = min(pareto(alpha) + 1, cap),
    out-degree = 1 + multinomial(A - S, w / sum(w))."""
    rng = np.random.default_rng(seed)
    S = int(num_states)
    w = np.minimum(rng.pareto(alpha, size=S) + 1.0, cap)
    deg = 1 + rng.multinomial(int(num_arcs) - S, w / w.sum())
    return _csr_from_degrees(rng, deg, vocab_size)


def random_small_graph(rng: np.random.Generator, num_states: int, vocab_size: int,
                       max_degree: int = 3, with_final: bool = False) -> Graph:
    """Tiny random FSA for exhaustive tests (each state gets 0..max_degree arcs)."""
    S = int(num_states)
    deg = rng.integers(0, max_degree + 1, size=S)
    if deg.sum() == 0:
        deg[0] = 1
    g = _csr_from_degrees(rng, deg, vocab_size, start=int(rng.integers(0, S)))
    if with_final:
        fin = np.log(rng.uniform(0.05, 1.0, size=S)).astype(np.float32)
        nonfinal = rng.uniform(size=S) < 0.4
        fin[nonfinal] = -np.inf
        g.final = fin
    return g


def make_model(rng: np.random.Generator, V: int, C: int, sigma: float) -> Model:
    E = (sigma * rng.standard_normal((V, C), dtype=np.float32)).astype(np.float32)
    conv = (sigma * rng.standard_normal((C, 2), dtype=np.float32)).astype(np.float32)
    W = (sigma * rng.standard_normal((V, C), dtype=np.float32)).astype(np.float32)
    b = (sigma * rng.standard_normal(V, dtype=np.float32)).astype(np.float32)
    return Model(V, C, E, conv, W, b)


def make_inputs(rng: np.random.Generator, B: int, T: int, C: int,
                length_range: Optional[tuple] = None) -> Inputs:
    if length_range is not None:
        lo, hi = length_range
        lengths = rng.integers(lo, hi + 1, size=B).astype(np.int32)
        Tmax = int(lengths.max()) if B else 0
    else:
        lengths = np.full(B, T, dtype=np.int32)
        Tmax = T
    enc = rng.standard_normal((B, Tmax, C), dtype=np.float32)
    for b in range(B):
        enc[b, lengths[b]:, :] = 0.0
    return Inputs(enc, lengths)


def make_graph(kind: str, V: int) -> Graph:
    if kind == "trivial":
        return trivial_graph(V)
    if kind == "uniform5k":
        return uniform_random_graph(5000, 100_000, V, seed=1)
    if kind == "powerlaw1m":
        return power_law_graph(1_000_000, 5_000_000, V, seed=1)
    raise ValueError(f"unknown graph kind {kind!r}")


def make_workload(name: str, seed: int = 0, B: Optional[int] = None):
    """Returns (workload, inputs, model, graph) for a named configuration.

    ``B`` overrides the batch size (the per-stream draws then differ from the full
    configuration, since the generator is shared)."""
    w = WORKLOADS[name]
    rng = np.random.default_rng(seed)
    inputs = make_inputs(rng, w.B if B is None else B, w.T, w.C, w.length_range)
    model = make_model(rng, w.V, w.C, w.sigma)
    graph = make_graph(w.graph, w.V)
    return w, inputs, model, graph
