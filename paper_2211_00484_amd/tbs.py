"""Python binding of libtbs.so (include/tbs.h): argument marshalling only.

Every step of the decode runs in the HIP library; torch supplies device memory
and the current HIP stream.  Importing this module does not load the library;
the first call does, and raises if ``libtbs.so`` has not been built.
"""
from __future__ import annotations

import atexit
import ctypes
import math
import os
import re
import weakref
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtbs.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "tbs.h")

TBS_JOINER_FP32, TBS_JOINER_BF16 = 0, 1
STATUS_NAMES = {0: "TBS_OK", -1: "TBS_EINVAL", -2: "TBS_ENOMEM", -3: "TBS_EDEVICE",
                -4: "TBS_ECAPACITY", -5: "TBS_EUNSUPPORTED"}

_P = ctypes.c_void_p
_I32 = ctypes.c_int32


class TbsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class KernelTime(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


KERNEL_NAMES = ("joiner", "search", "final", "stream", "stream_group", "hyp_step")
SCHEDULES = {"auto": 0, "frame": 1, "stream": 2, "stream1": 3}


class BeamParams(ctypes.Structure):
    _fields_ = [("beam", ctypes.c_float), ("max_states", ctypes.c_int32),
                ("max_contexts", ctypes.c_int32)]


_lib = None
# Set when the interpreter starts to exit: handles still open then are left to the
# process teardown instead of calling into the library (and HIP) from finalizers that
# may run after the runtime has begun shutting down.  Call close() to release earlier.
_exiting = False


def _at_exit():
    global _exiting
    _exiting = True


atexit.register(_at_exit)

_live = weakref.WeakSet()  # open handles (graphs, models, decode states, lattices)


def close_all():
    """Releases every handle still open: lattices and decode states first, then models
    and graphs (a lattice or state refers to its model).  For programs that want the
    device memory back before the interpreter exits."""
    order = {"Lattice": 0, "DecodeState": 1, "Model": 2, "Graph": 3}
    for obj in sorted(list(_live), key=lambda o: order.get(type(o).__name__, 4)):
        obj.close()


def declared_symbols() -> list:
    """Names of the functions declared in include/tbs.h."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(tbs_[a-z_0-9]+)\s*\(",
                                 text, flags=re.M)))


def lib():
    """The loaded library; raises if it is missing (there is no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(hipcc --offload-arch=gfx950); there is no CPU fallback")
    L = ctypes.CDLL(LIB_PATH)
    L.tbs_last_error.restype = ctypes.c_char_p
    L.tbs_last_error.argtypes = []
    L.tbs_graph_create.restype = _I32
    L.tbs_graph_create.argtypes = [_I32, _I32, _I32, _P, _P, _P, _P, _P, ctypes.POINTER(_P)]
    L.tbs_graph_create_trivial.restype = _I32
    L.tbs_graph_create_trivial.argtypes = [_I32, ctypes.POINTER(_P)]
    L.tbs_graph_destroy.restype = None
    L.tbs_graph_destroy.argtypes = [_P]
    L.tbs_model_create.restype = _I32
    L.tbs_model_create.argtypes = [_I32, _I32, _I32, _P, _P, _P, _P, _I32, _P, ctypes.POINTER(_P)]
    L.tbs_model_destroy.restype = None
    L.tbs_model_destroy.argtypes = [_P]
    L.tbs_decode.restype = _I32
    L.tbs_decode.argtypes = [_P, _P, ctypes.POINTER(BeamParams), _P, _P, _I32, _I32,
                             _P, _P, _P, _P, _P, _P, _P]
    L.tbs_decode_noalloc.restype = _I32
    L.tbs_decode_noalloc.argtypes = [_P, _P, ctypes.POINTER(BeamParams), _P, _P, _I32, _I32,
                                     _P, _P, _P, _P, _P, _P, _P]
    L.tbs_decode_graphs.restype = _I32
    L.tbs_decode_graphs.argtypes = [_P, _P, ctypes.POINTER(BeamParams), _P, _P, _I32, _I32,
                                    _P, _P, _P, _P, _P, _P, _P]
    L.tbs_model_set_schedule.restype = _I32
    L.tbs_model_set_schedule.argtypes = [_P, _I32]
    L.tbs_model_set_graph_capture.restype = _I32
    L.tbs_model_set_graph_capture.argtypes = [_P, _I32]
    L.tbs_model_graph_stats.restype = _I32
    L.tbs_model_graph_stats.argtypes = [_P, ctypes.POINTER(_I32), ctypes.POINTER(_I32)]
    L.tbs_model_set_exchange_spin_limit.restype = _I32
    L.tbs_model_set_exchange_spin_limit.argtypes = [_P, _I32]
    L.tbs_model_set_profiling.restype = _I32
    L.tbs_model_set_profiling.argtypes = [_P, _I32]
    L.tbs_model_read_profile.restype = _I32
    L.tbs_model_read_profile.argtypes = [_P, ctypes.POINTER(KernelTime)]
    L.tbs_joiner_logp.restype = _I32
    L.tbs_joiner_logp.argtypes = [_P, _P, _P, _I32, _P, _P]
    L.tbs_state_create.restype = _I32
    L.tbs_state_create.argtypes = [_P, _P, ctypes.POINTER(BeamParams), _I32, _I32, _P,
                                   ctypes.POINTER(_P)]
    L.tbs_state_create_graphs.restype = _I32
    L.tbs_state_create_graphs.argtypes = [_P, _P, ctypes.POINTER(BeamParams), _I32, _I32, _P,
                                          ctypes.POINTER(_P)]
    L.tbs_transducer_forward.restype = _I32
    L.tbs_transducer_forward.argtypes = [_I32, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P]
    L.tbs_hyp_search.restype = _I32
    L.tbs_hyp_search.argtypes = [_P, ctypes.POINTER(HypParams), _P, _P, _I32, _I32, _P, _P, _P,
                                 _P, _P]
    L.tbs_lattice_create.restype = _I32
    L.tbs_lattice_create.argtypes = [_P, _P, ctypes.POINTER(BeamParams), _P, _P, _I32, _I32, _P,
                                     ctypes.POINTER(_P)]
    L.tbs_lattice_create_graphs.restype = _I32
    L.tbs_lattice_create_graphs.argtypes = [_P, _P, ctypes.POINTER(BeamParams), _P, _P, _I32,
                                            _I32, _P, ctypes.POINTER(_P)]
    L.tbs_lattice_num_arcs.restype = _I32
    L.tbs_lattice_num_arcs.argtypes = [_P, ctypes.POINTER(ctypes.c_int64)]
    L.tbs_lattice_export.restype = _I32
    L.tbs_lattice_export.argtypes = [_P] + [_P] * 8 + [_P]
    L.tbs_lattice_nbest.restype = _I32
    L.tbs_lattice_nbest.argtypes = [_P, _I32, _P] + [_P] * 7 + [_P]
    L.tbs_lattice_destroy.restype = None
    L.tbs_lattice_destroy.argtypes = [_P]
    L.tbs_decode_chunk.restype = _I32
    L.tbs_decode_chunk.argtypes = [_P, _P, _P, _I32, _P, _P]
    L.tbs_state_finish.restype = _I32
    L.tbs_state_finish.argtypes = [_P, _P, _P, _P, _P, _P, _P]
    L.tbs_state_destroy.restype = None
    L.tbs_state_destroy.argtypes = [_P]
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise TbsError(status, lib().tbs_last_error().decode())


def _host_ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dev_ptr(t):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream_ptr(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Graph:
    """Device copy of an epsilon-free decoding graph (tbs_graph_create)."""

    def __init__(self, handle, num_states: int, vocab_size: int, max_out_degree: int):
        self._h = handle
        _live.add(self)
        self.num_states, self.vocab_size, self.max_out_degree = num_states, vocab_size, max_out_degree

    @classmethod
    def from_csr(cls, num_states, start, vocab_size, row_ptr, dest, label, score, final=None):
        rp = np.ascontiguousarray(row_ptr, dtype=np.int32)
        de = np.ascontiguousarray(dest, dtype=np.int32)
        la = np.ascontiguousarray(label, dtype=np.int32)
        sc = np.ascontiguousarray(score, dtype=np.float32)
        fi = None if final is None else np.ascontiguousarray(final, dtype=np.float32)
        h = _P()
        _check(lib().tbs_graph_create(int(num_states), int(start), int(vocab_size), _host_ptr(rp),
                                      _host_ptr(de), _host_ptr(la), _host_ptr(sc), _host_ptr(fi),
                                      ctypes.byref(h)))
        deg = int(np.max(np.diff(rp))) if len(rp) > 1 else 0
        return cls(h, int(num_states), int(vocab_size), deg)

    @classmethod
    def trivial(cls, vocab_size: int):
        h = _P()
        _check(lib().tbs_graph_create_trivial(int(vocab_size), ctypes.byref(h)))
        return cls(h, 1, int(vocab_size), int(vocab_size) - 1)

    @classmethod
    def from_synth(cls, g):
        return cls.from_csr(g.num_states, g.start, g.vocab_size, g.row_ptr, g.dest, g.label,
                            g.score, g.final)

    def close(self):
        if self._h is not None and _lib is not None and not _exiting:
            _lib.tbs_graph_destroy(self._h)
        self._h = None

    def __del__(self):
        self.close()


class Model:
    """Stateless decoder + joiner weights on the device (tbs_model_create)."""

    def __init__(self, vocab_size: int, dim: int, embed, conv, w_out, b_out=None,
                 dtype: str = "fp32", stream=None):
        import torch
        self._h = None
        dev = torch.device("cuda", torch.cuda.current_device())

        def dt(x):
            if x is None:
                return None
            if isinstance(x, np.ndarray):
                x = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
            return x.to(device=dev, dtype=torch.float32).contiguous()

        E, cv, W, b = dt(embed), dt(conv), dt(w_out), dt(b_out)
        code = {"fp32": TBS_JOINER_FP32, "bf16": TBS_JOINER_BF16}[dtype]
        h = _P()
        _check(lib().tbs_model_create(int(vocab_size), int(dim), 2, _dev_ptr(E), _dev_ptr(cv),
                                      _dev_ptr(W), _dev_ptr(b), code, _stream_ptr(stream),
                                      ctypes.byref(h)))
        self._h = h
        _live.add(self)
        self.vocab_size, self.dim, self.dtype = int(vocab_size), int(dim), dtype

    def set_schedule(self, schedule: str):
        """Frame-loop schedule for later decodes: "auto", "frame", "stream" (several
        workgroups per stream where possible) or "stream1" (one per stream)."""
        _check(lib().tbs_model_set_schedule(self._h, SCHEDULES[schedule]))

    def set_graph_capture(self, enable: bool):
        """Capture the frame schedule's frame loop in a HIP graph when a decode repeats
        the previous one's launch arguments (default on)."""
        _check(lib().tbs_model_set_graph_capture(self._h, int(bool(enable))))

    def graph_stats(self) -> tuple:
        """(captures, replays) of the frame-loop graph so far."""
        c, r = _I32(), _I32()
        _check(lib().tbs_model_graph_stats(self._h, ctypes.byref(c), ctypes.byref(r)))
        return int(c.value), int(r.value)

    def set_exchange_spin_limit(self, polls: int):
        """Poll budget of the grouped kernel's exchange waits (0 = default); a
        diagnostic for the timeout path."""
        _check(lib().tbs_model_set_exchange_spin_limit(self._h, int(polls)))

    def set_profiling(self, enable: bool):
        _check(lib().tbs_model_set_profiling(self._h, int(bool(enable))))

    def read_profile(self) -> dict:
        """{kernel: (launches, total_ms)} accumulated since profiling was enabled."""
        arr = (KernelTime * len(KERNEL_NAMES))()
        _check(lib().tbs_model_read_profile(self._h, arr))
        return {n: (int(arr[i].launches), float(arr[i].total_ms)) for i, n in enumerate(KERNEL_NAMES)}

    @classmethod
    def from_synth(cls, m, dtype: str = "fp32"):
        return cls(m.vocab_size, m.dim, m.embed, m.conv, m.w_out, m.b_out, dtype=dtype)

    def close(self):
        if self._h is not None and _lib is not None and not _exiting:
            _lib.tbs_model_destroy(self._h)
        self._h = None

    def __del__(self):
        self.close()


@dataclass
class DecodeOutput:
    tokens: "object"      # int32 [B, T] device
    num_tokens: "object"  # int32 [B]
    scores: "object"      # float64 [B]
    status: "object"      # int32 [B] or None
    arcs: "object"        # int32 [B, T] or None
    trace: "object"       # int32 [T+1, B, Ns, 4] or None

    def token_lists(self):
        tok = self.tokens.cpu().numpy()
        n = self.num_tokens.cpu().numpy()
        return [list(tok[b, : n[b]]) for b in range(tok.shape[0])]


def allocate_outputs(B: int, T: int, max_states: int, status=True, arcs=False, trace=False,
                     device=None) -> DecodeOutput:
    import torch
    dev = device or torch.device("cuda", torch.cuda.current_device())
    i32 = dict(dtype=torch.int32, device=dev)
    return DecodeOutput(
        tokens=torch.empty((B, T), **i32), num_tokens=torch.empty(B, **i32),
        scores=torch.empty(B, dtype=torch.float64, device=dev),
        status=torch.empty(B, **i32) if status else None,
        arcs=torch.empty((B, T), **i32) if arcs else None,
        trace=torch.empty((T + 1, B, max_states, 4), **i32) if trace else None)


def _graph_table(graphs, B: int):
    """Host array of B graph handles (kept alive by the caller's list)."""
    graphs = list(graphs)
    if len(graphs) != B:
        raise ValueError(f"need one graph per stream: {len(graphs)} graphs for B = {B}")
    return (_P * max(B, 1))(*[g._h for g in graphs])


def decode_into(model: Model, graph, encoder_out, lengths, beam: float, max_states: int,
                max_contexts: int, out: DecodeOutput, stream=None) -> DecodeOutput:
    """tbs_decode into preallocated outputs (stream-ordered; no synchronisation).
    ``graph`` is one Graph shared by every stream, or a list of B graphs, one per
    stream (tbs_decode_graphs)."""
    lens = np.ascontiguousarray(np.asarray(lengths), dtype=np.int32)
    B, T = int(encoder_out.shape[0]), int(encoder_out.shape[1])
    if encoder_out.dim() != 3 or encoder_out.shape[2] != model.dim:
        raise ValueError("encoder_out must be [B, T, dim]")
    if lens.shape != (B,):
        raise ValueError("lengths must have shape [B]")
    params = BeamParams(float(math.inf if beam is None else beam), int(max_states),
                        int(max_contexts))
    if isinstance(graph, Graph):
        fn, gh = lib().tbs_decode, graph._h
    else:
        fn, gh = lib().tbs_decode_graphs, _graph_table(graph, B)
    _check(fn(model._h, gh, ctypes.byref(params), _dev_ptr(encoder_out),
              _host_ptr(lens), B, T, _dev_ptr(out.tokens), _dev_ptr(out.num_tokens),
              _dev_ptr(out.scores), _dev_ptr(out.status), _dev_ptr(out.arcs),
              _dev_ptr(out.trace), _stream_ptr(stream)))
    return out


def decode_noalloc_into(model: Model, graph: Graph, encoder_out, lengths_dev, beam: float,
                        max_states: int, max_contexts: int, out: DecodeOutput,
                        stream=None) -> DecodeOutput:
    """tbs_decode_noalloc: tbs_decode with its workspace in the library's fixed device
    array (no allocation); ``lengths_dev`` is a device int32 tensor [B]."""
    B, T = int(encoder_out.shape[0]), int(encoder_out.shape[1])
    if encoder_out.dim() != 3 or encoder_out.shape[2] != model.dim:
        raise ValueError("encoder_out must be [B, T, dim]")
    if tuple(lengths_dev.shape) != (B,) or str(lengths_dev.dtype) != "torch.int32":
        raise ValueError("lengths_dev must be a device int32 tensor of shape [B]")
    params = BeamParams(float(math.inf if beam is None else beam), int(max_states),
                        int(max_contexts))
    _check(lib().tbs_decode_noalloc(model._h, graph._h, ctypes.byref(params),
                                    _dev_ptr(encoder_out), _dev_ptr(lengths_dev), B, T,
                                    _dev_ptr(out.tokens), _dev_ptr(out.num_tokens),
                                    _dev_ptr(out.scores), _dev_ptr(out.status),
                                    _dev_ptr(out.arcs), _dev_ptr(out.trace), _stream_ptr(stream)))
    return out


def decode(model: Model, graph, encoder_out, lengths, beam: float = math.inf,
           max_states: int = 4, max_contexts: int = 4, want_arcs: bool = False,
           want_trace: bool = False, stream=None) -> DecodeOutput:
    """Batched FSA-constrained one-symbol-per-frame beam search; outputs on the device.
    ``graph``: one Graph for every stream, or a list of one Graph per stream."""
    B, T = int(encoder_out.shape[0]), int(encoder_out.shape[1])
    out = allocate_outputs(B, T, max_states, status=True, arcs=want_arcs, trace=want_trace,
                           device=encoder_out.device)
    return decode_into(model, graph, encoder_out, lengths, beam, max_states, max_contexts, out,
                       stream)


def joiner_logp(model: Model, enc_rows, ctx, stream=None):
    """log P(. | ctx, enc row) [R, V] from the HIP joiner (tbs_joiner_logp)."""
    import torch
    R = int(enc_rows.shape[0])
    out = torch.empty((R, model.vocab_size), dtype=torch.float32, device=enc_rows.device)
    ctx = ctx.to(device=enc_rows.device, dtype=torch.int32).contiguous()
    _check(lib().tbs_joiner_logp(model._h, _dev_ptr(enc_rows.contiguous()), _dev_ptr(ctx), R,
                                 _dev_ptr(out), _stream_ptr(stream)))
    return out


class DecodeState:
    """Streaming decode (tbs_state_create / tbs_decode_chunk / tbs_state_finish):
    each chunk continues every stream from where it stopped; finish traces the best
    paths back over all decoded frames."""

    def __init__(self, model: Model, graph, B: int, max_frames: int,
                 beam: float = math.inf, max_states: int = 4, max_contexts: int = 4,
                 stream=None):
        """``graph``: one Graph for every stream, or a list of one Graph per stream."""
        self._h = None
        params = BeamParams(float(math.inf if beam is None else beam), int(max_states),
                            int(max_contexts))
        h = _P()
        if isinstance(graph, Graph):
            fn, gh = lib().tbs_state_create, graph._h
        else:
            graph = list(graph)
            fn, gh = lib().tbs_state_create_graphs, _graph_table(graph, int(B))
        _check(fn(model._h, gh, ctypes.byref(params), int(B), int(max_frames),
                  _stream_ptr(stream), ctypes.byref(h)))
        self._h = h
        _live.add(self)
        self._refs = (model, graph)  # the state must not outlive them
        self.B, self.max_frames, self.max_states = int(B), int(max_frames), int(max_states)

    def chunk(self, encoder_chunk, lengths, trace=None, stream=None):
        """Decode the next frames: encoder_chunk [B, Tc, C] on the device, lengths [B]
        frames per stream (host); trace: optional [max_frames+1, B, Ns, 4] int32 buffer."""
        lens = np.ascontiguousarray(np.asarray(lengths), dtype=np.int32)
        B, Tc = int(encoder_chunk.shape[0]), int(encoder_chunk.shape[1])
        if B != self.B or lens.shape != (B,):
            raise ValueError("encoder_chunk / lengths do not match the state's batch")
        _check(lib().tbs_decode_chunk(self._h, _dev_ptr(encoder_chunk.contiguous()),
                                      _host_ptr(lens), Tc, _dev_ptr(trace), _stream_ptr(stream)))

    def finish(self, want_arcs: bool = False, stream=None) -> DecodeOutput:
        out = allocate_outputs(self.B, self.max_frames, self.max_states, status=True,
                               arcs=want_arcs)
        _check(lib().tbs_state_finish(self._h, _dev_ptr(out.tokens), _dev_ptr(out.num_tokens),
                                      _dev_ptr(out.scores), _dev_ptr(out.status),
                                      _dev_ptr(out.arcs), _stream_ptr(stream)))
        return out

    def close(self):
        if self._h is not None and _lib is not None and not _exiting:
            _lib.tbs_state_destroy(self._h)
        self._h = None

    def __del__(self):
        self.close()


@dataclass
class NBestOutput:
    tokens: "object"         # int32 [B, T] device: the best label sequence, -1 padded
    num_tokens: "object"     # int32 [B]
    scores: "object"         # float64 [B]: its total log probability in the lattice
    num_unique: "object"     # int32 [B]: distinct sequences among the sampled paths
    unique_scores: "object"  # float64 [B, n]
    unique_first: "object"   # int32 [B, n]: the path that first gave each sequence
    paths: "object"          # int32 [B, n, T+1] or None

    def token_lists(self):
        tok = self.tokens.cpu().numpy()
        n = self.num_tokens.cpu().numpy()
        return [list(tok[b, : n[b]]) for b in range(tok.shape[0])]


class Lattice:
    """The search's lattice (tbs_lattice_create) and the n-best label-sequence search on it
    (tbs_lattice_nbest).  ``graph``: one Graph, or a list of one Graph per stream."""

    def __init__(self, model: Model, graph, encoder_out, lengths, beam: float = math.inf,
                 max_states: int = 4, max_contexts: int = 4, stream=None):
        self._h = None
        lens = np.ascontiguousarray(np.asarray(lengths), dtype=np.int32)
        B, T = int(encoder_out.shape[0]), int(encoder_out.shape[1])
        if encoder_out.dim() != 3 or encoder_out.shape[2] != model.dim:
            raise ValueError("encoder_out must be [B, T, dim]")
        if lens.shape != (B,):
            raise ValueError("lengths must have shape [B]")
        params = BeamParams(float(math.inf if beam is None else beam), int(max_states),
                            int(max_contexts))
        h = _P()
        if isinstance(graph, Graph):
            fn, gh = lib().tbs_lattice_create, graph._h
        else:
            graph = list(graph)
            fn, gh = lib().tbs_lattice_create_graphs, _graph_table(graph, B)
        _check(fn(model._h, gh, ctypes.byref(params), _dev_ptr(encoder_out.contiguous()),
                  _host_ptr(lens), B, T, _stream_ptr(stream), ctypes.byref(h)))
        self._h = h
        _live.add(self)
        self._refs = (model, graph)
        self.device = encoder_out.device
        self.B, self.T, self.max_states = B, T, int(max_states)
        self.lengths = lens

    def num_arcs(self) -> int:
        n = ctypes.c_int64(0)
        _check(lib().tbs_lattice_num_arcs(self._h, ctypes.byref(n)))
        return int(n.value)

    def export(self, stream=None) -> dict:
        """Device tensors: frame_off [B*T+1], arcs [A, 4] (src, dst, label, graph arc),
        weights [A], nodes [T+1, B, Ns, 4], alpha [B, T+1, Ns], final_w [B, Ns], total [B],
        status [B]."""
        import torch
        A, B, T, Ns, dev = self.num_arcs(), self.B, self.T, self.max_states, self.device
        out = {"frame_off": torch.empty(B * T + 1, dtype=torch.int64, device=dev),
               "arcs": torch.empty((A, 4), dtype=torch.int32, device=dev),
               "weights": torch.empty(A, dtype=torch.float32, device=dev),
               "nodes": torch.empty((T + 1, B, Ns, 4), dtype=torch.int32, device=dev),
               "alpha": torch.empty((B, T + 1, Ns), dtype=torch.float64, device=dev),
               "final_w": torch.empty((B, Ns), dtype=torch.float64, device=dev),
               "total": torch.empty(B, dtype=torch.float64, device=dev),
               "status": torch.empty(B, dtype=torch.int32, device=dev)}
        _check(lib().tbs_lattice_export(self._h, *[_dev_ptr(out[k]) for k in (
            "frame_off", "arcs", "weights", "nodes", "alpha", "final_w", "total", "status")],
            _stream_ptr(stream)))
        return out

    def nbest(self, num_paths: int, uniforms, want_paths: bool = False,
              stream=None) -> NBestOutput:
        """n-best label-sequence search; uniforms: float64 [B, num_paths, T+1] on the
        device, each in [0, 1)."""
        import torch
        B, T, n, dev = self.B, self.T, int(num_paths), self.device
        if tuple(uniforms.shape) != (B, n, T + 1) or uniforms.dtype != torch.float64:
            raise ValueError(f"uniforms must be float64 [{B}, {n}, {T + 1}]")
        i32 = dict(dtype=torch.int32, device=dev)
        out = NBestOutput(tokens=torch.empty((B, T), **i32), num_tokens=torch.empty(B, **i32),
                          scores=torch.empty(B, dtype=torch.float64, device=dev),
                          num_unique=torch.empty(B, **i32),
                          unique_scores=torch.empty((B, n), dtype=torch.float64, device=dev),
                          unique_first=torch.empty((B, n), **i32),
                          paths=torch.empty((B, n, T + 1), **i32) if want_paths else None)
        _check(lib().tbs_lattice_nbest(self._h, n, _dev_ptr(uniforms.contiguous()),
                                       _dev_ptr(out.tokens), _dev_ptr(out.num_tokens),
                                       _dev_ptr(out.scores), _dev_ptr(out.num_unique),
                                       _dev_ptr(out.unique_scores), _dev_ptr(out.unique_first),
                                       _dev_ptr(out.paths), _stream_ptr(stream)))
        return out

    def close(self):
        if self._h is not None and _lib is not None and not _exiting:
            _lib.tbs_lattice_destroy(self._h)
        self._h = None

    def __del__(self):
        self.close()


class HypParams(ctypes.Structure):
    _fields_ = [("beam_size", _I32), ("merge", _I32)]


MERGES = {"max": 0, "logadd": 1}


def hyp_search(model: Model, encoder_out, lengths, beam_size: int = 4, merge: str = "logadd",
               want_trace: bool = False, stream=None) -> DecodeOutput:
    """Full-sequence beam search with max-symbols 1 (tbs_hyp_search, Table 5's comparison
    search); outputs on the device; trace [T+1, B, beam_size, 2] (parent rank, label)."""
    import torch
    lens = np.ascontiguousarray(np.asarray(lengths), dtype=np.int32)
    B, T = int(encoder_out.shape[0]), int(encoder_out.shape[1])
    if encoder_out.dim() != 3 or encoder_out.shape[2] != model.dim:
        raise ValueError("encoder_out must be [B, T, dim]")
    if lens.shape != (B,):
        raise ValueError("lengths must have shape [B]")
    dev = encoder_out.device
    i32 = dict(dtype=torch.int32, device=dev)
    out = DecodeOutput(tokens=torch.empty((B, T), **i32), num_tokens=torch.empty(B, **i32),
                       scores=torch.empty(B, dtype=torch.float64, device=dev), status=None,
                       arcs=None,
                       trace=torch.empty((T + 1, B, int(beam_size), 2), **i32) if want_trace
                       else None)
    params = HypParams(int(beam_size), MERGES[merge])
    _check(lib().tbs_hyp_search(model._h, ctypes.byref(params),
                                _dev_ptr(encoder_out.contiguous()), _host_ptr(lens), B, T,
                                _dev_ptr(out.tokens), _dev_ptr(out.num_tokens),
                                _dev_ptr(out.scores), _dev_ptr(out.trace), _stream_ptr(stream)))
    return out


TRANSDUCER_KINDS = {"standard": 0, "modified": 1, "constrained": 2}


def transducer_forward(kind: str, blank, label, lengths, want_alpha: bool = False,
                       stream=None):
    """Forward recursion of the standard (eq. 1), modified (eq. 2) or constrained (eq. 3)
    transducer (tbs_transducer_forward).  blank [B, T, U+1] and label [B, T, U] float32 on
    the device; lengths [B, 2] int32 (frames, labels).  Returns (total [B] float64,
    alpha [B, T+1, U+1] float32 or None, status [B] int32)."""
    import torch
    B, T, U1 = (int(x) for x in blank.shape)
    U = U1 - 1
    if tuple(label.shape) != (B, T, U):
        raise ValueError("label must be [B, T, U]")
    dev = blank.device
    lengths = torch.as_tensor(lengths, dtype=torch.int32).reshape(B, 2).to(dev).contiguous()
    total = torch.empty(B, dtype=torch.float64, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    alpha = torch.empty((B, T + 1, U1), dtype=torch.float32, device=dev) if want_alpha else None
    _check(lib().tbs_transducer_forward(TRANSDUCER_KINDS[kind], _dev_ptr(blank.contiguous()),
                                        _dev_ptr(label.contiguous()) if U > 0 else None,
                                        _dev_ptr(lengths), B, T, U, _dev_ptr(total),
                                        _dev_ptr(alpha), _dev_ptr(status), _stream_ptr(stream)))
    return total, alpha, status
