"""C-ABI checks that need no GPU: the library loads, exports every function declared in
include/tbs.h, and rejects invalid arguments on the host before any device work."""
import ctypes
import math
import os
import subprocess

import numpy as np
import pytest

from paper_2211_00484_amd import tbs

EINVAL, EUNSUPPORTED = -1, -5


def test_library_exports_every_declared_symbol():
    L = tbs.lib()
    names = tbs.declared_symbols()
    assert "tbs_decode" in names and "tbs_graph_create" in names
    for n in names:
        assert hasattr(L, n), f"{n} is declared in tbs.h but not exported"
    out = subprocess.run(["nm", "-D", "--defined-only", tbs.LIB_PATH], capture_output=True, text=True)
    exported = {line.split()[-1] for line in out.stdout.splitlines() if " T " in line}
    assert set(names) <= exported


def _graph(S, start, V, rp, dest, label, score, final=None):
    L = tbs.lib()
    h = ctypes.c_void_p()
    arr = lambda a, t: None if a is None else np.ascontiguousarray(a, dtype=t)
    rp, dest, label, score, final = (arr(rp, np.int32), arr(dest, np.int32), arr(label, np.int32),
                                     arr(score, np.float32), arr(final, np.float32))
    p = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p)
    st = L.tbs_graph_create(S, start, V, p(rp), p(dest), p(label), p(score), p(final),
                            ctypes.byref(h))
    return st, L.tbs_last_error().decode(), h


@pytest.mark.parametrize("case,fragment", [
    (dict(S=0), "num_states"),
    (dict(start=3), "start_state"),
    (dict(V=1), "vocab_size"),
    (dict(V=70000), "vocab_size"),
    (dict(V=46341), "vocab_size"),   # contexts a * V + b would overflow int32
    (dict(rp=[1, 2, 3]), "row_ptr[0]"),
    (dict(rp=[0, 2, 1]), "decreases"),
    (dict(dest=[0, 2]), "dest[1]"),
    (dict(label=[0, 1]), "label[0]"),
    (dict(label=[1, 5]), "label[1]"),
    (dict(score=[0.0, math.nan]), "score[1]"),
    (dict(score=[math.inf, 0.0]), "score[0]"),
    (dict(final=[0.0, math.inf]), "final_score[1]"),
])
def test_graph_validation(case, fragment):
    args = dict(S=2, start=0, V=5, rp=[0, 1, 2], dest=[1, 0], label=[1, 2], score=[0.0, -1.0],
                final=None)
    args.update(case)
    st, msg, h = _graph(args["S"], args["start"], args["V"], args["rp"], args["dest"],
                        args["label"], args["score"], args["final"])
    assert st == EINVAL, msg
    assert fragment in msg
    assert not h.value


def test_model_validation_before_device_work():
    L = tbs.lib()
    h = ctypes.c_void_p()
    assert L.tbs_model_create(10, 8, 3, None, None, None, None, 0, None, ctypes.byref(h)) == EUNSUPPORTED
    assert L.tbs_model_create(10, 0, 2, None, None, None, None, 0, None, ctypes.byref(h)) == EINVAL
    assert L.tbs_model_create(10, 8, 2, None, None, None, None, 0, None, ctypes.byref(h)) == EINVAL
    assert "NULL" in L.tbs_last_error().decode()
    # contexts a * V + b are int32: V = 46,341 would overflow, 46,340 is the limit
    assert L.tbs_model_create(46341, 8, 2, None, None, None, None, 0, None, ctypes.byref(h)) == EINVAL
    assert "vocab_size" in L.tbs_last_error().decode()
    assert L.tbs_graph_create_trivial(46341, ctypes.byref(h)) == EINVAL
    assert L.tbs_model_create(46340, 8, 2, None, None, None, None, 0, None, ctypes.byref(h)) == EINVAL
    assert "NULL" in L.tbs_last_error().decode()


def test_decode_null_handles():
    L = tbs.lib()
    p = tbs.BeamParams(1.0, 4, 4)
    st = L.tbs_decode(None, None, ctypes.byref(p), None, None, 1, 1, None, None, None, None,
                      None, None, None)
    assert st == EINVAL
    assert L.tbs_joiner_logp(None, None, None, 1, None, None) == EINVAL
    st = L.tbs_decode_graphs(None, None, ctypes.byref(p), None, None, 1, 1, None, None, None,
                             None, None, None, None)
    assert st == EINVAL and "graphs is NULL" in L.tbs_last_error().decode()
    h = ctypes.c_void_p()
    assert L.tbs_state_create_graphs(None, None, ctypes.byref(p), 1, 1, None,
                                     ctypes.byref(h)) == EINVAL
    assert h.value is None
    assert L.tbs_transducer_forward(7, None, None, None, 1, 1, 1, None, None, None,
                                    None) == EINVAL
    assert L.tbs_transducer_forward(0, None, None, None, 1, 1, 1024, None, None, None,
                                    None) == -4
    hp = tbs.HypParams(4, 1)
    assert L.tbs_hyp_search(None, ctypes.byref(hp), None, None, 1, 1, None, None, None, None,
                            None) == EINVAL


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(tbs, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(tbs, "_lib", None)
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        tbs.lib()


def test_header_is_c_compatible(tmp_path):
    src = tmp_path / "t.c"
    src.write_text('#include "tbs.h"\nint main(void) { return TBS_OK; }\n')
    inc = os.path.join(os.path.dirname(tbs.HEADER_PATH))
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", inc, str(src), "-o",
                    str(tmp_path / "t")], check=True)
