"""Writes oracle regression fixtures (calls only the oracle and the input generators).

Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import math
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2211_00484_amd import synth  # noqa: E402

CASES = {
    # Tiny workload: B=2, T=20, C=32, V=16, trivial graph, max_states = max_contexts = 4.
    "tiny_seed0": dict(workload="tiny", seed=0, beam=math.inf, Ns=4, Nc=4, bf16=False),
    "tiny_seed0_bf16": dict(workload="tiny", seed=0, beam=math.inf, Ns=4, Nc=4, bf16=True),
    "tiny_seed3_beam1": dict(workload="tiny", seed=3, beam=1.0, Ns=6, Nc=3, bf16=False),
}


def run_case(c):
    w, inputs, model, graph = synth.make_workload(c["workload"], seed=c["seed"])
    res = oracle.decode(model, graph, inputs.encoder_out, inputs.lengths, c["beam"], c["Ns"],
                        c["Nc"], bf16=c["bf16"])
    return {"tokens": [[int(x) for x in tl] for tl in res.token_lists()], "scores": [float(s) for s in res.scores],
            "status": [int(s) for s in res.status], "trace": res.trace.tolist()}


def main():
    out = {}
    for name, c in CASES.items():
        d = dict(c)
        d["beam"] = "inf" if math.isinf(c["beam"]) else c["beam"]
        out[name] = {"params": d, "result": run_case(c)}
    with open(os.path.join(HERE, "oracle_tiny.json"), "w") as f:
        json.dump(out, f, separators=(",", ":"))


if __name__ == "__main__":
    main()
