"""Write the offline GSP/RCR tables and the App. C.1 thresholds of a workload.

    python tests/golden/make_tables.py prefill_4096 [zipf_256 ...]
    python tests/golden/make_tables.py stack_48      (tables of every layer; no tau)

Calls only the seeded generators (synth) and the CPU oracle: GSP by Alg. 2,
RCR by Alg. 3 (fp64, rounded once to fp32), and tau_q by the App. C.1 mapping
over one score pass of the workload's own prefill input (m_min = 1).  The GPU
tests and the benchmark read these files as inputs.
"""
from __future__ import annotations

import dataclasses
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import synth  # noqa: E402

QS = (0.1, 0.25, 0.5, 0.6)


def table_path(name: str, seed: int = 0) -> str:
    return os.path.join(HERE, f"tables_{name}_seed{seed}.json")


def make(name: str, seed: int = 0) -> dict:
    cfg = synth.config(name, seed=seed)
    t0 = time.time()
    L = synth.make_layer(cfg)
    t1 = time.time()
    tb = oracle.tables.build_tables(L)
    t2 = time.time()
    a_gsp, a_rcr = tb["a_gsp"], tb["a_rcr"]
    base = oracle.forward.moe_forward(L, cfg.k, a_gsp, a_rcr, tau=0.0, tokens=[])
    taus = oracle.tau.tau_table([base["c"]], 1, QS)
    t3 = time.time()
    out = {
        "config": dataclasses.asdict(cfg),
        "source": "oracle: Alg. 2 (GSP) and Alg. 3 (RCR) in fp64 rounded to fp32; tau by the "
                  "App. C.1 mapping over the c of every routed slot of this workload (m_min = 1)",
        "command": f"python tests/golden/make_tables.py {name}",
        "eps": 1e-6,
        "a_gsp": [float(v) for v in a_gsp],
        "a_rcr": [float(v) for v in a_rcr],
        "tau": {str(q): float(t) for q, t in taus.items()},
        "tau_f32": {str(q): float(np.float32(t)) for q, t in taus.items()},
        "seconds": {"generate": round(t1 - t0, 2), "tables": round(t2 - t1, 2),
                    "tau": round(t3 - t2, 2)},
    }
    with open(table_path(name, seed), "w") as f:
        json.dump(out, f, indent=1)
    return out


def make_stack(name: str = "stack_48", seed: int = 0) -> dict:
    """GSP/RCR tables of every layer of the stack (the threshold of a stack comes
    from its own score pass through the residual chain, so none is stored)."""
    cfg = synth.config(name, seed=seed)
    t0 = time.time()
    layers = []
    for li in range(synth.STACK_LAYERS):
        L = synth.make_layer(cfg.with_(T=16), layer=li)   # weights only matter here
        tb = oracle.tables.build_tables(L)
        layers.append({"a_gsp": [float(v) for v in tb["a_gsp"]], "a_rcr": [float(v) for v in tb["a_rcr"]]})
        print(f"layer {li} done at {time.time() - t0:.0f}s", flush=True)
    out = {"config": dataclasses.asdict(cfg), "layers_count": synth.STACK_LAYERS,
           "source": "oracle: Alg. 2 (GSP) and Alg. 3 (RCR) per layer in fp64 rounded to fp32; "
                     "layer l's weights are synth.make_layer(config, layer=l)",
           "command": f"python tests/golden/make_tables.py {name}", "eps": 1e-6, "layers": layers,
           "seconds": round(time.time() - t0, 1)}
    with open(table_path(name, seed), "w") as f:
        json.dump(out, f)
    return out


def load(name: str, seed: int = 0) -> dict:
    with open(table_path(name, seed)) as f:
        return json.load(f)


if __name__ == "__main__":
    for n in sys.argv[1:] or ["prefill_4096"]:
        if n.startswith("stack"):
            r = make_stack(n)
            print(n, r["seconds"])
            continue
        r = make(n)
        print(n, r["tau"], r["seconds"])
