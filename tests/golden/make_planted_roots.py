"""Writes planted_roots.json: for each planted-acceptance workload, a root
token whose token-by-token greedy continuation (the oracle's argmax decoding,
Sec. 2) has a top-1 minus top-2 logit margin of at least 2 tol at every step,
so a block of drafts taken from that continuation has only decisive accept
decisions. Calls only the oracle and the seeded input generator.

    python tests/golden/make_planted_roots.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle as orc  # noqa: E402
from paper_2510_13161_amd import synth  # noqa: E402

TOL = 2e-2
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "planted_roots.json")

# name -> (workload, layers, greedy steps whose margins must be decisive)
CASES = {
    "tiny_chain": (synth.WORKLOADS["tiny_chain"], None, 5),
    "14b_chain_l2": (synth.WORKLOADS["14b_chain"], 2, 9),
}


def margins(zs):
    s = np.sort(zs, axis=-1)
    return s[:, -1] - s[:, -2]


def search(w, layers, steps, tries=64):
    shape = w.model if layers is None else w.model.with_layers(layers)
    o = orc.Oracle(shape, synth.host_weights(shape, w.seed))
    L = int(w.ctx[0])
    ctx_cache = {l: (synth.host_ctx(shape, w.seed, l, "k", 0, L), synth.host_ctx(shape, w.seed, l, "v", 0, L))
                 for l in range(shape.n_layers)}
    roots = synth.rng(w.seed, "planted_root").integers(0, shape.vocab, size=tries)
    for i, root in enumerate(roots):
        y, zs = o.decode_greedy(int(root), L, steps, lambda l: ctx_cache[l], L)
        m = margins(zs)
        print(f"  root {int(root)}: min margin {m.min():.4f}", flush=True)
        if m.min() >= 2 * TOL:
            return {"root": int(root), "try": i, "steps": steps, "ctx": L, "layers": shape.n_layers,
                    "seed": w.seed, "min_margin": float(m.min()), "tokens": [int(t) for t in y]}
    raise RuntimeError("no root with decisive margins")


def main():
    out = {"tol_logit": TOL}
    for name, (w, layers, steps) in CASES.items():
        print(name, flush=True)
        out[name] = search(w, layers, steps)
    with open(OUT, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print("wrote", OUT)


if __name__ == "__main__":
    main()
