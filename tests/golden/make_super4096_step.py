"""Writes super4096_step.npz: the oracle's full training step (loss, energy,
forces, stress and the gradient of every parameter) on the 4096-atom
supercell workload (cubic a = 36.39 A, density 0.085, d = 64, T = 4), with
the seeded weights and targets of that workload. Calls only the oracle and
the seeded input generators; takes several minutes and ~16 GB of memory.

    python tests/golden/make_super4096_step.py
"""
import hashlib
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import graph as og  # noqa: E402
from oracle import model as om  # noqa: E402
from paper_2412_20796_amd import synth  # noqa: E402


def input_digest(b, params, targets):
    h = hashlib.sha256()
    for a in (b.atom_ptr, b.pos, b.lattice, b.Z, params, *targets):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def main():
    b, params, targets, d, T = synth.workload_inputs("super4096")
    graph = og.build_graph(b.atom_ptr, b.pos, b.lattice)
    loss, grad, (E, F, S), _ = om.step(om.HParams(d=d, n_layers=T), b, params.astype(np.float64), targets, graph=graph)
    np.savez_compressed(os.path.join(HERE, "super4096_step.npz"), loss=np.float64(loss), energy=E, forces=F.astype(np.float32),
                        stress=S, grad=grad.astype(np.float32), n_edges=len(graph["edge_dst"]),
                        inputs_sha256=input_digest(b, params, targets))


if __name__ == "__main__":
    main()
