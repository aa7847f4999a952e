"""Shared helpers of the GPU parity tests (no model arithmetic here)."""
import json
import os

import numpy as np

GRAPH_KEYS = ("edge_ptr", "edge_dst", "edge_img", "edge_rev", "bond_ptr", "bond_edge", "angle_ptr", "angle_b2")
ATOL, RTOL = 1e-5, 1e-4


def assert_close(got, ref, what=""):
    """|gpu - ref| <= 1e-5 + 1e-4 |ref| elementwise (ref from the fp64 oracle)."""
    got = np.asarray(got, dtype=np.float64).reshape(-1)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    err = np.abs(got - ref)
    bad = err > ATOL + RTOL * np.abs(ref)
    if bad.any():
        k = int(np.argmax(err - (ATOL + RTOL * np.abs(ref))))
        raise AssertionError("%s: %d/%d outside tolerance; worst at %d: gpu %.9g ref %.9g"
                             % (what, int(bad.sum()), bad.size, k, got[k], ref[k]))


def assert_graph_equal(gpu, ref):
    for k in GRAPH_KEYS:
        a = np.asarray(gpu[k])
        b = np.asarray(ref[k])
        assert a.size == b.size, (k, a.size, b.size)
        assert np.array_equal(a.reshape(b.shape), b), k


def subset_batch(batch, structs):
    """Batch made of the listed structures of `batch` (same fp32 data)."""
    from paper_2412_20796_amd.synth import Batch

    ptr = [0]
    pos, lat, Z = [], [], []
    for s in structs:
        a0, a1 = batch.atom_ptr[s], batch.atom_ptr[s + 1]
        pos.append(batch.pos[a0:a1])
        Z.append(batch.Z[a0:a1])
        lat.append(batch.lattice[s])
        ptr.append(ptr[-1] + a1 - a0)
    return Batch(np.asarray(ptr, np.int32), np.concatenate(pos), np.stack(lat), np.concatenate(Z))


def golden_reverse_pair_cell():
    """The two-atom cell of tests/golden/reverse_pair_cell.json as a batch."""
    from paper_2412_20796_amd.synth import Batch

    with open(os.path.join(os.path.dirname(__file__), "golden", "reverse_pair_cell.json")) as f:
        c = json.load(f)
    L = (np.eye(3, dtype=np.float32) * np.float32(c["lattice_a"]))[None]
    return Batch(np.array([0, 2], np.int32), np.asarray(c["pos"], np.float32), L, np.array([8, 25], np.int32)), c
