"""chgnet_build_graph_noalloc (static device scratch, no workspace) against
chgnet_build_graph with a workspace: identical graph arrays on two calls in a
row, the second with a smaller batch, and a batch beyond the static scratch
refused with CHGNET_EINVAL."""
import numpy as np
import pytest

from gpu_helpers import assert_graph_equal
from paper_2412_20796_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def bd():
    import torch

    from paper_2412_20796_amd import binding

    assert torch.cuda.is_available()
    binding.lib()
    return binding


def _both(bd, b):
    hp = bd.hparams()
    db = bd.DeviceBatch.from_host(b)
    g_ws = bd.DeviceGraph(b.n_atoms, 64, 16, 64)
    bd.build_graph(hp, db, g_ws, bd.Workspace())
    g_na = bd.DeviceGraph(b.n_atoms, 64, 16, 64)
    counts = bd.build_graph_noalloc(hp, db, g_na)
    return g_ws, g_na, counts


def test_noalloc_graph_matches_workspace_graph(bd):
    for name in ("heavytail64", "cubic8"):  # the second call is smaller
        b = synth.make_batch(name)
        g_ws, g_na, counts = _both(bd, b)
        assert counts == (g_ws.n_edges, g_ws.n_bonds, g_ws.n_angles), name
        assert_graph_equal(g_na.host(), g_ws.host())
        print(name, counts, flush=True)


def test_noalloc_graph_boundary_cells_and_limit(bd):
    b = synth.boundary_batch("atom")
    g_ws, g_na, _ = _both(bd, b)
    assert_graph_equal(g_na.host(), g_ws.host())
    # a batch needing more than the static scratch (64 bytes per atom) is
    # refused before any launch
    n = 140_000
    big = synth.Batch(np.array([0, n], np.int32), np.zeros((n, 3), np.float32),
                      (np.eye(3, dtype=np.float32) * 100.0)[None], np.ones(n, np.int32))
    hp = bd.hparams()
    db = bd.DeviceBatch.from_host(big)
    with pytest.raises(bd.ChgnetError) as e:
        bd.build_graph_noalloc(hp, db, bd.DeviceGraph(n, 64, 16, 64))
    assert e.value.code == bd.CHGNET_EINVAL and "static" in str(e.value)
