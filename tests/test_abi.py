"""The C-ABI library loads and exports every entry point of include/chgnet.h;
host-side argument checks (no GPU compute)."""
import ctypes
import os
import re

import pytest

from oracle import model as om

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "chgnet.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(chgnet_\w+)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def L():
    from paper_2412_20796_amd import binding

    if not os.path.exists(binding._LIB_PATH):
        pytest.fail("libchgnet.so not built; run __graft_entry__.build()")
    return binding


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert len(names) == 11
    lib = ctypes.CDLL(L._LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.EXPORTED)


def test_param_count_matches_oracle_layout(L):
    for d, T in ((64, 4), (128, 5), (64, 1), (128, 2)):
        assert L.param_count(L.hparams(d=d, n_layers=T)) == om.param_count(om.HParams(d=d, n_layers=T))
    assert L.param_count(L.hparams(d=64, n_layers=4)) == 405_001
    for d, T in ((64, 4), (128, 3)):
        ohp = om.HParams(d=d, n_layers=T, magmom=True)
        assert L.param_count(L.hparams(d=d, n_layers=T, magmom=True)) == om.param_count(ohp)
        assert L.param_count(L.hparams(d=d, n_layers=T, sequential=True)) == om.param_count(om.HParams(d=d, n_layers=T))


def test_workspace_size_monotone(L):
    hp = L.hparams()
    a = L.workspace_size(hp, 100, 1000, 100, 1000, 2)
    b = L.workspace_size(hp, 100, 2000, 100, 1000, 2)
    g = L.workspace_size(hp, 100, 0, 0, 0, 2)
    assert 0 < g < a < b


def test_workspace_holds_the_dual_number_buffers(L):
    """With the conservative readout the workspace also holds the buffers of
    the dual-number weight gradient: at least the value and tangent
    pre-activations of every gate of every layer, T x 2 x (E + 2A) x 2d
    floats, beyond the direct-head size."""
    N, E, B, A, S = 100, 1000, 100, 1000, 2
    base = L.workspace_size(L.hparams(), N, E, B, A, S)
    cons = L.workspace_size(L.hparams(conservative=True), N, E, B, A, S)
    assert cons - base >= 4 * 2 * (E + 2 * A) * 128 * 4


@pytest.mark.parametrize("kw", [dict(d=32), dict(d=96), dict(n_layers=0), dict(n_layers=17), dict(n_fourier=30),
                                dict(n_rbf=0), dict(n_rbf=65), dict(r_bond=7.0), dict(r_atom=25.0, r_bond=3.0),
                                dict(envelope_p=1), dict(magmom=2), dict(sequential=-1),
                                dict(conservative=3)])
def test_bad_hparams_rejected(L, kw):
    with pytest.raises(L.ChgnetError) as e:
        L.param_count(L.hparams(**kw))
    assert e.value.code == L.CHGNET_EINVAL


def test_null_arguments_rejected(L):
    hp = L.hparams()
    lib = L.lib()
    assert lib.chgnet_param_count(ctypes.byref(hp), None) == L.CHGNET_EINVAL
    assert lib.chgnet_build_graph(ctypes.byref(hp), None, None, None, 0, None) == L.CHGNET_EINVAL
    assert b"batch" in lib.chgnet_last_error_string()
    done = ctypes.c_int(7)
    assert lib.chgnet_md(ctypes.byref(hp), None, None, None, None, 1.0, 1, 0, ctypes.byref(done), None, 0,
                         None) == L.CHGNET_EINVAL
    assert done.value == 0
