"""Thin ctypes binding of libchgnet.so (the C interface in include/chgnet.h).

Argument marshalling only: torch tensors supply device memory and the HIP
stream; every step of the computation runs in the library's HIP kernels. The
library must be built (``python -m paper_2412_20796_amd.build_lib``); without
it every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libchgnet.so")
_lib = None

CHGNET_OK, CHGNET_EINVAL, CHGNET_ECAPACITY, CHGNET_EWORKSPACE, CHGNET_EHIP = 0, -1, -2, -3, -4
EXPORTED = ("chgnet_param_count", "chgnet_workspace_size", "chgnet_build_graph", "chgnet_build_graph_noalloc",
            "chgnet_forward",
            "chgnet_backward", "chgnet_step", "chgnet_md", "chgnet_last_error_string", "chgnet_profile_start",
            "chgnet_profile_stop")


class ChgnetError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("chgnet error %d: %s" % (code, msg))
        self.code = code


class HParams(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("n_rbf", ctypes.c_int32),
                ("n_fourier", ctypes.c_int32), ("envelope_p", ctypes.c_int32), ("r_atom", ctypes.c_float),
                ("r_bond", ctypes.c_float), ("magmom", ctypes.c_int32), ("sequential", ctypes.c_int32),
                ("conservative", ctypes.c_int32)]


class LossCfg(ctypes.Structure):
    _fields_ = [("w_energy", ctypes.c_float), ("w_force", ctypes.c_float), ("w_stress", ctypes.c_float),
                ("w_magmom", ctypes.c_float), ("huber_delta", ctypes.c_float)]


class MdState(ctypes.Structure):
    _fields_ = [("pos", ctypes.c_void_p), ("vel", ctypes.c_void_p), ("inv_mass", ctypes.c_void_p),
                ("forces", ctypes.c_void_p), ("energy", ctypes.c_void_p), ("stress", ctypes.c_void_p),
                ("skin", ctypes.c_float), ("cap_cand", ctypes.c_int64), ("n_cand", ctypes.c_int64),
                ("cand_ptr", ctypes.c_void_p), ("cand_dst", ctypes.c_void_p), ("cand_img", ctypes.c_void_p),
                ("ref_pos", ctypes.c_void_p), ("n_builds", ctypes.c_int32)]


class CBatch(ctypes.Structure):
    _fields_ = [("n_struct", ctypes.c_int32), ("n_atoms", ctypes.c_int32), ("atom_ptr", ctypes.c_void_p),
                ("pos", ctypes.c_void_p), ("lattice", ctypes.c_void_p), ("Z", ctypes.c_void_p)]


class CGraph(ctypes.Structure):
    _fields_ = [("cap_edges", ctypes.c_int64), ("cap_bonds", ctypes.c_int64), ("cap_angles", ctypes.c_int64),
                ("n_edges", ctypes.c_int64), ("n_bonds", ctypes.c_int64), ("n_angles", ctypes.c_int64),
                ("edge_ptr", ctypes.c_void_p), ("edge_dst", ctypes.c_void_p), ("edge_img", ctypes.c_void_p),
                ("edge_rev", ctypes.c_void_p), ("bond_ptr", ctypes.c_void_p), ("bond_edge", ctypes.c_void_p),
                ("angle_ptr", ctypes.c_void_p), ("angle_b2", ctypes.c_void_p)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError("libchgnet.so is not built (%s); run paper_2412_20796_amd/build_lib.py" % _LIB_PATH)
        L = ctypes.CDLL(_LIB_PATH)
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        L.chgnet_param_count.argtypes = [ctypes.POINTER(HParams), ctypes.POINTER(i64)]
        L.chgnet_workspace_size.argtypes = [ctypes.POINTER(HParams), i64, i64, i64, i64, i64,
                                            ctypes.POINTER(ctypes.c_size_t)]
        L.chgnet_build_graph.argtypes = [ctypes.POINTER(HParams), ctypes.POINTER(CBatch), ctypes.POINTER(CGraph), vp,
                                         ctypes.c_size_t, vp]
        L.chgnet_build_graph_noalloc.argtypes = [ctypes.POINTER(HParams), ctypes.POINTER(CBatch),
                                                 ctypes.POINTER(CGraph), vp]
        L.chgnet_forward.argtypes = [ctypes.POINTER(HParams), ctypes.POINTER(CBatch), ctypes.POINTER(CGraph), vp, vp,
                                     vp, vp, vp, ctypes.c_int, vp, ctypes.c_size_t, vp]
        L.chgnet_backward.argtypes = [ctypes.POINTER(HParams), ctypes.POINTER(CBatch), ctypes.POINTER(CGraph), vp, vp,
                                      vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.chgnet_step.argtypes = [ctypes.POINTER(HParams), ctypes.POINTER(CBatch), ctypes.POINTER(CGraph), vp, vp, vp,
                                  vp, vp, ctypes.POINTER(LossCfg), vp, vp, vp, vp, ctypes.POINTER(ctypes.c_float),
                                  vp, ctypes.c_size_t, vp]
        L.chgnet_md.argtypes = [ctypes.POINTER(HParams), ctypes.POINTER(CBatch), ctypes.POINTER(CGraph), vp,
                                ctypes.POINTER(MdState), ctypes.c_float, ctypes.c_int, ctypes.c_int,
                                ctypes.POINTER(ctypes.c_int), vp, ctypes.c_size_t, vp]
        L.chgnet_last_error_string.restype = ctypes.c_char_p
        L.chgnet_profile_start.argtypes = [ctypes.c_int]
        L.chgnet_profile_stop.argtypes = [ctypes.c_char_p, ctypes.c_size_t]
        for name in EXPORTED:
            if name != "chgnet_last_error_string":
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(code):
    if code != CHGNET_OK:
        raise ChgnetError(code, lib().chgnet_last_error_string().decode())


def hparams(d=64, n_layers=4, n_rbf=31, n_fourier=31, envelope_p=8, r_atom=6.0, r_bond=3.0, magmom=False,
            sequential=False, conservative=False) -> HParams:
    return HParams(d, n_layers, n_rbf, n_fourier, envelope_p, r_atom, r_bond, int(magmom), int(sequential),
                   int(conservative))


def param_count(hp: HParams) -> int:
    n = ctypes.c_int64()
    _check(lib().chgnet_param_count(ctypes.byref(hp), ctypes.byref(n)))
    return n.value


def workspace_size(hp: HParams, N, E, B, A, S) -> int:
    n = ctypes.c_size_t()
    _check(lib().chgnet_workspace_size(ctypes.byref(hp), N, E, B, A, S, ctypes.byref(n)))
    return n.value


def profile_start(max_launches=100000):
    _check(lib().chgnet_profile_start(max_launches))


def profile_stop():
    """{tag: (launches, total_ms)} of the launches since profile_start."""
    buf = ctypes.create_string_buffer(1 << 16)
    _check(lib().chgnet_profile_stop(buf, len(buf)))
    out = {}
    for line in buf.value.decode().splitlines():
        tag, n, ms = line.split()
        out[tag] = (int(n), float(ms))
    return out


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


@dataclass
class DeviceBatch:
    atom_ptr: torch.Tensor
    pos: torch.Tensor
    lattice: torch.Tensor
    Z: torch.Tensor

    @classmethod
    def from_host(cls, b, device="cuda"):
        return cls(torch.as_tensor(b.atom_ptr, dtype=torch.int32).to(device),
                   torch.as_tensor(b.pos, dtype=torch.float32).contiguous().to(device),
                   torch.as_tensor(b.lattice, dtype=torch.float32).contiguous().to(device),
                   torch.as_tensor(b.Z, dtype=torch.int32).to(device))

    @property
    def n_struct(self):
        return self.lattice.shape[0]

    @property
    def n_atoms(self):
        return self.pos.shape[0]

    def c(self) -> CBatch:
        return CBatch(self.n_struct, self.n_atoms, _ptr(self.atom_ptr), _ptr(self.pos), _ptr(self.lattice),
                      _ptr(self.Z))


class DeviceGraph:
    """Caller-owned graph arrays with capacities; grown on CHGNET_ECAPACITY."""

    def __init__(self, n_atoms, cap_edges, cap_bonds, cap_angles, device="cuda", with_angle_b2=True):
        i32 = dict(dtype=torch.int32, device=device)
        self.with_angle_b2 = with_angle_b2
        self.edge_ptr = torch.zeros(n_atoms + 1, **i32)
        self.bond_ptr = torch.zeros(n_atoms + 1, **i32)
        self.resize(cap_edges, cap_bonds, cap_angles, device)
        self.n_edges = self.n_bonds = self.n_angles = 0

    def resize(self, ce, cb, ca, device):
        i32 = dict(dtype=torch.int32, device=device)
        self.cap = (max(1, ce), max(1, cb), max(1, ca))
        self.edge_dst = torch.zeros(self.cap[0], **i32)
        self.edge_img = torch.zeros(self.cap[0], 3, **i32)
        self.edge_rev = torch.zeros(self.cap[0], **i32)
        self.bond_edge = torch.zeros(self.cap[1], **i32)
        self.angle_ptr = torch.zeros(self.cap[1] + 1, **i32)
        self.angle_b2 = torch.zeros(self.cap[2], **i32) if self.with_angle_b2 else None

    def c(self) -> CGraph:
        return CGraph(self.cap[0], self.cap[1], self.cap[2], self.n_edges, self.n_bonds, self.n_angles,
                      _ptr(self.edge_ptr), _ptr(self.edge_dst), _ptr(self.edge_img), _ptr(self.edge_rev),
                      _ptr(self.bond_ptr), _ptr(self.bond_edge), _ptr(self.angle_ptr), _ptr(self.angle_b2))

    def take_counts(self, cg: CGraph):
        self.n_edges, self.n_bonds, self.n_angles = cg.n_edges, cg.n_bonds, cg.n_angles

    def host(self):
        """Graph arrays trimmed to their sizes, as numpy (synchronises)."""
        E, B, A = self.n_edges, self.n_bonds, self.n_angles
        out = {"edge_ptr": self.edge_ptr, "edge_dst": self.edge_dst[:E], "edge_img": self.edge_img[:E],
               "edge_rev": self.edge_rev[:E], "bond_ptr": self.bond_ptr, "bond_edge": self.bond_edge[:B],
               "angle_ptr": self.angle_ptr[:B + 1]}
        if self.angle_b2 is not None:
            out["angle_b2"] = self.angle_b2[:A]
        return {k: v.cpu().numpy() for k, v in out.items()}

    @classmethod
    def from_host(cls, g, device="cuda"):
        N = len(g["edge_ptr"]) - 1
        E, B, A = len(g["edge_dst"]), len(g["bond_edge"]), int(g["angle_ptr"][-1])
        dg = cls(N, E, B, A, device)
        for k in ("edge_ptr", "edge_dst", "edge_img", "edge_rev", "bond_ptr", "bond_edge", "angle_ptr", "angle_b2"):
            src = torch.as_tensor(g[k], dtype=torch.int32).reshape(-1)
            getattr(dg, k).view(-1)[: src.numel()].copy_(src.to(device))
        dg.n_edges, dg.n_bonds, dg.n_angles = E, B, A
        return dg


class Workspace:
    """Caller-owned scratch buffer, grown on demand."""

    def __init__(self, device="cuda"):
        self.device = device
        self.buf = None

    def ensure(self, nbytes):
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=self.device)
        return self.buf

    @property
    def ptr(self):
        return ctypes.c_void_p(self.buf.data_ptr())

    @property
    def nbytes(self):
        return self.buf.numel()


def build_graph(hp: HParams, batch: DeviceBatch, graph: DeviceGraph, ws: Workspace):
    """chgnet_build_graph with a capacity retry. Returns (E, B, A)."""
    ws.ensure(workspace_size(hp, batch.n_atoms, 0, 0, 0, batch.n_struct))
    cb = batch.c()
    for _ in range(2):
        cg = graph.c()
        code = lib().chgnet_build_graph(ctypes.byref(hp), ctypes.byref(cb), ctypes.byref(cg), ws.ptr, ws.nbytes,
                                        _stream(batch.pos.device))
        graph.take_counts(cg)
        if code == CHGNET_ECAPACITY:
            graph.resize(int(cg.n_edges * 1.25) + 64, int(cg.n_bonds * 1.25) + 64, int(cg.n_angles * 1.25) + 64,
                         batch.pos.device)
            continue
        _check(code)
        return graph.n_edges, graph.n_bonds, graph.n_angles
    raise ChgnetError(CHGNET_ECAPACITY, "graph capacity retry failed")


def build_graph_noalloc(hp: HParams, batch: DeviceBatch, graph: DeviceGraph):
    """chgnet_build_graph_noalloc (the library's static scratch, no workspace)
    with a capacity retry. Returns (E, B, A)."""
    cb = batch.c()
    for _ in range(2):
        cg = graph.c()
        code = lib().chgnet_build_graph_noalloc(ctypes.byref(hp), ctypes.byref(cb), ctypes.byref(cg),
                                                _stream(batch.pos.device))
        graph.take_counts(cg)
        if code == CHGNET_ECAPACITY:
            graph.resize(int(cg.n_edges * 1.25) + 64, int(cg.n_bonds * 1.25) + 64, int(cg.n_angles * 1.25) + 64,
                         batch.pos.device)
            continue
        _check(code)
        return graph.n_edges, graph.n_bonds, graph.n_angles
    raise ChgnetError(CHGNET_ECAPACITY, "graph capacity retry failed")


def ensure_ws(hp, batch, graph, ws):
    ws.ensure(workspace_size(hp, batch.n_atoms, graph.cap[0], graph.cap[1], graph.cap[2], batch.n_struct))


def forward(hp, batch, graph, params, ws, save_for_backward=True):
    """(energy, forces, stress), plus magnetic moments with the head."""
    ensure_ws(hp, batch, graph, ws)
    dev = batch.pos.device
    S, N = batch.n_struct, batch.n_atoms
    energy = torch.empty(S, dtype=torch.float32, device=dev)
    forces = torch.empty(N, 3, dtype=torch.float32, device=dev)
    stress = torch.empty(S, 3, 3, dtype=torch.float32, device=dev)
    magmom = torch.empty(N, dtype=torch.float32, device=dev) if hp.magmom else None
    cb, cg = batch.c(), graph.c()
    _check(lib().chgnet_forward(ctypes.byref(hp), ctypes.byref(cb), ctypes.byref(cg), _ptr(params), _ptr(energy),
                                _ptr(forces), _ptr(stress), _ptr(magmom), int(save_for_backward), ws.ptr, ws.nbytes,
                                _stream(dev)))
    if hp.magmom:
        return energy, forces, stress, magmom
    return energy, forces, stress


def backward(hp, batch, graph, params, dE, dF, dS, ws, grad=None, dM=None):
    dev = batch.pos.device
    if grad is None:
        grad = torch.empty_like(params)
    cb, cg = batch.c(), graph.c()
    _check(lib().chgnet_backward(ctypes.byref(hp), ctypes.byref(cb), ctypes.byref(cg), _ptr(params),
                                 _ptr(dE.contiguous()), _ptr(dF.contiguous()), _ptr(dS.contiguous()),
                                 _ptr(None if dM is None else dM.contiguous()), _ptr(grad), ws.ptr, ws.nbytes,
                                 _stream(dev)))
    return grad


def step(hp, batch, graph, params, targets, ws, loss_w=(2.0, 1.5, 0.1, 0.1), huber_delta=0.0, grad=None, loss=None,
         adam=None):
    """One training step. targets = (E_target [S], F_target [N,3], S_target [S,3,3]) device tensors, plus
    M_target [N] with the magnetic-moment head. loss_w = energy, force, stress (, magmom) prefactors;
    huber_delta > 0 selects Huber's loss. adam = (m, v, (lr, b1, b2, eps, t)) or None. Returns (loss, grad)."""
    dev = batch.pos.device
    ensure_ws(hp, batch, graph, ws)
    if grad is None:
        grad = torch.empty_like(params)
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=dev)
    w = tuple(loss_w) + (0.0,) * (4 - len(loss_w))
    lw = LossCfg(w[0], w[1], w[2], w[3], huber_delta)
    mt = targets[3] if hp.magmom else None
    m = v = None
    ahp = None
    if adam is not None:
        m, v, h = adam
        ahp = (ctypes.c_float * 5)(*h)
    cb = batch.c()
    for _ in range(2):
        cg = graph.c()
        code = lib().chgnet_step(ctypes.byref(hp), ctypes.byref(cb), ctypes.byref(cg), _ptr(params),
                                 _ptr(targets[0]), _ptr(targets[1]), _ptr(targets[2]), _ptr(mt), ctypes.byref(lw),
                                 _ptr(loss), _ptr(grad), _ptr(m), _ptr(v), ahp, ws.ptr, ws.nbytes, _stream(dev))
        graph.take_counts(cg)
        if code == CHGNET_ECAPACITY:
            graph.resize(int(cg.n_edges * 1.25) + 64, int(cg.n_bonds * 1.25) + 64, int(cg.n_angles * 1.25) + 64, dev)
            ensure_ws(hp, batch, graph, ws)
            continue
        _check(code)
        return loss, grad
    raise ChgnetError(CHGNET_ECAPACITY, "graph capacity retry failed")


class MdList:
    """Device arrays of chgnet_md's candidate list (Verlet skin)."""

    def __init__(self, n_atoms, cap, device="cuda"):
        self.cap = int(cap)
        self.ptr = torch.zeros(n_atoms + 1, dtype=torch.int32, device=device)
        self.dst = torch.zeros(max(self.cap, 1), dtype=torch.int32, device=device)
        self.img = torch.zeros(max(self.cap, 1), 3, dtype=torch.int32, device=device)
        self.ref = torch.zeros(n_atoms, 3, dtype=torch.float32, device=device)
        self.n_builds = 0
        self.n_cand = 0

    def grow(self, n, device):
        self.cap = int(n * 1.25) + 64
        self.dst = torch.zeros(self.cap, dtype=torch.int32, device=device)
        self.img = torch.zeros(self.cap, 3, dtype=torch.int32, device=device)


def md(hp, batch, graph, params, vel, inv_mass, dt, n_steps, ws, forces=None, energy=None, stress=None, skin=0.0,
       cand=None):
    """n_steps of velocity-Verlet MD (chgnet_md) on batch.pos and vel in place, growing the graph (and the
    candidate list with skin > 0) when its capacity runs out. forces: [N,3] forces at batch.pos (computed
    first if None). cand: an MdList to use (one is made if None). Returns (forces, energy, stress)."""
    dev = batch.pos.device
    S, N = batch.n_struct, batch.n_atoms
    valid = forces is not None
    if forces is None:
        forces = torch.empty(N, 3, dtype=torch.float32, device=dev)
    if energy is None:
        energy = torch.empty(S, dtype=torch.float32, device=dev)
    if stress is None:
        stress = torch.empty(S, 3, 3, dtype=torch.float32, device=dev)
    if skin > 0 and cand is None:
        cand = MdList(N, 1024, dev)
    cb = batch.c()
    left = n_steps
    for _ in range(12):
        ensure_ws(hp, batch, graph, ws)
        st = MdState(_ptr(batch.pos).value, _ptr(vel).value, _ptr(inv_mass).value, _ptr(forces).value,
                     _ptr(energy).value, _ptr(stress).value, float(skin))
        if skin > 0:
            st.cap_cand, st.cand_ptr, st.cand_dst = cand.cap, _ptr(cand.ptr).value, _ptr(cand.dst).value
            st.cand_img, st.ref_pos = _ptr(cand.img).value, _ptr(cand.ref).value
        cg = graph.c()
        done = ctypes.c_int(0)
        code = lib().chgnet_md(ctypes.byref(hp), ctypes.byref(cb), ctypes.byref(cg), _ptr(params), ctypes.byref(st),
                               dt, left, int(valid), ctypes.byref(done), ws.ptr, ws.nbytes, _stream(dev))
        graph.take_counts(cg)
        left -= done.value
        valid = valid or done.value > 0
        if skin > 0:
            cand.n_builds += st.n_builds
            cand.n_cand = st.n_cand
        if code == CHGNET_ECAPACITY:
            if skin > 0 and st.n_cand > cand.cap:
                cand.grow(st.n_cand, dev)
            else:
                graph.resize(int(cg.n_edges * 1.25) + 64, int(cg.n_bonds * 1.25) + 64, int(cg.n_angles * 1.25) + 64,
                             dev)
            continue
        _check(code)
        return forces, energy, stress
    raise ChgnetError(CHGNET_ECAPACITY, "graph capacity retry failed")
