"""Benchmark: FastCHGNet training steps per second on one MI355X.

One step = chgnet_step on one batch: periodic graph build, forward (basis,
embeddings, T interaction blocks, energy/force/stress heads), weighted MSE
loss, backward for every weight and the Adam update, all in the HIP library.
Inputs (positions, lattices, atomic numbers, targets, weights) are seeded and
synthetic (the dataset is not available) and are resident in HBM before the
timed region.

Prints one JSON line (rank 0). Default workload: wide128, 128 random
triclinic crystals with 8-128 atoms each (log-uniform), d = 128, 5 layers
(the largest single-GPU configuration); the others are chosen by --workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_PEAK_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None, help="default: wide128 (training, inference), cubic8 (--md)")
    ap.add_argument("--magmom", action="store_true", help="model variant: magnetic-moment head and its loss term")
    ap.add_argument("--huber", type=float, default=0.0, help="model variant: Huber loss with this delta (0 = MSE)")
    ap.add_argument("--sequential", action="store_true", help="model variant: the Eq. (10) interaction block")
    ap.add_argument("--conservative", action="store_true",
                    help="forces and stress as derivatives of the energy (training: second derivatives)")
    ap.add_argument("--forward-only", action="store_true",
                    help="time inference (graph build + forward with the readout) instead of training steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="structures in the CPU oracle sample (0 = auto: the whole batch, or for wide128 four "
                         "structures at evenly spaced size quantiles)")
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--launch-timing-only", action="store_true",
                    help="after the warm-up steps, the timed steps with per-launch timing only (the library's side "
                         "stream then runs serialized, as in the roofline pass); prints the per-kernel figures only, "
                         "for profiling runs")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run a plain 256 MiB device copy (reference for HBM traffic counters)")
    ap.add_argument("--md", action="store_true",
                    help="time velocity-Verlet molecular dynamics (forward only) instead of training steps")
    ap.add_argument("--md-replicas", type=int, default=1, help="independent copies of the crystal stepped together")
    ap.add_argument("--md-skin", type=float, default=0.0,
                    help="MD neighbour-list reuse: Verlet skin in A (0 = full graph search every step)")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no GPU: reduce two rocprofv3 counter CSVs (FETCH_SIZE, WRITE_SIZE) to a markdown summary")
    args = ap.parse_args()
    if args.workload is None and not args.md:
        args.workload = "wide128"
    return args


def main():
    args = parse()
    if args.traffic_summary:
        # the counter runs wrote their CSVs into <dir>/run_counter_collection.csv
        cmd = ["rocprofv3 --pmc %s --output-format csv -d %s -o run -- python3 bench.py "
               "--workload %s --no-cpu-baseline --no-roofline --steps 3 --warmup 1 --calibrate-copy"
               % (c, os.path.dirname(path) or ".", args.workload)
               for c, path in zip(("FETCH_SIZE", "WRITE_SIZE"), args.traffic_summary)]
        cmd.append("python3 bench.py --workload %s --traffic-summary %s %s" % ((args.workload,) + tuple(args.traffic_summary)))
        print(traffic_summary(args.traffic_summary[0], args.traffic_summary[1], args.workload, cmd))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2412_20796_amd import binding as bd
    from paper_2412_20796_amd import synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.md:
        print(json.dumps(md_bench(args, bd, synth, dev)), flush=True)
        return
    b, params, targets, d, T = synth.workload_inputs(args.workload, magmom=args.magmom)
    hp = bd.hparams(d=d, n_layers=T, magmom=args.magmom, sequential=args.sequential, conservative=args.conservative)
    db = bd.DeviceBatch.from_host(b, dev)
    g = bd.DeviceGraph(b.n_atoms, 1024, 256, 1024, dev)
    ws = bd.Workspace(dev)
    p = torch.tensor(params, device=dev)
    m = torch.zeros_like(p)
    v = torch.zeros_like(p)
    tg = [torch.tensor(x, device=dev) for x in targets]
    grad = torch.empty_like(p)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    lr, b1, b2, eps = 3e-4, 0.9, 0.999, 1e-8

    step_no = [0]

    def one_step():
        step_no[0] += 1
        if args.forward_only:
            bd.build_graph(hp, db, g, ws)
            bd.forward(hp, db, g, p, ws)
            return
        bd.step(hp, db, g, p, tg, ws, loss_w=(2.0, 1.5, 0.1, 0.1), huber_delta=args.huber, grad=grad, loss=loss,
                adam=(m, v, (lr, b1, b2, eps, float(step_no[0]))))

    if args.calibrate_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.launch_timing_only:
        # warm-up steps unprofiled (their first launches include one-time
        # costs), then `steps` steps with every launch timed
        for _ in range(max(args.warmup, 1)):
            one_step()
        torch.cuda.synchronize()
        n = args.steps
        bd.profile_start(400 * n + 1000)
        for _ in range(n):
            one_step()
        torch.cuda.synchronize()
        prof = bd.profile_stop()
        E, B, A = g.n_edges, g.n_bonds, g.n_angles
        rl, rows = roofline(prof, n, dict(N=b.n_atoms, E=E, B=B, A=A, S=b.n_struct, D=d, T=T,
                                          fused_bwd=not args.sequential, workload=args.workload,
                                          R=hp.n_rbf, K=hp.n_fourier))
        print(json.dumps({"launch_timing_steps": n, "roofline": rl, "kernels": rows}), flush=True)
        return
    for _ in range(max(args.warmup, 1)):
        one_step()
    torch.cuda.synchronize()
    E, B, A = g.n_edges, g.n_bonds, g.n_angles

    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev[0].record()
    for k in range(args.steps):
        one_step()
        ev[k + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_mean = ev[0].elapsed_time(ev[-1]) / args.steps
    per_step = np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps)])
    ms = float(np.median(per_step))
    S = b.n_struct
    value = S / (ms * 1e-3)

    out = {
        "metric": ("inference structures/sec (graph + forward) on 1 MI355X" if args.forward_only
                   else "training structures/sec (fwd+bwd) on 1 MI355X"),
        "value": round(value, 2),
        "unit": "structures/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic (seeded crystals shaped like the paper's training set; random-init weights)",
        "timing": "median of per-step HIP events over the timed steps (mean in ms_per_step_mean)",
        "config": {"workload": args.workload, "structures": S, "atoms": b.n_atoms, "edges": E, "bonds": B,
                   "angles": A, "d": d, "layers": T, "parallelism": "single GPU",
                   "block": "Eq. 10 (sequential)" if args.sequential else "Eq. 11",
                   "loss": "Huber delta=%g" % args.huber if args.huber > 0 else "MSE",
                   "heads": "E, F, S, magmom" if args.magmom else "E, F, S",
                   "readout": "conservative (F = -dE/dr)" if args.conservative else "direct force/stress heads",
                   "step": "graph + forward" if args.forward_only else "graph + forward + loss + backward + Adam"},
        "edges_per_s": round(E / (ms * 1e-3), 1),
        "angles_per_s": round(A / (ms * 1e-3), 1),
        "ms_per_step_mean": round(ms_mean, 4),
        "ms_per_step_p10_p90": [round(float(np.percentile(per_step, 10)), 4),
                                round(float(np.percentile(per_step, 90)), 4)],
        "wall_s_timed": round(wall, 3),
        "final_loss": float(loss.cpu()[0]),
    }
    if not args.no_roofline:
        bd.profile_start(400 * args.steps + 1000)
        for _ in range(args.steps):
            one_step()
        torch.cuda.synchronize()
        prof = bd.profile_stop()
        out["roofline"], out["kernels"] = roofline(prof, args.steps, dict(N=b.n_atoms, E=E, B=B, A=A, S=S, D=d, T=T,
                                                                            fused_bwd=not args.sequential,
                                                                            workload=args.workload, R=hp.n_rbf,
                                                                            K=hp.n_fourier))
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_sample, variant=args)
    print(json.dumps(out), flush=True)


def md_bench(args, bd, synth, dev):
    """Molecular dynamics in the regime of the paper's Table 2: one small
    crystal (or R independent copies in one batch) stepped by chgnet_md; every
    step rebuilds the graph and runs the forward pass with the direct force
    and stress heads. K steps are timed as one call."""
    import numpy as np
    import torch

    workload = args.workload or "cubic8"
    b0, params, _, d, T = synth.workload_inputs(workload)
    R = max(1, args.md_replicas)
    if R > 1:
        n0 = b0.n_atoms
        b = synth.Batch(np.concatenate([[0], np.cumsum(np.tile(np.diff(b0.atom_ptr), R))]).astype(np.int32),
                        np.tile(b0.pos, (R, 1)), np.tile(b0.lattice, (R, 1, 1)), np.tile(b0.Z, R))
        assert b.n_atoms == R * n0
    else:
        b = b0
    rng = np.random.default_rng(17)
    hp = bd.hparams(d=d, n_layers=T, sequential=args.sequential, conservative=args.conservative)
    db = bd.DeviceBatch.from_host(b, dev)
    g = bd.DeviceGraph(b.n_atoms, 1024, 256, 1024, dev)
    ws = bd.Workspace(dev)
    p = torch.tensor(params, device=dev)
    vel = torch.tensor((rng.standard_normal((b.n_atoms, 3)) * 0.01).astype(np.float32), device=dev)
    inv_m = torch.tensor((1.0 / rng.uniform(6.0, 60.0, b.n_atoms)).astype(np.float32), device=dev)
    dt = 0.5
    skin = args.md_skin
    cand = bd.MdList(b.n_atoms, 4096, dev) if skin > 0 else None
    # a stream of its own (default priority): on it chgnet_md captures and
    # replays the forward pass of steps whose graph sizes repeat
    torch.cuda.synchronize()
    side = torch.cuda.Stream(dev)
    with torch.cuda.stream(side):
        F, E, S = bd.md(hp, db, g, p, vel, inv_m, dt, max(args.warmup, 1), ws, skin=skin, cand=cand)
        torch.cuda.synchronize()
        builds0 = cand.n_builds if cand else 0
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        wall0 = time.perf_counter()
        e0.record()
        bd.md(hp, db, g, p, vel, inv_m, dt, args.steps, ws, forces=F, energy=E, stress=S, skin=skin, cand=cand)
        e1.record()
        torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = e0.elapsed_time(e1) / args.steps
    return {
        "metric": "molecular-dynamics steps/sec on 1 MI355X",
        "value": round(1e3 / ms, 2), "unit": "steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp32", "data": "synthetic (seeded crystal, random velocities and masses; random-init weights)",
        "config": {"workload": "md-" + workload, "structures": b.n_struct, "atoms": b.n_atoms,
                   "replicas": R, "edges": g.n_edges, "bonds": g.n_bonds, "angles": g.n_angles, "d": d,
                   "layers": T, "integrator": "velocity Verlet, dt %.1f fs" % dt,
                   "neighbour_list": ("candidates within r + %.2f A, rebuilt %d times in the timed steps"
                                      % (skin, cand.n_builds - builds0)) if skin > 0 else "full search every step",
                   "block": "Eq. 10 (sequential)" if args.sequential else "Eq. 11",
                   "readout": "conservative (F = -dE/dr)" if args.conservative else "direct force/stress heads"},
        "atom_steps_per_s": round(b.n_atoms * 1e3 / ms, 1),
        "wall_ms_per_step": round(1e3 * wall / args.steps, 4),
        "paper_context": "one-step MD of an 8-atom LiMnO2 cell: 0.0077 s (FastCHGNet), 0.022 s (CHGNet), "
                         "on the paper's GPU (Table 2)",
    }


def algorithmic_cost(tag, z):
    """Algorithmic work of one step's launches of `tag`: ("mfma", flops) for
    the dense products, ("hbm", bytes) for gather/scatter/elementwise kernels.

    Per-unit figures (fp32, d = D): an angle of a layer with an angle update
    costs 8d^2 flops in its a-term (a [W_bond | W_angle], d -> 4d), 4d^2 in
    the last layer (bond conv only); an edge costs 4d^2 (e W, d -> 2d). The
    backward input gradients cost the same per unit, the weight gradients the
    same again (A^T B over the rows). Bytes count each array read or written
    once, gathered tables (per-atom and per-bond rows) once each."""
    N, E, B, A, D, T = z["N"], z["E"], z["B"], z["A"], z["D"], z["T"]
    Tang = T - 1  # layers with an angle update
    f = 4  # bytes per fp32
    if tag == "gemm_in_bwd" and z.get("fused_bwd"):
        # the edge and angle rows are formed by the fused gate backward; this
        # launch holds the atom rows and the bond rows (k = 8d, 6d last layer)
        return "mfma", T * N * 16 * D * D - N * 4 * D * D + Tang * B * 16 * D * D + B * 8 * D * D
    if tag == "gemm_in_bwd":
        return "mfma", T * (E * 4 * D * D + N * 16 * D * D) - N * 4 * D * D + Tang * A * 8 * D * D + A * 4 * D * D
    if tag == "tn_in":  # first-layer and output-layer weight gradients of every block
        return "mfma", (T * (E * 4 * D * D + N * 16 * D * D + B * 8 * D * D + (N + B) * 2 * D * D) - N * 4 * D * D
                        + Tang * (A * 8 * D * D + B * 8 * D * D) + A * 4 * D * D)
    if tag == "gemm_proj":
        return "mfma", T * (N * 16 * D * D + B * 8 * D * D) - N * 4 * D * D - B * 4 * D * D
    if tag == "gemm_bond_bwd":
        return "mfma", Tang * B * 16 * D * D + B * 8 * D * D
    if tag == "k_gate_fwd" and D != 64:
        # d = 128: the fused gate is bound by its product z = x W (+ b) of
        # every edge (d -> 2d) and, per angle, of the bond-conv and
        # angle-update gates (d -> 4d; d -> 2d in the last layer)
        return "mfma", T * E * 4 * D * D + Tang * A * 8 * D * D + A * 4 * D * D
    if tag == "k_gate_fwd" and D == 64:
        # pre-activations formed in the kernel (d = 64): per edge x (d) and
        # e^a (d) in, z kept for the backward (2d), message (d) and the copy
        # of x into e^{t+1} (d) out; per angle and gate x (d) in, z (2d) and
        # output (d) out, the angle gate also reads a (d). Tables: per-atom
        # terms N x 8d (6d last layer), per-bond terms B x 8d (4d), e^b B x d.
        lay = E * 6 * D + A * 9 * D + N * 8 * D + B * 9 * D
        last = E * 6 * D + A * 4 * D + N * 6 * D + B * 5 * D
        return "hbm", f * (Tang * lay + last)
    if tag == "k_gate_bwd" and z.get("fused_bwd") and D != 64:
        # d = 128: the fused backward gate is bound by its input-gradient
        # product dX = dz W^T of every edge (2d -> d) and, per angle, of the
        # bond-conv and angle-update gates (2 x 2d -> d; one gate in the last
        # layer): the same flops as the forward product
        return "mfma", T * E * 4 * D * D + Tang * A * 8 * D * D + A * 4 * D * D
    if tag == "k_gate_bwd" and z.get("fused_bwd"):
        # as below, plus the input gradients the kernel forms: per edge the
        # residual (d) in and de (d) out; per angle da (d) out and, in layers
        # with an angle update, the residual (d) in
        lay = E * 9 * D + A * 12 * D + N * 9 * D + B * 10 * D
        last = E * 9 * D + A * 6 * D + N * 7 * D + B * 6 * D
        return "hbm", f * (Tang * lay + last)
    if tag == "k_gate_bwd":
        # per edge: z (2d), e^a (d), d e^a (d) in; dz (2d), d e^a (d) out;
        # per angle and gate: z (2d) + upstream (d) in, dz (2d) out (the bond
        # gate's upstream is gathered, its t2 (d) written). Tables as in the
        # forward plus dm N x d, dmu B x d.
        lay = E * 7 * D + A * 10 * D + N * 9 * D + B * 10 * D
        last = E * 7 * D + A * 5 * D + N * 7 * D + B * 6 * D
        return "hbm", f * (Tang * lay + last)
    if tag == "k_bond_bwd_reduce":
        # dz read once from HBM (a row's second read, by its other bond, is
        # scheduled to hit L2), t2 read; DZ12 written
        return "hbm", f * (Tang * A * (4 * D + D) + A * (2 * D + D) + T * B * 8 * D)
    # training through the conservative readout: the dual-number pass (value
    # and tangent parts; a linear map costs twice its flops, the tangent-only
    # maps once)
    R, K = z.get("R", 31), z.get("K", 31)
    if tag == "kd_gemm":
        emb = 2 * (2 * E * R * D + B * R * D + A * K * D) + 8 * E * D * R + 4 * B * D * R
        heads = 4 * N * D * D + 8 * N * D * D
        # per layer: projections (atom blocks 4 or 3, bond blocks 4 or 2), the
        # edge and angle blocks, tangent updates; backward dm, dmu, the input
        # gradients of atoms (S, 4 or 3 blocks of 2d), edges, angles and bonds (T)
        lay = lambda ang: (8 * N * D * D * (4 if ang else 3) + 8 * B * D * D * (4 if ang else 2) + 8 * E * D * D
                           + 8 * A * D * D * (2 if ang else 1) + 2 * N * D * D + 2 * B * D * D
                           + 4 * N * D * D + 4 * B * D * D + 8 * N * D * D * (4 if ang else 3) + 8 * E * D * D
                           + 8 * A * D * D * (2 if ang else 1) + 8 * B * D * D * (4 if ang else 2))
        return "mfma", emb + heads + Tang * lay(True) + lay(False)
    if tag == "kd_tn":
        # X_t^T Y_v + X_v^T Y_t of every weight: heads, output linears, the
        # gate blocks (atom blocks over atoms, bond blocks over bonds, edge
        # and angle blocks over their rows), the embedding
        emb = 8 * E * R * D + 4 * B * R * D + 4 * A * K * D
        heads = 8 * N * D * D + 4 * N * D
        lay = lambda ang: (4 * N * D * D + 4 * B * D * D + 16 * N * D * D + 8 * E * D * D
                           + (8 * N * D * D + 16 * B * D * D + 8 * A * D * D) * (2 if ang else 1))
        return "mfma", emb + heads + Tang * lay(True) + lay(False)
    if tag == "kd_gate_fwd":
        # per row and gate: z (2d, both parts) in and out, phi (d, both
        # parts) out (the angle update: a tangent in, a' tangent out);
        # projection tables N x 8d and B x 8d, both parts, once
        lay = lambda ang: (E * 10 * D + A * 10 * D + (A * 10 * D if ang else 0) + N * 16 * D
                           + B * 16 * D * (1 if ang else 0.5))
        return "hbm", f * (Tang * lay(True) + lay(False))
    if tag == "kd_gate_bwd":
        # per row and gate: z (2d) and d phi (d) in, dz (2d) out, both parts
        # (the LayerNorm parameter terms stay in registers)
        lay = lambda ang: (E + A * (2 if ang else 1)) * 10 * D
        return "hbm", f * (Tang * lay(True) + lay(False))
    return None, None


def mandatory_cost(tag, z):
    """The method's own memory traffic (the mandatory forward bytes per unit
    and layer of the scope table: an edge reads e and e^a, 8d bytes; a bond
    of the bond graph reads and writes e_b, 8d; an angle reads and writes a,
    8d, plus 8 bytes of indices, or reads it only in the last layer, 4d + 8;
    atoms are negligible), attributed to the gate launch of each layer; the
    backward gate moves twice the forward (activations in, their gradients
    out). Dense products keep their flop count (the split GEMMs are the
    method's arithmetic). None where a kernel moves only this design's own
    intermediates."""
    bound, work = algorithmic_cost(tag, z)
    if bound == "mfma":
        return bound, work
    N, E, B, A, D, T = z["N"], z["E"], z["B"], z["A"], z["D"], z["T"]
    lay = E * 8 * D + B * 8 * D + A * (8 * D + 8)
    last = E * 8 * D + B * 8 * D + A * (4 * D + 8)
    if tag == "k_gate_fwd":
        return "hbm", (T - 1) * lay + last
    if tag == "k_gate_bwd":
        return "hbm", 2 * ((T - 1) * lay + last)
    return None, None


# rocprofv3 kernel symbols of each launch tag that has an algorithmic cost
# (a tag's call may launch several kernels: tn_in launches its 64 x 128 and
# its 64 x 64 wave-tile plans separately)
def tag_symbols(tag, d):
    return {
        "gemm_in_bwd": ["k_gemm<64, 2, 4>"],
        "tn_in": ["k_tn<1, true>", "k_tn<1, false>"],
        "k_gate_fwd": ["k_gate_fwd_mm<%d>" % d],
        "k_gate_bwd": ["k_gate_bwd_mm" if d == 64 else "k_gate_bwd_mm128"],
    }.get(tag)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_%s.md")
SOURCE_DIR = os.path.join(ROOT, "paper_2412_20796_amd", "csrc")


def source_digest():
    """sha256 over the HIP sources: traffic measured on other sources is stale."""
    import hashlib

    h = hashlib.sha256()
    for name in sorted(os.listdir(SOURCE_DIR)):
        if name.endswith((".hip", ".hpp")):
            h.update(name.encode())
            h.update(open(os.path.join(SOURCE_DIR, name), "rb").read())
    return h.hexdigest()


def measured_traffic(workload, tag):
    """HBM bytes per launch of `tag` from the committed counter summary, or
    None if there is none for this workload, the kernel, or these sources."""
    path = TRAFFIC_FILE % workload
    from paper_2412_20796_amd import synth

    syms = tag_symbols(tag, synth.WORKLOADS.get(workload, (0, 64, 0))[1])
    if syms is None or not os.path.exists(path):
        return None
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return None
    data = json.loads(text[start + 7:text.index("```", start + 7)])
    if data.get("source_sha256") != source_digest():
        return None
    # each kernel of the tag is launched once per call (those of a plan kind
    # the workload has no product for are absent)
    ks = [data["kernels"][s] for s in syms if s in data["kernels"]]
    return sum(k["fetch_bytes"] + k["write_bytes"] for k in ks) if ks else None


def traffic_summary(fetch_csv, write_csv, workload, command):
    """Reduce two rocprofv3 counter runs (FETCH_SIZE, WRITE_SIZE; KiB per
    dispatch) to bytes per dispatch for each kernel, each counter scaled by
    what it reads for the 256 MiB plain copy that --calibrate-copy launches
    first (the largest copy kernel in the run). Prints a markdown summary
    with a JSON block that roofline() reads."""
    import collections
    import csv

    def per_kernel(path, counter):
        d = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                d[r["Kernel_Name"].replace("chg::(anonymous namespace)::", "").split("(")[0].replace("void ", "")]\
                    .append(float(r["Counter_Value"]))
        return d

    fk, wk = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    copies = [k for k in fk if "copy" in k.lower() and not k.startswith("k_")]
    ck = max(copies, key=lambda k: max(fk[k]))
    ideal_kib = 256 * 1024
    sf, sw = ideal_kib / max(fk[ck]), ideal_kib / max(wk[ck])
    kern = {}
    for k in fk:
        if k == ck or k not in wk:
            continue
        F = sum(fk[k]) / len(fk[k]) * sf * 1024
        W = sum(wk[k]) / len(wk[k]) * sw * 1024
        kern[k] = {"dispatches": len(fk[k]), "fetch_bytes": round(F), "write_bytes": round(W)}
    data = {"workload": workload, "source_sha256": source_digest(), "calibration_kernel": ck,
            "fetch_scale": round(sf, 4), "write_scale": round(sw, 4), "kernels": kern}
    lines = ["# HBM traffic per dispatch, workload %s" % workload, "",
             "Commands (repository root, one MI355X):", ""]
    lines += ["    " + c for c in command]
    lines += ["", "Calibration: a 256 MiB device-to-device copy (%s) reads FETCH_SIZE %.0f KiB and "
              "WRITE_SIZE %.0f KiB; every kernel's counters are scaled by %.4f (fetch) and %.4f (write)."
              % (ck, max(fk[ck]), max(wk[ck]), sf, sw), "",
              "| kernel | dispatches | fetch MB/dispatch | write MB/dispatch |", "|---|---|---|---|"]
    for k, v in sorted(kern.items(), key=lambda kv: -(kv[1]["fetch_bytes"] + kv[1]["write_bytes"]) * kv[1]["dispatches"])[:20]:
        lines.append("| %s | %d | %.1f | %.1f |" % (k, v["dispatches"], v["fetch_bytes"] / 1e6, v["write_bytes"] / 1e6))
    lines += ["", "```json", json.dumps(data, indent=1), "```", ""]
    return "\n".join(lines)


def roofline(prof, steps, z):
    """Per-tag rates from the per-launch HIP events. `achieved` and `frac`
    count the method's mandatory work (mandatory_cost); the design_* fields
    count every array this implementation reads or writes (algorithmic_cost)."""
    rows = []
    for tag, (n, ms) in prof.items():
        bound, work = algorithmic_cost(tag, z)
        mbound, mwork = mandatory_cost(tag, z)
        per_step_ms = ms / steps
        row = {"tag": tag, "launches_per_step": n / steps, "ms_per_step": round(per_step_ms, 4),
               "avg_launch_us": round(1e3 * ms / max(n, 1), 2)}
        if bound:
            sec = ms * 1e-3 / steps
            if bound == "mfma":
                ach = work / sec / 1e12
                row.update(bound="mfma", achieved=round(ach, 3), unit="TFLOP/s", frac=round(ach / FP32_PEAK_TFLOPS, 4))
            else:
                dach = work / sec / 1e9
                row.update(bound="hbm", unit="GB/s", design_achieved=round(dach, 1),
                           design_frac=round(dach / HBM_PEAK_GBS, 4))
                if mbound:
                    ach = mwork / sec / 1e9
                    row.update(achieved=round(ach, 1), frac=round(ach / HBM_PEAK_GBS, 4))
        rows.append(row)
    rows.sort(key=lambda r: -r["ms_per_step"])
    dom = next(r for r in rows if "frac" in r)
    bound, work = algorithmic_cost(dom["tag"], z)
    _, mwork = mandatory_cost(dom["tag"], z)
    n_launch = dom["launches_per_step"]
    rl = {"kernel": dom["tag"], "bound": dom["bound"], "achieved": dom["achieved"],
          "peak": FP32_PEAK_TFLOPS if dom["bound"] == "mfma" else HBM_PEAK_GBS, "unit": dom["unit"],
          "frac": dom["frac"], "traffic": measured_traffic(z["workload"], dom["tag"]),
          "work_per_launch": mwork / n_launch, "work_unit": "flop" if bound == "mfma" else "byte",
          "work_basis": "the method's mandatory work per unit (split-GEMM flops; gate bytes: e, e^a, e_b, a "
                        "per layer), times the units of one launch",
          "design_work_per_launch": work / n_launch,
          "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
          "avg_launch_us": dom["avg_launch_us"], "launches_per_step": n_launch,
          "timing": "HIP events around every launch of the kernel on the library's stream, %d steps" % steps}
    if dom["bound"] == "hbm":
        rl.update(design_achieved=dom["design_achieved"], design_frac=dom["design_frac"])
    return rl, rows[:16]


def cpu_baseline(workload, sample, min_seconds=10.0, variant=None):
    """The CPU oracle (fp64 NumPy, untuned) on a bounded sample of the same
    workload: graph build, forward, loss and backward of `sample` structures
    taken at evenly spaced quantiles of the batch's size distribution (default:
    the whole batch, or four structures for wide128, whose full batch takes the
    oracle tens of minutes), repeated until min_seconds of CPU work and at
    least three times on the small workloads; reported in structures per
    second of that sample."""
    import numpy as np

    from oracle import model as om
    from paper_2412_20796_amd import synth

    mag = bool(variant and variant.magmom)
    b, params, targets, d, T = synth.workload_inputs(workload, magmom=mag)
    if sample <= 0:
        sample = 4 if workload == "wide128" else b.n_struct
    sample = min(sample, b.n_struct)
    sizes = np.diff(b.atom_ptr)
    order = np.argsort(sizes, kind="stable")
    picks = sorted(int(order[min(b.n_struct - 1, int((q + 0.5) * b.n_struct / sample))]) for q in range(sample))
    ptr = [0]
    for s in picks:
        ptr.append(ptr[-1] + int(sizes[s]))
    n = ptr[-1]
    atoms = np.concatenate([np.arange(b.atom_ptr[s], b.atom_ptr[s + 1]) for s in picks])
    sb = synth.Batch(np.asarray(ptr, np.int32), b.pos[atoms], b.lattice[picks], b.Z[atoms])
    tgt = (targets[0][picks], targets[1][atoms], targets[2][picks]) + ((targets[3][atoms],) if mag else ())
    min_reps = 3 if workload in ("cubic8", "triclinic40", "heavytail64") else 1
    fwd = bool(variant and variant.forward_only)
    hp = om.HParams(d=d, n_layers=T, magmom=mag, sequential=bool(variant and variant.sequential),
                    conservative=bool(variant and variant.conservative))
    delta = variant.huber if variant and variant.huber > 0 else None
    reps = 0
    t = time.perf_counter()
    n_edges = 0
    while True:
        if fwd:
            from oracle import graph as og

            graph = og.build_graph(sb.atom_ptr, sb.pos, sb.lattice, hp.r_atom, hp.r_bond)
            om.forward(hp, sb, graph, params.astype(np.float64))
        elif hp.conservative:
            # the loss gradient through F = -dE/dr: second derivatives by autograd
            from oracle import autodiff
            from oracle import graph as og

            graph = og.build_graph(sb.atom_ptr, sb.pos, sb.lattice, hp.r_atom, hp.r_bond)
            autodiff.loss_and_grad(hp, sb, graph, params.astype(np.float64), tgt, delta=delta)
        else:
            _, _, _, graph = om.step(hp, sb, params.astype(np.float64), tgt, delta=delta)
        n_edges = len(graph["edge_dst"])
        reps += 1
        dt = time.perf_counter() - t
        if (dt >= min_seconds and reps >= min_reps) or reps >= 20:
            break
    try:
        from threadpoolctl import threadpool_info

        threads = max(int(i.get("num_threads", 1)) for i in threadpool_info()) if threadpool_info() else 1
    except Exception:  # pragma: no cover - threadpoolctl is optional
        threads = 1
    return {"value": round(reps * sample / dt, 4), "unit": "structures/s", "cores": threads, "kind": "oracle",
            "host_cpus": len(os.sched_getaffinity(0)), "edges_per_s": round(reps * n_edges / dt, 1),
            "sample": "%d of the %d structures (%d atoms, %d edges; evenly spaced size quantiles), %d %s in %.1f s"
                      % (sample, b.n_struct, n, n_edges, reps, "inference(s) (graph, forward)" if fwd
                         else "full step(s) (graph, forward, loss, backward through F = -dE/dr by autograd)"
                         if hp.conservative else "full step(s) (graph, forward, loss, backward)", dt)}


if __name__ == "__main__":
    main()
