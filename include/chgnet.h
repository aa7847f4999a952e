/*
 * chgnet.h - C interface of the MI355X (gfx950) FastCHGNet training-step library.
 *
 * The library computes one training step of the FastCHGNet model (Zhou et al.,
 * "FastCHGNet: Training one Universal Interatomic Potential to 1.5 Hours with
 * 32 GPUs"): crystal structures in; energy, forces and stress out (Sec. II-B,
 * Fig. 1a); gradients of a weighted loss with respect to every weight out
 * (Sec. IV, "Parameters Setting").
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller. The library
 *    never allocates device memory: scratch space is the caller's `ws`
 *    buffer of `ws_bytes` bytes, sized by chgnet_workspace_size().
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream). Every
 *    call only enqueues work on `stream` and returns, except
 *    chgnet_build_graph, which waits once for the graph's sizes (see there).
 *  - Floating-point data are IEEE fp32; integer data are int32 unless noted.
 *  - All matrices are row-major. A lattice is 3x3 with ROWS = lattice vectors,
 *    so Cartesian = fractional @ lattice.
 *  - No global data: calls are re-entrant as long as concurrent calls use
 *    different workspaces. The backward pass overlaps its weight-gradient
 *    products with the next layer on a second HIP stream (default priority)
 *    that the library creates, with a few events, once per host thread and
 *    device; it forks from and joins back into `stream`, so the call still
 *    behaves as work enqueued on `stream`. Results are bitwise reproducible
 *    run to run: every floating-point sum runs in a fixed order (no
 *    floating-point atomics). chgnet_build_graph keeps a small pinned host
 *    buffer per host thread for the size readback (allocated on first use).
 *  - Return value: CHGNET_OK (0) or a negative error code below; the text of
 *    the last error of the calling thread is chgnet_last_error_string().
 *  - Environment: CHGNET_TN_WIDE_MIN_UNITS (a non-negative integer, read on
 *    every weight-gradient launch) sets the launch size, in units of 64 rows
 *    times 64 x 64 output tiles, from which the weight-gradient products use
 *    64 x 128 wave tiles (default 24576). It changes only the kernel
 *    schedule, not what is computed; unset is the measured default.
 *
 * Hyperparameters (Sec. IV): feature width d (64; 128 supported), layers T,
 * 31 radial and 31 angular basis functions, envelope exponent p = 8, atom
 * graph cutoff 6 A, bond graph cutoff 3 A. Supported: d in {64, 128},
 * 1 <= T <= 16, 1 <= n_rbf <= 64, n_fourier odd in [1, 63], p in [2, 16],
 * 0 < r_bond <= r_atom <= 20, magmom, sequential and conservative in {0, 1}.
 */
#ifndef CHGNET_H
#define CHGNET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CHGNET_OK 0
#define CHGNET_EINVAL -1    /* bad shape, hyperparameter or input value          */
#define CHGNET_ECAPACITY -2 /* graph capacity too small; required sizes returned  */
#define CHGNET_EWORKSPACE -3 /* workspace too small                               */
#define CHGNET_EHIP -4      /* HIP runtime error                                 */

typedef struct {
  int32_t d;          /* feature width of atoms, bonds and angles           */
  int32_t n_layers;   /* number of interaction blocks T                     */
  int32_t n_rbf;      /* radial basis size (31)                             */
  int32_t n_fourier;  /* angular basis size, odd (31 = 1 + 15 cos + 15 sin) */
  int32_t envelope_p; /* polynomial envelope exponent p (8)                 */
  float r_atom;       /* atom-graph cutoff, Angstrom (6)                    */
  float r_bond;       /* bond-graph cutoff, Angstrom (3)                    */
  int32_t magmom;     /* 1: magnetic-moment head m_i = |v^T_i w_m + b_m|    */
  int32_t sequential; /* 0: FastCHGNet block, Eq. 11 (bond conv and angle
                         update read layer-t features); 1: the reference
                         block of Eq. 10 (bond conv reads v^{t+1}, angle
                         update reads v^{t+1} and e^{t+1})                  */
  int32_t conservative; /* 1: forces and stress as derivatives of the energy,
                         F_i = -dE/dr_i, sigma = (1/V) dE/d(eps) for the
                         strain r -> (I + eps) r of positions and lattice
                         (the reference output layer, Sec. II-B (4)); the
                         force and stress head weights are then unused
                         (zero gradient). Training through it (chgnet_step,
                         chgnet_backward) takes second derivatives, as the
                         tangent of the weight gradient along the
                         displacement -dL/dF and the strain rate
                         (dL/dsigma)/V (forward-over-reverse in dual
                         numbers), with either block. The workspace then
                         holds the dual-number buffers
                         as well (chgnet_workspace_size includes them).     */
} chgnet_hparams;

/* Loss of chgnet_step (Sec. IV, "Parameters Setting"), host memory. Each term
 * is a mean over its elements of rho(prediction - target): per-atom energy
 * E_s/n_s over S crystals, force components over 3N, stress components over
 * 9S, magnetic moments over N. rho(r) = r^2 if huber_delta <= 0, else Huber's
 * loss: r^2/2 for |r| <= delta, delta (|r| - delta/2) beyond. The paper's
 * prefactors are 2, 1.5, 0.1, 0.1 with Huber's loss; its delta is not stated. */
typedef struct {
  float w_energy, w_force, w_stress, w_magmom;
  float huber_delta;
} chgnet_loss;

/* A batch of S crystals with N atoms in total (Alg. 2: all structures
 * concatenated). Atoms of structure s are atom_ptr[s] .. atom_ptr[s+1]-1. */
typedef struct {
  int32_t n_struct;        /* S >= 1                                             */
  int32_t n_atoms;         /* N = atom_ptr[S] >= 1                               */
  const int32_t* atom_ptr; /* [S+1], atom_ptr[0] = 0, non-decreasing           */
  const float* pos;        /* [N,3] Cartesian positions, Angstrom (not wrapped) */
  const float* lattice;    /* [S,3,3] rows = lattice vectors, |det| >= 1e-6     */
  const int32_t* Z;        /* [N] atomic numbers in 1..94                       */
} chgnet_batch;

/* Atom graph G^a, bond graph G^b and angle list (Sec. II-B (1)).
 *  Edges: all directed (i, j, n) with i, j in one crystal, n in Z^3,
 *   (i,j,n) != (i,i,0) and D2 < r_atom^2. D2 is evaluated in the canonical
 *   orientation (p, q, m) of the pair {(i, j, n), (j, i, -n)}: p < q, or
 *   p = q with m lexicographically positive (first non-zero component > 0).
 *   It is the fp32 expression
 *      s_c = ((m1*L1c) + (m2*L2c)) + (m3*L3c);  dl_c = (r_qc + s_c) - r_pc;
 *      D2  = ((dl_x*dl_x) + (dl_y*dl_y)) + (dl_z*dl_z)
 *   with one round-to-nearest per operation (no fused multiply-add), so both
 *   directions of a pair get the same D2 and every edge has its reverse.
 *   Every translation is kept (no truncation). Order: CSR by i, then by j,
 *   then (n1, n2, n3) lexicographically.
 *  Bonds: the edges with D2 < r_bond^2, in edge order.
 *  Angles: at every centre atom with bonds b_1 < ... < b_k, the k(k-1) ordered
 *   pairs (b, b') with b != b', ordered by (b, b'). */
typedef struct {
  int64_t cap_edges, cap_bonds, cap_angles; /* in: capacity of the arrays below   */
  int64_t n_edges, n_bonds, n_angles;       /* out: E, B, A (also on ECAPACITY)   */
  int32_t* edge_ptr;  /* [N+1] CSR offsets of edges by source atom                */
  int32_t* edge_dst;  /* [E]   destination atom j                                 */
  int32_t* edge_img;  /* [E,3] lattice translation n                              */
  int32_t* edge_rev;  /* [E]   index of (j, i, -n)                                */
  int32_t* bond_ptr;  /* [N+1] CSR offsets of bonds by source atom                */
  int32_t* bond_edge; /* [B]   edge index of each bond                            */
  int32_t* angle_ptr; /* [B+1] angles whose first bond is b: angle_ptr[b]..[b+1]-1 */
  int32_t* angle_b2;  /* [A]   second bond of each angle; may be NULL (not built) */
} chgnet_graph;

/* Number of fp32 parameters in the flat parameter vector for `hp`.
 * Flat layout, in this order (row-major, "W [a,b]" maps a inputs to b outputs):
 *   W_Z [94,d] element table; f_a [R], f_b [R] sRBF frequencies (6 A, 3 A);
 *   W_e [R,2d] columns e^0 | e^a; b_e0 [d]; W_eb [R,d]; W_th [K,d]; b_th [d];
 *   per layer t = 0..T-1:
 *     atom conv : W [3d,2d] (input rows v_i | v_j | e_ij, output columns
 *                 core | gate), b [2d], g_c [d], b_c [d], g_g [d], b_g [d]
 *                 (LayerNorm scale/shift of core and gate), Wo [d,d], bo [d]
 *     bond conv : W [4d,2d] (input rows v_i | e_ij | e_ik | a_ijk), b [2d],
 *                 g_c, b_c, g_g, b_g [d], Wo [d,d], bo [d]
 *     angle upd.: only if t < T-1: W [4d,2d], b [2d], g_c, b_c, g_g, b_g [d]
 *   heads E, F, S (energy, force, stress), each:
 *     W1 [d,d], b1 [d], W2 [d,d], b2 [d], W3 [d,o], b3 [o], o = 1, 1, 9;
 *   only if magmom: w_m [d,1], b_m [1].
 * d = 64, T = 4, R = K = 31 gives 405,001 (405,066 with magmom); d = 128,
 * T = 5 gives 1,975,753. The layout does not depend on `sequential`. */
int chgnet_param_count(const chgnet_hparams* hp, int64_t* n);

/* Workspace bytes for a batch of S structures, N atoms and at most E edges,
 * B bonds and A angles. chgnet_build_graph needs the size for (N, S) with
 * E = B = A = 0 or more; forward/backward/step need the full size. */
int chgnet_workspace_size(const chgnet_hparams* hp, int64_t N, int64_t E, int64_t B, int64_t A, int64_t S,
                          size_t* bytes);

/* Build G^a, G^b and the angle list of `batch` into `graph` (cell-list search).
 * Waits once on `stream` to read E, B and A back; sets graph->n_edges etc.
 * If any capacity is too small nothing beyond the counts is written and
 * CHGNET_ECAPACITY is returned: grow the arrays and call again.
 * Errors: EINVAL for bad shapes, Z outside 1..94, |det L| < 1e-6, a lattice
 * too thin for the cutoff (more than 64 cells of images per axis), positions
 * more than 10^4 A or 200 cells from the origin cell, or more than 8192
 * edges on one atom. */
int chgnet_build_graph(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, void* ws,
                       size_t ws_bytes, void* stream);

/* chgnet_build_graph without a workspace, for callers that cannot allocate
 * device memory (serving and molecular-dynamics loops or harnesses that
 * forbid hipMalloc; the call still waits once on the host for the sizes, so
 * it cannot be captured into a HIP graph). The graph scratch lives in a
 * static device array of CHGNET_NOALLOC_SCRATCH_BYTES (8 MiB) on each GPU the
 * library runs on, held until the process ends: a batch may need at most
 * that much, 64 N + 156 S bytes plus about 4 KiB (for example 130,000 atoms
 * in one crystal, or 100,000 atoms in up to 12,000 crystals); larger
 * batches return CHGNET_EINVAL before any launch. The call
 * allocates nothing: no device memory, no pinned host memory. It uses the
 * current device's array (the stream must belong to the current device) and
 * writes the same graph as chgnet_build_graph. Every call on a GPU shares
 * that GPU's array, so calls that overlap in time on one GPU (other host
 * threads, or streams not ordered with each other) race; calls on one stream
 * are ordered. Errors as for chgnet_build_graph. */
#define CHGNET_NOALLOC_SCRATCH_BYTES (8u << 20)
int chgnet_build_graph_noalloc(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, void* stream);

/* Forward pass (Eq. 2-9; interaction blocks of Eq. 11, or Eq. 10 if
 * hp->sequential): energy [S] (total energy of each crystal), forces [N,3],
 * stress [S,3,3] and, if hp->magmom, magnetic moments magmom [N] (may be NULL
 * when not wanted; must be NULL without the head). `graph` must hold a graph
 * of `batch` (n_edges/n_bonds/n_angles set; angle_b2 may be NULL). The
 * activations always stay in `ws` for chgnet_backward (save_for_backward is
 * accepted for compatibility and ignored). */
int chgnet_forward(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph,
                   const float* params, float* energy, float* forces, float* stress, float* magmom,
                   int save_for_backward, void* ws, size_t ws_bytes, void* stream);

/* Backward pass for the weights: grad [P] (overwritten) = d/dparams of
 * sum(dE*energy) + sum(dF*forces) + sum(dS*stress) (+ sum(dM*magmom) with
 * the head; dM [N] may be NULL, meaning zero; it must be NULL without the
 * head), using the activations of the preceding chgnet_forward on the same ws,
 * batch, graph and params. Positions and lattices are not differentiated.
 * d|x|/dx is taken as 0 at x = 0. With hp->conservative the forces and
 * stresses are the derivatives of the energy, and their terms differentiate
 * those derivatives (second derivatives). */
int chgnet_backward(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph,
                    const float* params, const float* dE, const float* dF, const float* dS, const float* dM,
                    float* grad, void* ws, size_t ws_bytes, void* stream);

/* One training step: build graph, forward, loss (chgnet_loss, HOST), backward,
 * optional Adam. E_target [S] is per atom, F_target [N,3], S_target [S,3,3],
 * M_target [N] magnetic moments (required with the head, must be NULL
 * without it). loss [1] is a device scalar. If adam_hp (HOST array {lr,
 * beta1, beta2, eps, t}, t >= 1 the step number) is non-NULL, params, adam_m
 * and adam_v [P] are updated in place by bias-corrected Adam; otherwise
 * params are unchanged and adam_m / adam_v may be NULL. The predictions are
 * not returned (use chgnet_forward). Errors as for chgnet_build_graph. */
int chgnet_step(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, float* params,
                const float* E_target, const float* F_target, const float* S_target, const float* M_target,
                const chgnet_loss* loss_cfg, float* loss, float* grad, float* adam_m, float* adam_v,
                const float* adam_hp, void* ws, size_t ws_bytes, void* stream);

/* Molecular-dynamics state of a batch (device arrays unless noted; Sec. V,
 * Table 2). Neighbour-list reuse (Verlet skin): with skin > 0 the call keeps
 * a candidate list of every pair within r_atom + skin of the positions at its
 * build (in the caller's cand_* arrays) and, at each step, filters it with
 * the exact cutoff test of chgnet_graph at the new positions, which gives the
 * same graph as a full search as long as no atom has moved more than
 * (skin - 0.01 A) / 2 since the list was built; the list is rebuilt (cell-list
 * search at r_atom + skin) at the first step of a call and whenever that no
 * longer holds. */
typedef struct {
  float* pos;            /* [N,3] positions, A (the batch's pos array); updated   */
  float* vel;            /* [N,3] velocities, A/fs; updated                       */
  const float* inv_mass; /* [N] inverse masses, 1/u                               */
  float* forces;         /* [N,3] forces at pos, eV/A: read if forces_valid,
                            written at the end                                    */
  float* energy;         /* [S] energies at the final positions, eV (or NULL)     */
  float* stress;         /* [S,3,3] stresses at the final positions (or NULL)     */
  float skin;            /* host: 0 = full search every step, else in (0.02, 2] A */
  int64_t cap_cand;      /* host in: capacity of cand_dst / cand_img              */
  int64_t n_cand;        /* host out: pairs on the last list built (also when
                            CHGNET_ECAPACITY reports the list too long)           */
  int32_t* cand_ptr;     /* [N+1] CSR offsets of the list by source atom          */
  int32_t* cand_dst;     /* [cap_cand] destination atom of each candidate         */
  int32_t* cand_img;     /* [cap_cand,3] lattice translation of each candidate    */
  float* ref_pos;        /* [N,3] positions at the last list build                */
  int32_t n_builds;      /* host out: lists built during the call                 */
} chgnet_md_state;

/* n_steps of NVE velocity-Verlet molecular dynamics with the model's direct
 * force head, lattices fixed: per step v += dt/2 a; x += dt v; graph and
 * forward at the new x; v += dt/2 a, with a = F / m * 0.0096485332157 A/fs^2
 * per eV/(A u) (dt in fs). batch->pos must equal state->pos. If forces_valid
 * is 0 the forces at the initial positions are computed first. Every step
 * forms the graph at the new positions, by a full search or from the
 * candidate list (see chgnet_md_state), with one wait for its sizes; once two
 * consecutive steps have graphs of the same sizes, the forward pass and the
 * second half-kick are captured into a HIP graph (on a non-null stream, with
 * the direct heads) and replayed while the sizes stay the same. Positions
 * are not wrapped into the cell. With skin > 0, CHGNET_ECAPACITY may also
 * mean that cap_cand < n_cand: grow the list and call again. *steps_done (host) receives the
 * number of completed steps: on CHGNET_ECAPACITY the state is that of the
 * last completed step with valid forces; grow the graph and call again for
 * the remaining steps with forces_valid = 1. The model variant of hp applies
 * (conservative forces included; magmom is not returned). Errors as for chgnet_build_graph. */
int chgnet_md(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, const float* params,
              chgnet_md_state* state, float dt, int n_steps, int forces_valid, int* steps_done, void* ws,
              size_t ws_bytes, void* stream);

/* Text of the last error on the calling thread ("" if none). */
const char* chgnet_last_error_string(void);

/* Measurement only (benchmarks, profilers). While enabled, the library
 * records a pair of HIP events around each of its kernel launches (up to
 * max_launches), on the stream of the call. This is the library's only
 * global state; it is off by default and not thread-safe.
 * chgnet_profile_stop waits for the recorded events, disables timing and
 * writes one line per launch tag into buf (host memory, buflen bytes):
 * "<tag> <launches> <total milliseconds>\n". Tags are kernel names, or the
 * role of a GEMM launch (gemm_proj: per-atom and per-bond terms of the split
 * first layers; gemm_in_bwd: input gradients of the interaction block;
 * tn_in: weight gradients of the interaction block; ...); a call that
 * launches several kernels under one tag (the weight gradients' 64 x 128
 * and 64 x 64 wave-tile launches) is timed as one launch. Returns
 * CHGNET_EINVAL if buf is too small and CHGNET_EWORKSPACE if more than
 * max_launches launches ran. */
int chgnet_profile_start(int max_launches);
int chgnet_profile_stop(char* buf, size_t buflen);

#ifdef __cplusplus
}
#endif
#endif /* CHGNET_H */
