// FastCHGNet forward, loss and weight backward on gfx950.
//
// Layer t follows Eq. (4)-(6) with the dependency-free inputs of Eq. (11):
// atom conv, bond conv and angle update all read (v^t, e^t, a^t). The
// GatedMLP inputs are concatenations [v_i, v_j, e_ij] and
// [v_i, e_ij, e_ik, a_ijk]; their first linear layer is split by input block
// so that only the edge term (e W) and the angle term (a W) are computed per
// edge / per angle, while the atom and bond terms are computed once per atom
// and per bond and gathered in the GEMM epilogue. Bond conv and angle update
// share their input (Eq. (11)) and their two weight blocks form one product.
//
// Aggregations are segmented sums over CSR ranges (edges by source atom,
// angles by first bond), one wavefront per segment, in a fixed order: no
// floating-point atomics anywhere, so results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "common.hpp"
#include "gemm.hpp"

namespace chg {

size_t graph_scratch_bytes(int64_t N, int64_t S);
int build_graph(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, void* ws, size_t ws_bytes,
                hipStream_t st);
int validate_batch(const chgnet_batch* b);

namespace {

constexpr float kLnEps = 1e-5f;
constexpr int kFreqRowsPerBlock = 64;  // rows per block in frequency-gradient kernel
constexpr int kReduceGroups = 32;      // first-level groups of the ordered partial-sum reduction
constexpr int64_t kTnPartFloats = 64ll << 20;

// logistic sigmoid; the hardware reciprocal (about 1 ulp) instead of an IEEE division
__device__ __forceinline__ float sigm(float x) { return __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }

__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <class T>
__device__ __forceinline__ int upper_bound_idx(const T* ptr, int n, T x) {
  // largest s in [0, n) with ptr[s] <= x (ptr non-decreasing, ptr[0] <= x)
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (ptr[mid] <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ void k_fill(float* __restrict__ p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

constexpr int kPackTensors = 128, kPackChunk = 2048;
struct PackTable {
  int n;
  int src[kPackTensors], dst[kPackTensors], len[kPackTensors];
  int chunk0[kPackTensors + 1];  // first chunk of each tensor; chunk0[n] = total
};

// Copy of the flat parameters with every tensor on a 16-byte boundary; one
// block per chunk of kPackChunk values of one tensor.
__global__ void __launch_bounds__(256) k_pack_params(PackTable t, const float* __restrict__ src, float* __restrict__ dst) {
  const int b = blockIdx.x;
  int lo = 0, hi = t.n;  // tensor k with chunk0[k] <= b < chunk0[k + 1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) / 2;
    if (t.chunk0[mid] <= b) lo = mid;
    else hi = mid;
  }
  const int base = (b - t.chunk0[lo]) * kPackChunk;
  const int n = min(kPackChunk, t.len[lo] - base);
  const float* s = src + t.src[lo] + base;
  float* d = dst + t.dst[lo] + base;
  for (int i = threadIdx.x; i < n; i += 256) d[i] = s[i];
}

// dst = src, n4 float4 values (16-byte aligned arrays), grid-stride
__global__ void __launch_bounds__(256) k_copy4(float4* __restrict__ dst, const float4* __restrict__ src, int64_t n4) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) dst[i] = src[i];
}

// ---------------------------------------------------------------------------
// Geometry (fp64) and basis expansions (Eq. 2, Alg. 2: whole batch at once).
// ---------------------------------------------------------------------------
// sRBF_n(r) = sqrt(2/c) sin(f_n r / c) / r * u(r / c), u the polynomial envelope.
__device__ __forceinline__ float envelope(float x, int p) {
  const float a = -0.5f * (p + 1) * (p + 2), b = (float)(p * (p + 2)), c = -0.5f * p * (p + 1);
  float xp = 1.0f;
  for (int k = 0; k < p; ++k) xp *= x;
  return 1.0f + xp * (a + x * (b + x * c));
}
__device__ __forceinline__ float srbf(float f, float d, float inv_c, int p) {
  return sqrtf(2.0f * inv_c) * sinf(f * d * inv_c) / d * envelope(d * inv_c, p);
}

// Cartesian vector from atom i to the image n of atom j (fp64).
__device__ __forceinline__ void edge_vector(int i, int j, const int* __restrict__ img, const float* __restrict__ L,
                                            const float* __restrict__ pos, double (&r)[3]) {
  const double n0 = img[0], n1 = img[1], n2 = img[2];
  for (int c = 0; c < 3; ++c)
    r[c] = (double)pos[3 * j + c] + (n0 * (double)L[c] + n1 * (double)L[3 + c] + n2 * (double)L[6 + c]) - (double)pos[3 * i + c];
}

// Geometry, bases and the atom embedding of a batch in one launch, by block
// range: atoms (structure index, v0 = W_Z[Z - 1]); edges, 256 a block
// (source atom, length, unit vector, then the block's sRBF rows at the atom
// cutoff); angles (first and second bond, centre atom; cos/sin of theta from
// (dot, |cross|) in fp64 and the Fourier basis by the complex-power
// recurrence (cos m t + i sin m t) = (cos t + i sin t)^m).
struct GeomArgs {
  int N, S, E, B, A, D, R, K, p, nb_atoms, nb_edges;
  float inv_ca;
  const int *atom_ptr, *Z, *edge_ptr, *edge_dst, *edge_img, *bond_ptr, *bond_edge, *angle_ptr;
  const float *pos, *lattice, *WZ, *freq_a;
  int *atom_struct, *edge_src, *ang_b1, *ang_b2, *ang_ctr;
  float *v0, *edge_len, *edge_xhat, *rbf_a, *ft;
};

__global__ void __launch_bounds__(256) k_geom(GeomArgs g) {
  __shared__ float dl[256];
  int blk = blockIdx.x;
  const int tid = threadIdx.x;
  if (blk < g.nb_atoms) {
    const int64_t t = (int64_t)blk * 256 + tid;
    if (t >= (int64_t)g.N * g.D) return;
    const int i = (int)(t / g.D), c = (int)(t % g.D);
    g.v0[t] = g.WZ[(int64_t)(g.Z[i] - 1) * g.D + c];
    if (c == 0) g.atom_struct[i] = upper_bound_idx(g.atom_ptr, g.S + 1, i);
    return;
  }
  blk -= g.nb_atoms;
  if (blk < g.nb_edges) {
    const int e0 = blk * 256, e = e0 + tid;
    float d = 1.0f;
    if (e < g.E) {
      const int i = upper_bound_idx(g.edge_ptr, g.N + 1, e);
      const int j = g.edge_dst[e];
      double r[3];
      edge_vector(i, j, g.edge_img + 3 * e, g.lattice + 9 * upper_bound_idx(g.atom_ptr, g.S + 1, i), g.pos, r);
      const double dd = sqrt(r[0] * r[0] + r[1] * r[1] + r[2] * r[2]);
      g.edge_src[e] = i;
      d = (float)dd;
      g.edge_len[e] = d;
      for (int c = 0; c < 3; ++c) g.edge_xhat[3 * e + c] = (float)(r[c] / dd);
    }
    dl[tid] = d;
    __syncthreads();
    const int ne = min(256, g.E - e0);
    float* out = g.rbf_a + (int64_t)e0 * g.R;
    for (int t = tid; t < ne * g.R; t += 256) out[t] = srbf(g.freq_a[t % g.R], dl[t / g.R], g.inv_ca, g.p);
    return;
  }
  blk -= g.nb_edges;
  const int a0 = blk * 256, al = a0 + tid;
  const int na = min(256, g.A - a0);
  // the block's Fourier rows go through LDS, so that they are written as
  // one contiguous run
  __shared__ float fts[256 * 32];
  if (al < g.A) {
    const int b1 = upper_bound_idx(g.angle_ptr, g.B + 1, al);
    const int i = upper_bound_idx(g.bond_ptr, g.N + 1, b1);
    const int k0 = g.bond_ptr[i];
    const int p = b1 - k0;
    const int q0 = al - g.angle_ptr[b1];
    const int b2 = k0 + (q0 < p ? q0 : q0 + 1);
    g.ang_b1[al] = b1;
    g.ang_b2[al] = b2;
    g.ang_ctr[al] = i;
    const float* L = g.lattice + 9 * upper_bound_idx(g.atom_ptr, g.S + 1, i);
    double r[2][3];
    const int es[2] = {g.bond_edge[b1], g.bond_edge[b2]};
    for (int s = 0; s < 2; ++s) edge_vector(i, g.edge_dst[es[s]], g.edge_img + 3 * es[s], L, g.pos, r[s]);
    const double dot = r[0][0] * r[1][0] + r[0][1] * r[1][1] + r[0][2] * r[1][2];
    const double cx = r[0][1] * r[1][2] - r[0][2] * r[1][1];
    const double cy = r[0][2] * r[1][0] - r[0][0] * r[1][2];
    const double cz = r[0][0] * r[1][1] - r[0][1] * r[1][0];
    const double cr = sqrt(cx * cx + cy * cy + cz * cz);
    const double h = sqrt(dot * dot + cr * cr);
    const double c1 = dot / h, s1 = cr / h;
    const int M = (g.K - 1) / 2;
    // n_fourier up to 32 is staged (the default 31); longer rows go straight out
    float* o = g.K <= 32 ? fts + tid * g.K : g.ft + (int64_t)al * g.K;
    const double inv_sqrt_pi = 0.56418958354775628695;
    o[0] = (float)(inv_sqrt_pi * 0.70710678118654752440);
    double cm = 1.0, sm = 0.0;
    for (int m = 1; m <= M; ++m) {
      const double cn = cm * c1 - sm * s1, sn = sm * c1 + cm * s1;
      cm = cn;
      sm = sn;
      o[m] = (float)(cm * inv_sqrt_pi);
      o[M + m] = (float)(sm * inv_sqrt_pi);
    }
  }
  if (g.K > 32) return;  // uniform over the block
  __syncthreads();
  float* out = g.ft + (int64_t)a0 * g.K;
  for (int t = tid; t < na * g.K; t += 256) out[t] = fts[t];
}

// Per bond (256 a block): source atom and the block's sRBF rows at the bond
// cutoff (from the edge lengths).
__global__ void __launch_bounds__(256) k_bond_geom(int B, int R, int p, float inv_c, const int* __restrict__ bond_edge,
                                                   const int* __restrict__ edge_src, const float* __restrict__ edge_len,
                                                   const float* __restrict__ freq, int* __restrict__ bond_src,
                                                   float* __restrict__ rbf_b) {
  __shared__ float dl[256];
  const int b0 = blockIdx.x * 256, b = b0 + threadIdx.x;
  float d = 1.0f;
  if (b < B) {
    const int e = bond_edge[b];
    bond_src[b] = edge_src[e];
    d = edge_len[e];
  }
  dl[threadIdx.x] = d;
  __syncthreads();
  const int nbk = min(256, B - b0);
  float* out = rbf_b + (int64_t)b0 * R;
  for (int t = threadIdx.x; t < nbk * R; t += 256) out[t] = srbf(freq[t % R], dl[t / R], inv_c, p);
}

// ---------------------------------------------------------------------------
// GatedMLP rows: phi = SiLU(LN_c(z_c)) * sigmoid(LN_g(z_g)).
// A row is held by LPR = d/CPL adjacent lanes with CPL core columns and the
// CPL matching gate columns each. Lane j of a row owns the float4 chunks at
// columns q*4*LPR + 4j (q < CPL/4), so one float4 load of a wavefront reads
// 4*LPR contiguous columns of every row it touches. LayerNorm statistics are
// sums over the LPR lanes by DPP permutes (no LDS traffic). A wavefront works
// on 64/LPR rows at a time.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <int LPR>
__device__ __forceinline__ float rowsum(float v) {
  static_assert(LPR == 4 || LPR == 8 || LPR == 16, "row of 4, 8 or 16 lanes");
  v += dpp<0xB1>(v);  // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);  // quad_perm [2,3,0,1]
  if (LPR >= 8) v += dpp<0x141>(v);   // row_half_mirror: pairs the two quads of 8 lanes
  if (LPR == 16) v += dpp<0x140>(v);  // row_mirror: pairs the two halves of 16 lanes
  return v;
}

template <int D, int CPL>
struct Lanes {
  static constexpr int LPR = D / CPL;   // lanes per row
  static constexpr int RPW = 64 / LPR;  // rows per wavefront pass
  static constexpr int NQ = CPL / 4;    // float4 chunks per lane
  static constexpr int STRIDE = 4 * LPR;
  // column of the lane's k-th value (lane j within its row)
  static __device__ __forceinline__ int col(int j, int k) { return (k >> 2) * STRIDE + 4 * j + (k & 3); }
};

template <int D, int CPL>
__device__ __forceinline__ void load_cols(const float* __restrict__ p, int j, float (&v)[CPL]) {
#pragma unroll
  for (int q = 0; q < CPL / 4; ++q) {
    const float4 t = *reinterpret_cast<const float4*>(p + q * Lanes<D, CPL>::STRIDE + 4 * j);
    v[4 * q] = t.x;
    v[4 * q + 1] = t.y;
    v[4 * q + 2] = t.z;
    v[4 * q + 3] = t.w;
  }
}
template <int D, int CPL>
__device__ __forceinline__ void store_cols(float* __restrict__ p, int j, const float (&v)[CPL]) {
#pragma unroll
  for (int q = 0; q < CPL / 4; ++q)
    *reinterpret_cast<float4*>(p + q * Lanes<D, CPL>::STRIDE + 4 * j) =
        make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
}

// Streaming variants for data touched once here and not again soon (the
// pre-activations saved for the backward pass, the copy into e^{t+1}):
// nontemporal accesses keep them from displacing cached table rows.
typedef float v4f __attribute__((ext_vector_type(4)));
template <int D, int CPL>
__device__ __forceinline__ void load_cols_nt(const float* __restrict__ p, int j, float (&v)[CPL]) {
#pragma unroll
  for (int q = 0; q < CPL / 4; ++q) {
    const v4f t = __builtin_nontemporal_load(reinterpret_cast<const v4f*>(p + q * Lanes<D, CPL>::STRIDE + 4 * j));
    v[4 * q] = t.x;
    v[4 * q + 1] = t.y;
    v[4 * q + 2] = t.z;
    v[4 * q + 3] = t.w;
  }
}
template <int D, int CPL>
__device__ __forceinline__ void store_cols_nt(float* __restrict__ p, int j, const float (&v)[CPL]) {
#pragma unroll
  for (int q = 0; q < CPL / 4; ++q) {
    const v4f t = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
    __builtin_nontemporal_store(t, reinterpret_cast<v4f*>(p + q * Lanes<D, CPL>::STRIDE + 4 * j));
  }
}

// Normalised core/gate (xc, xg) and 1/std (rc, rg) of one row; in place.
template <int D, int CPL>
__device__ __forceinline__ void ln_stats(float (&zc)[CPL], float (&zg)[CPL], float& rc, float& rg) {
  constexpr int LPR = Lanes<D, CPL>::LPR;
  float sc = 0.f, sg = 0.f;
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    sc += zc[k];
    sg += zg[k];
  }
  const float mc = rowsum<LPR>(sc) * (1.0f / D), mg = rowsum<LPR>(sg) * (1.0f / D);
  float vc = 0.f, vg = 0.f;
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    zc[k] -= mc;
    zg[k] -= mg;
    vc += zc[k] * zc[k];
    vg += zg[k] * zg[k];
  }
  // the argument is at least the LayerNorm epsilon: the hardware reciprocal
  // square root needs no denormal scaling
  rc = __builtin_amdgcn_rsqf(rowsum<LPR>(vc) * (1.0f / D) + kLnEps);
  rg = __builtin_amdgcn_rsqf(rowsum<LPR>(vg) * (1.0f / D) + kLnEps);
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    zc[k] *= rc;
    zg[k] *= rg;
  }
}

struct LnPtrs {
  const float *gc, *bc, *gg, *bg;
};

// Gathered terms of the split first linear layer: z = z_pre + sum_q
// add[q][idx_q[row]] (each a 2d-wide core | gate row), at most two (atom
// conv: source and destination atom; angle gates: first bond with its centre
// atom folded in, and second bond).
constexpr int kMaxAdds = 2;
struct GateAdds {
  int n;
  const float* p[kMaxAdds];
  int ld[kMaxAdds];
  const int* idx[kMaxAdds];
};

template <int D, int CPL>
__device__ __forceinline__ void load_z(const float* __restrict__ z, int ldz, int row, int j, float (&zc)[CPL],
                                       float (&zg)[CPL]) {
  load_cols_nt<D, CPL>(z + (int64_t)row * ldz, j, zc);
  load_cols_nt<D, CPL>(z + (int64_t)row * ldz + D, j, zg);
}

// Columns per lane of the row-layout backward gate.
constexpr int kBwdCpl = 8;

enum GateFwdMode { FWD_ATOM = 0, FWD_BOND = 1, FWD_ANGLE = 2 };

// Forward gate modes:
//   FWD_ATOM : out[row] = e^a[row] * phi            (atom conv message)
//   FWD_BOND : out[row] = e^b[b2[row]] * phi        (bond conv message)
//   FWD_ANGLE: out[row] = a[row] + phi              (angle update)

// Forward gate with its own pre-activation product: z = x W + b (+ the
// gathered terms) is formed tile by tile in LDS and never round-trips
// through HBM. Producer wave w keeps the fp32 MFMA B fragments of output
// columns [32w, 32w + 32) of W (d x 2d: core | gate) in registers; the x
// tile is staged in LDS; each producer forms its rows x 32 slice of z with
// 32x32x2 MFMAs (lane half h supplies k = 16h + i in step i of each 32-wide
// k block) and writes it to the z tile; the consumers' row-layout gate then
// reads z from LDS. d = 64: 64-row tiles, 4 producer and 8 consumer
// wavefronts; d = 128: 32-row tiles, 8 producers (256 columns) and 8
// consumers, 16 wavefronts of at most 128 VGPRs.
typedef float v16f __attribute__((ext_vector_type(16)));

struct GateMmJob {
  int mode, rows, tile0;
  const float* x;  // [rows, d]
  const float* W;  // [d, 2d] core | gate columns, row stride ldw
  int ldw;
  const float* bias;  // [2d]
  GateAdds ad;
  LnPtrs ln;
  const float* mulv;
  const int* mul_idx;
  float* out;
  float* zsave;  // optional [rows, ldzs]: the whole pre-activation z, kept for the backward pass
  int ldzs;
  float* xcopy;  // optional [rows, d]: a copy of x (the residual part of e^{t+1})
};
struct GateMmJobs {
  int n, ntiles;
  GateMmJob j[3];
};

constexpr int kMmCpl = 8;

// Wave priority of the consumer wavefronts in the fused gate kernels. The
// consumers' chains of dependent loads set the pace of a tile; ahead of the
// producers' MFMA stream in instruction issue they finish sooner (measured
// at d = 128: backward 1.34 -> 1.14 ms and forward 1.01 -> 0.96 ms per layer
// launch), while the producers, with a tile of slack, lose nothing.
constexpr int kConsumerPrio = 2;

template <int D>
struct MmCfg {
  static constexpr int Rows = D == 64 ? 64 : 32;  // rows per tile
  static constexpr int Prod = 2 * D / 32;         // producer waves: 32 z columns each
  static constexpr int Cons = 8;                  // consumer waves
  static constexpr int Threads = 64 * (Prod + Cons);
  static constexpr int Xld = D + 4;
  static constexpr int Zld = 2 * D + 4;
  static constexpr int KB = D / 32;    // 32-deep k blocks
  static constexpr int RS = Rows / 32;  // 32-row subtiles
  // x tile loads: every producer thread moves F floats of one row
  static constexpr int F = Rows * D / (64 * Prod);
  static constexpr int TPR = D / F;  // threads per x row
  static_assert(Cons * Lanes<D, kMmCpl>::RPW == Rows, "one consumer pass per tile");
  static_assert(F % 4 == 0 && Rows * TPR == 64 * Prod, "x tile split");
};
// kept for the backward gate kernel (d = 64 only)
constexpr int kMmRows = MmCfg<64>::Rows;
constexpr int kMmProducers = MmCfg<64>::Prod, kMmConsumers = MmCfg<64>::Cons;
constexpr int kMmThreads = MmCfg<64>::Threads;

// Gathered operands of one gate row (the atom/bond terms of the split first
// layer and the multiplier row), loaded one tile ahead of their use; the
// row indices are loaded one tile ahead of that.
struct GateRowIn {
  float ac[kMaxAdds][kMmCpl], ag[kMaxAdds][kMmCpl], mv[kMmCpl];
};

__device__ __forceinline__ void gate_mm_index(const GateMmJob& J, int row, int (&ix)[kMaxAdds + 1]) {
  const int r = min(row, J.rows - 1);
#pragma unroll
  for (int q = 0; q < kMaxAdds; ++q) ix[q] = q < J.ad.n ? J.ad.idx[q][r] : 0;
  ix[kMaxAdds] = J.mode == FWD_BOND ? J.mul_idx[r] : r;
}

template <int D>
__device__ __forceinline__ void gate_mm_gather(const GateMmJob& J, const int (&ix)[kMaxAdds + 1], GateRowIn& in) {
  constexpr int CPL = kMmCpl;
  const int j = (threadIdx.x & 63) % Lanes<D, CPL>::LPR;
#pragma unroll
  for (int q = 0; q < kMaxAdds; ++q) {
    if (q >= J.ad.n) break;
    const float* r = J.ad.p[q] + (int64_t)ix[q] * J.ad.ld[q];
    load_cols<D, CPL>(r, j, in.ac[q]);
    load_cols<D, CPL>(r + D, j, in.ag[q]);
  }
  load_cols<D, CPL>(J.mulv + (int64_t)ix[kMaxAdds] * D, j, in.mv);
}

// LayerNorm scale and shift (core and gate) of this lane's columns
struct GateLnRegs {
  float gc[kMmCpl], bc[kMmCpl], gg[kMmCpl], bg[kMmCpl];
};

template <int D, int MODE>
__device__ __forceinline__ void gate_mm_row(const GateMmJob& J, int row, int lr, const float* Zs, const GateRowIn& in,
                                            const GateLnRegs& ln) {
  constexpr int CPL = kMmCpl;
  using L = Lanes<D, CPL>;
  const int j = (threadIdx.x & 63) % L::LPR;
  if (row >= J.rows) return;
  float zc[CPL], zg[CPL], rc, rg;
  {
    // odd rows of the z tile hold the two 32-column halves of each 64-column
    // block swapped (written so by the producers): the two rows of a read
    // phase fall in different banks
    const float* zr = Zs + lr * MmCfg<D>::Zld;
    const int sw = (lr & 1) * 32;
#pragma unroll
    for (int q = 0; q < CPL / 4; ++q) {
      const int cc = (q * L::STRIDE + 4 * j) ^ sw;
      const float4 a = *reinterpret_cast<const float4*>(zr + cc);
      const float4 b = *reinterpret_cast<const float4*>(zr + D + cc);
      zc[4 * q] = a.x; zc[4 * q + 1] = a.y; zc[4 * q + 2] = a.z; zc[4 * q + 3] = a.w;
      zg[4 * q] = b.x; zg[4 * q + 1] = b.y; zg[4 * q + 2] = b.z; zg[4 * q + 3] = b.w;
    }
  }
#pragma unroll
  for (int q = 0; q < kMaxAdds; ++q) {
    if (q >= J.ad.n) break;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      zc[k] += in.ac[q][k];
      zg[k] += in.ag[q][k];
    }
  }
  if (J.zsave) {
    store_cols_nt<D, CPL>(J.zsave + (int64_t)row * J.ldzs, j, zc);
    store_cols_nt<D, CPL>(J.zsave + (int64_t)row * J.ldzs + D, j, zg);
  }
  ln_stats<D, CPL>(zc, zg, rc, rg);
  float o[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    const float yc = ln.gc[k] * zc[k] + ln.bc[k];
    const float yg = ln.gg[k] * zg[k] + ln.bg[k];
    const float phi = yc * sigm(yc) * sigm(yg);
    o[k] = MODE == FWD_ANGLE ? in.mv[k] + phi : in.mv[k] * phi;
  }
  store_cols<D, CPL>(J.out + (int64_t)row * D, j, o);
}

// Producer and consumer wavefronts: the producers form z of tile i (x tile
// and z tile double-buffered in LDS) while the consumers run the gate rows
// of tile i-1 and gather the operands of tile i; one block barrier per tile
// hands the buffers over. Producers and consumers run separate loops with
// the same number of block barriers, so each keeps only its own state.

// Producer pieces (threads 0 .. 64 Prod - 1). x tile loads: thread -> row
// tid / TPR, F columns at F (tid % TPR); rows past `rows` read as zero.
template <int D>
__device__ __forceinline__ void mm_fetch_x(const float* __restrict__ x, int rows, int row0,
                                           float4 (&v)[MmCfg<D>::F / 4]) {
  using C = MmCfg<D>;
  const int tid = threadIdx.x, row = row0 + tid / C::TPR, xc = C::F * (tid % C::TPR);
#pragma unroll
  for (int q = 0; q < C::F / 4; ++q) v[q] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (row < rows) {
    const float* p = x + (int64_t)row * D + xc;
#pragma unroll
    for (int q = 0; q < C::F / 4; ++q) v[q] = *reinterpret_cast<const float4*>(p + 4 * q);
  }
}
template <int D>
__device__ __forceinline__ void mm_store_x(float* X, const float4 (&v)[MmCfg<D>::F / 4]) {
  using C = MmCfg<D>;
  const int tid = threadIdx.x, xr = tid / C::TPR, xc = C::F * (tid % C::TPR);
#pragma unroll
  for (int q = 0; q < C::F / 4; ++q) *reinterpret_cast<float4*>(&X[xr * C::Xld + xc + 4 * q]) = v[q];
}
// the same x tile piece to global memory (rows past `rows` are skipped)
template <int D>
__device__ __forceinline__ void mm_copy_x(float* __restrict__ dst, int rows, int row0,
                                          const float4 (&v)[MmCfg<D>::F / 4]) {
  using C = MmCfg<D>;
  const int tid = threadIdx.x, row = row0 + tid / C::TPR, xc = C::F * (tid % C::TPR);
  if (row < rows) {
    float* p = dst + (int64_t)row * D + xc;
#pragma unroll
    for (int q = 0; q < C::F / 4; ++q) {
      const v4f t = {v[q].x, v[q].y, v[q].z, v[q].w};
      __builtin_nontemporal_store(t, reinterpret_cast<v4f*>(p + 4 * q));
    }
  }
}
// B fragments of W columns [32 wave, 32 wave + 32) and their bias
template <int D>
__device__ __forceinline__ void mm_load_w(const float* __restrict__ W, int ldw, const float* __restrict__ b, int wave,
                                          float (&bfr)[MmCfg<D>::KB][16], float& bias) {
  const int lane = threadIdx.x & 63, h = lane >> 5, col = 32 * wave + (lane & 31);
#pragma unroll
  for (int kb = 0; kb < MmCfg<D>::KB; ++kb)
#pragma unroll
    for (int e = 0; e < 16; ++e) bfr[kb][e] = W[(int64_t)(32 * kb + 16 * h + e) * ldw + col];
  bias = b[col];
}
// z slice (Rows x 32 columns) of one producer wave, X -> Z
template <int D>
__device__ __forceinline__ void mm_tile(const float* X, float* Z, const float (&bfr)[MmCfg<D>::KB][16], float bias,
                                        int wave) {
  using C = MmCfg<D>;
  const int lane = threadIdx.x & 63, h = lane >> 5, l32 = lane & 31;
  // the 32-row subtiles are independent accumulation chains
  v16f acc[C::RS];
#pragma unroll
  for (int s = 0; s < C::RS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[s][e] = 0.f;
#pragma unroll
  for (int kb = 0; kb < C::KB; ++kb) {
    float af[C::RS][16];
#pragma unroll
    for (int s = 0; s < C::RS; ++s) {
      const float* ap = &X[(32 * s + l32) * C::Xld + 32 * kb + 16 * h];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = *reinterpret_cast<const float4*>(ap + 4 * q);
        af[s][4 * q] = v.x; af[s][4 * q + 1] = v.y; af[s][4 * q + 2] = v.z; af[s][4 * q + 3] = v.w;
      }
    }
#pragma unroll
    for (int e = 0; e < 16; ++e)
#pragma unroll
      for (int s = 0; s < C::RS; ++s)
        acc[s] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[s][e], bfr[kb][e], acc[s], 0, 0, 0);
  }
#pragma unroll
  for (int s = 0; s < C::RS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      Z[(32 * s + 8 * (e >> 2) + 4 * h + (e & 3)) * C::Zld + ((32 * wave + l32) ^ ((e & 1) * 32))] = acc[s][e] + bias;
}

// One block per compute unit, walking tiles blockIdx.x, blockIdx.x +
// gridDim.x, ... of the concatenated jobs.
template <int D>
__global__ void __launch_bounds__(MmCfg<D>::Threads, 1) k_gate_fwd_mm(GateMmJobs J) {
  using C = MmCfg<D>;
  __shared__ __attribute__((aligned(16))) float Xs[2][C::Rows * C::Xld];
  __shared__ __attribute__((aligned(16))) float Zs[2][C::Rows * C::Zld];
  // LayerNorm parameters of every job: [job][gc, bc, gg, bg][d]
  __shared__ __attribute__((aligned(16))) float LnS[3][4][D];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int t = threadIdx.x; t < 3 * 4 * D; t += C::Threads) {
    const int jb = t / (4 * D), q = (t / D) % 4, c = t % D;
    if (jb < J.n) {
      const LnPtrs& ln = J.j[jb].ln;
      LnS[jb][q][c] = (q == 0 ? ln.gc : q == 1 ? ln.bc : q == 2 ? ln.gg : ln.bg)[c];
    }
  }
  auto job_of = [&](int tile) {
    int k = 0;
    while (k + 1 < J.n && tile >= J.j[k + 1].tile0) ++k;
    return k;
  };
  const int nt = (int)blockIdx.x < J.ntiles ? (J.ntiles - 1 - (int)blockIdx.x) / (int)gridDim.x + 1 : 0;
  if (nt == 0) return;
  auto tile_of = [&](int i) { return (int)blockIdx.x + i * (int)gridDim.x; };
  if (wave < C::Prod) {
    float4 xv[C::F / 4];
    auto fetch_x = [&](int tile) {
      const GateMmJob& jb = J.j[job_of(tile)];
      mm_fetch_x<D>(jb.x, jb.rows, (tile - jb.tile0) * C::Rows, xv);
    };
    auto copy_x = [&](int tile) {
      const GateMmJob& jb = J.j[job_of(tile)];
      if (jb.xcopy) mm_copy_x<D>(jb.xcopy, jb.rows, (tile - jb.tile0) * C::Rows, xv);
    };
    int cur = -1;
    float bfr[C::KB][16], bias = 0.f;
    fetch_x(tile_of(0));
    mm_store_x<D>(Xs[0], xv);
    copy_x(tile_of(0));
    if (nt > 1) fetch_x(tile_of(1));
    __syncthreads();
    for (int i = 0; i <= nt; ++i) {
      if (i < nt) {
        const int k = job_of(tile_of(i));
        if (k != cur) {
          cur = k;
          mm_load_w<D>(J.j[k].W, J.j[k].ldw, J.j[k].bias, wave, bfr, bias);
        }
        if (i + 1 < nt) {
          mm_store_x<D>(Xs[(i + 1) & 1], xv);
          copy_x(tile_of(i + 1));
          if (i + 2 < nt) fetch_x(tile_of(i + 2));
        }
        mm_tile<D>(Xs[i & 1], Zs[i & 1], bfr, bias, wave);
      }
      __syncthreads();
    }
  } else {
    __builtin_amdgcn_s_setprio(kConsumerPrio);
    // lane row within the tile; gathered operands of the next tile and row
    // indices of the one after
    using GL = Lanes<D, kMmCpl>;
    const int lr = (wave - C::Prod) * GL::RPW + lane / GL::LPR;
    auto row_of = [&](int tile, const GateMmJob& jb) { return (tile - jb.tile0) * C::Rows + lr; };
    GateRowIn in;
    GateLnRegs lnr;
    int lnjob = -1;
    int ix[kMaxAdds + 1];
    const GateMmJob& j0 = J.j[job_of(tile_of(0))];
    gate_mm_index(j0, row_of(tile_of(0), j0), ix);
    gate_mm_gather<D>(j0, ix, in);
    if (nt > 1) {
      const GateMmJob& j1 = J.j[job_of(tile_of(1))];
      gate_mm_index(j1, row_of(tile_of(1), j1), ix);
    }
    __syncthreads();
    for (int i = 0; i <= nt; ++i) {
      if (i > 0) {
        const int tile = tile_of(i - 1);
        const int k = job_of(tile);
        const GateMmJob& jb = J.j[k];
        if (k != lnjob) {
          lnjob = k;
          const int jl = lane % GL::LPR;
          load_cols<D, kMmCpl>(LnS[k][0], jl, lnr.gc);
          load_cols<D, kMmCpl>(LnS[k][1], jl, lnr.bc);
          load_cols<D, kMmCpl>(LnS[k][2], jl, lnr.gg);
          load_cols<D, kMmCpl>(LnS[k][3], jl, lnr.bg);
        }
        const int row = row_of(tile, jb);
        const float* Z = Zs[(i - 1) & 1];
        if (jb.mode == FWD_ATOM) gate_mm_row<D, FWD_ATOM>(jb, row, lr, Z, in, lnr);
        else if (jb.mode == FWD_BOND) gate_mm_row<D, FWD_BOND>(jb, row, lr, Z, in, lnr);
        else gate_mm_row<D, FWD_ANGLE>(jb, row, lr, Z, in, lnr);
        if (i < nt) {
          const GateMmJob& jn = J.j[job_of(tile_of(i))];
          gate_mm_gather<D>(jn, ix, in);
          if (i + 1 < nt) {
            const GateMmJob& jm = J.j[job_of(tile_of(i + 1))];
            gate_mm_index(jm, row_of(tile_of(i + 1), jm), ix);
          }
        }
      }
      __syncthreads();
    }
  }
}

enum GateBwdMode { BWD_ATOM = 0, BWD_BOND = 1, BWD_ANGLE = 2 };

// Backward gate: dz (2d values) from dphi, plus the LayerNorm parameter
// partial sums of the block (g_c, b_c, g_g, b_g; 4d values) into lnpart.
//   BWD_ATOM : dphi = dm[src] * e^a[row]; d e^a[row] += dm[src] * phi
//   BWD_BOND : w = dmu[b1] * e^b[b1]; dphi = w * e^b[b2]; t2[row] = w * phi
//   BWD_ANGLE: dphi = da'[row]
// Each block covers kGateRows rows.
constexpr int kGateRows = 128;
struct GateBwdJob {
  int mode, rows, ldz, lddz, block0;
  const float* z;  // the saved pre-activations [rows, ldz]
  LnPtrs ln;
  const float *up, *eb;
  const int *up_idx, *b2_idx;
  float *aux, *dz, *lnpart;
  int aux_acc;  // BWD_ATOM: add to aux (0: the first layer of the backward overwrites it)
};
struct GateBwdJobs {
  int n;
  GateBwdJob j[3];
};

// LDS staging of the per-lane LayerNorm partials: [4 sums][4 waves][RPW
// slots][d columns + 4 pad].
template <int D>
struct GateBwdLds {
  static constexpr int RPW = Lanes<D, kBwdCpl>::RPW;
  static constexpr int LD = D + 4;
  static constexpr int FLOATS = 4 * 4 * RPW * LD;
};

template <int D, int MODE>
__device__ __forceinline__ void gate_bwd_rows(int blk, const GateBwdJob& J, float* red) {
  const int rows = J.rows, ldz = J.ldz, lddz = J.lddz;
  const float* __restrict__ z = J.z;
  const LnPtrs& ln = J.ln;
  const float* __restrict__ up = J.up;
  const int* __restrict__ up_idx = J.up_idx;
  const float* __restrict__ eb = J.eb;
  const int* __restrict__ b2_idx = J.b2_idx;
  float* __restrict__ aux = J.aux;
  float* __restrict__ dz = J.dz;
  float* __restrict__ lnpart = J.lnpart;
  constexpr int CPL = kBwdCpl;
  using L = Lanes<D, CPL>;
  constexpr int LPR = L::LPR, RPW = L::RPW;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, slot = lane / LPR, j = lane % LPR;
  float acc[4][CPL];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int k = 0; k < CPL; ++k) acc[a][k] = 0.f;
  for (int it = 0; it < kGateRows / (4 * RPW); ++it) {
    const int row = blk * kGateRows + (it * 4 + wave) * RPW + slot;
    if (row >= rows) continue;
    float zc[CPL], zg[CPL], rc, rg;
    load_z<D, CPL>(z, ldz, row, j, zc, zg);
    ln_stats<D, CPL>(zc, zg, rc, rg);
    float u[CPL], w[CPL], dphi[CPL];
    if (MODE == BWD_ANGLE) {
      load_cols<D, CPL>(up + (int64_t)row * D, j, dphi);
    } else {
      const int64_t ur = up_idx[row];
      load_cols<D, CPL>(up + ur * D, j, u);
      if (MODE == BWD_ATOM) {
        load_cols<D, CPL>(eb + (int64_t)row * D, j, w);  // e^a of this edge
#pragma unroll
        for (int k = 0; k < CPL; ++k) dphi[k] = u[k] * w[k];
      } else {
        float e1[CPL], e2[CPL];
        load_cols<D, CPL>(eb + ur * D, j, e1);
        load_cols<D, CPL>(eb + (int64_t)b2_idx[row] * D, j, e2);
#pragma unroll
        for (int k = 0; k < CPL; ++k) {
          w[k] = u[k] * e1[k];
          dphi[k] = w[k] * e2[k];
        }
      }
    }
    float dyc[CPL], dyg[CPL], side[CPL];
    float s1c = 0.f, s2c = 0.f, s1g = 0.f, s2g = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int c = L::col(j, k);
      const float yc = ln.gc[c] * zc[k] + ln.bc[c];
      const float yg = ln.gg[c] * zg[k] + ln.bg[c];
      const float sc = sigm(yc), sg = sigm(yg);
      const float silu_c = yc * sc;
      side[k] = silu_c * sg;  // phi
      const float gy_c = dphi[k] * sg * sc * (1.0f + yc * (1.0f - sc));
      const float gy_g = dphi[k] * silu_c * sg * (1.0f - sg);
      acc[0][k] += gy_c * zc[k];
      acc[1][k] += gy_c;
      acc[2][k] += gy_g * zg[k];
      acc[3][k] += gy_g;
      dyc[k] = gy_c * ln.gc[c];
      dyg[k] = gy_g * ln.gg[c];
      s1c += dyc[k];
      s2c += dyc[k] * zc[k];
      s1g += dyg[k];
      s2g += dyg[k] * zg[k];
    }
    s1c = rowsum<LPR>(s1c) * (1.0f / D);
    s2c = rowsum<LPR>(s2c) * (1.0f / D);
    s1g = rowsum<LPR>(s1g) * (1.0f / D);
    s2g = rowsum<LPR>(s2g) * (1.0f / D);
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      dyc[k] = rc * (dyc[k] - s1c - zc[k] * s2c);
      dyg[k] = rg * (dyg[k] - s1g - zg[k] * s2g);
    }
    store_cols<D, CPL>(dz + (int64_t)row * lddz, j, dyc);
    store_cols<D, CPL>(dz + (int64_t)row * lddz + D, j, dyg);
    if (MODE == BWD_ATOM) {
      float de[CPL];
      if (J.aux_acc) {
        load_cols<D, CPL>(aux + (int64_t)row * D, j, de);
#pragma unroll
        for (int k = 0; k < CPL; ++k) de[k] += u[k] * side[k];
      } else {
#pragma unroll
        for (int k = 0; k < CPL; ++k) de[k] = u[k] * side[k];
      }
      store_cols<D, CPL>(aux + (int64_t)row * D, j, de);
    } else if (MODE == BWD_BOND) {
#pragma unroll
      for (int k = 0; k < CPL; ++k) side[k] *= w[k];
      store_cols<D, CPL>(aux + (int64_t)row * D, j, side);
    }
  }
  // LayerNorm partials: every lane stages its four partial rows in LDS, then
  // each thread sums one (sum, column) pair over the waves and row slots in
  // a fixed order.
  using S = GateBwdLds<D>;
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int q = 0; q < CPL / 4; ++q)
      *reinterpret_cast<float4*>(red + ((a * 4 + wave) * RPW + slot) * S::LD + q * L::STRIDE + 4 * j) =
          make_float4(acc[a][4 * q], acc[a][4 * q + 1], acc[a][4 * q + 2], acc[a][4 * q + 3]);
  __syncthreads();
  for (int t = threadIdx.x; t < 4 * D; t += 256) {
    const int a = t / D, c = t % D;
    float s = 0.f;
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int sl = 0; sl < RPW; ++sl) s += red[((a * 4 + w) * RPW + sl) * S::LD + c];
    lnpart[(int64_t)blk * 4 * D + t] = s;
  }
}

template <int D>
__global__ void __launch_bounds__(256) k_gate_bwd(GateBwdJobs J) {
  int k = 0;
  while (k + 1 < J.n && (int)blockIdx.x >= J.j[k + 1].block0) ++k;
  const GateBwdJob& jb = J.j[k];
  const int blk = blockIdx.x - jb.block0;
  __shared__ __align__(16) float red[GateBwdLds<D>::FLOATS];
  if (jb.mode == BWD_ATOM) gate_bwd_rows<D, BWD_ATOM>(blk, jb, red);
  else if (jb.mode == BWD_BOND) gate_bwd_rows<D, BWD_BOND>(blk, jb, red);
  else gate_bwd_rows<D, BWD_ANGLE>(blk, jb, red);
}

// ---------------------------------------------------------------------------
// Fused backward gates and input-gradient product (d = 64). A tile is 64
// rows: edges of the atom conv (one gate), or angles (the bond-conv gate and,
// in layers with an angle update, the angle-update gate of the same angles).
// Consumer wavefronts form dz of the tile's gates as k_gate_bwd does (stored
// to global memory for the weight gradients and the segment sums, and to an
// LDS tile); producer wavefronts then form the gradient of the rows' own
// input block, dX = sum over the gates of dz W_g^T (+ residual), with 16x16x4
// fp32 MFMAs. Producer p owns output columns [16p, 16p + 16) of all 64 rows;
// in step s of a 128-wide k block lane group q = lane / 16 supplies
// k = 32q + s for both operands, so a lane's B fragment of a gate is 32
// consecutive entries of one weight row, held in registers.
// LayerNorm parameter partials accumulate in a consumer's registers while
// its wavefront stays on one gate; when it changes gate (and at the end)
// they are summed over the wavefront's row slots and staged in LDS, and the
// block adds its wavefronts in a fixed order.
// ---------------------------------------------------------------------------
struct GateBwdMmJob {
  int rows, tile0, ngates;
  int gid[2];  // LayerNorm partial slot of each gate: 0 atom conv, 1 bond conv, 2 angle update
  GateBwdJob g[2];
  const float* W[2];  // rows of each gate's first-layer weight for this input block: [D][2D]
  const float* res;   // [rows, D] added to dX, or nullptr
  float* dx;          // [rows, D]
};
struct GateBwdMmJobs {
  int n, ntiles;
  GateBwdMmJob j[2];
  float* lnpart[3];  // by slot: [gridDim.x][4 * 64], or nullptr
};
constexpr int kBmLd = 256 + 4;

// Row indices of a consumer row: the upstream row and (bond gate) the second
// bond.
struct BwdMmIdx {
  int up, b2;
};
__device__ __forceinline__ void bwd_mm_index(const GateBwdJob& J, int row, BwdMmIdx& x) {
  x.up = J.mode == BWD_ANGLE ? row : J.up_idx[row];
  x.b2 = J.mode == BWD_BOND ? J.b2_idx[row] : 0;
}

// LayerNorm parameter partials of one pass (4 sums x 8 columns per lane,
// rows in the wavefront's 8 row slots, lane bits 3-5) summed over the slots
// and added to this wavefront's LDS slot wsum[4][64]. Reduce-scatter: each
// step pairs the values of two lanes differing in one slot bit, keeping one
// of two values' sums per lane (the lane-half swaps of gfx950, then a DPP
// rotate by 8 within a row of 16); afterwards lane (j, b3, b4, b5) holds sum
// a of column 32 b3 + 4 j + 2 b4 + b5 for a = 0..3, and is that slot's only
// writer (fixed order, no atomics race).
__device__ __forceinline__ float pl_sum32(float a, float b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pl_sum16(float a, float b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ void bwd_mm_ln_add(const float (&p)[32], float* wsum) {
  const int lane = threadIdx.x & 63;
  float w[16], x[8];
#pragma unroll
  for (int m = 0; m < 16; ++m) w[m] = pl_sum32(p[2 * m], p[2 * m + 1]);
#pragma unroll
  for (int m = 0; m < 8; ++m) x[m] = pl_sum16(w[2 * m], w[2 * m + 1]);
  const bool hi = (lane & 8) != 0;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const float keep = hi ? x[2 * m + 1] : x[2 * m], send = hi ? x[2 * m] : x[2 * m + 1];
    const float y = keep + dpp<0x128>(send);  // row_ror:8
    const int col = 32 * ((lane >> 3) & 1) + 4 * (lane & 7) + 2 * ((lane >> 4) & 1) + ((lane >> 5) & 1);
    wsum[m * 64 + col] += y;
  }
}

template <int D, int MODE>
__device__ __forceinline__ void gate_bwd_mm_row(const GateBwdJob& J, int row, const BwdMmIdx& x, int j,
                                                const float* lnS, float (&lp)[4 * kMmCpl], float* zrow) {
  constexpr int CPL = kMmCpl;
  constexpr int LPR = Lanes<D, CPL>::LPR;
  float zc[CPL], zg[CPL], rc, rg;
  load_cols_nt<D, CPL>(J.z + (int64_t)row * J.ldz, j, zc);
  load_cols_nt<D, CPL>(J.z + (int64_t)row * J.ldz + D, j, zg);
  // the running sum d e^a of this edge, loaded with the row's other inputs
  // (after the dz stores the load could not be moved ahead of them)
  float de[CPL];
  if (MODE == BWD_ATOM && J.aux_acc) load_cols<D, CPL>(J.aux + (int64_t)row * D, j, de);
  float u[CPL], w[CPL], dphi[CPL];
  if (MODE == BWD_ANGLE) {
    load_cols<D, CPL>(J.up + (int64_t)row * D, j, dphi);
  } else {
    const int64_t ur = x.up;
    load_cols<D, CPL>(J.up + ur * D, j, u);
    if (MODE == BWD_ATOM) {
      load_cols<D, CPL>(J.eb + (int64_t)row * D, j, w);  // e^a of this edge
#pragma unroll
      for (int k = 0; k < CPL; ++k) dphi[k] = u[k] * w[k];
    } else {
      float e1[CPL], e2[CPL];
      load_cols<D, CPL>(J.eb + ur * D, j, e1);
      load_cols<D, CPL>(J.eb + (int64_t)x.b2 * D, j, e2);
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        w[k] = u[k] * e1[k];
        dphi[k] = w[k] * e2[k];
      }
    }
  }
  ln_stats<D, CPL>(zc, zg, rc, rg);
  float gc[CPL], bc[CPL], gg[CPL], bg[CPL];
  load_cols<D, CPL>(lnS, j, gc);
  load_cols<D, CPL>(lnS + D, j, bc);
  load_cols<D, CPL>(lnS + 2 * D, j, gg);
  load_cols<D, CPL>(lnS + 3 * D, j, bg);
  float dyc[CPL], dyg[CPL], side[CPL];
  float s1c = 0.f, s2c = 0.f, s1g = 0.f, s2g = 0.f;
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    const float yc = gc[k] * zc[k] + bc[k];
    const float yg = gg[k] * zg[k] + bg[k];
    const float sc = sigm(yc), sg = sigm(yg);
    const float silu_c = yc * sc;
    side[k] = silu_c * sg;  // phi
    const float gy_c = dphi[k] * sg * sc * (1.0f + yc * (1.0f - sc));
    const float gy_g = dphi[k] * silu_c * sg * (1.0f - sg);
    lp[k] = gy_c * zc[k];
    lp[8 + k] = gy_c;
    lp[16 + k] = gy_g * zg[k];
    lp[24 + k] = gy_g;
    dyc[k] = gy_c * gc[k];
    dyg[k] = gy_g * gg[k];
    s1c += dyc[k];
    s2c += dyc[k] * zc[k];
    s1g += dyg[k];
    s2g += dyg[k] * zg[k];
  }
  s1c = rowsum<LPR>(s1c) * (1.0f / D);
  s2c = rowsum<LPR>(s2c) * (1.0f / D);
  s1g = rowsum<LPR>(s1g) * (1.0f / D);
  s2g = rowsum<LPR>(s2g) * (1.0f / D);
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    dyc[k] = rc * (dyc[k] - s1c - zc[k] * s2c);
    dyg[k] = rg * (dyg[k] - s1g - zg[k] * s2g);
  }
  store_cols<D, CPL>(J.dz + (int64_t)row * J.lddz, j, dyc);
  store_cols<D, CPL>(J.dz + (int64_t)row * J.lddz + D, j, dyg);
  // LDS tile: odd rows hold their two 32-column halves of each 64-column
  // block swapped (logical column c at c ^ 32), so that the two rows of a
  // write phase fall in different banks; the producers read with the same map
  {
    const int sw = (row & 1) * 32;
#pragma unroll
    for (int q = 0; q < CPL / 4; ++q) {
      const int cc = (q * Lanes<D, CPL>::STRIDE + 4 * j) ^ sw;
      *reinterpret_cast<float4*>(zrow + cc) = make_float4(dyc[4 * q], dyc[4 * q + 1], dyc[4 * q + 2], dyc[4 * q + 3]);
      *reinterpret_cast<float4*>(zrow + D + cc) = make_float4(dyg[4 * q], dyg[4 * q + 1], dyg[4 * q + 2], dyg[4 * q + 3]);
    }
  }
  if (MODE == BWD_ATOM) {
    if (J.aux_acc) {
#pragma unroll
      for (int k = 0; k < CPL; ++k) de[k] += u[k] * side[k];
    } else {
#pragma unroll
      for (int k = 0; k < CPL; ++k) de[k] = u[k] * side[k];
    }
    store_cols<D, CPL>(J.aux + (int64_t)row * D, j, de);
  } else if (MODE == BWD_BOND) {
#pragma unroll
    for (int k = 0; k < CPL; ++k) side[k] *= w[k];
    store_cols<D, CPL>(J.aux + (int64_t)row * D, j, side);
  }
}

// One block per compute unit, walking tiles blockIdx.x, blockIdx.x +
// gridDim.x, ... of the concatenated jobs; consumers fill the dz tile of
// tile i while producers multiply tile i - 1 (one block barrier per tile).
__global__ void __launch_bounds__(kMmThreads, 1) k_gate_bwd_mm(GateBwdMmJobs J) {
  __shared__ __attribute__((aligned(16))) float Zs[2][kMmRows * kBmLd];
  __shared__ __attribute__((aligned(16))) float LnS[2][2][4][64];
  __shared__ __attribute__((aligned(16))) float Wsum[3][kMmConsumers][4 * 64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int t = threadIdx.x; t < 2 * 2 * 4 * 64; t += kMmThreads) {
    const int jb = t / 512, g = (t / 256) % 2, q = (t / 64) % 4, c = t % 64;
    float v = 0.f;
    if (jb < J.n && g < J.j[jb].ngates) {
      const LnPtrs& ln = J.j[jb].g[g].ln;
      v = (q == 0 ? ln.gc : q == 1 ? ln.bc : q == 2 ? ln.gg : ln.bg)[c];
    }
    LnS[jb][g][q][c] = v;
  }
  for (int t = threadIdx.x; t < 3 * kMmConsumers * 4 * 64; t += kMmThreads) (&Wsum[0][0][0])[t] = 0.f;
  auto job_of = [&](int tile) {
    int k = 0;
    while (k + 1 < J.n && tile >= J.j[k + 1].tile0) ++k;
    return k;
  };
  // the grid never exceeds the tile count: every block has a tile
  const int nt = (J.ntiles - 1 - (int)blockIdx.x) / (int)gridDim.x + 1;
  auto tile_of = [&](int i) { return (int)blockIdx.x + i * (int)gridDim.x; };
  __syncthreads();
  if (wave < kMmProducers) {
    const int n = lane & 15, q4 = lane >> 4, col = 16 * wave + n;
    float bf[2][32];
    int cur = -1;
    // residual of output element (row 16 rt + 4 q4 + v, column col) of tile
    // ii, loaded one tile ahead
    float rv[4][4], rvn[4][4];
    auto load_res = [&](int ii) {
      if (ii >= nt) return;
      const int tile = tile_of(ii);
      const GateBwdMmJob& jb = J.j[job_of(tile)];
      const int row0 = (tile - jb.tile0) * kMmRows;
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = row0 + 16 * rt + 4 * q4 + v;
          rvn[rt][v] = (jb.res && row < jb.rows) ? jb.res[(int64_t)row * 64 + col] : 0.f;
        }
    };
    load_res(0);
    for (int i = 0; i <= nt; ++i) {
      if (i > 0) {
        const int tile = tile_of(i - 1);
        const int k = job_of(tile);
        const GateBwdMmJob& jb = J.j[k];
        const int ng = jb.ngates;
        if (k != cur) {
          cur = k;
#pragma unroll
          for (int g = 0; g < 2; ++g) {
            if (g < ng) {
              const float* wr = jb.W[g] + (int64_t)col * 128 + 32 * q4;
#pragma unroll
              for (int s4 = 0; s4 < 8; ++s4) {
                const float4 v = *reinterpret_cast<const float4*>(wr + 4 * s4);
                bf[g][4 * s4] = v.x; bf[g][4 * s4 + 1] = v.y; bf[g][4 * s4 + 2] = v.z; bf[g][4 * s4 + 3] = v.w;
              }
            }
          }
        }
        const int row0 = (tile - jb.tile0) * kMmRows;
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
          for (int v = 0; v < 4; ++v) rv[rt][v] = rvn[rt][v];
        load_res(i);
        v4f acc[4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) acc[rt] = v4f{0.f, 0.f, 0.f, 0.f};
        const float* Z = Zs[(i - 1) & 1];
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          if (g < ng) {
#pragma unroll
            for (int s4 = 0; s4 < 8; ++s4) {
              float4 a4[4];
#pragma unroll
              for (int rt = 0; rt < 4; ++rt)
                a4[rt] = *reinterpret_cast<const float4*>(Z + (16 * rt + n) * kBmLd + 128 * g +
                                                          ((32 * q4 + 4 * s4) ^ ((n & 1) * 32)));
#pragma unroll
              for (int rt = 0; rt < 4; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].x, bf[g][4 * s4], acc[rt], 0, 0, 0);
#pragma unroll
              for (int rt = 0; rt < 4; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].y, bf[g][4 * s4 + 1], acc[rt], 0, 0, 0);
#pragma unroll
              for (int rt = 0; rt < 4; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].z, bf[g][4 * s4 + 2], acc[rt], 0, 0, 0);
#pragma unroll
              for (int rt = 0; rt < 4; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].w, bf[g][4 * s4 + 3], acc[rt], 0, 0, 0);
            }
          }
        }
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = row0 + 16 * rt + 4 * q4 + v;
            if (row < jb.rows) jb.dx[(int64_t)row * 64 + col] = acc[rt][v] + rv[rt][v];
          }
      }
      __syncthreads();
    }
  } else {
    __builtin_amdgcn_s_setprio(kConsumerPrio);
    using GL = Lanes<64, kMmCpl>;
    const int cw = wave - kMmProducers, j = lane % GL::LPR, slot = lane / GL::LPR;
    // Every wavefront covers the same 8 rows of each of the tile's gates
    // (rows 8 cw + slot), one pass per gate; the row indices of a tile are
    // loaded one tile ahead.
    auto tile_job = [&](int ii) { return __builtin_amdgcn_readfirstlane(job_of(tile_of(ii))); };
    auto load_idx = [&](int ii, BwdMmIdx (&x)[2]) {
      if (ii >= nt) return;
      const int tile = tile_of(ii), k = tile_job(ii);
      const GateBwdMmJob& jb = J.j[k];
      const int row = (tile - jb.tile0) * kMmRows + 8 * cw + slot;
      if (row >= jb.rows) return;
      bwd_mm_index(jb.g[0], row, x[0]);
      if (jb.ngates > 1) bwd_mm_index(jb.g[1], row, x[1]);
    };
    BwdMmIdx xi[2] = {}, xn[2] = {};
    load_idx(0, xi);
    for (int i = 0; i <= nt; ++i) {
      if (i < nt) {
        load_idx(i + 1, xn);
        const int tile = tile_of(i), k = tile_job(i);
        const GateBwdMmJob& jb = J.j[k];
        const int lr = 8 * cw + slot;
        const int row = (tile - jb.tile0) * kMmRows + lr;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          if (g >= jb.ngates) break;
          const GateBwdJob& gj = jb.g[g];
          float lp[4 * kMmCpl];
#pragma unroll
          for (int q = 0; q < 4 * kMmCpl; ++q) lp[q] = 0.f;
          if (row < jb.rows) {
            const float* lnS = &LnS[k][g][0][0];
            float* zrow = Zs[i & 1] + lr * kBmLd + 128 * g;
            if (gj.mode == BWD_ATOM) gate_bwd_mm_row<64, BWD_ATOM>(gj, row, xi[g], j, lnS, lp, zrow);
            else if (gj.mode == BWD_BOND) gate_bwd_mm_row<64, BWD_BOND>(gj, row, xi[g], j, lnS, lp, zrow);
            else gate_bwd_mm_row<64, BWD_ANGLE>(gj, row, xi[g], j, lnS, lp, zrow);
          }
          bwd_mm_ln_add(lp, Wsum[jb.gid[g]][cw]);
        }
#pragma unroll
        for (int g = 0; g < 2; ++g) xi[g] = xn[g];
      }
      __syncthreads();
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < 3 * 4 * 64; t += kMmThreads) {
    const int gid = t / 256, c = t % 256;
    if (!J.lnpart[gid]) continue;
    float s = 0.f;
    for (int w = 0; w < kMmConsumers; ++w) s += Wsum[gid][w][c];
    J.lnpart[gid][(int64_t)blockIdx.x * 256 + c] = s;
  }
}

// LayerNorm parameter partials of one pass at d = 128 (4 sums x 8 columns
// per lane, rows in the wavefront's 4 row slots, lane bits 4-5) summed over
// the slots and added to this wavefront's LDS slot wsum[4][128]: the
// lane-half swaps reduce over bit 5 and then bit 4, after which lane
// (j, b4, b5) holds, for m = 0..7, sum m / 2 of column 64 (m % 2) + 4 j +
// 2 b4 + b5 and is that slot's only writer (fixed order, no atomics).
__device__ __forceinline__ void bwd_mm_ln_add128(const float (&p)[32], float* wsum) {
  const int lane = threadIdx.x & 63;
  float w[16];
#pragma unroll
  for (int m = 0; m < 16; ++m) w[m] = pl_sum32(p[2 * m], p[2 * m + 1]);
  const int base = 4 * (lane & 15) + 2 * ((lane >> 4) & 1) + ((lane >> 5) & 1);
#pragma unroll
  for (int m = 0; m < 8; ++m) wsum[(m >> 1) * 128 + 64 * (m & 1) + base] += pl_sum16(w[2 * m], w[2 * m + 1]);
}

// Fused backward gate at d = 128: the gate backward of a layer (dz, the
// LayerNorm parameter partials, d e^a / t2) and the input gradients of its
// own rows dX = sum_g dz_g W_g^T + residual in one launch, one 1024-thread
// block per compute unit. Every gate is a job of its own over 32-row tiles
// (atom conv over the edges; bond conv, then angle update over the angles);
// a block takes the row tiles r = blockIdx.x + k gridDim.x of every job, job
// by job, so it runs the angle update's tile r after the bond conv's tile r,
// and the angle update adds its product to the bond conv's dX of those rows
// (written and read back by the same lanes). Per tile the eight consumer
// wavefronts form dz (4 rows each, 16 lanes a row), store it for the weight
// gradients and segmented sums and into an LDS tile, while the eight
// producer wavefronts multiply the previous tile: each owns 16 output
// columns of all 32 rows (fp32 MFMA 16x16x4, two 16-row subtiles) and holds
// its 16 columns of the job's W^T (256 x 128) in registers, loaded once per
// job.
constexpr int kBm2Rows = 32, kBm2Ld = 256 + 4, kBm2Threads = 1024, kBm2Prod = 8, kBm2Cons = 8;

struct GateBwd128Job {
  int rows, ntiles, gid;  // gid: LayerNorm partial slot (0 atom conv, 1 bond conv, 2 angle update)
  GateBwdJob g;
  const float* W;    // [128, 256]: rows of the gate's first-layer weight for this input block
  const float* res;  // [rows, 128] added to dX, or nullptr
  float* dx;         // [rows, 128]
};
struct GateBwd128Jobs {
  int n;
  GateBwd128Job j[3];
  float* lnpart[3];  // by slot: [gridDim.x][4 * 128], or nullptr
};

__global__ void __launch_bounds__(kBm2Threads, 1) k_gate_bwd_mm128(GateBwd128Jobs J) {
  constexpr int D = 128;
  __shared__ __attribute__((aligned(16))) float Zs[2][kBm2Rows * kBm2Ld];
  __shared__ __attribute__((aligned(16))) float LnS[3][4][D];
  __shared__ __attribute__((aligned(16))) float Wsum[3][kBm2Cons][4 * D];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int t = threadIdx.x; t < 3 * 4 * D; t += kBm2Threads) {
    const int jb = t / (4 * D), q = (t / D) % 4, c = t % D;
    float v = 0.f;
    if (jb < J.n) {
      const LnPtrs& ln = J.j[jb].g.ln;
      v = (q == 0 ? ln.gc : q == 1 ? ln.bc : q == 2 ? ln.gg : ln.bg)[c];
    }
    LnS[jb][q][c] = v;
  }
  for (int t = threadIdx.x; t < 3 * kBm2Cons * 4 * D; t += kBm2Threads) (&Wsum[0][0][0])[t] = 0.f;
  const int b0 = (int)blockIdx.x, G = (int)gridDim.x;
  __syncthreads();
  if (wave < kBm2Prod) {
    const int n = lane & 15, q4 = lane >> 4, col = 16 * wave + n;
    int units = 0;  // tiles consumed so far (one block barrier each)
    for (int k = 0; k < J.n; ++k) {
      const GateBwd128Job& jb = J.j[k];
      if (b0 >= jb.ntiles) continue;
      // this lane's W^T entries: lane quad q4 supplies k = 64 qt + 16 q4 + s
      // in MFMA step s of quarter qt (the same map for A and B)
      float bq[4][16];
      {
        const float* wr = jb.W + (int64_t)col * (2 * D) + 16 * q4;
#pragma unroll
        for (int qt = 0; qt < 4; ++qt)
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float4 v = *reinterpret_cast<const float4*>(wr + 64 * qt + 4 * u);
            bq[qt][4 * u] = v.x; bq[qt][4 * u + 1] = v.y; bq[qt][4 * u + 2] = v.z; bq[qt][4 * u + 3] = v.w;
          }
      }
      for (int r = b0; r < jb.ntiles; r += G) {
        const int row0 = r * kBm2Rows;
        float rv[2][4];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = row0 + 16 * rt + 4 * q4 + v;
            rv[rt][v] = (jb.res && row < jb.rows) ? jb.res[(int64_t)row * D + col] : 0.f;
          }
        v4f acc[2];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) acc[rt] = v4f{0.f, 0.f, 0.f, 0.f};
        __syncthreads();  // the consumers have written this tile's dz
        const float* Z = Zs[units & 1];
        ++units;
#pragma unroll
        for (int qt = 0; qt < 4; ++qt)
#pragma unroll
          for (int s4 = 0; s4 < 4; ++s4) {
            float4 a4[2];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
              a4[rt] = *reinterpret_cast<const float4*>(Z + (16 * rt + n) * kBm2Ld +
                                                        ((64 * qt + 16 * q4 + 4 * s4) ^ ((n & 1) * 32)));
            const float* b = &bq[qt][4 * s4];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].x, b[0], acc[rt], 0, 0, 0);
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].y, b[1], acc[rt], 0, 0, 0);
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].z, b[2], acc[rt], 0, 0, 0);
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) acc[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[rt].w, b[3], acc[rt], 0, 0, 0);
          }
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = row0 + 16 * rt + 4 * q4 + v;
            if (row < jb.rows) jb.dx[(int64_t)row * D + col] = acc[rt][v] + rv[rt][v];
          }
      }
    }
    __syncthreads();  // matches the consumers' final barrier
  } else {
    __builtin_amdgcn_s_setprio(kConsumerPrio);
    using GL = Lanes<D, kMmCpl>;
    const int cw = wave - kBm2Prod, j = lane % GL::LPR, slot = lane / GL::LPR;
    const int lr = GL::RPW * cw + slot;  // row of the tile
    // the block's tiles in order: (job k, tile r); row indices loaded one
    // tile ahead
    auto next_unit = [&](int& k, int& r) {
      r += G;
      while (k < J.n && r >= J.j[k].ntiles) {
        ++k;
        r = b0;
      }
    };
    auto unit_idx = [&](int k, int r, BwdMmIdx& x) {
      if (k >= J.n) return;
      const int row = r * kBm2Rows + lr;
      if (row < J.j[k].rows) bwd_mm_index(J.j[k].g, row, x);
    };
    int k = 0, r = b0;
    while (k < J.n && r >= J.j[k].ntiles) {
      ++k;
      r = b0;
    }
    BwdMmIdx xcur{}, xnext{};
    unit_idx(k, r, xcur);
    int units = 0;
    while (k < J.n) {
      int kn = k, rn = r;
      next_unit(kn, rn);
      unit_idx(kn, rn, xnext);
      const GateBwd128Job& jb = J.j[k];
      const GateBwdJob& gj = jb.g;
      const int row = r * kBm2Rows + lr;
      float lp[4 * kMmCpl];
#pragma unroll
      for (int q = 0; q < 4 * kMmCpl; ++q) lp[q] = 0.f;
      if (row < jb.rows) {
        const BwdMmIdx x = xcur;
        const float* lnS = &LnS[k][0][0];
        float* zrow = Zs[units & 1] + lr * kBm2Ld;
        if (gj.mode == BWD_ATOM) gate_bwd_mm_row<D, BWD_ATOM>(gj, row, x, j, lnS, lp, zrow);
        else if (gj.mode == BWD_BOND) gate_bwd_mm_row<D, BWD_BOND>(gj, row, x, j, lnS, lp, zrow);
        else gate_bwd_mm_row<D, BWD_ANGLE>(gj, row, x, j, lnS, lp, zrow);
      }
      bwd_mm_ln_add128(lp, Wsum[jb.gid][cw]);
      xcur = xnext;
      k = kn;
      r = rn;
      __syncthreads();  // this tile's dz is complete
      ++units;
    }
    __syncthreads();  // the producers have read the last tile
  }
  __syncthreads();
  for (int t = threadIdx.x; t < 3 * 4 * D; t += kBm2Threads) {
    const int gid = t / (4 * D), c = t % (4 * D);
    if (!J.lnpart[gid]) continue;
    float s = 0.f;
    for (int w = 0; w < kBm2Cons; ++w) s += Wsum[gid][w][c];
    J.lnpart[gid][(int64_t)blockIdx.x * 4 * D + c] = s;
  }
}

// ---------------------------------------------------------------------------
// Readout MLPs (d = 64): the three layers of a head in one pass over its
// rows, h1 = x W1 + b1, a1 = SiLU(h1), h2 = a1 W2 + b2, a2 = SiLU(h2),
// o = a2 W3 + b3 (h1, a1, h2, a2 kept for the backward pass). A wavefront
// takes 32 rows at a time: fp32 MFMA 32x32x2 with each layer's weights
// loaded as B fragments just before it (cache-resident; lane half h supplies
// k = 32 kb + 16 h + e in step e of 32-wide k block kb), the activations passed between layers through a
// per-wavefront LDS tile, and the output layer as per-row dot products (each
// lane half sums its 32 k in order, then the halves are added).
// ---------------------------------------------------------------------------
struct HeadJob {
  int rows, tile0, out;
  const float *x, *W1, *b1, *W2, *b2, *W3, *b3;
  float *h1, *a1, *h2, *a2, *o;
};
struct HeadJobs {
  int n, ntiles;
  HeadJob j[3];
};
constexpr int kHdRows = 32, kHdLd = 64 + 4;

__device__ __forceinline__ void hd_bfrag(const float* __restrict__ W, int lane, float (&b)[2][2][16]) {
  const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) b[ct][kb][e] = W[(32 * kb + 16 * h + e) * 64 + 32 * ct + l32];
}

// one dense layer of a 32-row tile: acc[ct] = A W (A fragments af)
__device__ __forceinline__ void hd_layer(const float (&af)[2][16], const float (&b)[2][2][16], v16f (&acc)[2]) {
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[ct][e] = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int e = 0; e < 16; ++e)
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) acc[ct] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[kb][e], b[ct][kb][e], acc[ct], 0, 0, 0);
}

// bias and SiLU of a layer's tile: h and a to global memory (rows below
// `rows`), a to the wavefront's LDS tile
__device__ __forceinline__ void hd_epilogue(const v16f (&acc)[2], const float* __restrict__ bias, int rows, int row0,
                                            float* __restrict__ hout, float* __restrict__ aout, float* Tw, int lane) {
  const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int ct = 0; ct < 2; ++ct) {
    const int c = 32 * ct + l32;
    const float bc = bias[c];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int r = 8 * (j >> 2) + 4 * h + (j & 3);
      const float hv = acc[ct][j] + bc;
      const float av = hv * sigm(hv);
      if (row0 + r < rows) {
        hout[(int64_t)(row0 + r) * 64 + c] = hv;
        aout[(int64_t)(row0 + r) * 64 + c] = av;
      }
      Tw[r * kHdLd + c] = av;
    }
  }
}

// the wavefront's LDS writes are visible to all its lanes
__device__ __forceinline__ void hd_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__global__ void __launch_bounds__(256, 2) k_head_mlp(HeadJobs J) {
  __shared__ __attribute__((aligned(16))) float T[4][kHdRows * kHdLd];
  const int lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float* Tw = T[wave];
  float bf[2][2][16];
  const int nw = (int)gridDim.x * 4;
  for (int tile = (int)blockIdx.x * 4 + wave; tile < J.ntiles; tile += nw) {
    int k = 0;
    while (k + 1 < J.n && tile >= J.j[k + 1].tile0) ++k;
    k = __builtin_amdgcn_readfirstlane(k);
    const HeadJob& jb = J.j[k];
    hd_bfrag(jb.W1, lane, bf);
    const int row0 = (tile - jb.tile0) * kHdRows, row = row0 + l32;
    const bool valid = row < jb.rows;
    float af[2][16];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (valid) v = *reinterpret_cast<const float4*>(jb.x + (int64_t)row * 64 + 32 * kb + 16 * h + 4 * q);
        af[kb][4 * q] = v.x; af[kb][4 * q + 1] = v.y; af[kb][4 * q + 2] = v.z; af[kb][4 * q + 3] = v.w;
      }
    v16f acc[2];
    hd_layer(af, bf, acc);
    hd_epilogue(acc, jb.b1, jb.rows, row0, jb.h1, jb.a1, Tw, lane);
    hd_wave_sync();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = *reinterpret_cast<const float4*>(Tw + l32 * kHdLd + 32 * kb + 16 * h + 4 * q);
        af[kb][4 * q] = v.x; af[kb][4 * q + 1] = v.y; af[kb][4 * q + 2] = v.z; af[kb][4 * q + 3] = v.w;
      }
    hd_bfrag(jb.W2, lane, bf);
    hd_wave_sync();
    hd_layer(af, bf, acc);
    hd_epilogue(acc, jb.b2, jb.rows, row0, jb.h2, jb.a2, Tw, lane);
    hd_wave_sync();
    // output layer: lane (row l32, half h) sums k in [32 h, 32 h + 32)
    for (int c = 0; c < jb.out; ++c) {
      float s = 0.f;
#pragma unroll 8
      for (int kk = 0; kk < 32; ++kk) s += Tw[l32 * kHdLd + 32 * h + kk] * jb.W3[(32 * h + kk) * jb.out + c];
      s += __shfl_xor(s, 32);
      if (h == 0 && valid) jb.o[(int64_t)row * jb.out + c] = s + jb.b3[c];
    }
    hd_wave_sync();
  }
}

// Segmented row sums, several independent jobs per launch:
//   out[s] (+)= sum_{r in [ptr[s], ptr[s+1])} vals[idx(r)]; optionally
//   out2[s] = mul[s] * sum. WPS wavefronts per (segment, 64 columns) split the
// rows (wave w takes every WPS-th group of 4 rows) and their sums are added
// in wave order: the result does not depend on scheduling.
struct SegJob {
  int nseg, ncb, width, ld_in, ld_out, ld_mul, ld_out2, accumulate, block0;
  int wps;  // wavefronts per (segment, column block): 4 for long segments, 1 for short
  int lpr;  // set by the launch: 0, one column a lane; else lanes per row, four columns a lane
  // set by the launch on the first job of a pair: the pair's block count (a
  // multiple of 8); the two jobs' blocks are interleaved (see k_segsum)
  int pair;
  // optional output linear of the update (64-wide rows only): with y the
  // segment's result (out2 if set, else out), upd[urow(s)] = res[urow(s)]
  // + y Wo + bo, urow = upd_rows ? upd_rows[s] : s
  const float* Wo;
  const float* bo;
  const float* res;
  float* upd;
  const int* upd_rows;
  const int* ptr;
  const int* idx;
  const float* vals;
  float* out;
  const float* mul;
  float* out2;
};
struct SegJobs {
  int n;
  SegJob j[3];
};

template <int WPS>
__device__ __forceinline__ void segsum_block(const SegJob& S, float (*red)[64], int lb) {
  constexpr int SPB = 4 / WPS;  // (segment, column block) units per block
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int unit = lb * SPB + wave / WPS, w = wave % WPS;
  const int s = unit / S.ncb, c = (unit % S.ncb) * 64 + lane;
  const bool ok = s < S.nseg && c < S.width;
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  if (ok) {
    const int lo = S.ptr[s], hi = S.ptr[s + 1];
    int r = lo + 4 * w;
    for (; r + 3 < hi; r += 4 * WPS) {
      const int64_t i0 = S.idx ? S.idx[r] : r, i1 = S.idx ? S.idx[r + 1] : r + 1, i2 = S.idx ? S.idx[r + 2] : r + 2,
                    i3 = S.idx ? S.idx[r + 3] : r + 3;
      a0 += S.vals[i0 * S.ld_in + c];
      a1 += S.vals[i1 * S.ld_in + c];
      a2 += S.vals[i2 * S.ld_in + c];
      a3 += S.vals[i3 * S.ld_in + c];
    }
    // r is now the start of one of this wave's groups: its partial tail
    for (; r < hi; ++r) a0 += S.vals[(int64_t)(S.idx ? S.idx[r] : r) * S.ld_in + c];
  }
  float acc = (a0 + a1) + (a2 + a3);
  if (WPS > 1) {
    red[wave][lane] = acc;
    __syncthreads();
    if (w != 0) return;
    for (int q = 1; q < WPS; ++q) acc += red[wave + q][lane];
  }
  if (!ok) return;
  float* o = S.out + (int64_t)s * S.ld_out + c;
  *o = S.accumulate ? *o + acc : acc;
  float y = acc;
  if (S.out2) {
    y = S.mul[(int64_t)s * S.ld_mul + c] * acc;
    S.out2[(int64_t)s * S.ld_out2 + c] = y;
  }
  if (S.Wo) {
    // the wavefront holds the whole 64-wide row, lane c column c: out
    // column c = sum_k y_k Wo[k][c], y_k broadcast from lane k (fixed order,
    // two interleaved partial sums)
    const int64_t ur = S.upd_rows ? S.upd_rows[s] : s;
    float u0 = 0.f, u1 = 0.f;
#pragma unroll 8
    for (int k = 0; k < 64; k += 2) {
      const float y0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(y), k));
      const float y1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(y), k + 1));
      u0 += y0 * S.Wo[k * 64 + c];
      u1 += y1 * S.Wo[(k + 1) * 64 + c];
    }
    S.upd[ur * 64 + c] = (S.res[ur * 64 + c] + (u0 + u1)) + S.bo[c];
  }
}

// The same sums with four columns a lane (16-byte loads and stores): LPR
// lanes cover a row's column block of 4 LPR columns and a load instruction
// covers 64 / LPR rows. A wave takes groups of U instructions' rows; rows
// are clamped into the segment (the surplus is loaded and weighted 0), so
// every load of a group is issued at once, and with IDX the row indices of
// the wave's next group are loaded while the current group's rows are.
template <int WPS, int LPR, int U, bool IDX>
__device__ __forceinline__ void segsum_block4(const SegJob& S, float4 (*red4)[64], int lb) {
  constexpr int SPB = 4 / WPS, RPI = 64 / LPR, G = U * RPI;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int unit = lb * SPB + wave / WPS, w = wave % WPS;
  const int s = unit / S.ncb, sub = lane / LPR;
  const int c = (unit % S.ncb) * 4 * LPR + 4 * (lane % LPR);
  const bool ok = s < S.nseg && c < S.width;
  float4 a[U];
#pragma unroll
  for (int u = 0; u < U; ++u) a[u] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (ok) {
    const int lo = S.ptr[s], hi = S.ptr[s + 1];
    const float* __restrict__ vals = S.vals + c;
    int ix[U];
    auto rows_of = [&](int g) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = min(g + u * RPI + sub, hi - 1);
        ix[u] = IDX ? S.idx[r] : r;
      }
    };
    int g = lo + G * w;
    if (g < hi) rows_of(g);
    for (; g < hi; g += G * WPS) {
      int cur[U];
#pragma unroll
      for (int u = 0; u < U; ++u) cur[u] = ix[u];
      rows_of(g + G * WPS);
      float4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) x[u] = *reinterpret_cast<const float4*>(vals + (int64_t)cur[u] * S.ld_in);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float m = g + u * RPI + sub < hi ? 1.f : 0.f;
        a[u].x += m * x[u].x;
        a[u].y += m * x[u].y;
        a[u].z += m * x[u].z;
        a[u].w += m * x[u].w;
      }
    }
  }
  // fixed-order sums: the U partials, the lane groups of the other rows of an
  // instruction, then the WPS wavefronts
  float4 acc = a[0];
#pragma unroll
  for (int u = 1; u < U; ++u) {
    acc.x += a[u].x;
    acc.y += a[u].y;
    acc.z += a[u].z;
    acc.w += a[u].w;
  }
#pragma unroll
  for (int m = LPR; m < 64; m *= 2) {
    acc.x += __shfl_xor(acc.x, m);
    acc.y += __shfl_xor(acc.y, m);
    acc.z += __shfl_xor(acc.z, m);
    acc.w += __shfl_xor(acc.w, m);
  }
  if (WPS > 1) {
    red4[wave][lane] = acc;
    __syncthreads();
    if (w != 0) return;
    for (int q = 1; q < WPS; ++q) {
      const float4 t = red4[wave + q][lane];
      acc.x += t.x;
      acc.y += t.y;
      acc.z += t.z;
      acc.w += t.w;
    }
  }
  if (!ok || sub != 0) return;
  float4* o = reinterpret_cast<float4*>(S.out + (int64_t)s * S.ld_out + c);
  if (S.accumulate) {
    const float4 t = *o;
    acc.x += t.x;
    acc.y += t.y;
    acc.z += t.z;
    acc.w += t.w;
  }
  *o = acc;
  if (S.out2) {
    const float4 m = *reinterpret_cast<const float4*>(S.mul + (int64_t)s * S.ld_mul + c);
    *reinterpret_cast<float4*>(S.out2 + (int64_t)s * S.ld_out2 + c) =
        make_float4(m.x * acc.x, m.y * acc.y, m.z * acc.z, m.w * acc.w);
  }
}

template <int WPS, int U>
__device__ __forceinline__ void segsum_job(const SegJob& S, float4 (*red4)[64], int lb) {
  if (S.lpr == 0) segsum_block<WPS>(S, reinterpret_cast<float (*)[64]>(red4), lb);
  else if (S.idx) {
    if (S.lpr == 64) segsum_block4<WPS, 64, U, true>(S, red4, lb);
    else if (S.lpr == 32) segsum_block4<WPS, 32, U, true>(S, red4, lb);
    else segsum_block4<WPS, 16, U, true>(S, red4, lb);
  } else {
    if (S.lpr == 64) segsum_block4<WPS, 64, U, false>(S, red4, lb);
    else if (S.lpr == 32) segsum_block4<WPS, 32, U, false>(S, red4, lb);
    else segsum_block4<WPS, 16, U, false>(S, red4, lb);
  }
}

// Jobs of either segment length in one launch; each block runs its job's
// variant (the choice is uniform over the block).
__global__ void __launch_bounds__(256) k_segsum(SegJobs J) {
  __shared__ float4 red4[4][64];  // wavefront partials (WPS > 1)
  int k = 0;
  while (k + 1 < J.n && (int)blockIdx.x >= J.j[k + 1].block0) ++k;
  int lb = (int)blockIdx.x - J.j[k].block0;
  if (J.j[k].pair) {
    // a pair of sums over the same rows (a segment's out-edges, then its
    // in-edges through the reverse map): XCD x (blocks are dealt to the 8
    // XCDs in turn) takes the x-th eighth of the pair's blocks, in which the
    // two jobs alternate unit by unit, so a row read by its source atom's
    // block is read again by its destination atom's block, on the same XCD
    // and at about the same time
    const int l = (lb & 7) * (J.j[k].pair >> 3) + (lb >> 3);
    k += l & 1;
    lb = l >> 1;
  }
  if (J.j[k].wps == 4) segsum_job<4, 8>(J.j[k], red4, lb);
  else segsum_job<1, 4>(J.j[k], red4, lb);
}

// Per bond b (centre i, local index q among k bonds): DZ1 = sum over the
// angles (b, *) of dz, DZ2 = sum over the angles (*, b) of dz, and, if DEB,
// d eb_b += dmu_b * S_b + sum over the angles (*, b) of t2. One
// wavefront per bond; a lane owns CPL consecutive dz columns (dz rows have
// 4d floats, DZ12 rows 8d: DZ1 at column c, DZ2 at 4d + c) and TPL t2
// columns; two independent accumulators per sum (fixed order). Each angle
// row is read by two wavefronts (its first bond's and its second bond's);
// the rotated order below has both read it in the same step, so the second
// read hits L2 (wide128: 1.83 -> 1.07 GB fetched per launch).
template <int CPL, int TPL, bool DEB>
__global__ void __launch_bounds__(256) k_bond_bwd_reduce(int B, int D, const int* __restrict__ bond_src,
                                                         const int* __restrict__ bond_ptr, const int* __restrict__ angle_ptr,
                                                         const float* __restrict__ dzae, const float* __restrict__ t2,
                                                         const float* __restrict__ dmu, const float* __restrict__ ssum,
                                                         float* __restrict__ DZ12, float* __restrict__ deb, int deb_acc) {
  // blocks are dealt to the 8 XCDs in turn; XCD x takes the x-th eighth of
  // the bonds in order, so the bonds of a centre run on one XCD at once
  const int per = gridDim.x >> 3;
  const int blk = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  const int b = blk * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (b >= B) return;
  // the angles of the centre's bond p are rows angle_ptr[k0] + p (k - 1) ..,
  // one per other bond in order (the graph's angle order); angle_ptr[b] is
  // loaded beside bond_src[b], not after the centre's bond range
  const int64_t lo = angle_ptr[b];
  const int i = bond_src[b], k0 = bond_ptr[i], k = bond_ptr[i + 1] - k0, q = b - k0;
  const int64_t ap0 = lo - (int64_t)q * (k - 1);
  const int64_t ld = 4 * D;
  const int c = lane * CPL;
  float s1[2][CPL], s2[2][CPL], tt[2][TPL];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int x = 0; x < CPL; ++x) s1[u][x] = s2[u][x] = 0.f;
#pragma unroll
    for (int x = 0; x < TPL; ++x) tt[u][x] = 0.f;
  }
  // step t: angle (q, q + t) for DZ1 and angle (q - t, q) for DZ2 (bond
  // indices mod k); bond q + t reads the first row as its DZ2 term in the
  // same step, so the wavefronts of a centre share each row in L2
  int j1 = q, j2 = q;
#pragma unroll 2
  for (int t = 1; t < k; ++t) {
    j1 = j1 + 1 == k ? 0 : j1 + 1;
    j2 = j2 == 0 ? k - 1 : j2 - 1;
    const int u = t & 1;
    const int64_t r1 = lo + (j1 < q ? j1 : j1 - 1);
    const int64_t r2 = ap0 + (int64_t)j2 * (k - 1) + (q < j2 ? q : q - 1);
#pragma unroll
    for (int x = 0; x < CPL; ++x) {
      s1[u][x] += dzae[r1 * ld + c + x];
      s2[u][x] += dzae[r2 * ld + c + x];
    }
    if (DEB)
#pragma unroll
      for (int x = 0; x < TPL; ++x) tt[u][x] += t2[r2 * D + lane * TPL + x];
  }
#pragma unroll
  for (int x = 0; x < CPL; ++x) {
    DZ12[(int64_t)b * 8 * D + c + x] = s1[0][x] + s1[1][x];
    DZ12[(int64_t)b * 8 * D + 4 * D + c + x] = s2[0][x] + s2[1][x];
  }
  if (!DEB) return;
#pragma unroll
  for (int x = 0; x < TPL; ++x) {
    const int64_t o = (int64_t)b * D + lane * TPL + x;
    const float v = dmu[o] * ssum[o] + (tt[0][x] + tt[1][x]);
    deb[o] = deb_acc ? deb[o] + v : v;
  }
}

// ---------------------------------------------------------------------------
// Heads: per-structure energy and stress, per-atom forces (Eq. 7, 9).
// ---------------------------------------------------------------------------
__device__ void lattice_units(const float* Lf, double U[9], double& vol) {
  double L[9];
  for (int k = 0; k < 9; ++k) L[k] = (double)Lf[k];
  vol = fabs(L[0] * (L[4] * L[8] - L[5] * L[7]) - L[1] * (L[3] * L[8] - L[5] * L[6]) + L[2] * (L[3] * L[7] - L[4] * L[6]));
  for (int a = 0; a < 3; ++a) {
    const double n = sqrt(L[3 * a] * L[3 * a] + L[3 * a + 1] * L[3 * a + 1] + L[3 * a + 2] * L[3 * a + 2]);
    for (int c = 0; c < 3; ++c) U[3 * a + c] = L[3 * a + c] / n;
  }
}

__global__ void __launch_bounds__(256) k_struct_heads(int S, const int* __restrict__ atom_ptr, const float* __restrict__ lattice,
                                                      const float* __restrict__ oE, const float* __restrict__ oS,
                                                      float* __restrict__ energy, float* __restrict__ stress) {
  const int s = blockIdx.x;
  if (s >= S) return;  // uniform over the block
  __shared__ double red[10][256];
  double acc[10];
  for (int k = 0; k < 10; ++k) acc[k] = 0.0;
  for (int i = atom_ptr[s] + threadIdx.x; i < atom_ptr[s + 1]; i += 256) {
    acc[0] += oE[i];
    for (int k = 0; k < 9; ++k) acc[1 + k] += oS[(int64_t)i * 9 + k];
  }
  for (int k = 0; k < 10; ++k) red[k][threadIdx.x] = acc[k];
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off)
      for (int k = 0; k < 10; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    energy[s] = (float)red[0][0];
    double U[9], vol;
    lattice_units(lattice + 9 * s, U, vol);
    for (int x = 0; x < 3; ++x)
      for (int y = 0; y < 3; ++y) {
        double v = 0.0;
        for (int a = 0; a < 3; ++a)
          for (int b = 0; b < 3; ++b) v += red[1 + 3 * a + b][0] * U[3 * a + x] * U[3 * b + y];
        stress[9 * s + 3 * x + y] = (float)(v / vol);
      }
  }
}

// F_i = sum_e n_e xhat_e, n_e = (m_e + m_rev(e)) / 2; one wavefront per atom,
// lanes stride over its edges, fixed-order wave reduction.
__global__ void __launch_bounds__(256) k_forces(int N, const int* __restrict__ edge_ptr, const int* __restrict__ edge_rev,
                                                const float* __restrict__ oF, const float* __restrict__ xhat,
                                                float* __restrict__ forces) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= N) return;
  float f0 = 0.f, f1 = 0.f, f2 = 0.f;
  for (int e = edge_ptr[i] + lane; e < edge_ptr[i + 1]; e += 64) {
    const float n = 0.5f * (oF[e] + oF[edge_rev[e]]);
    f0 += n * xhat[3 * e];
    f1 += n * xhat[3 * e + 1];
    f2 += n * xhat[3 * e + 2];
  }
  f0 = wsum(f0);
  f1 = wsum(f1);
  f2 = wsum(f2);
  if (lane == 0) {
    forces[3 * i] = f0;
    forces[3 * i + 1] = f1;
    forces[3 * i + 2] = f2;
  }
}

// Magnetic moments: o_i = v_i . w_m + b_m, m_i = |o_i| (mag may be NULL); one
// wavefront per atom, fixed-order wave reduction. o is kept for the loss and
// the backward.
__global__ void __launch_bounds__(256) k_magmom(int N, int D, const float* __restrict__ v, const float* __restrict__ w,
                                                const float* __restrict__ b, float* __restrict__ om,
                                                float* __restrict__ mag) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= N) return;
  float s = 0.f;
  for (int c = lane; c < D; c += 64) s += v[(int64_t)i * D + c] * w[c];
  s = wsum(s);
  if (lane == 0) {
    const float o = s + b[0];
    om[i] = o;
    if (mag) mag[i] = fabsf(o);
  }
}

// g_i = dM_i sign(o_i) (sign(0) = 0); dv_i += g_i w_m.
__global__ void __launch_bounds__(256) k_magmom_bwd(int N, int D, const float* __restrict__ dM, const float* __restrict__ om,
                                                    const float* __restrict__ w, float* __restrict__ g,
                                                    float* __restrict__ dv) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= N) return;
  const float o = om[i];
  const float gi = o > 0.f ? dM[i] : o < 0.f ? -dM[i] : 0.f;
  if (lane == 0) g[i] = gi;
  for (int c = lane; c < D; c += 64) dv[(int64_t)i * D + c] += gi * w[c];
}

// Per-residual loss and derivative: squared error, or Huber's loss with
// threshold delta > 0 (r^2/2 inside [-delta, delta], linear beyond).
__device__ __forceinline__ double rho(double r, double delta, double& g) {
  if (delta <= 0.0) {
    g = 2.0 * r;
    return r * r;
  }
  if (fabs(r) <= delta) {
    g = r;
    return 0.5 * r * r;
  }
  g = r > 0.0 ? delta : -delta;
  return delta * (fabs(r) - 0.5 * delta);
}

// Loss (weighted mean errors, per-atom energy) and its gradient; one block,
// fp64 accumulation in a fixed order.
// one block; per-thread partial sums, then a fixed-order tree over the threads
constexpr int kLossThreads = 1024;
__global__ void __launch_bounds__(kLossThreads) k_loss(int S, int N, const int* __restrict__ atom_ptr, const float* __restrict__ energy,
                                              const float* __restrict__ forces, const float* __restrict__ stress,
                                              const float* __restrict__ om, const float* __restrict__ Et,
                                              const float* __restrict__ Ft, const float* __restrict__ St,
                                              const float* __restrict__ Mt, chgnet_loss lw, float* __restrict__ loss,
                                              float* __restrict__ dE, float* __restrict__ dF, float* __restrict__ dS,
                                              float* __restrict__ dM) {
  __shared__ double red[4][kLossThreads];
  const double delta = lw.huber_delta;
  double le = 0.0, lf = 0.0, ls = 0.0, lm = 0.0, g;
  for (int s = threadIdx.x; s < S; s += kLossThreads) {
    const double n = (double)(atom_ptr[s + 1] - atom_ptr[s]);
    le += rho((double)energy[s] / n - (double)Et[s], delta, g);
    dE[s] = (float)(lw.w_energy * g / n / S);
  }
  for (int k = threadIdx.x; k < 3 * N; k += kLossThreads) {
    lf += rho((double)forces[k] - (double)Ft[k], delta, g);
    dF[k] = (float)(lw.w_force * g / (3.0 * N));
  }
  for (int k = threadIdx.x; k < 9 * S; k += kLossThreads) {
    ls += rho((double)stress[k] - (double)St[k], delta, g);
    dS[k] = (float)(lw.w_stress * g / (9.0 * S));
  }
  if (om)
    for (int k = threadIdx.x; k < N; k += kLossThreads) {
      lm += rho(fabs((double)om[k]) - (double)Mt[k], delta, g);
      dM[k] = (float)(lw.w_magmom * g / N);
    }
  red[0][threadIdx.x] = le;
  red[1][threadIdx.x] = lf;
  red[2][threadIdx.x] = ls;
  red[3][threadIdx.x] = lm;
  __syncthreads();
  for (int off = kLossThreads / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off)
      for (int k = 0; k < 4; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    double l = lw.w_energy * red[0][0] / S + lw.w_force * red[1][0] / (3.0 * N) + lw.w_stress * red[2][0] / (9.0 * S);
    if (om) l += lw.w_magmom * red[3][0] / N;
    loss[0] = (float)l;
  }
}

// Upstream gradients of the head outputs.
__global__ void k_seed_atoms(int N, const int* __restrict__ atom_struct, const float* __restrict__ lattice,
                             const float* __restrict__ dE, const float* __restrict__ dS, float* __restrict__ doE,
                             float* __restrict__ doS) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  const int s = atom_struct[i];
  doE[i] = dE[s];
  double U[9], vol;
  lattice_units(lattice + 9 * s, U, vol);
  for (int a = 0; a < 3; ++a)
    for (int b = 0; b < 3; ++b) {
      double v = 0.0;
      for (int x = 0; x < 3; ++x)
        for (int y = 0; y < 3; ++y) v += (double)dS[9 * s + 3 * x + y] * U[3 * a + x] * U[3 * b + y];
      doS[(int64_t)i * 9 + 3 * a + b] = (float)(v / vol);
    }
}

__global__ void k_seed_edges(int E, const int* __restrict__ edge_src, const float* __restrict__ dF,
                             const float* __restrict__ xhat, float* __restrict__ dn) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int i = edge_src[e];
  dn[e] = dF[3 * i] * xhat[3 * e] + dF[3 * i + 1] * xhat[3 * e + 1] + dF[3 * i + 2] * xhat[3 * e + 2];
}

__global__ void k_seed_edges2(int E, const int* __restrict__ edge_rev, const float* __restrict__ dn, float* __restrict__ doF) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < E) doF[e] = 0.5f * (dn[e] + dn[edge_rev[e]]);
}

// Gradient of the element table W_Z: row z - 1 gets the sum of dv0 over the
// atoms with Z = z. One block per element; wavefront w scans the w-th eighth
// of the atoms (Z of 8 x 64 atoms loaded at once) and adds the rows of its
// matches in atom order, up to 8 rows' loads issued together; the eight
// partial sums are added in wavefront order.
constexpr int kEmbZWaves = 8;
__global__ void __launch_bounds__(64 * kEmbZWaves) k_embed_bwd_Z(int N, int D, const int* __restrict__ Z,
                                                                 const float* __restrict__ dv0, float* __restrict__ gWZ) {
  __shared__ float red[kEmbZWaves][2][64];
  const int z = blockIdx.x + 1, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lo = (int)((int64_t)N * w / kEmbZWaves), hi = (int)((int64_t)N * (w + 1) / kEmbZWaves);
  float acc0 = 0.f, acc1 = 0.f;
  for (int base = lo; base < hi; base += 512) {
    int zz[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = base + 64 * u + lane;
      zz[u] = i < hi ? Z[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      unsigned long long m = __ballot(zz[u] == z);
      const int b0 = base + 64 * u;
      while (m) {
        int rows[8];
        int nr = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          rows[q] = 0;
          if (m) {
            rows[q] = b0 + __ffsll(m) - 1;
            m &= m - 1;
            nr = q + 1;
          }
        }
        float v0[8], v1[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          v0[q] = v1[q] = 0.f;
          if (q < nr) {
            const int64_t row = (int64_t)rows[q] * D;
            v0[q] = dv0[row + lane];
            if (D > 64) v1[q] = dv0[row + 64 + lane];
          }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (q < nr) {
            acc0 += v0[q];
            if (D > 64) acc1 += v1[q];
          }
      }
    }
  }
  red[w][0][lane] = acc0;
  red[w][1][lane] = acc1;
  __syncthreads();
  if (w != 0) return;
  for (int q = 1; q < kEmbZWaves; ++q) {
    acc0 += red[q][0][lane];
    acc1 += red[q][1][lane];
  }
  gWZ[(int64_t)(z - 1) * D + lane] += acc0;
  if (D > 64) gWZ[(int64_t)(z - 1) * D + 64 + lane] += acc1;
}

// Partial sums over rows of d sRBF_n * d sRBF_n / d f_n.
// d(loss)/d f_n of the radial basis: sum over rows of drbf[row, n] times
// d rbf_n / d f_n. A wavefront pass covers 64 / NP rows x NP basis slots
// (NP = 32 or 64 >= R); 64 rows per block; per-block sums into part[block].
__global__ void __launch_bounds__(256) k_rbf_fgrad(int rows, const int* __restrict__ idx, const float* __restrict__ len,
                                                   const float* __restrict__ freq, int R, float cutoff, int p,
                                                   const float* __restrict__ drbf, float* __restrict__ part) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int np = R <= 32 ? 32 : 64, rpp = 64 / np;  // basis slots and rows per pass
  const int n = lane % np, rs = lane / np;
  float acc = 0.f;
  if (n < R) {
    const float inv_c = 1.0f / cutoff, pre = sqrtf(2.0f * inv_c) * inv_c, f = freq[n];
    const int r0 = blockIdx.x * kFreqRowsPerBlock + wave * (kFreqRowsPerBlock / 4);
    for (int rr = rs; rr < kFreqRowsPerBlock / 4; rr += rpp) {
      const int row = r0 + rr;
      if (row >= rows) break;
      const float d = len[idx ? idx[row] : row];
      acc += drbf[(int64_t)row * R + n] * pre * cosf(f * d * inv_c) * envelope(d * inv_c, p);
    }
  }
  // the rpp row slots of a wave hold the same n: fold them, then the waves
  if (np == 32) acc += __shfl_xor(acc, 32);
  if (lane < np) red[wave][lane] = acc;
  __syncthreads();
  if ((int)threadIdx.x < R)
    part[(int64_t)blockIdx.x * R + threadIdx.x] = ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) + red[3][threadIdx.x];
}

__global__ void k_adam(int64_t P, float* __restrict__ params, const float* __restrict__ grad, float* __restrict__ m,
                       float* __restrict__ v, float lr, float b1, float b2, float eps, float c1, float c2) {
  const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= P) return;
  const float g = grad[k];
  const float mk = b1 * m[k] + (1.0f - b1) * g;
  const float vk = b2 * v[k] + (1.0f - b2) * g * g;
  m[k] = mk;
  v[k] = vk;
  params[k] -= lr * (mk / c1) / (sqrtf(vk / c2) + eps);
}

// ---------------------------------------------------------------------------
// Conservative readout: F = -dE/dr, sigma = (1/V) dE/d(eps), from the
// gradients of E with respect to the radial bases (drbf) and the angular
// basis (dft). g_e = dE/dr_e is formed per edge; fp64 arithmetic.
// ---------------------------------------------------------------------------
// sum_n drbf_n d sRBF_n / dr at r (product rule on sin(f r/c) (1/r) u(r/c))
__device__ double drbf_dr(const float* __restrict__ drbf, const float* __restrict__ freq, int R, double r, double c,
                          int p) {
  const double x = r / c;
  double xp1 = 1.0;  // x^(p-1)
  for (int k = 0; k < p - 1; ++k) xp1 *= x;
  const double u = 1.0 + xp1 * x * (-0.5 * (p + 1) * (p + 2) + x * ((double)p * (p + 2) - x * 0.5 * p * (p + 1)));
  const double du = -0.5 * p * (p + 1) * (p + 2) * xp1 * (1.0 - x) * (1.0 - x);
  const double pre = sqrt(2.0 / c);
  double acc = 0.0;
  for (int n = 0; n < R; ++n) {
    const double f = freq[n];
    double sa, ca;
    sincos(f * x, &sa, &ca);
    acc += (double)drbf[n] * pre * (ca * f / c / r * u - sa / (r * r) * u + sa / r * du / c);
  }
  return acc;
}

// g_e = (sum_n drbf_a d sRBF_n(6 A) / dr) r_e / |r_e|
__global__ void k_cons_edges(int E, const float* __restrict__ len, const float* __restrict__ xhat,
                             const float* __restrict__ drbf_a, const float* __restrict__ freq, int R, float cutoff,
                             int p, float* __restrict__ gvec) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const double gd = drbf_dr(drbf_a + (int64_t)e * R, freq, R, len[e], cutoff, p);
  for (int c = 0; c < 3; ++c) gvec[3 * e + c] = (float)(gd * xhat[3 * e + c]);
}

// Per angle: g_theta = sum_k dft_k d FT_k / d theta; p1 = g_theta d theta / d r1,
// p2 = g_theta d theta / d r2 with d theta / d r1 = (c r1 / |r1|^2 - r2) / s
// (c = r1.r2, s = |r1 x r2|; zero when s = 0).
__global__ void k_cons_angles(int A, const int* __restrict__ ang_b1, const int* __restrict__ ang_b2,
                              const int* __restrict__ bond_edge, const int* __restrict__ ang_ctr,
                              const int* __restrict__ edge_dst, const int* __restrict__ edge_img,
                              const int* __restrict__ atom_struct, const float* __restrict__ pos,
                              const float* __restrict__ lattice, const float* __restrict__ dft, int K,
                              float* __restrict__ pang) {
  const int al = blockIdx.x * blockDim.x + threadIdx.x;
  if (al >= A) return;
  const int i = ang_ctr[al];
  const float* L = lattice + 9 * atom_struct[i];
  double r[2][3];
  const int es[2] = {bond_edge[ang_b1[al]], bond_edge[ang_b2[al]]};
  for (int q = 0; q < 2; ++q) {
    const int e = es[q], j = edge_dst[e];
    const double n0 = edge_img[3 * e], n1 = edge_img[3 * e + 1], n2 = edge_img[3 * e + 2];
    for (int c = 0; c < 3; ++c)
      r[q][c] = (double)pos[3 * j + c] + (n0 * (double)L[c] + n1 * (double)L[3 + c] + n2 * (double)L[6 + c]) - (double)pos[3 * i + c];
  }
  const double dot = r[0][0] * r[1][0] + r[0][1] * r[1][1] + r[0][2] * r[1][2];
  const double cx = r[0][1] * r[1][2] - r[0][2] * r[1][1];
  const double cy = r[0][2] * r[1][0] - r[0][0] * r[1][2];
  const double cz = r[0][0] * r[1][1] - r[0][1] * r[1][0];
  const double sn = sqrt(cx * cx + cy * cy + cz * cz);
  const double h = sqrt(dot * dot + sn * sn);
  const double c1 = dot / h, s1 = sn / h;
  const int M = (K - 1) / 2;
  const float* d = dft + (int64_t)al * K;
  const double inv_sqrt_pi = 0.56418958354775628695;
  double gth = 0.0, cm = 1.0, sm = 0.0;
  for (int m = 1; m <= M; ++m) {
    const double cn = cm * c1 - sm * s1, snn = sm * c1 + cm * s1;
    cm = cn;
    sm = snn;
    gth += m * inv_sqrt_pi * (-(double)d[m] * sm + (double)d[M + m] * cm);
  }
  const double inv_s = sn > 0.0 ? 1.0 / sn : 0.0;
  const double n1 = r[0][0] * r[0][0] + r[0][1] * r[0][1] + r[0][2] * r[0][2];
  const double n2 = r[1][0] * r[1][0] + r[1][1] * r[1][1] + r[1][2] * r[1][2];
  for (int c = 0; c < 3; ++c) {
    pang[6 * (int64_t)al + c] = (float)(gth * (dot * r[0][c] / n1 - r[1][c]) * inv_s);
    pang[6 * (int64_t)al + 3 + c] = (float)(gth * (dot * r[1][c] / n2 - r[0][c]) * inv_s);
  }
}

// Per bond b (edge e): g_e += (sum_n drbf_b d sRBF_n(3 A) / dr) r_e / |r_e|
// + sum over angles (b, *) of p1 + sum over angles (*, b) of p2 (fixed order).
__global__ void k_cons_bonds(int B, const int* __restrict__ bond_edge, const int* __restrict__ bond_src,
                             const int* __restrict__ bond_ptr, const int* __restrict__ angle_ptr,
                             const float* __restrict__ len, const float* __restrict__ xhat,
                             const float* __restrict__ drbf_b, const float* __restrict__ freq, int R, float cutoff,
                             int p, const float* __restrict__ pang, float* __restrict__ gvec) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int e = bond_edge[b];
  const double gd = drbf_dr(drbf_b + (int64_t)b * R, freq, R, len[e], cutoff, p);
  double g[3];
  for (int c = 0; c < 3; ++c) g[c] = gd * xhat[3 * e + c];
  for (int al = angle_ptr[b]; al < angle_ptr[b + 1]; ++al)
    for (int c = 0; c < 3; ++c) g[c] += pang[6 * (int64_t)al + c];
  const int i = bond_src[b], k0 = bond_ptr[i], k = bond_ptr[i + 1] - k0, q = b - k0;
  for (int pp = 0; pp < k; ++pp) {
    if (pp == q) continue;
    const int64_t al = angle_ptr[k0 + pp] + (q < pp ? q : q - 1);
    for (int c = 0; c < 3; ++c) g[c] += pang[6 * al + 3 + c];
  }
  for (int c = 0; c < 3; ++c) gvec[3 * e + c] += (float)g[c];
}

// F_i = sum over edges e leaving i of (g_e - g_rev(e)); one wavefront per atom.
__global__ void __launch_bounds__(256) k_cons_forces(int N, const int* __restrict__ edge_ptr,
                                                     const int* __restrict__ edge_rev, const float* __restrict__ gvec,
                                                     float* __restrict__ forces) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= N) return;
  float f[3] = {0.f, 0.f, 0.f};
  for (int e = edge_ptr[i] + lane; e < edge_ptr[i + 1]; e += 64) {
    const int r = edge_rev[e];
    for (int c = 0; c < 3; ++c) f[c] += gvec[3 * e + c] - gvec[3 * r + c];
  }
  for (int c = 0; c < 3; ++c) f[c] = wsum(f[c]);
  if (lane == 0)
    for (int c = 0; c < 3; ++c) forces[3 * i + c] = f[c];
}

// sigma_s = (1/V_s) sum over the edges of crystal s of g_e r_e^T; one block per crystal.
__global__ void __launch_bounds__(256) k_cons_stress(int S, const int* __restrict__ atom_ptr,
                                                     const int* __restrict__ edge_ptr, const float* __restrict__ len,
                                                     const float* __restrict__ xhat, const float* __restrict__ gvec,
                                                     const float* __restrict__ lattice, float* __restrict__ stress) {
  const int s = blockIdx.x;
  if (s >= S) return;  // uniform over the block
  __shared__ double red[9][256];
  double acc[9];
  for (int k = 0; k < 9; ++k) acc[k] = 0.0;
  for (int e = edge_ptr[atom_ptr[s]] + threadIdx.x; e < edge_ptr[atom_ptr[s + 1]]; e += 256) {
    const double l = len[e];
    for (int a = 0; a < 3; ++a)
      for (int b = 0; b < 3; ++b) acc[3 * a + b] += (double)gvec[3 * e + a] * l * (double)xhat[3 * e + b];
  }
  for (int k = 0; k < 9; ++k) red[k][threadIdx.x] = acc[k];
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off)
      for (int k = 0; k < 9; ++k) red[k][threadIdx.x] += red[k][threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x < 9) {
    double U[9], vol;
    lattice_units(lattice + 9 * s, U, vol);
    stress[9 * s + threadIdx.x] = (float)(red[threadIdx.x][0] / vol);
  }
}

// ---------------------------------------------------------------------------
// Velocity Verlet (NVE, fixed lattices). h = dt/2 times the acceleration of
// 1 eV/A on 1 u in A/fs^2.
// ---------------------------------------------------------------------------
// first half kick and drift into the trial state: v' = v + h F / m, x' = x + dt v'
__global__ void k_md_kick_drift(int n3, const float* __restrict__ pos, const float* __restrict__ vel,
                                const float* __restrict__ F, const float* __restrict__ inv_mass, float h, float dt,
                                float* __restrict__ pos2, float* __restrict__ vel2) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= n3) return;
  const float v = vel[k] + h * inv_mass[k / 3] * F[k];
  vel2[k] = v;
  pos2[k] = pos[k] + dt * v;
}

// second half kick with the new forces, and commit of the trial positions
__global__ void k_md_kick_commit(int n3, const float* __restrict__ pos2, const float* __restrict__ vel2,
                                 const float* __restrict__ F, const float* __restrict__ inv_mass, float h,
                                 float* __restrict__ pos, float* __restrict__ vel) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= n3) return;
  vel[k] = vel2[k] + h * inv_mass[k / 3] * F[k];
  pos[k] = pos2[k];
}

// ---------------------------------------------------------------------------
// Workspace carving.
// ---------------------------------------------------------------------------
struct Dims {
  int64_t N, S, E, B, A;
  int D, T, R, K;
};

struct Acts {
  int *atom_struct, *edge_src, *bond_src, *ang_b1, *ang_b2, *ang_ctr;
  float *edge_len, *edge_xhat, *rbf_a, *rbf_b, *ft, *ea, *eb;
  float* v[kMaxLayers + 1];
  float* e[kMaxLayers + 1];
  float* a[kMaxLayers];
  float *zv[kMaxLayers], *zae[kMaxLayers], *m[kMaxLayers], *ssum[kMaxLayers], *mu[kMaxLayers];
  float *msg, *msgb, *Xa[kMaxLayers], *Xb[kMaxLayers];
  float *hE1, *aE1, *hE2, *aE2, *hS1, *aS1, *hS2, *aS2, *hF1, *aF1, *hF2, *aF2, *oE, *oS, *oF, *oM, *gM;
  float* dvf;  // gradient of v^{t+1} including the sequential block's bond and angle inputs
  // two copies of the per-layer backward intermediates, alternating by layer,
  // so a layer's weight gradients can run while the next layer is formed
  float *dzv_pp[2], *dzae_pp[2], *AT_pp[2], *DZ12_pp[2], *dvf_pp[2];
  // backward
  // the gradient of e^t rotates through three copies: the fused backward
  // gate of layer t writes it while the weight gradients of layer t + 1 may
  // still read the copy of e^{t+2}
  float *dv[2], *de[3], *da[2], *dm, *dmu, *dzv, *dzae, *t2, *AT, *DZ12, *dea, *deb;
  float *doE, *doS, *dn, *doF, *dh2E, *dh2S, *dh2F, *dh1ES, *dh1F, *drbf_a, *drbf_b;
  float *lnpart, *tnpart, *fpart, *Pal;
  double* red2;
  int64_t lnpart_stride;
  int64_t tnpart_cap;
  // loss
  float *dE, *dF, *dS, *dM, *out_E, *out_F, *out_S, *out_M;
  // molecular dynamics: trial positions and velocities
  float *md_pos, *md_vel;
  // conservative readout: dE/d FT [A,K], dE/dr_e [E,3], per-angle d theta terms [A,6]
  float *dft, *gvec, *pang;
};

void carve_acts(Arena& ar, const Dims& m, Acts& a, int64_t n_params_aligned) {
  const int64_t N = m.N, S = m.S, E = m.E, B = m.B, A = m.A, D = m.D, R = m.R, K = m.K;
  a.Pal = ar.take<float>(n_params_aligned);
  // carved before anything that depends on the graph sizes: the same address
  // for every graph of the batch
  a.md_pos = ar.take<float>(3 * N);
  a.md_vel = ar.take<float>(3 * N);
  a.atom_struct = ar.take<int>(N);
  a.edge_src = ar.take<int>(E);
  a.bond_src = ar.take<int>(B);
  a.ang_b1 = ar.take<int>(A);
  a.ang_b2 = ar.take<int>(A);
  a.ang_ctr = ar.take<int>(A);
  a.edge_len = ar.take<float>(E);
  a.edge_xhat = ar.take<float>(3 * E);
  a.rbf_a = ar.take<float>(E * R);
  a.rbf_b = ar.take<float>(B * R);
  a.ft = ar.take<float>(A * K);
  a.ea = ar.take<float>(E * D);
  a.eb = ar.take<float>(B * D);
  for (int t = 0; t <= m.T; ++t) {
    a.v[t] = ar.take<float>(N * D);
    a.e[t] = ar.take<float>(E * D);
  }
  for (int t = 0; t < m.T; ++t) {
    a.a[t] = ar.take<float>(A * D);
    a.zv[t] = ar.take<float>(E * 2 * D);
    a.zae[t] = ar.take<float>(A * 4 * D);
    a.m[t] = ar.take<float>(N * D);
    a.ssum[t] = ar.take<float>(B * D);
    a.mu[t] = ar.take<float>(B * D);
  }
  a.msg = ar.take<float>(E * D);
  a.msgb = ar.take<float>(A * D);
  for (int t = 0; t < m.T; ++t) {
    a.Xa[t] = ar.take<float>(N * 8 * D);
    a.Xb[t] = ar.take<float>(B * 8 * D);
  }
  float** atom_heads[] = {&a.hE1, &a.aE1, &a.hE2, &a.aE2, &a.hS1, &a.aS1, &a.hS2, &a.aS2};
  for (auto p : atom_heads) *p = ar.take<float>(N * D);
  float** edge_heads[] = {&a.hF1, &a.aF1, &a.hF2, &a.aF2};
  for (auto p : edge_heads) *p = ar.take<float>(E * D);
  a.oE = ar.take<float>(N);
  a.oS = ar.take<float>(N * 9);
  a.oF = ar.take<float>(E);
  a.oM = ar.take<float>(N);
  a.gM = ar.take<float>(N);
  for (int k = 0; k < 2; ++k) a.dvf_pp[k] = ar.take<float>(N * D);
  a.dvf = a.dvf_pp[0];
  for (int k = 0; k < 2; ++k) {
    a.dv[k] = ar.take<float>(N * D);
    a.da[k] = ar.take<float>(A * D);
  }
  for (int k = 0; k < 3; ++k) a.de[k] = ar.take<float>(E * D);
  a.dm = ar.take<float>(N * D);
  a.dmu = ar.take<float>(B * D);
  for (int k = 0; k < 2; ++k) {
    a.dzv_pp[k] = ar.take<float>(E * 2 * D);
    a.dzae_pp[k] = ar.take<float>(A * 4 * D);
    a.AT_pp[k] = ar.take<float>(N * 8 * D);
    a.DZ12_pp[k] = ar.take<float>(B * 8 * D);
  }
  a.dzv = a.dzv_pp[0];
  a.dzae = a.dzae_pp[0];
  a.AT = a.AT_pp[0];
  a.DZ12 = a.DZ12_pp[0];
  a.t2 = ar.take<float>(A * D);
  a.dea = ar.take<float>(E * D);
  a.deb = ar.take<float>(B * D);
  a.doE = ar.take<float>(N);
  a.doS = ar.take<float>(N * 9);
  a.dn = ar.take<float>(E);
  a.doF = ar.take<float>(E);
  a.dh2E = ar.take<float>(N * D);
  a.dh2S = ar.take<float>(N * D);
  a.dh2F = ar.take<float>(E * D);
  a.dh1ES = ar.take<float>(N * 2 * D);
  a.dh1F = ar.take<float>(E * D);
  a.drbf_a = ar.take<float>(E * R);
  a.drbf_b = ar.take<float>(B * R);
  const int64_t gate_blocks = std::max<int64_t>(cdiv(std::max<int64_t>(std::max(E, A), 1), kGateRows), 256);
  a.lnpart_stride = gate_blocks * 4 * D;
  // LayerNorm parameter partials of every gate of every layer (reduced
  // together at the end of the backward)
  a.lnpart = ar.take<float>(3 * m.T * a.lnpart_stride);
  a.red2 = ar.take<double>((int64_t)kMaxReduceJobs * kReduceGroups * 8 * 128);  // per job: 32 groups x <= 1024 columns
  a.tnpart_cap = kTnPartFloats;
  a.tnpart = ar.take<float>(a.tnpart_cap);
  a.fpart = ar.take<float>(2 * cdiv(std::max(E, (int64_t)1), kFreqRowsPerBlock) * R);
  a.dE = ar.take<float>(S);
  a.dF = ar.take<float>(3 * N);
  a.dS = ar.take<float>(9 * S);
  a.dM = ar.take<float>(N);
  a.out_E = ar.take<float>(S);
  a.out_F = ar.take<float>(3 * N);
  a.out_S = ar.take<float>(9 * S);
  a.out_M = ar.take<float>(N);
  a.dft = ar.take<float>(A * K);
  a.gvec = ar.take<float>(3 * E);
  a.pang = ar.take<float>(6 * A);
}

// ---------------------------------------------------------------------------
// Host-side helpers for building GEMM problem lists.
// ---------------------------------------------------------------------------
GemmProblem gp(int64_t M, int64_t Nc, float* C, int ldc) {
  GemmProblem p{};
  p.M = (int)M;
  p.N = (int)Nc;
  p.C = C;
  p.ldc = ldc;
  return p;
}
void seg(GemmProblem& p, const float* A, int lda, int a_col, int K, const float* B, int ldb, int trans) {
  GemmSeg& s = p.seg[p.nseg++];
  s.A = A;
  s.lda = lda;
  s.a_col = a_col;
  s.K = K;
  s.B = B;
  s.ldb = ldb;
  s.trans = trans;
}

int run_gemms(const std::vector<GemmProblem>& ps, hipStream_t st, const char* tag) {
  GemmBatch b{};
  for (const auto& p : ps) {
    if (p.M <= 0 || p.N <= 0) continue;
    b.p[b.n++] = p;
    if (b.n == kMaxGemmProblems) {
      CHG_TRY(gemm_launch(b, st, tag));
      b.n = 0;
    }
  }
  if (b.n) CHG_TRY(gemm_launch(b, st, tag));
  return CHGNET_OK;
}

TnProblem tp(int64_t R, int M, int Nn, const float* X, int ldx, int x_col, const int* x_rows, const float* Y, int ldy,
             int y_col, const int* y_rows, float* out, int ld_out) {
  TnProblem p{};
  p.R = (int)R;
  p.M = M;
  p.N = Nn;
  p.X = X;
  p.ldx = ldx;
  p.x_col = x_col;
  p.x_rows = x_rows;
  p.Y = Y;
  p.ldy = ldy;
  p.y_col = y_col;
  p.y_rows = y_rows;
  p.out = out;
  p.ld_out = ld_out;
  return p;
}

TnProblem split_out(TnProblem p, int owidth, float* o1, float* o2 = nullptr, float* o3 = nullptr) {
  p.owidth = owidth;
  p.outs[1] = o1;
  p.outs[2] = o2;
  p.outs[3] = o3;
  return p;
}

int run_tns(const std::vector<TnProblem>& ps, const Acts& a, hipStream_t st, const char* tag) {
  TnBatch b{};
  for (const auto& p : ps) {
    b.p[b.n++] = p;
    if (b.n == kMaxTnProblems) {
      CHG_TRY(tn_launch(b, a.tnpart, a.tnpart_cap, st, tag));
      b.n = 0;
    }
  }
  if (b.n) CHG_TRY(tn_launch(b, a.tnpart, a.tnpart_cap, st, tag));
  return CHGNET_OK;
}

int fill(float* p, int64_t n, float v, hipStream_t st) {
  if (n <= 0) return CHGNET_OK;
  KLAUNCH(st, "k_fill", k_fill<<<(unsigned)cdiv(n, 256), 256, 0, st>>>(p, n, v));
  return CHGNET_OK;
}

SegJob seg_job(int64_t nseg, const int* ptr, const int* idx, const float* vals, int ld_in, int width, float* out,
               int ld_out, const float* mul = nullptr, int ld_mul = 0, float* out2 = nullptr, int ld_out2 = 0) {
  SegJob j{};
  j.nseg = (int)nseg;
  j.ncb = (int)cdiv(width, 64);
  j.ptr = ptr;
  j.idx = idx;
  j.vals = vals;
  j.ld_in = ld_in;
  j.width = width;
  j.out = out;
  j.ld_out = ld_out;
  j.mul = mul;
  j.ld_mul = ld_mul;
  j.out2 = out2;
  j.ld_out2 = ld_out2;
  return j;
}

// wps: wavefronts per segment (4 for long segments such as the edges of an
// atom, 1 for short ones such as the angles of a bond)
// wps: wavefronts per (segment, column block) for jobs that do not set
// their own (4 for long segments such as the edges of an atom, 1 for short
// ones such as the angles of a bond)
int segsum_launch(SegJobs J, int wps, hipStream_t st) {
  SegJobs K{};
  int blocks = 0;
  auto al16 = [](const void* p, int ld) { return ((uintptr_t)p & 15) == 0 && (ld & 3) == 0; };
  for (int i = 0; i < J.n; ++i) {
    if (J.j[i].nseg <= 0) continue;
    SegJob& q = K.j[K.n];
    q = J.j[i];
    q.block0 = blocks;
    if (q.wps != 1 && q.wps != 4) q.wps = wps;
    if (q.Wo && (q.width != 64 || q.ncb != 1))
      return fail(CHGNET_EINVAL, "segsum: the fused output linear needs 64-wide rows");
    // four columns a lane where rows and pointers allow 16-byte accesses
    q.lpr = 0;
    const bool vec = !q.Wo && q.width % 4 == 0 && al16(q.vals, q.ld_in) && al16(q.out, q.ld_out) &&
                     (!q.out2 || (al16(q.out2, q.ld_out2) && al16(q.mul, q.ld_mul)));
    if (vec && (q.width >= 256 || 256 % q.width == 0) && q.width >= 64) {
      q.lpr = std::min(64, q.width / 4);
      q.ncb = (int)cdiv(q.width, 4 * q.lpr);
    }
    blocks += (int)cdiv((int64_t)q.nseg * q.ncb, 4 / q.wps);
    K.n++;
  }
  // pairs: a plain job and the next over the same rows through an index
  // (the reverse map) share one interleaved block range
  blocks = 0;
  for (int i = 0; i < K.n; ++i) {
    SegJob& q = K.j[i];
    q.block0 = blocks;
    q.pair = 0;
    const int nb = (int)cdiv((int64_t)q.nseg * q.ncb, 4 / q.wps);
    if (i + 1 < K.n && blocks % 8 == 0) {
      const SegJob& r = K.j[i + 1];
      if (!q.idx && r.idx && r.ptr == q.ptr && r.vals == q.vals && r.nseg == q.nseg && r.ncb == q.ncb &&
          r.wps == q.wps && r.lpr == q.lpr && !q.Wo && !r.Wo) {
        q.pair = (int)(8 * cdiv(2 * (int64_t)nb, 8));
        blocks += q.pair;
        K.j[i + 1].block0 = blocks;
        K.j[i + 1].pair = 0;
        ++i;
        continue;
      }
    }
    blocks += nb;
  }
  if (blocks == 0) return CHGNET_OK;
  KLAUNCH(st, "k_segsum", k_segsum<<<blocks, 256, 0, st>>>(K));
  return CHGNET_OK;
}

int pack_params(const ParamLayout& L, const ParamLayout& La, const float* P, float* Pal, hipStream_t st) {
  for (int k0 = 0; k0 < L.ntensors; k0 += kPackTensors) {
    PackTable t{};
    int chunks = 0;
    for (int k = k0; k < L.ntensors && t.n < kPackTensors; ++k, ++t.n) {
      t.src[t.n] = (int)L.toff[k];
      t.dst[t.n] = (int)La.toff[k];
      t.len[t.n] = (int)L.tlen[k];
      t.chunk0[t.n] = chunks;
      chunks += (int)cdiv(std::max<int64_t>(L.tlen[k], 1), kPackChunk);
    }
    t.chunk0[t.n] = chunks;
    KLAUNCH(st, "k_pack_params", k_pack_params<<<chunks, 256, 0, st>>>(t, P, Pal));
  }
  return CHGNET_OK;
}

// Launch the gates of one layer (forward) as one multi-job kernel.
// Launch the fused forward gates of one layer: a persistent grid of one
// block per compute unit.
int gate_fwd_mm_launch(int D, GateMmJobs J, hipStream_t st) {
  const int rows_per_tile = D == 64 ? MmCfg<64>::Rows : MmCfg<128>::Rows;
  GateMmJobs K{};
  int tiles = 0;
  for (int i = 0; i < J.n; ++i) {
    if (J.j[i].rows <= 0) continue;
    K.j[K.n] = J.j[i];
    K.j[K.n].tile0 = tiles;
    tiles += (int)cdiv(J.j[i].rows, rows_per_tile);
    K.n++;
  }
  K.ntiles = tiles;
  if (tiles == 0) return CHGNET_OK;
  const int grid = std::min(tiles, 256);
  if (D == 64) KLAUNCH(st, "k_gate_fwd", k_gate_fwd_mm<64><<<grid, MmCfg<64>::Threads, 0, st>>>(K));
  else KLAUNCH(st, "k_gate_fwd", k_gate_fwd_mm<128><<<grid, MmCfg<128>::Threads, 0, st>>>(K));
  return CHGNET_OK;
}

GateMmJob mm_job(int D, int mode, int64_t rows, const float* x, const float* W, const float* bias, const GateAdds& ad,
                 LnPtrs ln, const float* mulv, const int* idx, float* out, float* zsave, int ldzs) {
  GateMmJob j{};
  j.mode = mode;
  j.rows = (int)rows;
  j.x = x;
  j.W = W;
  j.ldw = 2 * D;
  j.bias = bias;
  j.ad = ad;
  j.ln = ln;
  j.mulv = mulv;
  j.mul_idx = idx;
  j.out = out;
  j.zsave = zsave;
  j.ldzs = ldzs;
  return j;
}

GateBwdJob bwd_job(int mode, int64_t rows, const float* z, int ldz, LnPtrs ln, const float* up,
                   const int* up_idx, const float* eb, const int* b2_idx, float* aux, float* dz, int lddz) {
  GateBwdJob j{};
  j.mode = mode;
  j.rows = (int)rows;
  j.z = z;
  j.ldz = ldz;
  j.ln = ln;
  j.up = up;
  j.up_idx = up_idx;
  j.eb = eb;
  j.b2_idx = b2_idx;
  j.aux = aux;
  j.dz = dz;
  j.lddz = lddz;
  return j;
}

// Backward gates of one layer in one launch, then one launch reducing each
// job's LayerNorm partials into ln_grad[k].
// Job i writes its LayerNorm parameter partials to slot[i] (lnpart slots of
// 3 x T); with ln_grad their reductions into ln_grad[i] are appended to
// `defer`, to run after the whole backward.
int gate_bwd_launch(int D, GateBwdJobs J, float* const* ln_grad, const int* slot, const Acts& a,
                    std::vector<ReduceJob>& defer, hipStream_t st) {
  GateBwdJobs K{};
  int blocks = 0;
  for (int i = 0; i < J.n; ++i) {
    if (J.j[i].rows <= 0) continue;
    const int nb = (int)cdiv(J.j[i].rows, kGateRows);
    K.j[K.n] = J.j[i];
    K.j[K.n].block0 = blocks;
    K.j[K.n].lnpart = a.lnpart + (int64_t)slot[i] * a.lnpart_stride;
    if (ln_grad) defer.push_back(ReduceJob{K.j[K.n].lnpart, nb, 4 * D, 4 * D, ln_grad[i]});
    blocks += nb;
    K.n++;
  }
  if (blocks == 0) return CHGNET_OK;
  if (D == 64) KLAUNCH(st, "k_gate_bwd", k_gate_bwd<64><<<blocks, 256, 0, st>>>(K));
  else KLAUNCH(st, "k_gate_bwd", k_gate_bwd<128><<<blocks, 256, 0, st>>>(K));
  return CHGNET_OK;
}

// Launch the fused backward gates and their input-gradient products of one
// layer: a persistent grid of at most one block per compute unit.
// slot[gid] is the lnpart slot of gate id gid (0 atom conv, 1 bond conv, 2
// angle update); with ln_grad, each used slot's reduction into ln_grad[gid]
// is appended to `defer`.
int gate_bwd_mm_launch(int D, GateBwdMmJobs J, float* const* ln_grad, const int* slot, const Acts& a,
                       std::vector<ReduceJob>& defer, hipStream_t st) {
  bool used[3] = {false, false, false};
  auto ln_slots = [&](int grid, float** lnpart) -> int {
    if ((int64_t)grid * 4 * D > a.lnpart_stride)
      return fail(CHGNET_EINVAL, "gate_bwd_mm: LayerNorm partial slots too small");
    for (int gid = 0; gid < 3; ++gid) {
      lnpart[gid] = nullptr;
      if (!used[gid] || !ln_grad) continue;
      lnpart[gid] = a.lnpart + (int64_t)slot[gid] * a.lnpart_stride;
      defer.push_back(ReduceJob{lnpart[gid], grid, 4 * D, 4 * D, ln_grad[gid]});
    }
    return CHGNET_OK;
  };
  if (D == 128) {
    // one job per gate; a job's later gates add to the dX its first wrote
    GateBwd128Jobs K{};
    int maxt = 0;
    for (int i = 0; i < J.n; ++i) {
      const GateBwdMmJob& q = J.j[i];
      if (q.rows <= 0) continue;
      for (int g = 0; g < q.ngates; ++g) {
        if (K.n == 3) return fail(CHGNET_EINVAL, "gate_bwd_mm: more than three gates");
        GateBwd128Job& k = K.j[K.n++];
        k.rows = q.rows;
        k.ntiles = (int)cdiv(q.rows, kBm2Rows);
        k.gid = q.gid[g];
        k.g = q.g[g];
        k.W = q.W[g];
        k.res = g == 0 ? q.res : q.dx;
        k.dx = q.dx;
        used[k.gid] = true;
        maxt = std::max(maxt, k.ntiles);
      }
    }
    if (maxt == 0) return CHGNET_OK;
    const int grid = std::min(maxt, 256);
    if (int rc = ln_slots(grid, K.lnpart)) return rc;
    KLAUNCH(st, "k_gate_bwd", k_gate_bwd_mm128<<<grid, kBm2Threads, 0, st>>>(K));
    return CHGNET_OK;
  }
  GateBwdMmJobs K{};
  int tiles = 0;
  for (int i = 0; i < J.n; ++i) {
    if (J.j[i].rows <= 0) continue;
    K.j[K.n] = J.j[i];
    K.j[K.n].tile0 = tiles;
    tiles += (int)cdiv(J.j[i].rows, kMmRows);
    for (int g = 0; g < J.j[i].ngates; ++g) used[J.j[i].gid[g]] = true;
    K.n++;
  }
  K.ntiles = tiles;
  if (tiles == 0) return CHGNET_OK;
  const int grid = std::min(tiles, 256);
  if (int rc = ln_slots(grid, K.lnpart)) return rc;
  KLAUNCH(st, "k_gate_bwd", k_gate_bwd_mm<<<grid, kMmThreads, 0, st>>>(K));
  return CHGNET_OK;
}

GateAdds adds(int n, const float* p0, int ld0, const int* i0, const float* p1, int ld1, const int* i1) {
  GateAdds a{};
  a.n = n;
  a.p[0] = p0; a.ld[0] = ld0; a.idx[0] = i0;
  a.p[1] = p1; a.ld[1] = ld1; a.idx[1] = i1;
  return a;
}

LnPtrs ln_ptrs(const float* P, const GatedOffsets& g) { return LnPtrs{P + g.g_c, P + g.b_c, P + g.g_g, P + g.b_g}; }

struct Ctx {
  const chgnet_hparams* hp;
  const chgnet_batch* batch;
  const chgnet_graph* graph;
  Dims dm;
  ParamLayout L;   // public layout (gradients)
  ParamLayout La;  // aligned layout of the internal weight copy (reads)
  Acts a;
  char* ws;        // workspace, and the bytes the activations use of it
  size_t ws_bytes, ws_used;
  bool save_z = true;  // keep the gate pre-activations for a backward pass
};

int make_ctx(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph, void* ws, size_t ws_bytes,
             Ctx& c) {
  CHG_TRY(validate_hparams(hp));
  CHG_TRY(validate_batch(batch));
  if (!graph) return fail(CHGNET_EINVAL, "graph is NULL");
  if (graph->n_edges < 0 || graph->n_bonds < 0 || graph->n_angles < 0 || graph->n_bonds > graph->n_edges)
    return fail(CHGNET_EINVAL, "graph sizes are invalid");
  if (!graph->edge_ptr || !graph->bond_ptr || !graph->angle_ptr ||
      (graph->n_edges > 0 && (!graph->edge_dst || !graph->edge_img || !graph->edge_rev)) ||
      (graph->n_bonds > 0 && !graph->bond_edge))
    return fail(CHGNET_EINVAL, "graph arrays missing");
  c.hp = hp;
  c.batch = batch;
  c.graph = graph;
  c.dm = Dims{batch->n_atoms, batch->n_struct, graph->n_edges, graph->n_bonds, graph->n_angles,
              hp->d, hp->n_layers, hp->n_rbf, hp->n_fourier};
  c.L = make_layout(*hp, 1);
  c.La = make_layout(*hp, 4);
  Arena ar{static_cast<char*>(ws), ws_bytes, 0};
  ar.used = graph_scratch_bytes(c.dm.N, c.dm.S);
  carve_acts(ar, c.dm, c.a, c.La.total);
  if (!ws || !ar.ok()) return fail(CHGNET_EWORKSPACE, "workspace too small (query chgnet_workspace_size)");
  c.ws = static_cast<char*>(ws);
  c.ws_bytes = ws_bytes;
  c.ws_used = ar.used;
  return CHGNET_OK;
}

// ---------------------------------------------------------------------------
// Forward.
// ---------------------------------------------------------------------------
int forward_impl(Ctx& c, const float* Pflat, float* energy, float* forces, float* stress, float* magmom,
                 hipStream_t st, bool pack = true) {
  const Dims& m = c.dm;
  Acts& a = c.a;
  const ParamLayout& L = c.La;
  if (pack) CHG_TRY(pack_params(c.L, c.La, Pflat, a.Pal, st));
  const float* P = a.Pal;
  const chgnet_graph& g = *c.graph;
  const chgnet_batch& bt = *c.batch;
  const int D = m.D;
  const int64_t N = m.N, S = m.S, E = m.E, B = m.B, A = m.A;

  // geometry, bases and v0 (Eq. 2)
  {
    GeomArgs ga{};
    ga.N = (int)N; ga.S = (int)S; ga.E = (int)E; ga.B = (int)B; ga.A = (int)A; ga.D = D; ga.R = m.R; ga.K = m.K;
    ga.p = c.hp->envelope_p;
    ga.inv_ca = 1.0f / c.hp->r_atom;
    ga.nb_atoms = (int)cdiv(N * D, 256);
    ga.nb_edges = (int)cdiv(E, 256);
    ga.atom_ptr = bt.atom_ptr; ga.Z = bt.Z; ga.edge_ptr = g.edge_ptr; ga.edge_dst = g.edge_dst; ga.edge_img = g.edge_img;
    ga.bond_ptr = g.bond_ptr; ga.bond_edge = g.bond_edge; ga.angle_ptr = g.angle_ptr;
    ga.pos = bt.pos; ga.lattice = bt.lattice; ga.WZ = P + L.W_Z; ga.freq_a = P + L.f_a;
    ga.atom_struct = a.atom_struct; ga.edge_src = a.edge_src; ga.ang_b1 = a.ang_b1; ga.ang_b2 = a.ang_b2; ga.ang_ctr = a.ang_ctr;
    ga.v0 = a.v[0]; ga.edge_len = a.edge_len; ga.edge_xhat = a.edge_xhat; ga.rbf_a = a.rbf_a; ga.ft = a.ft;
    const int64_t blocks = ga.nb_atoms + ga.nb_edges + cdiv(A, 256);
    KLAUNCH(st, "k_geom", k_geom<<<(unsigned)blocks, 256, 0, st>>>(ga));
  }
  if (B > 0)
    KLAUNCH(st, "k_bond_geom", k_bond_geom<<<(unsigned)cdiv(B, 256), 256, 0, st>>>((int)B, m.R, c.hp->envelope_p,
                                                                              1.0f / c.hp->r_bond, g.bond_edge, a.edge_src,
                                                                              a.edge_len, P + L.f_b, a.bond_src, a.rbf_b));
  {
    std::vector<GemmProblem> ps;
    GemmProblem p = gp(E, D, a.e[0], D);
    seg(p, a.rbf_a, m.R, 0, m.R, P + L.W_e, 2 * D, 0);
    p.bias = P + L.b_e0;
    ps.push_back(p);
    p = gp(E, D, a.ea, D);
    seg(p, a.rbf_a, m.R, 0, m.R, P + L.W_e + D, 2 * D, 0);
    ps.push_back(p);
    p = gp(B, D, a.eb, D);
    seg(p, a.rbf_b, m.R, 0, m.R, P + L.W_eb, D, 0);
    ps.push_back(p);
    p = gp(A, D, a.a[0], D);
    seg(p, a.ft, m.K, 0, m.K, P + L.W_th, D, 0);
    p.bias = P + L.b_th;
    ps.push_back(p);
    CHG_TRY(run_gemms(ps, st, "gemm_embed"));
  }

  const bool seq = c.hp->sequential != 0;
  for (int t = 0; t < m.T; ++t) {
    const LayerOffsets& lo = L.layer[t];
    const bool ang = lo.has_angle;
    const float* Wav = P + lo.av.W;
    const float* Wbe = P + lo.be.W;
    const float* Wan = P + lo.an.W;
    // Atom terms of the split first linear layers, Xa blocks k0..k1-1:
    // 0 atom conv v_i, 1 atom conv v_j, 2 bond conv centre, 3 angle centre.
    auto proj_atoms = [&](int k0, int k1, const float* vin) -> int {
      std::vector<GemmProblem> ps;
      for (int k = k0; k < k1; ++k) {
        if (k == 3 && !ang) break;
        const float* W = k == 0 ? Wav : k == 1 ? Wav + D * 2 * D : k == 2 ? Wbe : Wan;
        GemmProblem p = gp(N, 2 * D, a.Xa[t] + k * 2 * D, 8 * D);
        seg(p, vin, D, 0, D, W, 2 * D, 0);
        ps.push_back(p);
      }
      return run_gemms(ps, st, "gemm_proj");
    };
    // Bond terms, Xb blocks in `mask`: 0 bond-conv role b1, 1 angle role b1,
    // 2 bond-conv role b2, 3 angle role b2.
    auto proj_bonds = [&](int mask, const float* ein) -> int {
      std::vector<GemmProblem> ps;
      for (int k = 0; k < 4; ++k) {
        if (!((mask >> k) & 1) || ((k & 1) && !ang)) continue;
        const float* W = (k & 1 ? Wan : Wbe) + (k < 2 ? 1 : 2) * D * 2 * D;
        GemmProblem p = gp(B, 2 * D, a.Xb[t] + k * 2 * D, 8 * D);
        p.a_rows = g.bond_edge;
        seg(p, ein, D, 0, D, W, 2 * D, 0);
        if (k < 2) {
          // the centre atom of an angle is the source atom of its first bond:
          // its term is folded into the first-bond row
          p.res = a.Xa[t] + (4 + 2 * k) * D;
          p.res_ld = 8 * D;
          p.res_rows = a.bond_src;
        }
        ps.push_back(p);
      }
      return run_gemms(ps, st, "gemm_proj");
    };
    const GateAdds ad_av = adds(2, a.Xa[t], 8 * D, a.edge_src, a.Xa[t] + 2 * D, 8 * D, g.edge_dst);
    const GateAdds ad_be = adds(2, a.Xb[t], 8 * D, a.ang_b1, a.Xb[t] + 4 * D, 8 * D, a.ang_b2);
    const GateAdds ad_an = adds(2, a.Xb[t] + 2 * D, 8 * D, a.ang_b1, a.Xb[t] + 6 * D, 8 * D, a.ang_b2);
    const float* Wx_av = Wav + 2 * D * 2 * D;  // rows of e_ij
    const float* Wx_be = Wbe + 3 * D * 2 * D;  // rows of a_ijk
    const float* Wx_an = Wan + 3 * D * 2 * D;
    // GatedMLPs: bit 0 atom conv, bit 1 bond conv, bit 2 angle update
    auto gates = [&](int which) -> int {
      if (!ang) which &= 3;
      // pre-activations formed inside the gate kernel; z kept for a backward
      // pass unless the caller asked for none
      GateMmJobs J{};
      float* zv = c.save_z ? a.zv[t] : nullptr;
      float* zae = c.save_z ? a.zae[t] : nullptr;
      if (which & 1) {
        J.j[J.n] = mm_job(D, FWD_ATOM, E, a.e[t], Wx_av, P + lo.av.b, ad_av, ln_ptrs(P, lo.av), a.ea, nullptr, a.msg,
                          zv, 2 * D);
        J.j[J.n++].xcopy = a.e[t + 1];  // e^{t+1} = e^t outside G^b (the bond rows are updated after)
      }
      if (which & 2)
        J.j[J.n++] = mm_job(D, FWD_BOND, A, a.a[t], Wx_be, P + lo.be.b, ad_be, ln_ptrs(P, lo.be), a.eb, a.ang_b2,
                            a.msgb, zae, 4 * D);
      if (which & 4)
        J.j[J.n++] = mm_job(D, FWD_ANGLE, A, a.a[t], Wx_an, P + lo.an.b, ad_an, ln_ptrs(P, lo.an), a.a[t], nullptr,
                            a.a[t + 1], zae ? zae + 2 * D : nullptr, 4 * D);
      return gate_fwd_mm_launch(D, J, st);
    };
    // messages: m_i = sum over out-edges of e^a * phi_v; mu_b = eb_b * sum over
    // angles (b, b2) of eb_b2 * phi_e
    // at d = 64 the same launch applies the output linears of the updates
    // (v' = v + m Wo + bo; e'_b = e_b + mu Wo + bo): a wavefront holds a row
    const bool fuse_upd = D == 64;
    auto messages = [&](int which) -> int {
      SegJobs J{};
      if (which & 1) {
        SegJob& q = J.j[J.n++];
        q = seg_job(N, g.edge_ptr, nullptr, a.msg, D, D, a.m[t], D);
        q.wps = 4;
        if (fuse_upd) {
          q.Wo = P + lo.av_Wo;
          q.bo = P + lo.av_bo;
          q.res = a.v[t];
          q.upd = a.v[t + 1];
        }
      }
      if (which & 2) {
        SegJob& q = J.j[J.n++];
        q = seg_job(B, g.angle_ptr, nullptr, a.msgb, D, D, a.ssum[t], D, a.eb, D, a.mu[t], D);
        q.wps = 1;
        if (fuse_upd) {
          q.Wo = P + lo.be_Wo;
          q.bo = P + lo.be_bo;
          q.res = a.e[t];
          q.upd = a.e[t + 1];
          q.upd_rows = g.bond_edge;
        }
      }
      return segsum_launch(J, 4, st);
    };
    // updates: v' = v + m Wo + bo; e' = e (+ mu Wo + bo on bonds)
    auto updates = [&](int which) -> int {
      if (fuse_upd) return CHGNET_OK;  // done by the message launch (and the copy by the atom-conv gate)
      std::vector<GemmProblem> ps;
      if (which & 1) {
        GemmProblem p = gp(N, D, a.v[t + 1], D);
        seg(p, a.m[t], D, 0, D, P + lo.av_Wo, D, 0);
        p.bias = P + lo.av_bo;
        p.res = a.v[t];
        p.res_ld = D;
        ps.push_back(p);
      }
      if (which & 2) {
        // the atom-conv gate launch wrote e^{t+1} = e^t; the bond rows follow
        GemmProblem p = gp(B, D, a.e[t + 1], D);
        seg(p, a.mu[t], D, 0, D, P + lo.be_Wo, D, 0);
        p.bias = P + lo.be_bo;
        p.res = a.e[t];
        p.res_ld = D;
        p.res_rows = g.bond_edge;
        p.c_rows = g.bond_edge;
        ps.push_back(p);
      }
      return run_gemms(ps, st, "gemm_update");
    };
    if (!seq) {
      // Eq. (11): the three modules read layer-t features and run together
      CHG_TRY(proj_atoms(0, 4, a.v[t]));
      CHG_TRY(proj_bonds(15, a.e[t]));
      CHG_TRY(gates(7));
      CHG_TRY(messages(3));
      CHG_TRY(updates(3));
    } else {
      // Eq. (10): atom conv, then bond conv on v^{t+1}, then the angle update
      // on v^{t+1} and e^{t+1}
      CHG_TRY(proj_atoms(0, 2, a.v[t]));
      CHG_TRY(gates(1));
      CHG_TRY(messages(1));
      CHG_TRY(updates(1));
      CHG_TRY(proj_atoms(2, 4, a.v[t + 1]));
      CHG_TRY(proj_bonds(5, a.e[t]));
      CHG_TRY(gates(2));
      CHG_TRY(messages(2));
      CHG_TRY(updates(2));
      if (ang) {
        CHG_TRY(proj_bonds(10, a.e[t + 1]));
        CHG_TRY(gates(4));
      }
    }
  }

  // heads: MLP d -> d -> d -> out with SiLU (d = 128: three GEMM launches)
  if (D != 64) {
    const HeadOffsets &hE = L.head[0], &hF = L.head[1], &hS = L.head[2];
    const float* vT = a.v[m.T];
    const float* eT = a.e[m.T];
    std::vector<GemmProblem> ps;
    struct Lay { const float* in; int64_t M; const HeadOffsets* h; float *h1, *a1, *h2, *a2, *o; };
    Lay ls[3] = {{vT, N, &hE, a.hE1, a.aE1, a.hE2, a.aE2, a.oE},
                 {vT, N, &hS, a.hS1, a.aS1, a.hS2, a.aS2, a.oS},
                 {eT, E, &hF, a.hF1, a.aF1, a.hF2, a.aF2, a.oF}};
    for (auto& l : ls) {
      GemmProblem p = gp(l.M, D, l.h1, D);
      seg(p, l.in, D, 0, D, P + l.h->W1, D, 0);
      p.bias = P + l.h->b1;
      p.act = ACT_SILU_OUT;
      p.C2 = l.a1;
      p.ldc2 = D;
      ps.push_back(p);
    }
    CHG_TRY(run_gemms(ps, st, "gemm_head1"));
    ps.clear();
    for (auto& l : ls) {
      GemmProblem p = gp(l.M, D, l.h2, D);
      seg(p, l.a1, D, 0, D, P + l.h->W2, D, 0);
      p.bias = P + l.h->b2;
      p.act = ACT_SILU_OUT;
      p.C2 = l.a2;
      p.ldc2 = D;
      ps.push_back(p);
    }
    CHG_TRY(run_gemms(ps, st, "gemm_head2"));
    ps.clear();
    for (auto& l : ls) {
      GemmProblem p = gp(l.M, l.h->out, l.o, l.h->out);
      seg(p, l.a2, D, 0, D, P + l.h->W3, l.h->out, 0);
      p.bias = P + l.h->b3;
      ps.push_back(p);
    }
    CHG_TRY(run_gemms(ps, st, "gemm_head3"));
  }
  if (D == 64) {
    // heads: MLP d -> d -> d -> out with SiLU, the three layers in one launch
    const HeadOffsets &hE = L.head[0], &hF = L.head[1], &hS = L.head[2];
    HeadJobs J{};
    int tiles = 0;
    auto add = [&](const float* x, int64_t rows, const HeadOffsets& h, float* h1, float* a1, float* h2, float* a2, float* o) {
      if (rows <= 0) return;
      HeadJob& q = J.j[J.n++];
      q = HeadJob{(int)rows, tiles, h.out, x, P + h.W1, P + h.b1, P + h.W2, P + h.b2, P + h.W3, P + h.b3, h1, a1, h2, a2, o};
      tiles += (int)cdiv(rows, kHdRows);
    };
    add(a.e[m.T], E, hF, a.hF1, a.aF1, a.hF2, a.aF2, a.oF);
    add(a.v[m.T], N, hE, a.hE1, a.aE1, a.hE2, a.aE2, a.oE);
    add(a.v[m.T], N, hS, a.hS1, a.aS1, a.hS2, a.aS2, a.oS);
    J.ntiles = tiles;
    const int blocks = (int)std::min<int64_t>(cdiv(tiles, 4), 512);
    KLAUNCH(st, "k_head_mlp", k_head_mlp<<<blocks, 256, 0, st>>>(J));
  }
  KLAUNCH(st, "k_struct_heads", k_struct_heads<<<(unsigned)S, 256, 0, st>>>((int)S, bt.atom_ptr, bt.lattice, a.oE, a.oS, energy, stress));
  KLAUNCH(st, "k_forces", k_forces<<<(unsigned)cdiv(N, 4), 256, 0, st>>>((int)N, g.edge_ptr, g.edge_rev, a.oF, a.edge_xhat, forces));
  if (c.hp->magmom)
    KLAUNCH(st, "k_magmom", k_magmom<<<(unsigned)cdiv(N, 4), 256, 0, st>>>((int)N, D, a.v[m.T], P + L.M_W, P + L.M_b,
                                                                            a.oM, magmom));
  return CHGNET_OK;
}

// ---------------------------------------------------------------------------
// Backward (weights only).
// ---------------------------------------------------------------------------
// Weight gradients run on a second stream of the device (default priority),
// forked from and joined back into the caller's stream by events; one set
// per host thread and device, created on first use.
struct SideStream {
  hipStream_t side = nullptr;
  hipEvent_t ready[kMaxLayers], done[kMaxLayers], heads, embed, fin;
};

int side_stream(SideStream*& out) {
  constexpr int kMaxDevices = 64;
  thread_local SideStream cache[kMaxDevices];
  int dev = 0;
  CHG_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(CHGNET_EHIP, "device index out of range");
  SideStream& ss = cache[dev];
  if (!ss.side) {
    CHG_HIP(hipStreamCreateWithFlags(&ss.side, hipStreamNonBlocking));
    auto mk = [](hipEvent_t& e) { return hipEventCreateWithFlags(&e, hipEventDisableTiming); };
    for (int t = 0; t < kMaxLayers; ++t) {
      CHG_HIP(mk(ss.ready[t]));
      CHG_HIP(mk(ss.done[t]));
    }
    CHG_HIP(mk(ss.heads));
    CHG_HIP(mk(ss.embed));
    CHG_HIP(mk(ss.fin));
  }
  out = &ss;
  return CHGNET_OK;
}

// the side stream waits for everything enqueued on st so far
int side_fork(SideStream& ss, hipStream_t st, hipEvent_t e) {
  CHG_HIP(hipEventRecord(e, st));
  CHG_HIP(hipStreamWaitEvent(ss.side, e, 0));
  return CHGNET_OK;
}

// G == nullptr: input gradients only (no weight gradients); dft_out != nullptr:
// also dE/d FT = da^0 W_th^T [A,K] for the conservative readout.
int backward_impl(Ctx& c, const float* Pflat, bool repack, const float* dE, const float* dF, const float* dS,
                  const float* dM, float* G, hipStream_t st, float* dft_out = nullptr) {
  const Dims& m = c.dm;
  Acts& a = c.a;
  const ParamLayout& L = c.La;   // reads from the aligned weight copy
  const ParamLayout& Lg = c.L;   // gradients in the public layout
  if (repack) CHG_TRY(pack_params(c.L, c.La, Pflat, a.Pal, st));
  const float* P = a.Pal;
  const chgnet_graph& g = *c.graph;
  const chgnet_batch& bt = *c.batch;
  const int D = m.D;
  const int64_t N = m.N, E = m.E, B = m.B, A = m.A;

  const bool wg = G != nullptr;
  SideStream* ssp = nullptr;
  if (wg) {
    CHG_TRY(fill(G, Lg.total, 0.f, st));
    CHG_TRY(side_stream(ssp));
  }
  std::vector<ReduceJob> reduce_jobs;  // ordered partial sums, run at the end
  SideStream no_side;
  if (wg && prof_active()) {
    // per-launch timing: everything on the caller's stream, so each
    // launch's duration is its own
    no_side = *ssp;
    no_side.side = st;
    ssp = &no_side;
  }
  SideStream& ss = wg ? *ssp : no_side;

  // heads
  KLAUNCH(st, "k_seed_atoms", k_seed_atoms<<<(unsigned)cdiv(N, 256), 256, 0, st>>>((int)N, a.atom_struct, bt.lattice, dE, dS, a.doE, a.doS));
  if (E > 0) {
    KLAUNCH(st, "k_seed_edges", k_seed_edges<<<(unsigned)cdiv(E, 256), 256, 0, st>>>((int)E, a.edge_src, dF, a.edge_xhat, a.dn));
    KLAUNCH(st, "k_seed_edges2", k_seed_edges2<<<(unsigned)cdiv(E, 256), 256, 0, st>>>((int)E, g.edge_rev, a.dn, a.doF));
  }
  int cur = 0, ecur = 0;  // dv and da alternate between two copies, de rotates through three
  {
    const HeadOffsets &hE = L.head[0], &hF = L.head[1], &hS = L.head[2];
    struct Lay {
      const float* in;
      int64_t M;
      const HeadOffsets* h;
      const HeadOffsets* hg;
      const float *h1, *a1, *h2, *a2, *dout;
      float *dh2, *dh1base;
      int dh1col, ld1;
    };
    Lay ls[3] = {{a.v[m.T], N, &hE, &Lg.head[0], a.hE1, a.aE1, a.hE2, a.aE2, a.doE, a.dh2E, a.dh1ES, 0, 2 * D},
                 {a.v[m.T], N, &hS, &Lg.head[2], a.hS1, a.aS1, a.hS2, a.aS2, a.doS, a.dh2S, a.dh1ES, D, 2 * D},
                 {a.e[m.T], E, &hF, &Lg.head[1], a.hF1, a.aF1, a.hF2, a.aF2, a.doF, a.dh2F, a.dh1F, 0, D}};
    std::vector<GemmProblem> ps;
    for (auto& l : ls) {
      GemmProblem p = gp(l.M, D, l.dh2, D);
      seg(p, l.dout, l.h->out, 0, l.h->out, P + l.h->W3, l.h->out, 1);
      p.act = ACT_DSILU_MUL;
      p.mul = l.h2;
      p.mul_ld = D;
      ps.push_back(p);
    }
    CHG_TRY(run_gemms(ps, st, "gemm_head_bwd2"));
    ps.clear();
    for (auto& l : ls) {
      GemmProblem p = gp(l.M, D, l.dh1base + l.dh1col, l.ld1);
      seg(p, l.dh2, D, 0, D, P + l.h->W2, D, 1);
      p.act = ACT_DSILU_MUL;
      p.mul = l.h1;
      p.mul_ld = D;
      ps.push_back(p);
    }
    CHG_TRY(run_gemms(ps, st, "gemm_head_bwd1"));
    ps.clear();
    {
      GemmProblem p = gp(N, D, a.dv[cur], D);
      seg(p, a.dh1ES, 2 * D, 0, D, P + hE.W1, D, 1);
      seg(p, a.dh1ES, 2 * D, D, D, P + hS.W1, D, 1);
      ps.push_back(p);
      p = gp(E, D, a.de[ecur], D);
      seg(p, a.dh1F, D, 0, D, P + hF.W1, D, 1);
      ps.push_back(p);
      CHG_TRY(run_gemms(ps, st, "gemm_head_bwd0"));
    }
    const bool mag = c.hp->magmom && dM;
    if (mag)
      KLAUNCH(st, "k_magmom_bwd", k_magmom_bwd<<<(unsigned)cdiv(N, 4), 256, 0, st>>>((int)N, D, dM, a.oM, P + L.M_W, a.gM,
                                                                                      a.dv[cur]));
    std::vector<TnProblem> ts;
    for (auto& l : ls) {
      const int o = l.h->out;
      ts.push_back(tp(l.M, D, o, l.a2, D, 0, nullptr, l.dout, o, 0, nullptr, G + l.hg->W3, o));
      ts.push_back(tp(l.M, 1, o, nullptr, 0, 0, nullptr, l.dout, o, 0, nullptr, G + l.hg->b3, o));
      ts.push_back(tp(l.M, D, D, l.a1, D, 0, nullptr, l.dh2, D, 0, nullptr, G + l.hg->W2, D));
      ts.push_back(tp(l.M, 1, D, nullptr, 0, 0, nullptr, l.dh2, D, 0, nullptr, G + l.hg->b2, D));
    }
    // first layers: energy and stress heads share the input v^T
    ts.push_back(split_out(tp(N, D, 2 * D, a.v[m.T], D, 0, nullptr, a.dh1ES, 2 * D, 0, nullptr, G + Lg.head[0].W1, D), D,
                           G + Lg.head[2].W1));
    ts.push_back(split_out(tp(N, 1, 2 * D, nullptr, 0, 0, nullptr, a.dh1ES, 2 * D, 0, nullptr, G + Lg.head[0].b1, D), D,
                           G + Lg.head[2].b1));
    ts.push_back(tp(E, D, D, a.e[m.T], D, 0, nullptr, a.dh1F, D, 0, nullptr, G + Lg.head[1].W1, D));
    ts.push_back(tp(E, 1, D, nullptr, 0, 0, nullptr, a.dh1F, D, 0, nullptr, G + Lg.head[1].b1, D));
    if (mag) {
      ts.push_back(tp(N, D, 1, a.v[m.T], D, 0, nullptr, a.gM, 1, 0, nullptr, G + Lg.M_W, 1));
      ts.push_back(tp(N, 1, 1, nullptr, 0, 0, nullptr, a.gM, 1, 0, nullptr, G + Lg.M_b, 1));
    }
    if (wg) {
      CHG_TRY(side_fork(ss, st, ss.heads));
      CHG_TRY(run_tns(ts, a, ss.side, "tn_heads"));
    }
  }

  // interaction blocks in reverse
  const bool seq = c.hp->sequential != 0;
  // with the Eq. 11 block the gate backward also forms the input gradients
  // of the edge and angle rows (k_gate_bwd_mm, k_gate_bwd_mm128)
  const bool fused = !seq;
  for (int t = m.T - 1; t >= 0; --t) {
    const LayerOffsets& lo = L.layer[t];
    const LayerOffsets& lg = Lg.layer[t];
    const bool ang = lo.has_angle;
    const int W4 = ang ? 4 * D : 2 * D;
    a.dzv = a.dzv_pp[t & 1];
    a.dzae = a.dzae_pp[t & 1];
    a.AT = a.AT_pp[t & 1];
    a.DZ12 = a.DZ12_pp[t & 1];
    a.dvf = a.dvf_pp[t & 1];
    const float* Wav = P + lo.av.W;
    const float* Wbe = P + lo.be.W;
    const float* Wan = P + lo.an.W;
    const int nx = 1 - cur, enx = (ecur + 1) % 3;
    std::vector<GemmProblem> ps;
    std::vector<TnProblem> ts;
    // GatedMLP backward: bit 0 atom conv, bit 1 bond conv, bit 2 angle update
    auto gates = [&](int which) -> int {
      if (!ang) which &= 3;
      GateBwdJobs J{};
      float* lg_out[3];
      int slot[3];
      if (which & 2) {
        slot[J.n] = 3 * t;
        lg_out[J.n] = G + lg.be.g_c;
        J.j[J.n++] = bwd_job(BWD_BOND, A, a.zae[t], 4 * D, ln_ptrs(P, lo.be), a.dmu, a.ang_b1, a.eb, a.ang_b2,
                             a.t2, a.dzae, 4 * D);
      }
      if (which & 1) {
        slot[J.n] = 3 * t + 1;
        lg_out[J.n] = G + lg.av.g_c;
        J.j[J.n++] = bwd_job(BWD_ATOM, E, a.zv[t], 2 * D, ln_ptrs(P, lo.av), a.dm, a.edge_src, a.ea, nullptr,
                             a.dea, a.dzv, 2 * D);
        J.j[J.n - 1].aux_acc = t < m.T - 1;  // the first layer of the backward starts d e^a
      }
      if (which & 4) {
        slot[J.n] = 3 * t + 2;
        lg_out[J.n] = G + lg.an.g_c;
        J.j[J.n++] = bwd_job(BWD_ANGLE, A, a.zae[t] + 2 * D, 4 * D, ln_ptrs(P, lo.an), a.da[cur], nullptr,
                             nullptr, nullptr, nullptr, a.dzae + 2 * D, 4 * D);
      }
      return gate_bwd_launch(D, J, wg ? lg_out : nullptr, slot, a, reduce_jobs, st);
    };
    // fused gate backward and edge/angle input gradients: edges
    // de(e^t) = de(e^{t+1}) + dz_v W_av,e^T; angles da(a^t) = da(a^{t+1}) +
    // dz_b W_be,a^T + dz_a W_an,a^T (no angle update in the last layer)
    auto gates_mm = [&]() -> int {
      GateBwdMmJobs J{};
      {
        GateBwdMmJob& q = J.j[J.n++];
        q.rows = (int)E;
        q.ngates = 1;
        q.gid[0] = 0;
        q.g[0] = bwd_job(BWD_ATOM, E, a.zv[t], 2 * D, ln_ptrs(P, lo.av), a.dm, a.edge_src, a.ea, nullptr, a.dea,
                         a.dzv, 2 * D);
        q.g[0].aux_acc = t < m.T - 1;  // the first layer of the backward starts d e^a
        q.W[0] = Wav + 2 * D * 2 * D;
        q.res = a.de[ecur];
        q.dx = a.de[enx];
      }
      {
        GateBwdMmJob& q = J.j[J.n++];
        q.rows = (int)A;
        q.ngates = ang ? 2 : 1;
        q.gid[0] = 1;
        q.g[0] = bwd_job(BWD_BOND, A, a.zae[t], 4 * D, ln_ptrs(P, lo.be), a.dmu, a.ang_b1, a.eb, a.ang_b2, a.t2,
                         a.dzae, 4 * D);
        q.W[0] = Wbe + 3 * D * 2 * D;
        if (ang) {
          q.gid[1] = 2;
          q.g[1] = bwd_job(BWD_ANGLE, A, a.zae[t] + 2 * D, 4 * D, ln_ptrs(P, lo.an), a.da[cur], nullptr, nullptr,
                           nullptr, nullptr, a.dzae + 2 * D, 4 * D);
          q.W[1] = Wan + 3 * D * 2 * D;
          q.res = a.da[cur];
        }
        q.dx = a.da[nx];
      }
      const int slot[3] = {3 * t + 1, 3 * t, 3 * t + 2};
      if (!wg) return gate_bwd_mm_launch(D, J, nullptr, slot, a, reduce_jobs, st);
      float* lg_out[3] = {G + lg.av.g_c, G + lg.be.g_c, G + lg.an.g_c};
      return gate_bwd_mm_launch(D, J, lg_out, slot, a, reduce_jobs, st);
    };
    // per-bond sums of dz over the bond's two angle roles (DZ12) from `ncols`
    // columns of dzae starting at col0; with_deb also forms d e^b
    auto bond_reduce = [&](int col0, int ncols, bool with_deb) -> int {
      if (B <= 0) return CHGNET_OK;
      const unsigned nb = (unsigned)(8 * cdiv(B, 32));  // a multiple of 8 (one share per XCD)
      const int cpl = ncols / 64;
      const float* dz = a.dzae + col0;
      float* dz12 = a.DZ12 + col0;
      const int acc = t < m.T - 1;
#define BOND_REDUCE(CPL, TPL, DEB)                                                                                \
  KLAUNCH(st, "k_bond_bwd_reduce", k_bond_bwd_reduce<CPL, TPL, DEB><<<nb, 256, 0, st>>>((int)B, D, a.bond_src,      \
                                     g.bond_ptr, g.angle_ptr, dz, a.t2, a.dmu, a.ssum[t], dz12, a.deb, acc))
      if (with_deb) {
        if (cpl == 2) BOND_REDUCE(2, 1, true);
        else if (cpl == 4 && D == 64) BOND_REDUCE(4, 1, true);
        else if (cpl == 4) BOND_REDUCE(4, 2, true);
        else BOND_REDUCE(8, 2, true);
      } else {
        if (cpl == 2) BOND_REDUCE(2, 1, false);
        else BOND_REDUCE(4, 2, false);
      }
#undef BOND_REDUCE
      return CHGNET_OK;
    };
    // output linears of the atom and bond updates: dm = dv' Wo^T, dmu = de'_b Wo^T
    auto out_bwd = [&](const float* dvo, bool atoms, bool bonds) -> int {
      std::vector<GemmProblem> q;
      if (atoms) {
        GemmProblem p = gp(N, D, a.dm, D);
        seg(p, dvo, D, 0, D, P + lo.av_Wo, D, 1);
        q.push_back(p);
      }
      if (bonds) {
        GemmProblem p = gp(B, D, a.dmu, D);
        p.a_rows = g.bond_edge;
        seg(p, a.de[ecur], D, 0, D, P + lo.be_Wo, D, 1);
        q.push_back(p);
      }
      return run_gemms(q, st, "gemm_out_bwd");
    };
    SegJobs sj{};
    if (!seq) {
      CHG_TRY(out_bwd(a.dv[cur], true, true));
      CHG_TRY(fused ? gates_mm() : gates(7));
      CHG_TRY(bond_reduce(0, W4, true));
      sj.j[sj.n++] = seg_job(N, g.edge_ptr, nullptr, a.dzv, 2 * D, 2 * D, a.AT, 8 * D);
      sj.j[sj.n++] = seg_job(N, g.edge_ptr, g.edge_rev, a.dzv, 2 * D, 2 * D, a.AT + 2 * D, 8 * D);
      sj.j[sj.n++] = seg_job(N, g.bond_ptr, nullptr, a.DZ12, 8 * D, W4, a.AT + 4 * D, 8 * D);
      CHG_TRY(segsum_launch(sj, 4, st));
    } else {
      // Eq. (10), in reverse: the angle update read e^{t+1} (its bond terms
      // join de', the gradient of e^{t+1}) and v^{t+1}; the bond conv read
      // v^{t+1}; both centre terms join dvf, the gradient of v^{t+1}, before
      // the atom conv.
      if (ang) {
        CHG_TRY(gates(4));
        CHG_TRY(bond_reduce(2 * D, 2 * D, false));
        GemmProblem p = gp(B, D, a.de[ecur], D);
        p.c_rows = g.bond_edge;
        p.accumulate = 1;
        seg(p, a.DZ12, 8 * D, 2 * D, 2 * D, Wan + D * 2 * D, 2 * D, 1);
        seg(p, a.DZ12, 8 * D, 6 * D, 2 * D, Wan + 2 * D * 2 * D, 2 * D, 1);
        ps.push_back(p);
        CHG_TRY(run_gemms(ps, st, "gemm_bond_bwd"));
        ps.clear();
      }
      CHG_TRY(out_bwd(nullptr, false, true));
      CHG_TRY(gates(2));
      CHG_TRY(bond_reduce(0, 2 * D, true));
      sj.j[sj.n++] = seg_job(N, g.bond_ptr, nullptr, a.DZ12, 8 * D, W4, a.AT + 4 * D, 8 * D);
      CHG_TRY(segsum_launch(sj, 4, st));
      GemmProblem p = gp(N, D, a.dvf, D);
      seg(p, a.AT, 8 * D, 4 * D, 2 * D, Wbe, 2 * D, 1);
      if (ang) seg(p, a.AT, 8 * D, 6 * D, 2 * D, Wan, 2 * D, 1);
      p.res = a.dv[cur];
      p.res_ld = D;
      ps.push_back(p);
      CHG_TRY(run_gemms(ps, st, "gemm_in_bwd"));
      ps.clear();
      CHG_TRY(out_bwd(a.dvf, true, false));
      CHG_TRY(gates(1));
      sj = SegJobs{};
      sj.j[sj.n++] = seg_job(N, g.edge_ptr, nullptr, a.dzv, 2 * D, 2 * D, a.AT, 8 * D);
      sj.j[sj.n++] = seg_job(N, g.edge_ptr, g.edge_rev, a.dzv, 2 * D, 2 * D, a.AT + 2 * D, 8 * D);
      CHG_TRY(segsum_launch(sj, 4, st));
    }
    // gradient of v^{t+1} as seen by the atom update
    const float* dvo = seq ? a.dvf : a.dv[cur];
    ts.push_back(tp(N, D, D, a.m[t], D, 0, nullptr, dvo, D, 0, nullptr, G + lg.av_Wo, D));
    ts.push_back(tp(N, 1, D, nullptr, 0, 0, nullptr, dvo, D, 0, nullptr, G + lg.av_bo, D));
    ts.push_back(tp(B, D, D, a.mu[t], D, 0, nullptr, a.de[ecur], D, 0, g.bond_edge, G + lg.be_Wo, D));
    ts.push_back(tp(B, 1, D, nullptr, 0, 0, nullptr, a.de[ecur], D, 0, g.bond_edge, G + lg.be_bo, D));
    // weight gradients of the first linear layers
    {
      const float* vt = a.v[t];
      const float* et = a.e[t];
      if (!seq) {
        // v^T [dP | dQ | DZa_bond | DZa_angle] -> atom-role blocks of the three first layers
        ts.push_back(split_out(tp(N, D, (ang ? 8 : 6) * D, vt, D, 0, nullptr, a.AT, 8 * D, 0, nullptr, G + lg.av.W, 2 * D),
                               2 * D, G + lg.av.W + D * 2 * D, G + lg.be.W, ang ? G + lg.an.W : nullptr));
      } else {
        // the atom conv read v^t; the bond conv and angle update read v^{t+1}
        ts.push_back(split_out(tp(N, D, 4 * D, vt, D, 0, nullptr, a.AT, 8 * D, 0, nullptr, G + lg.av.W, 2 * D), 2 * D,
                               G + lg.av.W + D * 2 * D));
        ts.push_back(split_out(tp(N, D, (ang ? 4 : 2) * D, a.v[t + 1], D, 0, nullptr, a.AT, 8 * D, 4 * D, nullptr,
                                  G + lg.be.W, 2 * D),
                               2 * D, ang ? G + lg.an.W : nullptr));
      }
      ts.push_back(tp(E, D, 2 * D, et, D, 0, nullptr, a.dzv, 2 * D, 0, nullptr, G + lg.av.W + 2 * D * 2 * D, 2 * D));
      // biases: sum over atoms of dP (= sum over edges of dz) and of DZa
      ts.push_back(tp(N, 1, 2 * D, nullptr, 0, 0, nullptr, a.AT, 8 * D, 0, nullptr, G + lg.av.b, 2 * D));
      ts.push_back(split_out(tp(N, 1, (ang ? 4 : 2) * D, nullptr, 0, 0, nullptr, a.AT, 8 * D, 4 * D, nullptr, G + lg.be.b, 2 * D),
                             2 * D, ang ? G + lg.an.b : nullptr));
      if (ang && !seq) {
        // e_b^T [DZ1_bond | DZ1_angle | DZ2_bond | DZ2_angle]
        ts.push_back(split_out(tp(B, D, 8 * D, et, D, 0, g.bond_edge, a.DZ12, 8 * D, 0, nullptr, G + lg.be.W + D * 2 * D, 2 * D),
                               2 * D, G + lg.an.W + D * 2 * D, G + lg.be.W + 2 * D * 2 * D, G + lg.an.W + 2 * D * 2 * D));
      } else {
        ts.push_back(tp(B, D, 2 * D, et, D, 0, g.bond_edge, a.DZ12, 8 * D, 0, nullptr, G + lg.be.W + D * 2 * D, 2 * D));
        ts.push_back(tp(B, D, 2 * D, et, D, 0, g.bond_edge, a.DZ12, 8 * D, 4 * D, nullptr, G + lg.be.W + 2 * D * 2 * D, 2 * D));
        if (ang) {
          // the angle update of Eq. (10) read e^{t+1}
          const float* et1 = a.e[t + 1];
          ts.push_back(tp(B, D, 2 * D, et1, D, 0, g.bond_edge, a.DZ12, 8 * D, 2 * D, nullptr, G + lg.an.W + D * 2 * D, 2 * D));
          ts.push_back(tp(B, D, 2 * D, et1, D, 0, g.bond_edge, a.DZ12, 8 * D, 6 * D, nullptr, G + lg.an.W + 2 * D * 2 * D,
                          2 * D));
        }
      }
      if (ang) {
        // a^T [dz_bond | dz_angle]
        ts.push_back(split_out(tp(A, D, 4 * D, a.a[t], D, 0, nullptr, a.dzae, 4 * D, 0, nullptr, G + lg.be.W + 3 * D * 2 * D, 2 * D),
                               2 * D, G + lg.an.W + 3 * D * 2 * D));
      } else {
        ts.push_back(tp(A, D, 2 * D, a.a[t], D, 0, nullptr, a.dzae, 4 * D, 0, nullptr, G + lg.be.W + 3 * D * 2 * D, 2 * D));
      }
    }
    // input gradients (they overwrite dv of the layer above, which its weight
    // gradients read; the three copies of de leave the one they read alone)
    if (wg && t + 1 < m.T) CHG_HIP(hipStreamWaitEvent(st, ss.done[t + 1], 0));
    {
      GemmProblem p = gp(N, D, a.dv[nx], D);
      seg(p, a.AT, 8 * D, 0, 2 * D, Wav, 2 * D, 1);
      seg(p, a.AT, 8 * D, 2 * D, 2 * D, Wav + D * 2 * D, 2 * D, 1);
      if (!seq) {
        seg(p, a.AT, 8 * D, 4 * D, 2 * D, Wbe, 2 * D, 1);
        if (ang) seg(p, a.AT, 8 * D, 6 * D, 2 * D, Wan, 2 * D, 1);
      }
      p.res = dvo;
      p.res_ld = D;
      ps.push_back(p);
    }
    if (!fused) {
      GemmProblem p = gp(E, D, a.de[enx], D);
      seg(p, a.dzv, 2 * D, 0, 2 * D, Wav + 2 * D * 2 * D, 2 * D, 1);
      p.res = a.de[ecur];
      p.res_ld = D;
      ps.push_back(p);
      p = gp(A, D, a.da[nx], D);
      seg(p, a.dzae, 4 * D, 0, 2 * D, Wbe + 3 * D * 2 * D, 2 * D, 1);
      if (ang) {
        seg(p, a.dzae, 4 * D, 2 * D, 2 * D, Wan + 3 * D * 2 * D, 2 * D, 1);
        p.res = a.da[cur];
        p.res_ld = D;
      }
      ps.push_back(p);
    }
    {
      // fused: the atom rows' product shares the launch of the bond rows'
      // (both direct-load, k = 8d)
      if (!fused) {
        CHG_TRY(run_gemms(ps, st, "gemm_in_bwd"));
        ps.clear();
      }
      GemmProblem p = gp(B, D, a.de[enx], D);
      p.c_rows = g.bond_edge;
      p.accumulate = 1;
      seg(p, a.DZ12, 8 * D, 0, 2 * D, Wbe + D * 2 * D, 2 * D, 1);
      seg(p, a.DZ12, 8 * D, 4 * D, 2 * D, Wbe + 2 * D * 2 * D, 2 * D, 1);
      if (ang && !seq) {
        seg(p, a.DZ12, 8 * D, 2 * D, 2 * D, Wan + D * 2 * D, 2 * D, 1);
        seg(p, a.DZ12, 8 * D, 6 * D, 2 * D, Wan + 2 * D * 2 * D, 2 * D, 1);
      }
      ps.push_back(p);
      CHG_TRY(run_gemms(ps, st, fused ? "gemm_in_bwd" : "gemm_bond_bwd"));
      ps.clear();
    }
    // the weight gradients of this layer run on the side stream, overlapping
    // the gate backward of the next layer; the buffers they read are not
    // written again before the wait on done(t) in the next layer (the
    // intermediates alternate between two copies by layer)
    if (wg) {
      CHG_TRY(side_fork(ss, st, ss.ready[t]));
      CHG_TRY(run_tns(ts, a, ss.side, "tn_in"));
      CHG_HIP(hipEventRecord(ss.done[t], ss.side));
    }
    ts.clear();
    cur = nx;
    ecur = enx;
  }

  // embeddings
  if (wg) KLAUNCH(st, "k_embed_bwd_Z", k_embed_bwd_Z<<<94, 64 * kEmbZWaves, 0, st>>>((int)N, D, bt.Z, a.dv[cur], G + Lg.W_Z));
  {
    std::vector<TnProblem> ts;
    ts.push_back(tp(E, m.R, D, a.rbf_a, m.R, 0, nullptr, a.de[ecur], D, 0, nullptr, G + Lg.W_e, 2 * D));
    ts.push_back(tp(E, m.R, D, a.rbf_a, m.R, 0, nullptr, a.dea, D, 0, nullptr, G + Lg.W_e + D, 2 * D));
    ts.push_back(tp(E, 1, D, nullptr, 0, 0, nullptr, a.de[ecur], D, 0, nullptr, G + Lg.b_e0, D));
    ts.push_back(tp(B, m.R, D, a.rbf_b, m.R, 0, nullptr, a.deb, D, 0, nullptr, G + Lg.W_eb, D));
    ts.push_back(tp(A, m.K, D, a.ft, m.K, 0, nullptr, a.da[cur], D, 0, nullptr, G + Lg.W_th, D));
    ts.push_back(tp(A, 1, D, nullptr, 0, 0, nullptr, a.da[cur], D, 0, nullptr, G + Lg.b_th, D));
    if (wg) {
      CHG_TRY(side_fork(ss, st, ss.embed));
      CHG_TRY(run_tns(ts, a, ss.side, "tn_embed"));
    }
    std::vector<GemmProblem> ps;
    GemmProblem p = gp(E, m.R, a.drbf_a, m.R);
    seg(p, a.de[ecur], D, 0, D, P + L.W_e, 2 * D, 1);
    seg(p, a.dea, D, 0, D, P + L.W_e + D, 2 * D, 1);
    ps.push_back(p);
    p = gp(B, m.R, a.drbf_b, m.R);
    seg(p, a.deb, D, 0, D, P + L.W_eb, D, 1);
    ps.push_back(p);
    if (dft_out) {
      p = gp(A, m.K, dft_out, m.K);
      seg(p, a.da[cur], D, 0, D, P + L.W_th, D, 1);
      ps.push_back(p);
    }
    CHG_TRY(run_gemms(ps, st, "gemm_embed_bwd"));
    if (!wg) return CHGNET_OK;
    float* fpart_b = a.fpart + cdiv(std::max(E, (int64_t)1), kFreqRowsPerBlock) * m.R;
    if (E > 0) {
      const int64_t nb = cdiv(E, kFreqRowsPerBlock);
      KLAUNCH(st, "k_rbf_fgrad", k_rbf_fgrad<<<(unsigned)nb, 256, 0, st>>>((int)E, nullptr, a.edge_len, P + L.f_a, m.R, c.hp->r_atom,
                                                c.hp->envelope_p, a.drbf_a, a.fpart));
      reduce_jobs.push_back(ReduceJob{a.fpart, (int)nb, m.R, m.R, G + Lg.f_a});
    }
    if (B > 0) {
      const int64_t nb = cdiv(B, kFreqRowsPerBlock);
      KLAUNCH(st, "k_rbf_fgrad", k_rbf_fgrad<<<(unsigned)nb, 256, 0, st>>>((int)B, g.bond_edge, a.edge_len, P + L.f_b, m.R, c.hp->r_bond,
                                                c.hp->envelope_p, a.drbf_b, fpart_b));
      reduce_jobs.push_back(ReduceJob{fpart_b, (int)nb, m.R, m.R, G + Lg.f_b});
    }
    // every LayerNorm and frequency gradient: ordered sums of the partials
    for (size_t i0 = 0; i0 < reduce_jobs.size(); i0 += kMaxReduceJobs) {
      ReduceJobs R{};
      for (size_t i = i0; i < reduce_jobs.size() && R.n < kMaxReduceJobs; ++i) R.j[R.n++] = reduce_jobs[i];
      CHG_TRY(reduce_rows_multi(R, a.red2, st));
    }
  }
  // join: later work on the caller's stream sees every weight gradient
  CHG_HIP(hipEventRecord(ss.fin, ss.side));
  CHG_HIP(hipStreamWaitEvent(st, ss.fin, 0));
  return CHGNET_OK;
}

#include "dual.hpp"

}  // namespace

// Conservative readout after a forward pass: the backward of E with respect
// to the inputs of the bases (no weight gradients), then dE/dr_e per edge,
// forces and stresses.
int conservative_impl(Ctx& c, float* forces, float* stress, hipStream_t st) {
  Acts& a = c.a;
  const Dims& m = c.dm;
  const ParamLayout& L = c.La;
  const float* P = a.Pal;
  const chgnet_graph& g = *c.graph;
  const chgnet_batch& bt = *c.batch;
  const int64_t N = m.N, S = m.S, E = m.E, B = m.B, A = m.A;
  CHG_TRY(fill(a.dE, S, 1.f, st));
  CHG_TRY(fill(a.dF, 3 * N, 0.f, st));
  CHG_TRY(fill(a.dS, 9 * S, 0.f, st));
  CHG_TRY(backward_impl(c, nullptr, false, a.dE, a.dF, a.dS, nullptr, nullptr, st, a.dft));
  const int p = c.hp->envelope_p;
  if (E > 0)
    KLAUNCH(st, "k_cons", k_cons_edges<<<(unsigned)cdiv(E, 256), 256, 0, st>>>((int)E, a.edge_len, a.edge_xhat, a.drbf_a,
                                                                              P + L.f_a, m.R, c.hp->r_atom, p, a.gvec));
  if (A > 0)
    KLAUNCH(st, "k_cons", k_cons_angles<<<(unsigned)cdiv(A, 256), 256, 0, st>>>((int)A, a.ang_b1, a.ang_b2, g.bond_edge,
                                                                               a.ang_ctr, g.edge_dst, g.edge_img,
                                                                               a.atom_struct, bt.pos, bt.lattice, a.dft,
                                                                               m.K, a.pang));
  if (B > 0)
    KLAUNCH(st, "k_cons", k_cons_bonds<<<(unsigned)cdiv(B, 256), 256, 0, st>>>((int)B, g.bond_edge, a.bond_src, g.bond_ptr,
                                                                              g.angle_ptr, a.edge_len, a.edge_xhat,
                                                                              a.drbf_b, P + L.f_b, m.R, c.hp->r_bond, p,
                                                                              a.pang, a.gvec));
  KLAUNCH(st, "k_cons", k_cons_forces<<<(unsigned)cdiv(N, 4), 256, 0, st>>>((int)N, g.edge_ptr, g.edge_rev, a.gvec, forces));
  KLAUNCH(st, "k_cons", k_cons_stress<<<(unsigned)S, 256, 0, st>>>((int)S, bt.atom_ptr, g.edge_ptr, a.edge_len,
                                                                      a.edge_xhat, a.gvec, bt.lattice, stress));
  return CHGNET_OK;
}

// Forward pass with the readout the hyperparameters select.
int forward_full(Ctx& c, const float* Pflat, float* energy, float* forces, float* stress, float* magmom,
                 hipStream_t st, bool pack = true) {
  if (c.hp->conservative) c.save_z = true;  // its readout runs the backward of E
  CHG_TRY(forward_impl(c, Pflat, energy, forces, stress, magmom, st, pack));
  if (c.hp->conservative) CHG_TRY(conservative_impl(c, forces, stress, st));
  return CHGNET_OK;
}

size_t acts_bytes(const chgnet_hparams& hp, int64_t N, int64_t E, int64_t B, int64_t A, int64_t S) {
  Arena ar;
  Acts a;
  Dims m{N, S, E, B, A, hp.d, hp.n_layers, hp.n_rbf, hp.n_fourier};
  carve_acts(ar, m, a, make_layout(hp, 4).total);
  if (hp.conservative) {
    // dual-number buffers of the weight gradient through the conservative readout
    DualBufs d;
    carve_dual(ar, m, make_layout(hp, 1).total, d);
  }
  return align_up(ar.used, 256);
}

int forward_entry(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph, const float* params,
                  float* energy, float* forces, float* stress, float* magmom, int save_for_backward, void* ws,
                  size_t ws_bytes, hipStream_t st) {
  Ctx c;
  CHG_TRY(make_ctx(hp, batch, graph, ws, ws_bytes, c));
  if (!params || !energy || !forces || !stress) return fail(CHGNET_EINVAL, "forward: null output or params");
  c.save_z = save_for_backward != 0;
  if (magmom && !hp->magmom) return fail(CHGNET_EINVAL, "forward: magmom output without the magnetic-moment head");
  return forward_full(c, params, energy, forces, stress, magmom, st);
}

int backward_entry(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph, const float* params,
                   const float* dE, const float* dF, const float* dS, const float* dM, float* grad, void* ws,
                   size_t ws_bytes, hipStream_t st) {
  Ctx c;
  CHG_TRY(make_ctx(hp, batch, graph, ws, ws_bytes, c));
  if (!params || !dE || !dF || !dS || !grad) return fail(CHGNET_EINVAL, "backward: null argument");
  if (dM && !hp->magmom) return fail(CHGNET_EINVAL, "backward: dM without the magnetic-moment head");
  if (hp->conservative) {
    CHG_TRY(pack_params(c.L, c.La, params, c.a.Pal, st));
    return cons_grad_impl(c, dE, dF, dS, dM, grad, st);
  }
  return backward_impl(c, params, true, dE, dF, dS, dM, grad, st);
}

int step_entry(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, float* params,
               const float* E_t, const float* F_t, const float* S_t, const float* M_t, const chgnet_loss* loss_cfg,
               float* loss, float* grad, float* adam_m, float* adam_v, const float* adam_hp, void* ws,
               size_t ws_bytes, hipStream_t st) {
  if (!params || !E_t || !F_t || !S_t || !loss_cfg || !loss || !grad) return fail(CHGNET_EINVAL, "step: null argument");
  CHG_TRY(validate_hparams(hp));
  if ((M_t != nullptr) != (hp->magmom != 0))
    return fail(CHGNET_EINVAL, "step: M_target is required with the magnetic-moment head and only with it");
  if (!std::isfinite(loss_cfg->huber_delta)) return fail(CHGNET_EINVAL, "step: huber_delta is not finite");
  if (adam_hp && (!adam_m || !adam_v || !(adam_hp[4] >= 1.0f)))
    return fail(CHGNET_EINVAL, "step: Adam needs m, v and a step number t >= 1");
  {
    // the weight copy sits at the start of the activations, at an address
    // that does not depend on the graph: pack it before the graph build so
    // the device has work while the host waits for the graph sizes
    CHG_TRY(validate_batch(batch));
    Arena ar{static_cast<char*>(ws), ws_bytes, 0};
    ar.used = graph_scratch_bytes(batch->n_atoms, batch->n_struct);
    Acts a0;
    Dims d0{batch->n_atoms, batch->n_struct, 0, 0, 0, hp->d, hp->n_layers, hp->n_rbf, hp->n_fourier};
    const ParamLayout L1 = make_layout(*hp, 1), L4 = make_layout(*hp, 4);
    carve_acts(ar, d0, a0, L4.total);
    if (!ws || !ar.ok()) return fail(CHGNET_EWORKSPACE, "workspace too small (query chgnet_workspace_size)");
    CHG_TRY(pack_params(L1, L4, params, a0.Pal, st));
  }
  CHG_TRY(build_graph(hp, batch, graph, ws, ws_bytes, st));
  Ctx c;
  CHG_TRY(make_ctx(hp, batch, graph, ws, ws_bytes, c));
  float* e_out = c.a.out_E;
  float* f_out = c.a.out_F;
  float* s_out = c.a.out_S;
  CHG_TRY(forward_impl(c, params, e_out, f_out, s_out, nullptr, st, false));
  if (hp->conservative) CHG_TRY(conservative_impl(c, f_out, s_out, st));
  const bool mag = hp->magmom != 0;
  KLAUNCH(st, "k_loss", k_loss<<<1, kLossThreads, 0, st>>>((int)c.dm.S, (int)c.dm.N, batch->atom_ptr, e_out, f_out, s_out,
                                                   mag ? c.a.oM : nullptr, E_t, F_t, S_t, M_t, *loss_cfg, loss, c.a.dE,
                                                   c.a.dF, c.a.dS, c.a.dM));
  if (hp->conservative) CHG_TRY(cons_grad_impl(c, c.a.dE, c.a.dF, c.a.dS, mag ? c.a.dM : nullptr, grad, st));
  else CHG_TRY(backward_impl(c, params, false, c.a.dE, c.a.dF, c.a.dS, mag ? c.a.dM : nullptr, grad, st));
  if (adam_hp) {
    const float lr = adam_hp[0], b1 = adam_hp[1], b2 = adam_hp[2], eps = adam_hp[3], t = adam_hp[4];
    const float c1 = 1.0f - powf(b1, t), c2 = 1.0f - powf(b2, t);
    KLAUNCH(st, "k_adam", k_adam<<<(unsigned)cdiv(c.L.total, 256), 256, 0, st>>>(c.L.total, params, grad, adam_m, adam_v, lr, b1, b2, eps, c1, c2));
  }
  return CHGNET_OK;
}

int md_build_candidates(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_md_state* s, chgnet_graph* graph,
                        void* ws, size_t ws_bytes, hipStream_t st);
int md_filter_graph(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_md_state* s,
                    chgnet_graph* graph, void* ws, size_t ws_bytes, hipStream_t st, bool* stale);

// Ends a stream capture begun by the caller and turns it into an executable
// graph (nullptr and the error of `code` if the captured work failed).
int end_capture(hipStream_t st, int code, hipGraphExec_t* exec) {
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(st, &g);
  if (code != CHGNET_OK) {
    if (g) (void)hipGraphDestroy(g);
    return code;
  }
  if (e != hipSuccess) return fail(CHGNET_EHIP, std::string("hipStreamEndCapture: ") + hipGetErrorString(e));
  const hipError_t e2 = hipGraphInstantiate(exec, g, nullptr, nullptr, 0);
  (void)hipGraphDestroy(g);
  if (e2 != hipSuccess) return fail(CHGNET_EHIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(e2));
  return CHGNET_OK;
}

int md_entry(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, const float* params,
             chgnet_md_state* s, float dt, int n_steps, int forces_valid, int* steps_done, void* ws,
             size_t ws_bytes, hipStream_t st) {
  if (steps_done) *steps_done = 0;
  CHG_TRY(validate_hparams(hp));
  if (!batch || !s || !params || !steps_done) return fail(CHGNET_EINVAL, "md: null argument");
  if (!s->pos || !s->vel || !s->inv_mass || !s->forces || s->pos != batch->pos)
    return fail(CHGNET_EINVAL, "md: state arrays missing or state->pos != batch->pos");
  if (!(dt > 0.f) || !std::isfinite(dt) || n_steps < 0) return fail(CHGNET_EINVAL, "md: need dt > 0 and n_steps >= 0");
  const bool reuse = s->skin != 0.f;
  if (reuse && (!(s->skin > 0.02f) || !(s->skin <= 2.0f) || !(hp->r_atom + s->skin <= 20.0f)))
    return fail(CHGNET_EINVAL, "md: the skin must be 0 or in (0.02, 2] A with r_atom + skin <= 20");
  if (reuse && (!s->cand_ptr || !s->ref_pos || s->cap_cand < 0 || (s->cap_cand > 0 && (!s->cand_dst || !s->cand_img))))
    return fail(CHGNET_EINVAL, "md: the candidate list needs cand_ptr, cand_dst, cand_img and ref_pos");
  s->n_builds = 0;
  // 1 eV / (A u) in A / fs^2: e / u * 1e10 m/s^2 = e / u * 1e-10 A/fs^2 (CODATA 2018 e and u)
  constexpr double kAccel = 1.602176634e-19 / 1.66053906660e-27 * 1e-10;
  const float h = (float)(0.5 * (double)dt * kAccel);
  const int n3 = 3 * batch->n_atoms;
  const unsigned nb = (unsigned)cdiv(n3, 256);
  chgnet_batch trial = *batch;
  bool packed = false, have_list = false;
  // the graph at b's positions: a full search, or the filtered candidate list
  // (rebuilt at the first step of the call and whenever an atom has moved
  // too far since its build)
  auto graph_at = [&](const chgnet_batch* b) -> int {
    if (!reuse) return build_graph(hp, b, graph, ws, ws_bytes, st);
    for (int attempt = 0; attempt < 2; ++attempt) {
      if (!have_list) {
        CHG_TRY(md_build_candidates(hp, b, s, graph, ws, ws_bytes, st));
        have_list = true;
      }
      bool stale = false;
      CHG_TRY(md_filter_graph(hp, b, s, graph, ws, ws_bytes, st, &stale));
      if (!stale) return CHGNET_OK;
      have_list = false;
    }
    return fail(CHGNET_EHIP, "md: a fresh candidate list was reported stale");
  };
  auto forward_at = [&](const chgnet_batch* b) -> int {
    Ctx c;
    CHG_TRY(make_ctx(hp, b, graph, ws, ws_bytes, c));
    c.save_z = false;  // no backward pass follows (the conservative readout keeps its own)
    CHG_TRY(forward_full(c, params, s->energy ? s->energy : c.a.out_E, s->forces, s->stress ? s->stress : c.a.out_S,
                         nullptr, st, !packed));
    packed = true;
    return CHGNET_OK;
  };
  if (!forces_valid) {
    CHG_TRY(graph_at(batch));
    CHG_TRY(forward_at(batch));
  }
  // trial positions and velocities sit in the workspace at an address that
  // does not depend on the graph sizes; a step that runs out of graph
  // capacity leaves the caller's state at the last completed step
  float *pos2, *vel2;
  {
    CHG_TRY(validate_batch(batch));
    Arena ar{static_cast<char*>(ws), ws_bytes, 0};
    ar.used = graph_scratch_bytes(batch->n_atoms, batch->n_struct);
    Acts a;
    Dims d0{batch->n_atoms, batch->n_struct, 0, 0, 0, hp->d, hp->n_layers, hp->n_rbf, hp->n_fourier};
    carve_acts(ar, d0, a, make_layout(*hp, 4).total);
    if (!ws || !ar.ok()) return fail(CHGNET_EWORKSPACE, "workspace too small (query chgnet_workspace_size)");
    pos2 = a.md_pos;
    vel2 = a.md_vel;
  }
  // The forward pass and the second half-kick of a step depend on the graph
  // only through its sizes (the arrays are read from memory, the workspace
  // layout follows the sizes), so once two consecutive steps have the same
  // sizes that part is captured into a HIP graph and replayed while they
  // stay the same. Not with the conservative readout (its backward forks a
  // second stream), a null stream or per-launch timing.
  const bool can_capture = st != nullptr && !prof_active() && !hp->conservative;
  hipGraphExec_t exec = nullptr;
  int64_t exec_sizes[3] = {-1, -1, -1}, prev[3] = {-1, -1, -1};
  auto commit = [&]() -> int {
    KLAUNCH(st, "k_md", k_md_kick_commit<<<nb, 256, 0, st>>>(n3, pos2, vel2, s->forces, s->inv_mass, h, s->pos, s->vel));
    return CHGNET_OK;
  };
  auto run_steps = [&]() -> int {
    for (int k = 0; k < n_steps; ++k) {
      KLAUNCH(st, "k_md", k_md_kick_drift<<<nb, 256, 0, st>>>(n3, s->pos, s->vel, s->forces, s->inv_mass, h, dt, pos2, vel2));
      trial.pos = pos2;
      CHG_TRY(graph_at(&trial));
      const int64_t sz[3] = {graph->n_edges, graph->n_bonds, graph->n_angles};
      const bool same_prev = sz[0] == prev[0] && sz[1] == prev[1] && sz[2] == prev[2];
      const bool same_exec = exec && sz[0] == exec_sizes[0] && sz[1] == exec_sizes[1] && sz[2] == exec_sizes[2];
      if (can_capture && packed && !same_exec && same_prev) {
        if (exec) {
          CHG_HIP(hipGraphExecDestroy(exec));
          exec = nullptr;
        }
        CHG_HIP(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
        int code = forward_at(&trial);
        if (code == CHGNET_OK) code = commit();
        CHG_TRY(end_capture(st, code, &exec));
        for (int q = 0; q < 3; ++q) exec_sizes[q] = sz[q];
        CHG_HIP(hipGraphLaunch(exec, st));
      } else if (can_capture && same_exec) {
        CHG_HIP(hipGraphLaunch(exec, st));
      } else {
        CHG_TRY(forward_at(&trial));
        CHG_TRY(commit());
      }
      for (int q = 0; q < 3; ++q) prev[q] = sz[q];
      *steps_done = k + 1;
    }
    return CHGNET_OK;
  };
  const int code = run_steps();
  if (exec) (void)hipGraphExecDestroy(exec);
  return code;
}

}  // namespace chg
