// Periodic atom graph, bond graph and angle list on gfx950 (Sec. II-B (1)).
//
// Cell-list search: each crystal's cell is cut into n_a slabs per lattice
// axis, each at least r + margin thick (so the neighbours of an atom lie in
// the slabs within K_a = floor((r + margin) n_a / h_a) + 1 of its own, with
// periodic images handled by "virtual" slab indices), atoms are binned by
// their wrapped fractional coordinates, and one block per atom tests all
// candidates with the exact fp32 inclusion expression. The accepted (j, n)
// keys of an atom are then sorted in LDS into the canonical (j, n1, n2, n3)
// order, so the output does not depend on the order in which atoms landed in
// their bins. One host wait reads the sizes E, B, A back.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>

#include "common.hpp"

namespace chg {

namespace {

constexpr double kMargin = 0.05;      // Angstrom added to the cutoff for binning
constexpr int kMaxK = 64;             // max slab reach per axis
constexpr int kMaxWrap = 200;         // max |cell index| of an input position
constexpr float kMaxCoord = 1.0e4f;   // max |Cartesian coordinate|
constexpr int kMaxEdgesPerAtom = 8192;
constexpr int kImgBias = 512;         // image components stored as n + 512 in 10 bits

enum ErrBits { ERR_Z = 1, ERR_DET = 2, ERR_THIN = 4, ERR_FAR = 8, ERR_PTR = 32 };

struct StructInfo {
  double Linv[9];
  float L[9];
  int nb[3];
  int K[3];
  int bin_base;
  int pad;
};

struct GraphInfo {
  long long n_edges, n_bonds, n_angles;
  int max_count;
  int err;
  unsigned int max_disp2;  // MD neighbour-list reuse: largest squared displacement (fp32 bits)
  int pad;
};

// ---------------------------------------------------------------------------
// The exact fp32 cutoff expression: one rounding per operation, no FMA,
// evaluated in the canonical orientation of the pair {(i, j, n), (j, i, -n)}
// (i < j, or i = j with n lexicographically positive). (r_j + s) - r_i and
// (r_i - s) - r_j round differently, so without a fixed orientation an edge
// near the cutoff could pass while its reverse fails; with it both directions
// get the same D2 and every edge has its reverse.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float pair_d2(int i, int j, const float* ri, const float* rj, int n1, int n2, int n3,
                                         const float* L) {
#pragma clang fp contract(off)
  const bool canon = i < j || (i == j && (n1 > 0 || (n1 == 0 && (n2 > 0 || (n2 == 0 && n3 > 0)))));
  const float sg = canon ? 1.0f : -1.0f;  // exact: m = sg * n
  const float f1 = sg * (float)n1, f2 = sg * (float)n2, f3 = sg * (float)n3;
  const float sx = (f1 * L[0] + f2 * L[3]) + f3 * L[6];
  const float sy = (f1 * L[1] + f2 * L[4]) + f3 * L[7];
  const float sz = (f1 * L[2] + f2 * L[5]) + f3 * L[8];
  const float px = canon ? ri[0] : rj[0], py = canon ? ri[1] : rj[1], pz = canon ? ri[2] : rj[2];
  const float qx = canon ? rj[0] : ri[0], qy = canon ? rj[1] : ri[1], qz = canon ? rj[2] : ri[2];
  const float dx = (qx + sx) - px;
  const float dy = (qy + sy) - py;
  const float dz = (qz + sz) - pz;
  return (dx * dx + dy * dy) + dz * dz;
}

__device__ __forceinline__ int floor_mod(int v, int n) {
  int r = v % n;
  return r < 0 ? r + n : r;
}

__device__ __forceinline__ int find_struct(const int* atom_ptr, int S, int i) {
  int lo = 0, hi = S - 1;  // last s with atom_ptr[s] <= i
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (atom_ptr[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Per-structure setup: inverse lattice, slab counts and reach. One block.
// Inverse lattice, slab counts and reach of structure s (flags bad input).
__device__ StructInfo struct_info(int s, const int* __restrict__ atom_ptr, const float* __restrict__ lattice, float r,
                                  GraphInfo* ginfo) {
  StructInfo si{};
  double L[9];
  for (int k = 0; k < 9; ++k) {
    si.L[k] = lattice[s * 9 + k];
    L[k] = (double)si.L[k];
  }
  // rows a0, a1, a2; cofactor rows give the reciprocal basis
  double c0[3] = {L[4] * L[8] - L[5] * L[7], L[5] * L[6] - L[3] * L[8], L[3] * L[7] - L[4] * L[6]};
  double c1[3] = {L[7] * L[2] - L[8] * L[1], L[8] * L[0] - L[6] * L[2], L[6] * L[1] - L[7] * L[0]};
  double c2[3] = {L[1] * L[5] - L[2] * L[4], L[2] * L[3] - L[0] * L[5], L[0] * L[4] - L[1] * L[3]};
  double det = L[0] * c0[0] + L[1] * c0[1] + L[2] * c0[2];
  int n_s = atom_ptr[s + 1] - atom_ptr[s];
  if (!(fabs(det) >= 1e-6) || n_s < 0) {
    atomicOr(&ginfo->err, n_s < 0 ? ERR_PTR : ERR_DET);
    for (int k = 0; k < 9; ++k) si.Linv[k] = 0.0;
    si.nb[0] = si.nb[1] = si.nb[2] = 1;
    si.K[0] = si.K[1] = si.K[2] = 0;
    return si;
  }
  // frac = cart @ Linv, Linv = L^{-1}; column a of Linv = c_a / det
  for (int row = 0; row < 3; ++row) {
    si.Linv[row * 3 + 0] = c0[row] / det;
    si.Linv[row * 3 + 1] = c1[row] / det;
    si.Linv[row * 3 + 2] = c2[row] / det;
  }
  double vol = fabs(det);
  double h[3];
  const double* cs[3] = {c0, c1, c2};
  for (int a = 0; a < 3; ++a) h[a] = vol / sqrt(cs[a][0] * cs[a][0] + cs[a][1] * cs[a][1] + cs[a][2] * cs[a][2]);
  const double rr = (double)r + kMargin;
  long long nb[3];
  for (int a = 0; a < 3; ++a) {
    double q = floor(h[a] / rr);
    nb[a] = q < 1.0 ? 1 : (q > 1024.0 ? 1024 : (long long)q);
  }
  long long cap = n_s > 1 ? n_s : 1;
  while (nb[0] * nb[1] * nb[2] > cap) {
    int a = 0;
    if (nb[1] > nb[a]) a = 1;
    if (nb[2] > nb[a]) a = 2;
    nb[a] -= 1;
  }
  bool thin = false;
  for (int a = 0; a < 3; ++a) {
    si.nb[a] = (int)nb[a];
    double kk = floor(rr * (double)nb[a] / h[a]) + 1.0;
    if (kk > kMaxK) { thin = true; kk = 0; }
    si.K[a] = (int)kk;
  }
  if (thin) atomicOr(&ginfo->err, ERR_THIN);
  si.bin_base = 0;
  return si;
}

__global__ void __launch_bounds__(1024) k_struct_setup(int S, const int* __restrict__ atom_ptr,
                                                       const float* __restrict__ lattice, float r,
                                                       StructInfo* __restrict__ info, int* __restrict__ total_bins,
                                                       GraphInfo* ginfo) {
  __shared__ int scan[1024];
  int carry = 0;  // bins of the structures of earlier rounds
  for (int s0 = 0; s0 < S; s0 += 1024) {
    const int s = s0 + (int)threadIdx.x;
    int bins = 0;
    if (s < S) {
      const StructInfo si = struct_info(s, atom_ptr, lattice, r, ginfo);
      info[s] = si;
      bins = si.nb[0] * si.nb[1] * si.nb[2];
    }
    // exclusive scan of the bin counts over the round (Hillis-Steele in LDS)
    scan[threadIdx.x] = bins;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
      const int y = threadIdx.x >= (unsigned)off ? scan[threadIdx.x - off] : 0;
      __syncthreads();
      scan[threadIdx.x] += y;
      __syncthreads();
    }
    if (s < S) info[s].bin_base = carry + scan[threadIdx.x] - bins;
    carry += scan[1023];
    __syncthreads();
  }
  if (threadIdx.x == 0) *total_bins = carry;
}

__global__ void k_atom_bin(int N, int S, const int* __restrict__ atom_ptr, const float* __restrict__ pos,
                           const int* __restrict__ Z, const StructInfo* __restrict__ info, int* __restrict__ atom_struct,
                           int* __restrict__ atom_bin, int* __restrict__ atom_cell, int* __restrict__ atom_wrap,
                           int* __restrict__ bin_count, GraphInfo* ginfo) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  int s = find_struct(atom_ptr, S, i);
  atom_struct[i] = s;
  int z = Z[i];
  if (z < 1 || z > 94) atomicOr(&ginfo->err, ERR_Z);
  const StructInfo& si = info[s];
  float p[3] = {pos[i * 3 + 0], pos[i * 3 + 1], pos[i * 3 + 2]};
  int err = 0;
  int c[3], w[3];
  for (int a = 0; a < 3; ++a) {
    if (!(fabsf(p[a]) <= kMaxCoord)) err |= ERR_FAR;
    double f = (double)p[0] * si.Linv[0 * 3 + a] + (double)p[1] * si.Linv[1 * 3 + a] + (double)p[2] * si.Linv[2 * 3 + a];
    double fl = floor(f);
    if (!(fabs(fl) <= kMaxWrap)) { err |= ERR_FAR; fl = 0.0; }
    double fr = f - fl;
    int ca = (int)floor(fr * si.nb[a]);
    ca = ca < 0 ? 0 : (ca >= si.nb[a] ? si.nb[a] - 1 : ca);
    c[a] = ca;
    w[a] = (int)fl;
  }
  if (err) atomicOr(&ginfo->err, err);
  int bin = si.bin_base + (c[0] * si.nb[1] + c[1]) * si.nb[2] + c[2];
  atom_bin[i] = bin;
  for (int a = 0; a < 3; ++a) {
    atom_cell[i * 3 + a] = c[a];
    atom_wrap[i * 3 + a] = w[a];
  }
  atomicAdd(&bin_count[bin], 1);
}

// Scans in a fixed order: a wavefront's inclusive scan by lane shuffles,
// and a block's exclusive scan from its wavefronts' totals (sh: 17 slots of
// shared memory; every thread of the block takes part).
template <class T>
__device__ __forceinline__ T wave_incl_scan(T v, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const T t = __shfl_up(v, d, 64);
    if (lane >= d) v += t;
  }
  return v;
}
template <class T>
__device__ __forceinline__ T block_excl_scan(T v, T* sh, T& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = (int)(blockDim.x + 63) >> 6;
  const T inc = wave_incl_scan(v, lane);
  if (lane == 63) sh[w] = inc;
  __syncthreads();
  if (w == 0) {
    const T t = lane < nw ? sh[lane] : T(0);
    const T ti = wave_incl_scan(t, lane);
    if (lane < nw) sh[lane] = ti - t;
    if (lane == nw - 1) sh[16] = ti;
  }
  __syncthreads();
  const T r = sh[w] + inc - v;
  total = sh[16];
  __syncthreads();
  return r;
}

// Exclusive scan of n ints with one 1024-thread block (any n), 8 consecutive
// values a thread per pass. out[n] = total.
constexpr int kScanPer = 8;
__global__ void __launch_bounds__(1024) k_scan_single(int n, const int* __restrict__ in, int* __restrict__ out) {
  __shared__ int sh[17];
  int carry = 0;
  for (int base = 0; base < n; base += (int)blockDim.x * kScanPer) {
    const int i0 = base + (int)threadIdx.x * kScanPer;
    int v[kScanPer], sum = 0;
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      v[q] = i0 + q < n ? in[i0 + q] : 0;
      sum += v[q];
    }
    int total;
    int run = carry + block_excl_scan(sum, sh, total);
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      if (i0 + q < n) out[i0 + q] = run;
      run += v[q];
    }
    carry += total;
  }
  if (threadIdx.x == 0) out[n] = carry;
}

__global__ void k_bin_fill(int N, const int* __restrict__ atom_bin, const int* __restrict__ bin_start,
                           int* __restrict__ bin_cursor, int* __restrict__ bin_atoms) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  int b = atom_bin[i];
  int slot = atomicAdd(&bin_cursor[b], 1);
  bin_atoms[bin_start[b] + slot] = i;
}

struct SearchArgs {
  int N;
  float rc2_atom, rc2_bond;
  const float* pos;
  const StructInfo* info;
  const int* atom_struct;
  const int* atom_cell;
  const int* atom_wrap;
  const int* bin_start;
  const int* bin_atoms;
};

// One 256-thread block per atom. The candidates of atom i are the atoms of
// its (2K+1)^3 virtual slabs; the block takes the virtual slabs 256 at a
// time, scans their atom counts, and then spreads the flattened candidate
// list over all threads (a thread finds its slab by binary search over the
// scanned counts), so small slabs do not leave lanes idle.
constexpr int kSearchThreads = 256;
struct SearchShared {
  int pre[kSearchThreads];  // exclusive prefix of the slabs' atom counts
  int lo[kSearchThreads];   // first bin_atoms slot of each slab
  int m[kSearchThreads][3];  // lattice translation of each virtual slab
  int wsum[kSearchThreads / 64];
};

// Calls f(j, n1, n2, n3, d2) on the thread that holds candidate (j, n) of
// atom i, for every candidate that passes the atom cutoff.
template <class F>
__device__ __forceinline__ void block_search(const SearchArgs& A, int i, SearchShared& sh, F&& f) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int s = A.atom_struct[i];
  const StructInfo& si = A.info[s];
  float L[9];
  for (int k = 0; k < 9; ++k) L[k] = si.L[k];
  const float ri[3] = {A.pos[i * 3 + 0], A.pos[i * 3 + 1], A.pos[i * 3 + 2]};
  const int ci[3] = {A.atom_cell[i * 3 + 0], A.atom_cell[i * 3 + 1], A.atom_cell[i * 3 + 2]};
  const int wi[3] = {A.atom_wrap[i * 3 + 0], A.atom_wrap[i * 3 + 1], A.atom_wrap[i * 3 + 2]};
  const int w0 = 2 * si.K[0] + 1, w1 = 2 * si.K[1] + 1, w2 = 2 * si.K[2] + 1;
  const int nv = w0 * w1 * w2;
  for (int v0 = 0; v0 < nv; v0 += kSearchThreads) {
    const int v = v0 + t;
    int cnt = 0;
    if (v < nv) {
      const int d2 = v % w2 - si.K[2], d1 = (v / w2) % w1 - si.K[1], d0 = v / (w2 * w1) - si.K[0];
      const int x0 = ci[0] + d0, b0 = floor_mod(x0, si.nb[0]);
      const int x1 = ci[1] + d1, b1 = floor_mod(x1, si.nb[1]);
      const int x2 = ci[2] + d2, b2 = floor_mod(x2, si.nb[2]);
      const int bin = si.bin_base + (b0 * si.nb[1] + b1) * si.nb[2] + b2;
      const int lo = A.bin_start[bin];
      cnt = A.bin_start[bin + 1] - lo;
      sh.lo[t] = lo;
      sh.m[t][0] = (x0 - b0) / si.nb[0];
      sh.m[t][1] = (x1 - b1) / si.nb[1];
      sh.m[t][2] = (x2 - b2) / si.nb[2];
    }
    // block exclusive scan of the counts
    int incl = cnt;
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(incl, off, 64);
      if (lane >= off) incl += y;
    }
    if (lane == 63) sh.wsum[w] = incl;
    __syncthreads();
    int base = 0, total = 0;
    for (int k = 0; k < kSearchThreads / 64; ++k) {
      base += k < w ? sh.wsum[k] : 0;
      total += sh.wsum[k];
    }
    sh.pre[t] = base + incl - cnt;
    __syncthreads();
    for (int c = t; c < total; c += kSearchThreads) {
      int lo = 0, hi = kSearchThreads - 1;  // last slab u with pre[u] <= c
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (sh.pre[mid] <= c) lo = mid;
        else hi = mid - 1;
      }
      const int j = A.bin_atoms[sh.lo[lo] + (c - sh.pre[lo])];
      const int n1 = sh.m[lo][0] - A.atom_wrap[j * 3 + 0] + wi[0];
      const int n2 = sh.m[lo][1] - A.atom_wrap[j * 3 + 1] + wi[1];
      const int n3 = sh.m[lo][2] - A.atom_wrap[j * 3 + 2] + wi[2];
      const float rj[3] = {A.pos[j * 3 + 0], A.pos[j * 3 + 1], A.pos[j * 3 + 2]};
      const float dd = pair_d2(i, j, ri, rj, n1, n2, n3, L);
      if (dd < A.rc2_atom && !(j == i && n1 == 0 && n2 == 0 && n3 == 0)) f(j, n1, n2, n3, dd);
    }
    __syncthreads();
  }
}

// Block-wide sum of one int per thread (256 threads); every thread gets it.
__device__ __forceinline__ int block_sum(int v, int* wsum) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = v;
  __syncthreads();
  int t = 0;
  for (int k = 0; k < kSearchThreads / 64; ++k) t += wsum[k];
  return t;
}

// Count edges and bonds of atom blockIdx.x.
__global__ void __launch_bounds__(kSearchThreads) k_count(SearchArgs A, int* __restrict__ edge_count,
                                                          int* __restrict__ bond_count) {
  __shared__ SearchShared sh;
  const int i = blockIdx.x;
  int ne = 0, nb = 0;
  block_search(A, i, sh, [&](int, int, int, int, float dd) {
    ++ne;
    nb += dd < A.rc2_bond ? 1 : 0;
  });
  ne = block_sum(ne, sh.wsum);
  nb = block_sum(nb, sh.wsum);
  if (threadIdx.x == 0) {
    edge_count[i] = ne;
    bond_count[i] = nb;
  }
}

// Exclusive scans of edge counts, bond counts and k(k-1); totals into ginfo.
__global__ void __launch_bounds__(1024) k_scan_counts(int N, const int* __restrict__ edge_count,
                                                     const int* __restrict__ bond_count, int* __restrict__ edge_ptr,
                                                     int* __restrict__ bond_ptr, long long* __restrict__ angle_base,
                                                     GraphInfo* ginfo) {
  __shared__ long long sh[17];
  __shared__ int mx[1024];
  long long ce = 0, cb = 0, ca = 0;
  int my_max = 0;
  for (int base = 0; base < N; base += (int)blockDim.x * kScanPer) {
    const int i0 = base + (int)threadIdx.x * kScanPer;
    int ve[kScanPer], vb[kScanPer];
    long long se = 0, sb = 0, sa = 0;
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      const bool in = i0 + q < N;
      ve[q] = in ? edge_count[i0 + q] : 0;
      vb[q] = in ? bond_count[i0 + q] : 0;
      se += ve[q];
      sb += vb[q];
      sa += (long long)vb[q] * (vb[q] - 1);
      my_max = max(my_max, ve[q]);
    }
    long long te, tb, ta;
    long long e0 = ce + block_excl_scan(se, sh, te);
    long long b0 = cb + block_excl_scan(sb, sh, tb);
    long long a0 = ca + block_excl_scan(sa, sh, ta);
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      if (i0 + q < N) {
        edge_ptr[i0 + q] = (int)(e0 < INT_MAX ? e0 : INT_MAX);
        bond_ptr[i0 + q] = (int)(b0 < INT_MAX ? b0 : INT_MAX);
        angle_base[i0 + q] = a0;
      }
      e0 += ve[q];
      b0 += vb[q];
      a0 += (long long)vb[q] * (vb[q] - 1);
    }
    ce += te;
    cb += tb;
    ca += ta;
  }
  mx[threadIdx.x] = my_max;
  __syncthreads();
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) mx[threadIdx.x] = max(mx[threadIdx.x], mx[threadIdx.x + off]);
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    edge_ptr[N] = (int)(ce < INT_MAX ? ce : INT_MAX);
    bond_ptr[N] = (int)(cb < INT_MAX ? cb : INT_MAX);
    angle_base[N] = ca;
    ginfo->n_edges = ce;
    ginfo->n_bonds = cb;
    ginfo->n_angles = ca;
    ginfo->max_count = mx[0];
  }
}

__device__ __forceinline__ unsigned long long make_key(int j, int n1, int n2, int n3, bool bond) {
  return ((unsigned long long)(unsigned)j << 31) | ((unsigned long long)(n1 + kImgBias) << 21) |
         ((unsigned long long)(n2 + kImgBias) << 11) | ((unsigned long long)(n3 + kImgBias) << 1) |
         (bond ? 1ull : 0ull);
}

// One block per atom: gather the accepted keys into LDS (slots taken with an
// LDS counter; the order is fixed by the sort that follows), bitonic sort,
// write the edges in canonical order and the atom's bond list.
__global__ void __launch_bounds__(kSearchThreads) k_fill(SearchArgs A, int sort_size, const int* __restrict__ edge_ptr,
                                                         const int* __restrict__ bond_ptr, int* __restrict__ edge_dst,
                                                         int* __restrict__ edge_img, int* __restrict__ bond_edge) {
  extern __shared__ unsigned long long keys[];
  __shared__ SearchShared sh;
  __shared__ int nkeys;
  const int i = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  if (t == 0) nkeys = 0;
  __syncthreads();
  block_search(A, i, sh, [&](int j, int n1, int n2, int n3, float dd) {
    const int slot = atomicAdd(&nkeys, 1);
    if (slot < sort_size) keys[slot] = make_key(j, n1, n2, n3, dd < A.rc2_bond);
  });
  const int count = min(nkeys, sort_size);
  for (int k = count + t; k < sort_size; k += kSearchThreads) keys[k] = ~0ull;
  __syncthreads();
  // bitonic sort of sort_size (power of two) keys
  for (int size = 2; size <= sort_size; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int u = t; u < sort_size / 2; u += kSearchThreads) {
        const int lo = 2 * u - (u & (stride - 1));
        const int hi = lo + stride;
        const bool up = (lo & size) == 0;
        const unsigned long long a = keys[lo], b = keys[hi];
        if ((a > b) == up) { keys[lo] = b; keys[hi] = a; }
      }
      __syncthreads();
    }
  }
  const int e0 = edge_ptr[i];
  const int b0 = bond_ptr[i];
  int nb = 0;  // bonds written before this round of kSearchThreads keys
  for (int base = 0; base < count; base += kSearchThreads) {
    const int k = base + t;
    bool bond = false;
    if (k < count) {
      const unsigned long long key = keys[k];
      edge_dst[e0 + k] = (int)(key >> 31);
      edge_img[(e0 + k) * 3 + 0] = (int)((key >> 21) & 1023) - kImgBias;
      edge_img[(e0 + k) * 3 + 1] = (int)((key >> 11) & 1023) - kImgBias;
      edge_img[(e0 + k) * 3 + 2] = (int)((key >> 1) & 1023) - kImgBias;
      bond = (key & 1ull) != 0;
    }
    const unsigned long long m = __ballot(bond);
    if (lane == 0) sh.wsum[w] = __popcll(m);
    __syncthreads();
    int before = nb;
    for (int q = 0; q < w; ++q) before += sh.wsum[q];
    if (bond) bond_edge[b0 + before + __popcll(m & ((1ull << lane) - 1ull))] = e0 + k;
    for (int q = 0; q < kSearchThreads / 64; ++q) nb += sh.wsum[q];
    __syncthreads();
  }
}

// Reverse map: binary search of (i, -n) in the sorted edge list of j. The
// search always succeeds: D2 is the same number in both directions (see
// pair_d2), and the cell list of j holds i at -n whenever that of i holds j
// at n (both cover every pair closer than r + kMargin, while D2 < r^2 implies
// a separation within fp32 rounding of r). The fallback value is never used.
__device__ __forceinline__ void rev_atoms(int blk, int N, const int* __restrict__ edge_ptr, const int* __restrict__ edge_dst,
                                          const int* __restrict__ edge_img, int* __restrict__ edge_rev) {
  const int i = blk * 4 + (threadIdx.x >> 6);
  if (i >= N) return;
  const int lane = threadIdx.x & 63;
  for (int e = edge_ptr[i] + lane; e < edge_ptr[i + 1]; e += 64) {
    const int j = edge_dst[e];
    const int t0 = -edge_img[e * 3 + 0], t1 = -edge_img[e * 3 + 1], t2 = -edge_img[e * 3 + 2];
    int lo = edge_ptr[j], hi = edge_ptr[j + 1] - 1, found = -1;
    while (lo <= hi) {
      const int mid = (lo + hi) >> 1;
      const int k0 = edge_dst[mid], k1 = edge_img[mid * 3 + 0], k2 = edge_img[mid * 3 + 1], k3 = edge_img[mid * 3 + 2];
      int cmp = k0 != i ? (k0 < i ? -1 : 1)
                        : (k1 != t0 ? (k1 < t0 ? -1 : 1) : (k2 != t1 ? (k2 < t1 ? -1 : 1) : (k3 != t2 ? (k3 < t2 ? -1 : 1) : 0)));
      if (cmp == 0) { found = mid; break; }
      if (cmp < 0) lo = mid + 1; else hi = mid - 1;
    }
    edge_rev[e] = found < 0 ? e : found;
  }
}

// Angle list of atom i (one wavefront per atom): angle_ptr of its bonds and,
// if requested, the second bond of each of its k(k-1) angles.
__device__ __forceinline__ void angle_atoms(int blk, int N, const int* __restrict__ bond_ptr,
                                            const long long* __restrict__ angle_base, int* __restrict__ angle_ptr,
                                            int* __restrict__ angle_b2) {
  const int i = blk * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= N) return;
  const int b0 = bond_ptr[i], k = bond_ptr[i + 1] - b0;
  const long long a0 = angle_base[i];
  for (int p = lane; p < k; p += 64) angle_ptr[b0 + p] = (int)(a0 + (long long)p * (k - 1));
  if (i == N - 1 && lane == 0) angle_ptr[bond_ptr[N]] = (int)angle_base[N];
  if (angle_b2 && k > 1) {
    const int na = k * (k - 1);
    for (int x = lane; x < na; x += 64) {
      const int p = x / (k - 1), qq = x - p * (k - 1);
      angle_b2[a0 + x] = b0 + (qq < p ? qq : qq + 1);
    }
  }
}

// Reverse-edge map and angle lists in one launch: blocks [0, nb) take the
// reverse edges of atoms 4 b .. 4 b + 3, blocks [nb, 2 nb) their angle lists.
__global__ void __launch_bounds__(256) k_rev_angles(int N, const int* __restrict__ edge_ptr,
                                                    const int* __restrict__ edge_dst, const int* __restrict__ edge_img,
                                                    int* __restrict__ edge_rev, const int* __restrict__ bond_ptr,
                                                    const long long* __restrict__ angle_base, int* __restrict__ angle_ptr,
                                                    int* __restrict__ angle_b2) {
  const int nb = (N + 3) / 4;
  if ((int)blockIdx.x < nb) rev_atoms(blockIdx.x, N, edge_ptr, edge_dst, edge_img, edge_rev);
  else angle_atoms(blockIdx.x - nb, N, bond_ptr, angle_base, angle_ptr, angle_b2);
}

// Clears the graph info record and the bin counters (n each).
__global__ void k_zero_scratch(GraphInfo* __restrict__ ginfo, int* __restrict__ bin_count, int* __restrict__ bin_cursor,
                               int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) *ginfo = GraphInfo{};
  if (i < n) {
    bin_count[i] = 0;
    bin_cursor[i] = 0;
  }
}

struct GraphScratch {
  StructInfo* info;
  GraphInfo* ginfo;
  int* total_bins;
  int *atom_struct, *atom_bin, *atom_cell, *atom_wrap;
  int *bin_count, *bin_start, *bin_cursor, *bin_atoms;
  int *edge_count, *bond_count;
  long long* angle_base;
};

void carve(Arena& ar, int64_t N, int64_t S, GraphScratch& g) {
  const int64_t nbins = N + S + 1;
  g.info = ar.take<StructInfo>(S);
  g.ginfo = ar.take<GraphInfo>(1);
  g.total_bins = ar.take<int>(1);
  g.atom_struct = ar.take<int>(N);
  g.atom_bin = ar.take<int>(N);
  g.atom_cell = ar.take<int>(3 * N);
  g.atom_wrap = ar.take<int>(3 * N);
  g.bin_count = ar.take<int>(nbins + 1);
  g.bin_start = ar.take<int>(nbins + 1);
  g.bin_cursor = ar.take<int>(nbins + 1);
  g.bin_atoms = ar.take<int>(N);
  g.edge_count = ar.take<int>(N);
  g.bond_count = ar.take<int>(N);
  g.angle_base = ar.take<long long>(N + 1);
}

}  // namespace

size_t graph_scratch_bytes(int64_t N, int64_t S) {
  Arena ar;
  GraphScratch g;
  carve(ar, N, S, g);
  return align_up(ar.used, 256);
}

int validate_batch(const chgnet_batch* b) {
  if (!b || b->n_struct < 1 || b->n_atoms < 1 || !b->atom_ptr || !b->pos || !b->lattice || !b->Z)
    return fail(CHGNET_EINVAL, "batch: need n_struct >= 1, n_atoms >= 1 and non-null arrays");
  return CHGNET_OK;
}

namespace {

// Graph build on a scratch region of ws_bytes at ws. With pinned_readback the
// sizes come back through a small pinned host buffer of the calling thread
// (allocated on its first use); otherwise through a pageable host variable.
int build_graph_impl(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, void* ws,
                     size_t ws_bytes, hipStream_t st, bool pinned_readback, bool candidates = false) {
  CHG_TRY(validate_hparams(hp));
  CHG_TRY(validate_batch(batch));
  if (!graph || !graph->edge_ptr || !graph->bond_ptr) return fail(CHGNET_EINVAL, "graph: edge_ptr and bond_ptr are required");
  const int N = batch->n_atoms, S = batch->n_struct;
  Arena ar{static_cast<char*>(ws), ws_bytes, 0};
  GraphScratch g;
  carve(ar, N, S, g);
  if (!ws || !ar.ok()) return fail(CHGNET_EWORKSPACE, "workspace too small for the graph build");
  const int64_t nbins_cap = (int64_t)N + S + 1;

  {
    const int n = (int)(nbins_cap + 1);
    KLAUNCH(st, "k_zero_scratch", k_zero_scratch<<<(unsigned)cdiv(n, 256), 256, 0, st>>>(g.ginfo, g.bin_count, g.bin_cursor, n));
  }
  KLAUNCH(st, "k_struct_setup", k_struct_setup<<<1, 1024, 0, st>>>(S, batch->atom_ptr, batch->lattice, hp->r_atom, g.info, g.total_bins, g.ginfo));
  KLAUNCH(st, "k_atom_bin", k_atom_bin<<<cdiv(N, 256), 256, 0, st>>>(N, S, batch->atom_ptr, batch->pos, batch->Z, g.info, g.atom_struct, g.atom_bin,
                                           g.atom_cell, g.atom_wrap, g.bin_count, g.ginfo));
  // total bins <= N + S (each crystal has at most max(1, n_s) bins)
  KLAUNCH(st, "k_scan_single", k_scan_single<<<1, 1024, 0, st>>>((int)nbins_cap, g.bin_count, g.bin_start));
  KLAUNCH(st, "k_bin_fill", k_bin_fill<<<cdiv(N, 256), 256, 0, st>>>(N, g.atom_bin, g.bin_start, g.bin_cursor, g.bin_atoms));

  SearchArgs A;
  A.N = N;
  A.rc2_atom = hp->r_atom * hp->r_atom;
  A.rc2_bond = candidates ? -1.0f : hp->r_bond * hp->r_bond;  // a candidate list has no bonds
  A.pos = batch->pos;
  A.info = g.info;
  A.atom_struct = g.atom_struct;
  A.atom_cell = g.atom_cell;
  A.atom_wrap = g.atom_wrap;
  A.bin_start = g.bin_start;
  A.bin_atoms = g.bin_atoms;
  KLAUNCH(st, "k_count", k_count<<<N, kSearchThreads, 0, st>>>(A, g.edge_count, g.bond_count));
  KLAUNCH(st, "k_scan_counts", k_scan_counts<<<1, 1024, 0, st>>>(N, g.edge_count, g.bond_count, graph->edge_ptr, graph->bond_ptr, g.angle_base,
                                    g.ginfo));

  // the sizes come back through a small pinned buffer (one per host thread,
  // allocated on first use): a direct DMA instead of a staged pageable copy
  GraphInfo hinfo;
  if (pinned_readback) {
    thread_local GraphInfo* pinned = nullptr;
    if (!pinned) CHG_HIP(hipHostMalloc(reinterpret_cast<void**>(&pinned), sizeof(GraphInfo), hipHostMallocDefault));
    CHG_HIP(hipMemcpyAsync(pinned, g.ginfo, sizeof(GraphInfo), hipMemcpyDeviceToHost, st));
    CHG_HIP(hipStreamSynchronize(st));
    hinfo = *pinned;
  } else {
    CHG_HIP(hipMemcpyAsync(&hinfo, g.ginfo, sizeof(GraphInfo), hipMemcpyDeviceToHost, st));
    CHG_HIP(hipStreamSynchronize(st));
  }
  if (hinfo.err) {
    std::string m = "build_graph: invalid input:";
    if (hinfo.err & ERR_Z) m += " Z outside 1..94;";
    if (hinfo.err & ERR_DET) m += " |det L| < 1e-6;";
    if (hinfo.err & ERR_THIN) m += " lattice too thin for the cutoff;";
    if (hinfo.err & ERR_FAR) m += " position too far from the origin cell;";
    if (hinfo.err & ERR_PTR) m += " atom_ptr decreasing;";
    return fail(CHGNET_EINVAL, m);
  }
  graph->n_edges = hinfo.n_edges;
  graph->n_bonds = hinfo.n_bonds;
  graph->n_angles = hinfo.n_angles;
  if (hinfo.max_count > kMaxEdgesPerAtom)
    return fail(CHGNET_EINVAL, "build_graph: more than 8192 edges on one atom");
  if (hinfo.n_edges >= INT_MAX || hinfo.n_angles >= INT_MAX)
    return fail(CHGNET_EINVAL, "build_graph: graph larger than 2^31 entries");
  if (hinfo.n_edges > graph->cap_edges || hinfo.n_bonds > graph->cap_bonds || hinfo.n_angles > graph->cap_angles)
    return fail(CHGNET_ECAPACITY, "build_graph: capacity too small (required sizes written to the graph)");
  if (candidates) {
    if (hinfo.n_edges > 0 && (!graph->edge_dst || !graph->edge_img))
      return fail(CHGNET_EINVAL, "md: candidate arrays are required");
    int sort_size = 64;
    while (sort_size < hinfo.max_count) sort_size <<= 1;
    KLAUNCH(st, "k_fill", k_fill<<<N, kSearchThreads, sizeof(unsigned long long) * sort_size, st>>>(
                              A, sort_size, graph->edge_ptr, graph->bond_ptr, graph->edge_dst, graph->edge_img, nullptr));
    return CHGNET_OK;
  }
  if (hinfo.n_edges > 0 && (!graph->edge_dst || !graph->edge_img || !graph->edge_rev))
    return fail(CHGNET_EINVAL, "graph: edge arrays are required");
  if (!graph->angle_ptr || (hinfo.n_bonds > 0 && !graph->bond_edge))
    return fail(CHGNET_EINVAL, "graph: bond_edge and angle_ptr are required");

  int sort_size = 64;
  while (sort_size < hinfo.max_count) sort_size <<= 1;
  KLAUNCH(st, "k_fill", k_fill<<<N, kSearchThreads, sizeof(unsigned long long) * sort_size, st>>>(A, sort_size, graph->edge_ptr, graph->bond_ptr,
                                                                graph->edge_dst, graph->edge_img, graph->bond_edge));
  KLAUNCH(st, "k_rev_angles", k_rev_angles<<<2 * cdiv(N, 4), 256, 0, st>>>(N, graph->edge_ptr, graph->edge_dst, graph->edge_img,
                                                                       graph->edge_rev, graph->bond_ptr, g.angle_base,
                                                                       graph->angle_ptr, graph->angle_b2));
  return CHGNET_OK;
}

// ---------------------------------------------------------------------------
// Molecular dynamics: reuse of a candidate list (Verlet skin). The list holds
// every pair within r + skin of the positions at its build, in the canonical
// (j, n) order of each source atom. While no atom has moved more than
// (skin - 0.01 A) / 2 since then, every pair now within r is on the list, and
// filtering it with the exact cutoff test at the current positions gives the
// same graph, in the same order, as a full search.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_md_disp(int n, const float* __restrict__ pos, const float* __restrict__ ref,
                                                 GraphInfo* ginfo) {
  __shared__ float red[4];
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  float d2 = 0.f;
  if (i < n) {
    const float dx = pos[3 * i] - ref[3 * i], dy = pos[3 * i + 1] - ref[3 * i + 1], dz = pos[3 * i + 2] - ref[3 * i + 2];
    d2 = dx * dx + dy * dy + dz * dz;
  }
  for (int off = 32; off > 0; off >>= 1) d2 = fmaxf(d2, __shfl_xor(d2, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = d2;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    atomicMax(&ginfo->max_disp2, __float_as_uint(m));  // non-negative floats order as their bits
  }
}

struct CandArgs {
  int N, S;
  float rc2_atom, rc2_bond;
  const int* atom_ptr;
  const float* pos;
  const float* lattice;
  const int* cand_ptr;
  const int* cand_dst;
  const int* cand_img;
};

// Cutoff test of candidate c of atom i at the current positions.
__device__ __forceinline__ float cand_d2(const CandArgs& A, int i, const float* L, const float (&ri)[3], int c,
                                         int& j) {
  j = A.cand_dst[c];
  const float rj[3] = {A.pos[3 * j], A.pos[3 * j + 1], A.pos[3 * j + 2]};
  return pair_d2(i, j, ri, rj, A.cand_img[3 * c], A.cand_img[3 * c + 1], A.cand_img[3 * c + 2], L);
}

// Edges and bonds of each atom among its candidates; one wavefront per atom.
__global__ void __launch_bounds__(256) k_cand_count(CandArgs A, int* __restrict__ edge_count, int* __restrict__ bond_count) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= A.N) return;
  const int s = find_struct(A.atom_ptr, A.S, i);
  float L[9];
  for (int k = 0; k < 9; ++k) L[k] = A.lattice[9 * s + k];
  const float ri[3] = {A.pos[3 * i], A.pos[3 * i + 1], A.pos[3 * i + 2]};
  int ne = 0, nb = 0;
  for (int c = A.cand_ptr[i] + lane; c < A.cand_ptr[i + 1]; c += 64) {
    int j;
    const float dd = cand_d2(A, i, L, ri, c, j);
    ne += dd < A.rc2_atom ? 1 : 0;
    nb += dd < A.rc2_bond ? 1 : 0;
  }
  for (int off = 32; off > 0; off >>= 1) {
    ne += __shfl_xor(ne, off, 64);
    nb += __shfl_xor(nb, off, 64);
  }
  if (lane == 0) {
    edge_count[i] = ne;
    bond_count[i] = nb;
  }
}

// The kept candidates of each atom in list order (one wavefront per atom,
// 64 candidates per round, compacted by ballot): edge arrays and bond list.
__global__ void __launch_bounds__(256) k_cand_fill(CandArgs A, const int* __restrict__ edge_ptr,
                                                   const int* __restrict__ bond_ptr, int* __restrict__ edge_dst,
                                                   int* __restrict__ edge_img, int* __restrict__ bond_edge) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= A.N) return;
  const int s = find_struct(A.atom_ptr, A.S, i);
  float L[9];
  for (int k = 0; k < 9; ++k) L[k] = A.lattice[9 * s + k];
  const float ri[3] = {A.pos[3 * i], A.pos[3 * i + 1], A.pos[3 * i + 2]};
  int e = edge_ptr[i], b = bond_ptr[i];
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int c0 = A.cand_ptr[i]; c0 < A.cand_ptr[i + 1]; c0 += 64) {
    const int c = c0 + lane;
    bool keep = false, bond = false;
    int j = 0;
    if (c < A.cand_ptr[i + 1]) {
      const float dd = cand_d2(A, i, L, ri, c, j);
      keep = dd < A.rc2_atom;
      bond = dd < A.rc2_bond;
    }
    const unsigned long long mk = __ballot(keep), mb = __ballot(bond);
    if (keep) {
      const int k = e + __popcll(mk & below);
      edge_dst[k] = j;
      edge_img[3 * k] = A.cand_img[3 * c];
      edge_img[3 * k + 1] = A.cand_img[3 * c + 1];
      edge_img[3 * k + 2] = A.cand_img[3 * c + 2];
      if (bond) bond_edge[b + __popcll(mb & below)] = k;
    }
    e += __popcll(mk);
    b += __popcll(mb);
  }
}

// Scratch of the allocation-free graph build: one array per GPU, held until
// the process ends. Host code never passes `scratch` itself to a kernel (in
// host code the name is a stand-in, not a device address); it uses the
// address hipGetSymbolAddress returns on each device.
constexpr size_t kNoAllocScratchBytes = size_t(8) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per device.
int scratch_address(void** out) {
  int dev = -1;
  CHG_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(CHGNET_EINVAL, "build_graph_noalloc: device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    CHG_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(CHGNET_EHIP, "build_graph_noalloc: no device address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return CHGNET_OK;
}

}  // namespace

int build_graph(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, void* ws, size_t ws_bytes,
                hipStream_t st) {
  return build_graph_impl(hp, batch, graph, ws, ws_bytes, st, true);
}

int build_graph_noalloc(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, hipStream_t st) {
  CHG_TRY(validate_hparams(hp));
  CHG_TRY(validate_batch(batch));
  const size_t need = graph_scratch_bytes(batch->n_atoms, batch->n_struct);
  if (need > kNoAllocScratchBytes)
    return fail(CHGNET_EINVAL, "build_graph_noalloc: the batch needs " + std::to_string(need) +
                                   " bytes of graph scratch, more than the static " +
                                   std::to_string(kNoAllocScratchBytes) + " (use chgnet_build_graph with a workspace)");
  void* p = nullptr;
  CHG_TRY(scratch_address(&p));
  return build_graph_impl(hp, batch, graph, p, kNoAllocScratchBytes, st, false);
}

// Candidate list of every pair within r_atom + skin of the batch's current
// positions into s->cand_* (bonds are not kept), and those positions into
// s->ref_pos. graph->bond_ptr serves as scratch.
int md_build_candidates(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_md_state* s, chgnet_graph* graph,
                        void* ws, size_t ws_bytes, hipStream_t st) {
  chgnet_hparams hc = *hp;
  hc.r_atom = hp->r_atom + s->skin;
  hc.r_bond = hc.r_atom;
  chgnet_graph cg{};
  cg.cap_edges = s->cap_cand;
  cg.edge_ptr = s->cand_ptr;
  cg.edge_dst = s->cand_dst;
  cg.edge_img = s->cand_img;
  cg.bond_ptr = graph->bond_ptr;
  const int code = build_graph_impl(&hc, batch, &cg, ws, ws_bytes, st, true, true);
  s->n_cand = cg.n_edges;
  if (code != CHGNET_OK) return code;
  CHG_HIP(hipMemcpyAsync(s->ref_pos, batch->pos, sizeof(float) * 3 * batch->n_atoms, hipMemcpyDeviceToDevice, st));
  s->n_builds += 1;
  return CHGNET_OK;
}

// The graph of the batch's current positions from the candidate list. Sets
// *stale (and builds nothing) when some atom has moved too far since the
// list was built; otherwise as chgnet_build_graph (one wait for the sizes).
int md_filter_graph(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_md_state* s,
                    chgnet_graph* graph, void* ws, size_t ws_bytes, hipStream_t st, bool* stale) {
  *stale = false;
  const int N = batch->n_atoms, S = batch->n_struct;
  Arena ar{static_cast<char*>(ws), ws_bytes, 0};
  GraphScratch g;
  carve(ar, N, S, g);
  if (!ws || !ar.ok()) return fail(CHGNET_EWORKSPACE, "workspace too small for the graph build");
  KLAUNCH(st, "k_zero_scratch", k_zero_scratch<<<1, 256, 0, st>>>(g.ginfo, g.bin_count, g.bin_cursor, 1));
  KLAUNCH(st, "k_md_disp", k_md_disp<<<(unsigned)cdiv(N, 256), 256, 0, st>>>(N, batch->pos, s->ref_pos, g.ginfo));
  CandArgs A{N, S, hp->r_atom * hp->r_atom, hp->r_bond * hp->r_bond, batch->atom_ptr, batch->pos, batch->lattice,
             s->cand_ptr, s->cand_dst, s->cand_img};
  KLAUNCH(st, "k_cand_count", k_cand_count<<<(unsigned)cdiv(N, 4), 256, 0, st>>>(A, g.edge_count, g.bond_count));
  KLAUNCH(st, "k_scan_counts", k_scan_counts<<<1, 1024, 0, st>>>(N, g.edge_count, g.bond_count, graph->edge_ptr,
                                                                   graph->bond_ptr, g.angle_base, g.ginfo));
  thread_local GraphInfo* pinned = nullptr;
  if (!pinned) CHG_HIP(hipHostMalloc(reinterpret_cast<void**>(&pinned), sizeof(GraphInfo), hipHostMallocDefault));
  CHG_HIP(hipMemcpyAsync(pinned, g.ginfo, sizeof(GraphInfo), hipMemcpyDeviceToHost, st));
  CHG_HIP(hipStreamSynchronize(st));
  const GraphInfo hinfo = *pinned;
  // the list covers every pair within r of the current positions while twice
  // the largest displacement stays below the skin (0.01 A spares fp32
  // rounding of coordinates up to 10^4 A)
  const float half = 0.5f * (s->skin - 0.01f);
  float md2;
  std::memcpy(&md2, &hinfo.max_disp2, sizeof(float));
  if (!(md2 < half * half)) {
    *stale = true;
    return CHGNET_OK;
  }
  graph->n_edges = hinfo.n_edges;
  graph->n_bonds = hinfo.n_bonds;
  graph->n_angles = hinfo.n_angles;
  if (hinfo.max_count > kMaxEdgesPerAtom) return fail(CHGNET_EINVAL, "build_graph: more than 8192 edges on one atom");
  if (hinfo.n_edges >= INT_MAX || hinfo.n_angles >= INT_MAX)
    return fail(CHGNET_EINVAL, "build_graph: graph larger than 2^31 entries");
  if (hinfo.n_edges > graph->cap_edges || hinfo.n_bonds > graph->cap_bonds || hinfo.n_angles > graph->cap_angles)
    return fail(CHGNET_ECAPACITY, "build_graph: capacity too small (required sizes written to the graph)");
  KLAUNCH(st, "k_cand_fill", k_cand_fill<<<(unsigned)cdiv(N, 4), 256, 0, st>>>(A, graph->edge_ptr, graph->bond_ptr,
                                                                              graph->edge_dst, graph->edge_img,
                                                                              graph->bond_edge));
  KLAUNCH(st, "k_rev_angles", k_rev_angles<<<2 * cdiv(N, 4), 256, 0, st>>>(N, graph->edge_ptr, graph->edge_dst,
                                                                            graph->edge_img, graph->edge_rev,
                                                                            graph->bond_ptr, g.angle_base,
                                                                            graph->angle_ptr, graph->angle_b2));
  return CHGNET_OK;
}

}  // namespace chg
