// Weight gradient of a loss on the conservative readout (Sec. II-B (4): F =
// -dE/dr, sigma = (1/V) dE/d eps). Such a loss depends on first derivatives
// of E, so its gradient needs second derivatives. With the loss gradients
// l_E, l_F, l_sigma of the outputs, the displacement u_i = -l_F,i of every
// atom and the strain rate U_s = l_sigma,s / V_s of every crystal,
//
//   dL/dtheta = sum_s l_E,s dE_s/dtheta + d/dtheta D_(u,U) E_tot,
//
// where D_(u,U) E_tot is the derivative of the total energy along r -> r +
// h u, eps -> h U. Both terms are the derivative at h = 0 of
//
//   sum_s (1 + h l_E,s) dE_s/dtheta (theta; r + h u, eps = h U),
//
// so the forward pass and the weight backward run here in dual numbers
// (value, tangent), seeded with the edge-vector tangent u_j - u_i + U_s r_ij
// and the energy seeds (1, l_E,s); the gradient is the tangent part of the
// weight gradient. Values of the forward activations are the forward pass's
// own; tangents, and both parts of every backward quantity, are kept in
// separate arrays of the same shape (value array, tangent array). The linear
// maps (embedding, gated-MLP inputs, output linears, heads) run on the GEMM
// and weight-gradient kernels, once per part; the gates, the messages and
// the per-atom and per-bond sums of the pre-activation gradients have their
// own kernels here. Eq. (11) blocks
// (sequential = 0). The magnetic-moment loss term is first order: its output
// takes the seed (0, l_M,i), which adds its ordinary backward to the tangent
// part.

struct Dn {
  float v, t;
};
__device__ __forceinline__ Dn operator+(Dn a, Dn b) { return {a.v + b.v, a.t + b.t}; }
__device__ __forceinline__ Dn operator-(Dn a, Dn b) { return {a.v - b.v, a.t - b.t}; }
__device__ __forceinline__ Dn operator*(Dn a, Dn b) { return {a.v * b.v, a.v * b.t + a.t * b.v}; }
__device__ __forceinline__ Dn operator*(float s, Dn a) { return {s * a.v, s * a.t}; }
__device__ __forceinline__ Dn operator+(Dn a, float s) { return {a.v + s, a.t}; }
__device__ __forceinline__ Dn operator+(float s, Dn a) { return {s + a.v, a.t}; }
__device__ __forceinline__ Dn operator-(float s, Dn a) { return {s - a.v, -a.t}; }
__device__ __forceinline__ Dn dn_recip(Dn a) {
  const float r = 1.0f / a.v;
  return {r, -a.t * r * r};
}
__device__ __forceinline__ Dn dn_sqrt(Dn a) {
  const float r = sqrtf(a.v);
  return {r, 0.5f * a.t / r};
}
__device__ __forceinline__ Dn dn_sin(Dn a) { return {sinf(a.v), cosf(a.v) * a.t}; }
__device__ __forceinline__ Dn dn_cos(Dn a) { return {cosf(a.v), -sinf(a.v) * a.t}; }
__device__ __forceinline__ Dn dn_sigm(Dn a) {
  const float s = 1.0f / (1.0f + expf(-a.v));
  return {s, s * (1.0f - s) * a.t};
}
// silu'(x) = s (1 + x (1 - s)), s = sigmoid(x)
__device__ __forceinline__ Dn dn_dsilu(Dn a) {
  const Dn s = dn_sigm(a);
  return s * (1.0f + a * (1.0f - s));
}
__device__ __forceinline__ Dn dn_atan2(Dn y, Dn x) {
  const float q = x.v * x.v + y.v * y.v;
  return {atan2f(y.v, x.v), (x.v * y.t - y.v * x.t) / q};
}
// polynomial envelope u(x) = 1 - (p+1)(p+2)/2 x^p + p(p+2) x^(p+1) - p(p+1)/2 x^(p+2)
__device__ __forceinline__ Dn dn_envelope(Dn x, int p) {
  Dn xp = x;
  for (int k = 1; k < p; ++k) xp = xp * x;
  const Dn xp1 = xp * x, xp2 = xp1 * x;
  return 1.0f - ((0.5f * (p + 1) * (p + 2)) * xp - (float)(p * (p + 2)) * xp1 + (0.5f * p * (p + 1)) * xp2);
}
// sRBF_n(d) = sqrt(2/c) sin(f_n d / c) / d * u(d / c), and its derivative in f_n
__device__ __forceinline__ Dn dn_srbf(Dn d, float f, float inv_c, int p) {
  const Dn x = inv_c * d;
  return sqrtf(2.0f * inv_c) * (dn_sin(f * x) * dn_recip(d) * dn_envelope(x, p));
}
__device__ __forceinline__ Dn dn_srbf_df(Dn d, float f, float inv_c, int p) {
  const Dn x = inv_c * d;
  return (sqrtf(2.0f * inv_c) * inv_c) * (dn_cos(f * x) * dn_envelope(x, p));
}
__device__ __forceinline__ float dn_wsum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ Dn dn_wsum(Dn x) { return {dn_wsum(x.v), dn_wsum(x.t)}; }

// ---------------------------------------------------------------------------
// Tangents of the geometry and the bases.
// ---------------------------------------------------------------------------
// Per edge: r_ij = |r| xhat, its tangent u_j - u_i + U_s r_ij (u = -l_F, U =
// l_sigma / V), the length tangent and the sRBF row tangent at the atom cutoff.
__global__ void __launch_bounds__(256) kd_edges(int E, int R, int p, float inv_c, const int* __restrict__ src,
                                                const int* __restrict__ dst, const int* __restrict__ astruct,
                                                const float* __restrict__ len, const float* __restrict__ xhat,
                                                const float* __restrict__ lattice, const float* __restrict__ dF,
                                                const float* __restrict__ dS, const float* __restrict__ f,
                                                float* __restrict__ rdot, float* __restrict__ ddot,
                                                float* __restrict__ rbf_t) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= E) return;
  const int i = src[e], j = dst[e], s = astruct[i];
  const float l = len[e];
  const float* L = lattice + 9 * (int64_t)s;
  const float vol = fabsf(L[0] * (L[4] * L[8] - L[5] * L[7]) - L[1] * (L[3] * L[8] - L[5] * L[6]) +
                          L[2] * (L[3] * L[7] - L[4] * L[6]));
  const float* U = dS + 9 * (int64_t)s;
  float r[3], dd = 0.f;
  for (int c = 0; c < 3; ++c) r[c] = l * xhat[3 * (int64_t)e + c];
  for (int a = 0; a < 3; ++a) {
    const float rd = -(dF[3 * (int64_t)j + a] - dF[3 * (int64_t)i + a]) + (U[3 * a] * r[0] + U[3 * a + 1] * r[1] + U[3 * a + 2] * r[2]) / vol;
    rdot[3 * (int64_t)e + a] = rd;
    dd += xhat[3 * (int64_t)e + a] * rd;
  }
  ddot[e] = dd;
  for (int n = 0; n < R; ++n) rbf_t[(int64_t)e * R + n] = dn_srbf(Dn{l, dd}, f[n], inv_c, p).t;
}

// Per bond: sRBF row tangent at the bond cutoff (the bond's edge length).
__global__ void __launch_bounds__(256) kd_bonds(int B, int R, int p, float inv_c, const int* __restrict__ bond_edge,
                                                const float* __restrict__ len, const float* __restrict__ ddot,
                                                const float* __restrict__ f, float* __restrict__ rbf_t) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  const int e = bond_edge[b];
  for (int n = 0; n < R; ++n) rbf_t[(int64_t)b * R + n] = dn_srbf(Dn{len[e], ddot[e]}, f[n], inv_c, p).t;
}

// Per angle: theta = atan2(|r1 x r2|, r1 . r2) and the Fourier row tangent
// (columns: constant, cos m theta, sin m theta); d theta = 0 where the two
// bonds are collinear.
__global__ void __launch_bounds__(256) kd_angles(int A, int K, const int* __restrict__ b1, const int* __restrict__ b2,
                                                 const int* __restrict__ bond_edge, const float* __restrict__ len,
                                                 const float* __restrict__ xhat, const float* __restrict__ rdot,
                                                 float* __restrict__ ft_t) {
  const int al = blockIdx.x * 256 + threadIdx.x;
  if (al >= A) return;
  const int64_t e1 = bond_edge[b1[al]], e2 = bond_edge[b2[al]];
  Dn r1[3], r2[3];
  for (int c = 0; c < 3; ++c) {
    r1[c] = Dn{len[e1] * xhat[3 * e1 + c], rdot[3 * e1 + c]};
    r2[c] = Dn{len[e2] * xhat[3 * e2 + c], rdot[3 * e2 + c]};
  }
  const Dn cx = r1[1] * r2[2] - r1[2] * r2[1];
  const Dn cy = r1[2] * r2[0] - r1[0] * r2[2];
  const Dn cz = r1[0] * r2[1] - r1[1] * r2[0];
  const Dn c2 = cx * cx + cy * cy + cz * cz;
  const Dn sn = c2.v > 0.f ? dn_sqrt(c2) : Dn{0.f, 0.f};
  const Dn th = dn_atan2(sn, r1[0] * r2[0] + r1[1] * r2[1] + r1[2] * r2[2]);
  const int M = (K - 1) / 2;
  const float inv_sqrt_pi = 0.56418958354775628695f;
  float* o = ft_t + (int64_t)al * K;
  o[0] = 0.f;
  for (int m = 1; m <= M; ++m) {
    o[m] = -m * sinf(m * th.v) * th.t * inv_sqrt_pi;
    o[M + m] = m * cosf(m * th.v) * th.t * inv_sqrt_pi;
  }
}

// ---------------------------------------------------------------------------
// Gathered blocks of the gated-MLP inputs [v_i | v_j | e_ij] and [v_i | e_ij |
// e_ik | a_ijk]. The first linear layer of a gate is split by input block:
// atom and bond blocks are multiplied once per atom or bond (projections,
// rows of 8d: four blocks of 2d) and their rows are gathered into the
// pre-activation by the gate kernel; in the backward pass the
// pre-activation gradients are first summed per atom (S) and per bond (T),
// in the graph's CSR orders (no atomics), and multiplied there.
// ---------------------------------------------------------------------------
// A block per atom i and block q of S (both parts): S[i] = [sum over the
// out-edges e of dz_av[e] | of dz_av[rev e] (the edges that end at i) | sum
// over the angles centred on i of dz_be | of dz_an]; the four wavefronts
// take every fourth row and their sums are added in a fixed order.
constexpr int kDzMaxCols = 4;  // 2d / 64 columns a lane
__global__ void __launch_bounds__(256) kd_dz_atoms(int N, int D, int q0, int nblk, const int* __restrict__ ep,
                                                   const int* __restrict__ rev, const int* __restrict__ bp,
                                                   const int* __restrict__ ap, const float* __restrict__ zav,
                                                   const float* __restrict__ zat, const float* __restrict__ zbv,
                                                   const float* __restrict__ zbt, const float* __restrict__ znv,
                                                   const float* __restrict__ znt, float* __restrict__ sv,
                                                   float* __restrict__ st) {
  __shared__ float red[4][2][kDzMaxCols * 64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t i = blockIdx.x / nblk;
  if (i >= N) return;  // uniform over the block
  const int q = q0 + (int)(blockIdx.x % nblk);
  const int W2 = 2 * D, nc = W2 / 64;
  int64_t r0, r1;
  const float *xv, *xt;
  if (q < 2) {
    r0 = ep[i];
    r1 = ep[i + 1];
    xv = zav;
    xt = zat;
  } else {
    r0 = ap[bp[i]];
    r1 = ap[bp[i + 1]];
    xv = q == 2 ? zbv : znv;
    xt = q == 2 ? zbt : znt;
  }
  float av[kDzMaxCols] = {}, at[kDzMaxCols] = {};
  for (int64_t r = r0 + wv; r < r1; r += 4) {
    const int64_t o = (q == 1 ? (int64_t)rev[r] : r) * W2 + lane;
#pragma unroll
    for (int k = 0; k < kDzMaxCols; ++k)
      if (k < nc) {
        av[k] += xv[o + 64 * k];
        at[k] += xt[o + 64 * k];
      }
  }
#pragma unroll
  for (int k = 0; k < kDzMaxCols; ++k)
    if (k < nc) {
      red[wv][0][lane + 64 * k] = av[k];
      red[wv][1][lane + 64 * k] = at[k];
    }
  __syncthreads();
  for (int c = threadIdx.x; c < 2 * W2; c += 256) {
    const int pl = c / W2, cc = c % W2;
    const float v = ((red[0][pl][cc] + red[1][pl][cc]) + red[2][pl][cc]) + red[3][pl][cc];
    (pl ? st : sv)[i * 4 * W2 + q * W2 + cc] = v;
  }
}

// a wavefront per bond b (both parts): T[b] = [sum over the angles whose
// first bond is b of dz_be | over the angles whose second bond is b | the
// same two of dz_an]. At a centre atom with bonds b0 .. b0 + k - 1 the block
// of bond p lists the other k - 1 bonds in increasing order, so the angle
// (p, q) is the reverse of (q, p) and sits at position q - b0 (minus one if q
// > p) of p's block: the second-bond sums read the reverses of b's own angles.
__global__ void __launch_bounds__(256) kd_dz_bonds(int B, int D, int which, const int* __restrict__ ap,
                                                   const int* __restrict__ bsrc, const int* __restrict__ bp,
                                                   const int* __restrict__ b2, const float* __restrict__ zbv,
                                                   const float* __restrict__ zbt, const float* __restrict__ znv,
                                                   const float* __restrict__ znt, float* __restrict__ tv,
                                                   float* __restrict__ tt) {
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= B) return;
  const int W2 = 2 * D;
  const int64_t b0 = bp[bsrc[w]], qq = w - b0;
  for (int c = lane; c < W2; c += 64) {
    float s[8] = {};
    for (int64_t a = ap[w]; a < ap[w + 1]; ++a) {
      const int64_t p = b2[a], pp = p - b0;
      const int64_t o = a * W2 + c, o2 = (ap[p] + (qq < pp ? qq : qq - 1)) * W2 + c;
      if (which & 1) {
        s[0] += zbv[o];
        s[1] += zbt[o];
        s[2] += zbv[o2];
        s[3] += zbt[o2];
      }
      if (which & 2) {
        s[4] += znv[o];
        s[5] += znt[o];
        s[6] += znv[o2];
        s[7] += znt[o2];
      }
    }
    const int64_t o = w * 4 * W2 + c;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (!(which & (k < 2 ? 1 : 2))) continue;
      tv[o + k * W2] = s[2 * k];
      tt[o + k * W2] = s[2 * k + 1];
    }
  }
}

// ---------------------------------------------------------------------------
// Gated MLP (Sec. II-B (3)): phi = SiLU(LN_c(z_c)) * sigmoid(LN_g(z_g)), one
// wavefront a row, d / 64 columns a lane.
// ---------------------------------------------------------------------------
constexpr int kDnMaxV = 2;  // d <= 128
constexpr int kDnGateWaves = 4096;  // wavefronts of the gate kernels: one resident round, 4 a SIMD

struct DnGate {
  int64_t rows;
  // [rows, 2d] pre-activations; the forward adds the rows idx[k][r] of the
  // projections add[k] (rows of 8d) to the edge or angle block's product and
  // stores the sum
  float *zv, *zt;
  int nadd;
  const float *addv[3], *addt[3];
  const int* idx[3];
  const float *gc, *bc, *gg, *bg;
  // forward: phi -> (pv, pt), or with res_t: pt = res_t + phi tangent (a + phi)
  float *pv, *pt;
  const float* res_t;
  // backward: d phi in (dpv, dpt) -> dz (dzv, dzt) and the tangents of the
  // LayerNorm parameter terms summed per wavefront, lnp [waves, 4d]
  const float *dpv, *dpt;
  float *dzv, *dzt, *lnp;
};
struct DnGates {
  int n;
  int64_t start[4];  // prefix sums of the jobs' rows; start[n] = total
  DnGate j[3];
};

template <int MV>
__device__ __forceinline__ void dn_ln(const Dn (&z)[MV], int V, int D, Dn (&xh)[MV], Dn& rstd) {
  Dn s{0.f, 0.f};
#pragma unroll
  for (int i = 0; i < MV; ++i)
    if (i < V) s = s + z[i];
  const Dn mu = (1.0f / D) * dn_wsum(s);
  Dn q{0.f, 0.f};
#pragma unroll
  for (int i = 0; i < MV; ++i)
    if (i < V) q = q + (z[i] - mu) * (z[i] - mu);
  rstd = dn_recip(dn_sqrt((1.0f / D) * dn_wsum(q) + kLnEps));
#pragma unroll
  for (int i = 0; i < MV; ++i) xh[i] = (z[i] - mu) * rstd;
}

// Raw inputs of one forward row (lane's columns): z core/gate value and
// tangent, and the gathered projection rows, summed only when the row is
// computed, so that the loads of the next row are in flight meanwhile.
template <int V>
struct DnFwdRaw {
  float z[4][V];
  float a[3][4][V];
};
template <int V>
__device__ __forceinline__ void dn_fwd_load(const DnGate& q, int64_t r, const int64_t (&ro)[3], int D, int lane,
                                            DnFwdRaw<V>& x) {
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const int64_t o = r * 2 * D + lane + 64 * i;
    x.z[0][i] = q.zv[o];
    x.z[1][i] = q.zt[o];
    x.z[2][i] = q.zv[o + D];
    x.z[3][i] = q.zt[o + D];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      if (k >= q.nadd) break;
      const int64_t c = ro[k] + lane + 64 * i;
      x.a[k][0][i] = q.addv[k][c];
      x.a[k][1][i] = q.addt[k][c];
      x.a[k][2][i] = q.addv[k][c + D];
      x.a[k][3][i] = q.addt[k][c + D];
    }
  }
}
__device__ __forceinline__ void dn_fwd_index(const DnGate& q, int64_t r, int D, int64_t (&ro)[3]) {
#pragma unroll
  for (int k = 0; k < 3; ++k) ro[k] = k < q.nadd ? (int64_t)q.idx[k][r] * 8 * D : 0;
}

// Forward of the gates: every wavefront walks the rows w, w + W, ... of each
// job, loading row r + W (and the gather indices of r + 2W) before it
// computes row r.
template <int V>
__global__ void __launch_bounds__(256) kd_gate_fwd(DnGates J) {
  constexpr int D = 64 * V;
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6), W = (int64_t)gridDim.x * 4;
  for (int job = 0; job < J.n; ++job) {
    const DnGate& q = J.j[job];
    if (w >= q.rows) continue;
    int64_t ro[3], ron[3];
    DnFwdRaw<V> cur, nxt;
    dn_fwd_index(q, w, D, ro);
    if (w + W < q.rows) dn_fwd_index(q, w + W, D, ron);
    dn_fwd_load(q, w, ro, D, lane, cur);
    for (int64_t r = w; r < q.rows; r += W) {
      if (r + W < q.rows) {
        dn_fwd_load(q, r + W, ron, D, lane, nxt);
        if (r + 2 * W < q.rows) dn_fwd_index(q, r + 2 * W, D, ron);
      }
      Dn zc[V], zg[V], xc[V], xg[V], rc, rg;
#pragma unroll
      for (int i = 0; i < V; ++i) {
        zc[i] = Dn{cur.z[0][i], cur.z[1][i]};
        zg[i] = Dn{cur.z[2][i], cur.z[3][i]};
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          if (k >= q.nadd) break;
          zc[i] = zc[i] + Dn{cur.a[k][0][i], cur.a[k][1][i]};
          zg[i] = zg[i] + Dn{cur.a[k][2][i], cur.a[k][3][i]};
        }
      }
      if (q.nadd > 0) {
#pragma unroll
        for (int i = 0; i < V; ++i) {
          const int64_t o = r * 2 * D + lane + 64 * i;
          q.zv[o] = zc[i].v;
          q.zt[o] = zc[i].t;
          q.zv[o + D] = zg[i].v;
          q.zt[o + D] = zg[i].t;
        }
      }
      dn_ln(zc, V, D, xc, rc);
      dn_ln(zg, V, D, xg, rg);
#pragma unroll
      for (int i = 0; i < V; ++i) {
        const int c = lane + 64 * i;
        const Dn yc = q.gc[c] * xc[i] + q.bc[c];
        const Dn yg = q.gg[c] * xg[i] + q.bg[c];
        const Dn ph = yc * dn_sigm(yc) * dn_sigm(yg);
        const int64_t o = r * D + c;
        if (q.res_t) {
          q.pt[o] = q.res_t[o] + ph.t;
        } else {
          q.pv[o] = ph.v;
          q.pt[o] = ph.t;
        }
      }
      cur = nxt;
    }
  }
}

// Backward of the gates: every wavefront walks the rows w, w + W, ... of each
// job (W wavefronts in the grid), loading row r + W before it computes row
// r, and keeps the tangents of its rows' LayerNorm parameter terms in
// registers; it writes them once per job, as row w of lnp [W, 4d]:
// dy_c xhat_c | dy_c | dy_g xhat_g | dy_g.
template <int V>
struct DnBwdRaw {
  float z[4][V];
  float dp[2][V];
};
template <int V>
__device__ __forceinline__ void dn_bwd_load(const DnGate& q, int64_t r, int lane, DnBwdRaw<V>& x) {
  constexpr int D = 64 * V;
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const int64_t o = r * 2 * D + lane + 64 * i, op = r * D + lane + 64 * i;
    x.z[0][i] = q.zv[o];
    x.z[1][i] = q.zt[o];
    x.z[2][i] = q.zv[o + D];
    x.z[3][i] = q.zt[o + D];
    x.dp[0][i] = q.dpv[op];
    x.dp[1][i] = q.dpt[op];
  }
}

template <int V>
__device__ __forceinline__ void dn_gate_bwd_row(const DnGate& q, int64_t r, int lane, const DnBwdRaw<V>& x,
                                                float (&acc)[4][V]) {
  constexpr int D = 64 * V;
  Dn zc[V], zg[V], xc[V], xg[V], rc, rg;
#pragma unroll
  for (int i = 0; i < V; ++i) {
    zc[i] = Dn{x.z[0][i], x.z[1][i]};
    zg[i] = Dn{x.z[2][i], x.z[3][i]};
  }
  dn_ln(zc, V, D, xc, rc);
  dn_ln(zg, V, D, xg, rg);
  Dn gc[V], gg[V];
  Dn s1c{0.f, 0.f}, s2c{0.f, 0.f}, s1g{0.f, 0.f}, s2g{0.f, 0.f};
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const int c = lane + 64 * i;
    const Dn dp{x.dp[0][i], x.dp[1][i]};
    const Dn yc = q.gc[c] * xc[i] + q.bc[c];
    const Dn yg = q.gg[c] * xg[i] + q.bg[c];
    const Dn sc = dn_sigm(yc), sg = dn_sigm(yg);
    const Dn dyc = dp * sg * (sc * (1.0f + yc * (1.0f - sc)));
    const Dn dyg = dp * (yc * sc) * sg * (1.0f - sg);
    acc[0][i] += (dyc * xc[i]).t;
    acc[1][i] += dyc.t;
    acc[2][i] += (dyg * xg[i]).t;
    acc[3][i] += dyg.t;
    gc[i] = q.gc[c] * dyc;
    gg[i] = q.gg[c] * dyg;
    s1c = s1c + gc[i];
    s2c = s2c + gc[i] * xc[i];
    s1g = s1g + gg[i];
    s2g = s2g + gg[i] * xg[i];
  }
  const float inv = 1.0f / D;
  s1c = inv * dn_wsum(s1c);
  s2c = inv * dn_wsum(s2c);
  s1g = inv * dn_wsum(s1g);
  s2g = inv * dn_wsum(s2g);
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const int64_t o = r * 2 * D + lane + 64 * i;
    const Dn dc = rc * (gc[i] - s1c - xc[i] * s2c);
    const Dn dg = rg * (gg[i] - s1g - xg[i] * s2g);
    q.dzv[o] = dc.v;
    q.dzt[o] = dc.t;
    q.dzv[o + D] = dg.v;
    q.dzt[o + D] = dg.t;
  }
}

template <int V>
__global__ void __launch_bounds__(256) kd_gate_bwd(DnGates J) {
  constexpr int D = 64 * V;
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6), W = (int64_t)gridDim.x * 4;
  for (int k = 0; k < J.n; ++k) {
    const DnGate& q = J.j[k];
    float acc[4][V] = {};
    DnBwdRaw<V> cur, nxt;
    if (w < q.rows) dn_bwd_load(q, w, lane, cur);
    for (int64_t r = w; r < q.rows; r += W) {
      if (r + W < q.rows) dn_bwd_load(q, r + W, lane, nxt);
      dn_gate_bwd_row(q, r, lane, cur, acc);
      cur = nxt;
    }
#pragma unroll
    for (int i = 0; i < V; ++i)
#pragma unroll
      for (int u = 0; u < 4; ++u) q.lnp[w * 4 * D + u * D + lane + 64 * i] = acc[u][i];
  }
}

// ---------------------------------------------------------------------------
// Messages (Eq. 4, 5) and their backward.
// ---------------------------------------------------------------------------
// m_i = sum over the edges e of atom i (CSR by source) of e^a_e * phi_e: a
// block per atom, its four wavefronts take every fourth edge and their sums
// are added in a fixed order
__global__ void __launch_bounds__(256) kd_msg_atoms(int N, int D, const int* __restrict__ ep,
                                                    const float* __restrict__ eav, const float* __restrict__ eat,
                                                    const float* __restrict__ pv, const float* __restrict__ pt,
                                                    float* __restrict__ mv, float* __restrict__ mt) {
  __shared__ float red[4][2][kDnMaxV * 64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t i = blockIdx.x;
  if (i >= N) return;  // uniform over the block
  float sv[kDnMaxV] = {}, st[kDnMaxV] = {};
  for (int64_t e = ep[i] + wv; e < ep[i + 1]; e += 4) {
#pragma unroll
    for (int k = 0; k < kDnMaxV; ++k) {
      if (k >= D / 64) break;
      const int64_t o = e * D + lane + 64 * k;
      const Dn x = Dn{eav[o], eat[o]} * Dn{pv[o], pt[o]};
      sv[k] += x.v;
      st[k] += x.t;
    }
  }
#pragma unroll
  for (int k = 0; k < kDnMaxV; ++k) {
    red[wv][0][lane + 64 * k] = sv[k];
    red[wv][1][lane + 64 * k] = st[k];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < 2 * D; c += 256) {
    const int pl = c / D, cc = c % D;
    const float v = ((red[0][pl][cc] + red[1][pl][cc]) + red[2][pl][cc]) + red[3][pl][cc];
    (pl ? mt : mv)[i * D + cc] = v;
  }
}

// s_b = sum over the angles (b, b2) of e^b_b2 * phi; mu_b = e^b_b * s_b
__global__ void __launch_bounds__(256) kd_msg_bonds(int B, int D, const int* __restrict__ ap, const int* __restrict__ b2,
                                                    const float* __restrict__ ebv, const float* __restrict__ ebt,
                                                    const float* __restrict__ pv, const float* __restrict__ pt,
                                                    float* __restrict__ sv, float* __restrict__ st,
                                                    float* __restrict__ uv, float* __restrict__ ut) {
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= B) return;
  for (int c = lane; c < D; c += 64) {
    Dn s{0.f, 0.f};
    for (int64_t a = ap[w]; a < ap[w + 1]; ++a) {
      const int64_t o2 = (int64_t)b2[a] * D + c, o = a * D + c;
      s = s + Dn{ebv[o2], ebt[o2]} * Dn{pv[o], pt[o]};
    }
    const Dn u = Dn{ebv[w * D + c], ebt[w * D + c]} * s;
    sv[w * D + c] = s.v;
    st[w * D + c] = s.t;
    uv[w * D + c] = u.v;
    ut[w * D + c] = u.t;
  }
}

// per edge: d phi = dm_src * e^a; d e^a += dm_src * phi
__global__ void __launch_bounds__(256) kd_bwd_atoms(int64_t n, int D, const int* __restrict__ src,
                                                    const float* __restrict__ dmv, const float* __restrict__ dmt,
                                                    const float* __restrict__ eav, const float* __restrict__ eat,
                                                    const float* __restrict__ pv, const float* __restrict__ pt,
                                                    float* __restrict__ dpv, float* __restrict__ dpt,
                                                    float* __restrict__ deav, float* __restrict__ deat) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t so = (int64_t)src[i / D] * D + i % D;
  const Dn dm{dmv[so], dmt[so]};
  const Dn dp = dm * Dn{eav[i], eat[i]};
  const Dn g = dm * Dn{pv[i], pt[i]};
  dpv[i] = dp.v;
  dpt[i] = dp.t;
  deav[i] += g.v;
  deat[i] += g.t;
}

// per bond: d e^b += d mu * s; d s = d mu * e^b
__global__ void __launch_bounds__(256) kd_bwd_bonds(int64_t n, const float* __restrict__ dmuv,
                                                    const float* __restrict__ dmut, const float* __restrict__ sv,
                                                    const float* __restrict__ st, const float* __restrict__ ebv,
                                                    const float* __restrict__ ebt, float* __restrict__ debv,
                                                    float* __restrict__ debt, float* __restrict__ dsv,
                                                    float* __restrict__ dst) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const Dn du{dmuv[i], dmut[i]};
  const Dn g = du * Dn{sv[i], st[i]};
  const Dn ds = du * Dn{ebv[i], ebt[i]};
  debv[i] += g.v;
  debt[i] += g.t;
  dsv[i] = ds.v;
  dst[i] = ds.t;
}

// per angle (b1, b2): d phi = d s_b1 * e^b_b2
__global__ void __launch_bounds__(256) kd_bwd_angles(int64_t n, int D, const int* __restrict__ b1,
                                                     const int* __restrict__ b2, const float* __restrict__ dsv,
                                                     const float* __restrict__ dst, const float* __restrict__ ebv,
                                                     const float* __restrict__ ebt, float* __restrict__ dpv,
                                                     float* __restrict__ dpt) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t a = i / D, c = i % D;
  const int64_t o1 = (int64_t)b1[a] * D + c, o2 = (int64_t)b2[a] * D + c;
  const Dn dp = Dn{dsv[o1], dst[o1]} * Dn{ebv[o2], ebt[o2]};
  dpv[i] = dp.v;
  dpt[i] = dp.t;
}

// per bond q: d e^b_q += sum over the angles (p, q) whose second bond is q of
// d s_p * phi_(p,q). The angles of a centre atom with bonds b0 .. b0 + k - 1
// form one block, bond p's row listing the other bonds in order, so (p, q)
// sits at angle_ptr[p] + (q - b0) - (q > p); the sum runs over p in order
// (no atomics, the same result every run).
__global__ void __launch_bounds__(256) kd_bwd_b2(int64_t n, int D, const int* __restrict__ bond_src,
                                                 const int* __restrict__ bond_ptr, const int* __restrict__ angle_ptr,
                                                 const float* __restrict__ dsv, const float* __restrict__ dst,
                                                 const float* __restrict__ pv, const float* __restrict__ pt,
                                                 float* __restrict__ debv, float* __restrict__ debt) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int q = (int)(i / D), c = (int)(i % D);
  const int ctr = bond_src[q], b0 = bond_ptr[ctr], b1 = bond_ptr[ctr + 1];
  Dn acc{0.f, 0.f};
  for (int p = b0; p < b1; ++p) {
    if (p == q) continue;
    const int64_t a = (int64_t)angle_ptr[p] + (q - b0) - (q > p ? 1 : 0);
    acc = acc + Dn{dsv[(int64_t)p * D + c], dst[(int64_t)p * D + c]} * Dn{pv[a * D + c], pt[a * D + c]};
  }
  debv[i] += acc.v;
  debt[i] += acc.t;
}

// ---------------------------------------------------------------------------
// Energy head (Eq. 7-9 readout MLP) and the remaining weight terms.
// ---------------------------------------------------------------------------
// tangent of a = SiLU(h): silu'(h) h_t
__global__ void __launch_bounds__(256) kd_act(int64_t n, const float* __restrict__ hv, const float* __restrict__ ht,
                                              float* __restrict__ at) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  at[i] = dn_dsilu(Dn{hv[i], 0.f}).v * ht[i];
}

// seed (1, l_E,s) of every atom's energy output o; d a2 = seed W3^T, d h2 = d a2 * silu'(h2)
__global__ void __launch_bounds__(256) kd_head_seed(int64_t n, int D, const int* __restrict__ astruct,
                                                    const float* __restrict__ dE, const float* __restrict__ W3,
                                                    const float* __restrict__ h2v, const float* __restrict__ h2t,
                                                    float* __restrict__ dov, float* __restrict__ dot,
                                                    float* __restrict__ dhv, float* __restrict__ dht) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t a = i / D;
  const int c = (int)(i % D);
  const Dn sd{1.0f, dE[astruct[a]]};
  if (c == 0) {
    dov[a] = sd.v;
    dot[a] = sd.t;
  }
  const Dn g = (W3[c] * sd) * dn_dsilu(Dn{h2v[i], h2t[i]});
  dhv[i] = g.v;
  dht[i] = g.t;
}

// d h = d a * silu'(h), in place
__global__ void __launch_bounds__(256) kd_act_bwd(int64_t n, const float* __restrict__ hv, const float* __restrict__ ht,
                                                  float* __restrict__ dv, float* __restrict__ dt) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const Dn g = Dn{dv[i], dt[i]} * dn_dsilu(Dn{hv[i], ht[i]});
  dv[i] = g.v;
  dt[i] = g.t;
}

// tangent of d sRBF / d rbf_n * d sRBF_n / d f_n per row (edge, or bond through its edge)
__global__ void __launch_bounds__(256) kd_freq(int64_t n, int R, int p, float inv_c, const int* __restrict__ rows,
                                               const float* __restrict__ len, const float* __restrict__ ddot,
                                               const float* __restrict__ f, const float* __restrict__ drv,
                                               const float* __restrict__ drt, float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t r = i / R;
  const int k = (int)(i % R);
  const int64_t e = rows ? rows[r] : r;
  out[i] = (Dn{drv[i], drt[i]} * dn_srbf_df(Dn{len[e], ddot[e]}, f[k], inv_c, p)).t;
}

__global__ void __launch_bounds__(256) kd_add(int64_t n, float* __restrict__ a, const float* __restrict__ b) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) a[i] += b[i];
}

// ---------------------------------------------------------------------------
// Buffers (after the activations in the workspace, with the conservative
// readout only) and the host driver.
// ---------------------------------------------------------------------------
struct DualBufs {
  // forward tangents
  float *rdot, *ddot, *rbfa_t, *rbfb_t, *ft_t, *ea_t, *eb_t;
  float *v_t[kMaxLayers + 1], *e_t[kMaxLayers + 1], *a_t[kMaxLayers + 1];
  // per layer, [0] value and [1] tangent: pre-activations, gate outputs and
  // messages
  float *zav[kMaxLayers][2], *zbe[kMaxLayers][2], *zan[kMaxLayers][2];
  float *pav[kMaxLayers][2], *pbe[kMaxLayers][2], *m[kMaxLayers][2], *ss[kMaxLayers][2], *mu[kMaxLayers][2];
  float *h1_t, *a1_t, *h2_t, *a2_t;
  // backward, [0] value and [1] tangent
  float *dov[2], *dh2[2], *dh1[2], *dv[2], *de[2], *da[2], *dea[2], *deb[2], *dm[2], *dmu[2], *dss[2];
  float *dpav[2], *dpbe[2], *dzav[2], *dzbe[2], *dzan[2], *drbfa[2], *drbfb[2];
  // projections of the atom and bond blocks (forward) and the per-atom and
  // per-bond sums of the pre-activation gradients (backward), rows of 8d
  float *PA[2], *PB[2], *S[2], *T[2];
  float *lnav, *lnbe, *lnan, *fpa, *fpb, *gB;
};

void carve_dual(Arena& ar, const Dims& m, int64_t n_params, DualBufs& d) {
  const int64_t N = m.N, E = m.E, B = m.B, A = m.A, D = m.D, R = m.R, K = m.K;
  auto f = [&](int64_t n) { return ar.take<float>(n); };
  d.rdot = f(3 * E);
  d.ddot = f(E);
  d.rbfa_t = f(E * R);
  d.rbfb_t = f(B * R);
  d.ft_t = f(A * K);
  d.ea_t = f(E * D);
  d.eb_t = f(B * D);
  for (int t = 0; t <= m.T; ++t) {
    d.v_t[t] = f(N * D);
    d.e_t[t] = f(E * D);
    d.a_t[t] = t < m.T ? f(A * D) : nullptr;
  }
  for (int t = 0; t < m.T; ++t)
    for (int k = 0; k < 2; ++k) {
      d.zav[t][k] = f(E * 2 * D);
      d.zbe[t][k] = f(A * 2 * D);
      d.zan[t][k] = f(A * 2 * D);
      d.pav[t][k] = f(E * D);
      d.pbe[t][k] = f(A * D);
      d.m[t][k] = f(N * D);
      d.ss[t][k] = f(B * D);
      d.mu[t][k] = f(B * D);
    }
  d.h1_t = f(N * D);
  d.a1_t = f(N * D);
  d.h2_t = f(N * D);
  d.a2_t = f(N * D);
  for (int k = 0; k < 2; ++k) {
    d.dov[k] = f(N);
    d.dh2[k] = f(N * D);
    d.dh1[k] = f(N * D);
    d.dv[k] = f(N * D);
    d.de[k] = f(E * D);
    d.da[k] = f(A * D);
    d.dea[k] = f(E * D);
    d.deb[k] = f(B * D);
    d.dm[k] = f(N * D);
    d.dmu[k] = f(B * D);
    d.dss[k] = f(B * D);
    d.dpav[k] = f(E * D);
    d.dpbe[k] = f(A * D);
    d.dzav[k] = f(E * 2 * D);
    d.dzbe[k] = f(A * 2 * D);
    d.dzan[k] = f(A * 2 * D);
    d.PA[k] = f(N * 8 * D);
    d.PB[k] = f(B * 8 * D);
    d.S[k] = f(N * 8 * D);
    d.T[k] = f(B * 8 * D);
    d.drbfa[k] = f(E * R);
    d.drbfb[k] = f(B * R);
  }
  d.lnav = f(kDnGateWaves * 4 * D);
  d.lnbe = f(kDnGateWaves * 4 * D);
  d.lnan = f(kDnGateWaves * 4 * D);
  d.fpa = f(E * R);
  d.fpb = f(B * R);
  d.gB = f(n_params);
}

// The tangent problem of a linear map whose value problem is p: tangent
// inputs per segment, no bias, the residual's tangent.
GemmProblem tangent_of(GemmProblem p, std::initializer_list<const float*> at, float* ct, const float* res_t) {
  int k = 0;
  for (const float* x : at) p.seg[k++].A = x;
  p.C = ct;
  p.bias = nullptr;
  p.res = res_t;
  return p;
}

unsigned dn_blocks(int64_t n) { return (unsigned)cdiv(std::max<int64_t>(n, 1), 256); }

// G (public layout, overwritten) = tangent of the weight gradient described
// at the top of this file, for the loss gradients dE [S], dF [N,3], dS [S,9]
// and, with the moment head, dM [N] (may be null: zero). Needs the
// activations of forward_impl with the same weights (a.Pal) and positions.
int cons_grad_impl(Ctx& c, const float* dE, const float* dF, const float* dS, const float* dM, float* G,
                   hipStream_t st) {
  const Dims& m = c.dm;
  Acts& a = c.a;
  const ParamLayout& L = c.La;
  const ParamLayout& Lg = c.L;
  const float* P = a.Pal;
  const chgnet_graph& g = *c.graph;
  const chgnet_batch& bt = *c.batch;
  const int D = m.D, R = m.R, K = m.K, pe = c.hp->envelope_p;
  const int64_t N = m.N, E = m.E, B = m.B, A = m.A;
  DualBufs d;
  {
    Arena ar{c.ws, c.ws_bytes, c.ws_used};
    carve_dual(ar, m, Lg.total, d);
    if (!ar.ok()) return fail(CHGNET_EWORKSPACE, "workspace too small (query chgnet_workspace_size)");
  }
  float* gB = d.gB;
  CHG_TRY(fill(G, Lg.total, 0.f, st));
  CHG_TRY(fill(gB, Lg.total, 0.f, st));
  const float inv_ca = 1.0f / c.hp->r_atom, inv_cb = 1.0f / c.hp->r_bond;

  // tangents of the geometry and bases
  if (E > 0)
    KLAUNCH(st, "kd_geom", kd_edges<<<dn_blocks(E), 256, 0, st>>>((int)E, R, pe, inv_ca, a.edge_src, g.edge_dst, a.atom_struct,
                                                                  a.edge_len, a.edge_xhat, bt.lattice, dF, dS, P + L.f_a,
                                                                  d.rdot, d.ddot, d.rbfa_t));
  if (B > 0)
    KLAUNCH(st, "kd_geom", kd_bonds<<<dn_blocks(B), 256, 0, st>>>((int)B, R, pe, inv_cb, g.bond_edge, a.edge_len, d.ddot,
                                                                  P + L.f_b, d.rbfb_t));
  if (A > 0)
    KLAUNCH(st, "kd_geom", kd_angles<<<dn_blocks(A), 256, 0, st>>>((int)A, K, a.ang_b1, a.ang_b2, g.bond_edge, a.edge_len,
                                                                   a.edge_xhat, d.rdot, d.ft_t));
  {
    std::vector<GemmProblem> ps;
    GemmProblem p = gp(E, D, d.e_t[0], D);
    seg(p, d.rbfa_t, R, 0, R, P + L.W_e, 2 * D, 0);
    ps.push_back(p);
    p = gp(E, D, d.ea_t, D);
    seg(p, d.rbfa_t, R, 0, R, P + L.W_e + D, 2 * D, 0);
    ps.push_back(p);
    p = gp(B, D, d.eb_t, D);
    seg(p, d.rbfb_t, R, 0, R, P + L.W_eb, D, 0);
    ps.push_back(p);
    p = gp(A, D, d.a_t[0], D);
    seg(p, d.ft_t, K, 0, K, P + L.W_th, D, 0);
    ps.push_back(p);
    CHG_TRY(run_gemms(ps, st, "kd_gemm"));
  }
  CHG_TRY(fill(d.v_t[0], N * D, 0.f, st));

  // forward tangents through the interaction blocks (Eq. 11)
  auto gates = [&](DnGates& J, bool fwd) -> int {
    J.start[0] = 0;
    for (int k = 0; k < J.n; ++k) J.start[k + 1] = J.start[k] + J.j[k].rows;
    if (fwd) {
      if (J.start[J.n] > 0)
      {
        if (D == 64) KLAUNCH(st, "kd_gate_fwd", kd_gate_fwd<1><<<(unsigned)(kDnGateWaves / 4), 256, 0, st>>>(J));
        else KLAUNCH(st, "kd_gate_fwd", kd_gate_fwd<2><<<(unsigned)(kDnGateWaves / 4), 256, 0, st>>>(J));
      }
    } else {
      // every wavefront writes its LayerNorm terms, also for jobs without rows
      if (D == 64) KLAUNCH(st, "kd_gate_bwd", kd_gate_bwd<1><<<(unsigned)(kDnGateWaves / 4), 256, 0, st>>>(J));
      else KLAUNCH(st, "kd_gate_bwd", kd_gate_bwd<2><<<(unsigned)(kDnGateWaves / 4), 256, 0, st>>>(J));
    }
    return CHGNET_OK;
  };
  const int64_t WB = (int64_t)D * 2 * D;  // one d-row input block of a gate's first layer
  const bool seq = c.hp->sequential != 0;
  // Modules of a layer, by bit: 1 atom conv (Eq. 4), 2 bond conv (Eq. 5), 4
  // angle update (Eq. 6). Under Eq. (11) all three read layer-t features and
  // run together; under Eq. (10) they run in order, the bond conv reading
  // v^{t+1} and the angle update v^{t+1} and e^{t+1}.
  for (int t = 0; t < m.T; ++t) {
    const LayerOffsets& lo = L.layer[t];
    const bool ang = lo.has_angle;
    const float *Wav = P + lo.av.W, *Wbe = P + lo.be.W, *Wan = P + lo.an.W;
    // projections of the modules' atom blocks (v W_av0 | v W_av1 | v W_be0 |
    // v W_an0, from vin) and bond blocks (e_b W_be1 | e_b W_be2 | e_b W_an1 |
    // e_b W_an2, from ein); the edge and angle blocks with the bias into z
    auto project = [&](int which, const float* vv, const float* vt, const float* ev, const float* et) -> int {
      std::vector<GemmProblem> ps;
      const float* Wa[4] = {Wav, Wav + WB, Wbe, Wan};
      for (int k = 0; k < 4; ++k) {
        if (!(which & (k < 2 ? 1 : k == 2 ? 2 : 4))) continue;
        GemmProblem p = gp(N, 2 * D, d.PA[0] + k * 2 * D, 8 * D);
        seg(p, vv, D, 0, D, Wa[k], 2 * D, 0);
        ps.push_back(p);
        ps.push_back(tangent_of(p, {vt}, d.PA[1] + k * 2 * D, nullptr));
      }
      const float* Wb[4] = {Wbe + WB, Wbe + 2 * WB, Wan + WB, Wan + 2 * WB};
      for (int k = 0; k < 4; ++k) {
        if (!(which & (k < 2 ? 2 : 4))) continue;
        GemmProblem p = gp(B, 2 * D, d.PB[0] + k * 2 * D, 8 * D);
        p.a_rows = g.bond_edge;
        seg(p, ev, D, 0, D, Wb[k], 2 * D, 0);
        ps.push_back(p);
        ps.push_back(tangent_of(p, {et}, d.PB[1] + k * 2 * D, nullptr));
      }
      if (which & 1) {
        GemmProblem p = gp(E, 2 * D, d.zav[t][0], 2 * D);
        seg(p, a.e[t], D, 0, D, Wav + 2 * WB, 2 * D, 0);
        p.bias = P + lo.av.b;
        ps.push_back(p);
        ps.push_back(tangent_of(p, {d.e_t[t]}, d.zav[t][1], nullptr));
      }
      if (which & 2) {
        GemmProblem p = gp(A, 2 * D, d.zbe[t][0], 2 * D);
        seg(p, a.a[t], D, 0, D, Wbe + 3 * WB, 2 * D, 0);
        p.bias = P + lo.be.b;
        ps.push_back(p);
        ps.push_back(tangent_of(p, {d.a_t[t]}, d.zbe[t][1], nullptr));
      }
      if (which & 4) {
        GemmProblem p = gp(A, 2 * D, d.zan[t][0], 2 * D);
        seg(p, a.a[t], D, 0, D, Wan + 3 * WB, 2 * D, 0);
        p.bias = P + lo.an.b;
        ps.push_back(p);
        ps.push_back(tangent_of(p, {d.a_t[t]}, d.zan[t][1], nullptr));
      }
      return run_gemms(ps, st, "kd_gemm");
    };
    auto gates_fwd = [&](int which) -> int {
      DnGates J{};
      const GatedOffsets* go[3] = {&lo.av, &lo.be, &lo.an};
      float* zs[3][2] = {{d.zav[t][0], d.zav[t][1]}, {d.zbe[t][0], d.zbe[t][1]}, {d.zan[t][0], d.zan[t][1]}};
      for (int k = 0; k < 3; ++k) {
        if (!(which & (1 << k))) continue;
        DnGate& q = J.j[J.n++];
        q.rows = k == 0 ? E : A;
        q.zv = zs[k][0];
        q.zt = zs[k][1];
        q.gc = P + go[k]->g_c;
        q.bc = P + go[k]->b_c;
        q.gg = P + go[k]->g_g;
        q.bg = P + go[k]->b_g;
        // gathered projections: atom conv v_i, v_j; bond conv and angle
        // update the centre atom, first and second bond
        const int pa = k == 0 ? 0 : k == 1 ? 4 * D : 6 * D, pb = k == 1 ? 0 : 4 * D;
        const int* ix[3] = {k == 0 ? a.edge_src : a.ang_ctr, k == 0 ? g.edge_dst : a.ang_b1, a.ang_b2};
        q.nadd = k == 0 ? 2 : 3;
        for (int u = 0; u < q.nadd; ++u) {
          const bool atom = u == 0 || k == 0;
          const int col = k == 0 ? 2 * D * u : atom ? pa : pb + 2 * D * (u - 1);
          q.addv[u] = (atom ? d.PA[0] : d.PB[0]) + col;
          q.addt[u] = (atom ? d.PA[1] : d.PB[1]) + col;
          q.idx[u] = ix[u];
        }
        if (k == 0) {
          q.pv = d.pav[t][0];
          q.pt = d.pav[t][1];
        } else if (k == 1) {
          q.pv = d.pbe[t][0];
          q.pt = d.pbe[t][1];
        } else {
          q.pt = d.a_t[t + 1];
          q.res_t = d.a_t[t];
        }
      }
      return gates(J, true);
    };
    auto messages = [&](int which) -> int {
      if ((which & 1) && N > 0)
        KLAUNCH(st, "kd_msg", kd_msg_atoms<<<(unsigned)N, 256, 0, st>>>((int)N, D, g.edge_ptr, a.ea, d.ea_t, d.pav[t][0],
                                                                        d.pav[t][1], d.m[t][0], d.m[t][1]));
      if ((which & 2) && B > 0)
        KLAUNCH(st, "kd_msg", kd_msg_bonds<<<(unsigned)cdiv(B, 4), 256, 0, st>>>((int)B, D, g.angle_ptr, a.ang_b2, a.eb,
                                                                                 d.eb_t, d.pbe[t][0], d.pbe[t][1],
                                                                                 d.ss[t][0], d.ss[t][1], d.mu[t][0],
                                                                                 d.mu[t][1]));
      return CHGNET_OK;
    };
    // v' = v + m Wo + bo; e' = e, bonds e'_b = e_b + mu Wo + bo (tangents)
    auto updates = [&](int which) -> int {
      if ((which & 2) && E > 0) {
        const int64_t n4 = E * D / 4;
        KLAUNCH(st, "k_copy", k_copy4<<<(unsigned)std::min<int64_t>(cdiv(n4, 256), 4096), 256, 0, st>>>(
                                  reinterpret_cast<float4*>(d.e_t[t + 1]), reinterpret_cast<const float4*>(d.e_t[t]), n4));
      }
      std::vector<GemmProblem> ps;
      if (which & 1) {
        GemmProblem p = gp(N, D, d.v_t[t + 1], D);
        seg(p, d.m[t][1], D, 0, D, P + lo.av_Wo, D, 0);
        p.res = d.v_t[t];
        p.res_ld = D;
        ps.push_back(p);
      }
      if (which & 2) {
        GemmProblem p = gp(B, D, d.e_t[t + 1], D);
        seg(p, d.mu[t][1], D, 0, D, P + lo.be_Wo, D, 0);
        p.res = d.e_t[t];
        p.res_ld = D;
        p.res_rows = g.bond_edge;
        p.c_rows = g.bond_edge;
        ps.push_back(p);
      }
      return run_gemms(ps, st, "kd_gemm");
    };
    if (!seq) {
      CHG_TRY(project(ang ? 7 : 3, a.v[t], d.v_t[t], a.e[t], d.e_t[t]));
      CHG_TRY(gates_fwd(ang ? 7 : 3));
      CHG_TRY(messages(3));
      CHG_TRY(updates(3));
    } else {
      CHG_TRY(project(1, a.v[t], d.v_t[t], a.e[t], d.e_t[t]));
      CHG_TRY(gates_fwd(1));
      CHG_TRY(messages(1));
      CHG_TRY(updates(1));
      CHG_TRY(project(2, a.v[t + 1], d.v_t[t + 1], a.e[t], d.e_t[t]));
      CHG_TRY(gates_fwd(2));
      CHG_TRY(messages(2));
      CHG_TRY(updates(2));
      if (ang) {
        CHG_TRY(project(4, a.v[t + 1], d.v_t[t + 1], a.e[t + 1], d.e_t[t + 1]));
        CHG_TRY(gates_fwd(4));
      }
    }
  }

  // energy head tangents: h1 = v W1 + b1, a1 = SiLU(h1), h2 = a1 W2 + b2, a2 = SiLU(h2)
  const HeadOffsets& hE = L.head[0];
  const HeadOffsets& hEg = Lg.head[0];
  const int64_t ND = N * D;
  auto gemm1 = [&](int64_t M, int Nc, float* C, int ldc, const float* Ain, int lda, int Kd, const float* W, int ldw,
                   int trans) -> int {
    std::vector<GemmProblem> ps;
    GemmProblem p = gp(M, Nc, C, ldc);
    seg(p, Ain, lda, 0, Kd, W, ldw, trans);
    ps.push_back(p);
    return run_gemms(ps, st, "kd_gemm");
  };
  CHG_TRY(gemm1(N, D, d.h1_t, D, d.v_t[m.T], D, D, P + hE.W1, D, 0));
  KLAUNCH(st, "kd_head", kd_act<<<dn_blocks(ND), 256, 0, st>>>(ND, a.hE1, d.h1_t, d.a1_t));
  CHG_TRY(gemm1(N, D, d.h2_t, D, d.a1_t, D, D, P + hE.W2, D, 0));
  KLAUNCH(st, "kd_head", kd_act<<<dn_blocks(ND), 256, 0, st>>>(ND, a.hE2, d.h2_t, d.a2_t));

  // backward in dual numbers; weight terms: X_t^T Y_v into G, X_v^T Y_t into gB
  std::vector<TnProblem> ts;
  auto crossc = [&](int64_t Rr, int M, int Nn, const float* xv, const float* xt, int ldx, const int* xr,
                    const float* const* y, int ldy, int ycol, const int* yr, int64_t off, int ld_out) {
    if (Rr <= 0) return;
    ts.push_back(tp(Rr, M, Nn, xt, ldx, 0, xr, y[0], ldy, ycol, yr, G + off, ld_out));
    ts.push_back(tp(Rr, M, Nn, xv, ldx, 0, xr, y[1], ldy, ycol, yr, gB + off, ld_out));
  };
  auto cross = [&](int64_t Rr, int M, int Nn, const float* xv, const float* xt, int ldx, const int* xr, const float* const* y,
                   int ldy, const int* yr, int64_t off, int ld_out) {
    crossc(Rr, M, Nn, xv, xt, ldx, xr, y, ldy, 0, yr, off, ld_out);
  };
  auto colsum = [&](int64_t Rr, int Nn, const float* yt, int ldy, const int* yr, int64_t off) {
    if (Rr <= 0) return;
    ts.push_back(tp(Rr, 1, Nn, nullptr, 0, 0, nullptr, yt, ldy, 0, yr, gB + off, Nn));
  };
  auto flush = [&]() -> int {
    const int r = run_tns(ts, a, st, "kd_tn");
    ts.clear();
    return r;
  };
  auto gemm2 = [&](int64_t M, int Nc, float* const* C, int ldc, float* const* Ain, int lda, int Kd, const float* W, int ldw,
                   int trans, const int* a_rows) -> int {
    std::vector<GemmProblem> ps;
    GemmProblem p = gp(M, Nc, C[0], ldc);
    p.a_rows = a_rows;
    seg(p, Ain[0], lda, 0, Kd, W, ldw, trans);
    ps.push_back(p);
    ps.push_back(tangent_of(p, {Ain[1]}, C[1], nullptr));
    return run_gemms(ps, st, "kd_gemm");
  };

  KLAUNCH(st, "kd_head", kd_head_seed<<<dn_blocks(ND), 256, 0, st>>>(ND, D, a.atom_struct, dE, P + hE.W3, a.hE2, d.h2_t,
                                                                      d.dov[0], d.dov[1], d.dh2[0], d.dh2[1]));
  const float* a2p[2] = {a.aE2, d.a2_t};
  cross(N, D, 1, a2p[0], a2p[1], D, nullptr, d.dov, 1, nullptr, hEg.W3, 1);
  colsum(N, 1, d.dov[1], 1, nullptr, hEg.b3);
  CHG_TRY(gemm2(N, D, d.dh1, D, d.dh2, D, D, P + hE.W2, D, 1, nullptr));
  KLAUNCH(st, "kd_head", kd_act_bwd<<<dn_blocks(ND), 256, 0, st>>>(ND, a.hE1, d.h1_t, d.dh1[0], d.dh1[1]));
  cross(N, D, D, a.aE1, d.a1_t, D, nullptr, d.dh2, D, nullptr, hEg.W2, D);
  colsum(N, D, d.dh2[1], D, nullptr, hEg.b2);
  CHG_TRY(gemm2(N, D, d.dv, D, d.dh1, D, D, P + hE.W1, D, 1, nullptr));
  cross(N, D, D, a.v[m.T], d.v_t[m.T], D, nullptr, d.dh1, D, nullptr, hEg.W1, D);
  colsum(N, D, d.dh1[1], D, nullptr, hEg.b1);
  if (c.hp->magmom && dM) {
    // m_i = |v_i w_m + b_m| with the seed (0, l_M,i): its first-order
    // backward, in the tangent part only
    KLAUNCH(st, "kd_head", k_magmom_bwd<<<(unsigned)cdiv(N, 4), 256, 0, st>>>((int)N, D, dM, a.oM, P + L.M_W, a.gM,
                                                                            d.dv[1]));
    ts.push_back(tp(N, D, 1, a.v[m.T], D, 0, nullptr, a.gM, 1, 0, nullptr, gB + Lg.M_W, 1));
    ts.push_back(tp(N, 1, 1, nullptr, 0, 0, nullptr, a.gM, 1, 0, nullptr, gB + Lg.M_b, 1));
  }
  CHG_TRY(flush());
  for (int k = 0; k < 2; ++k) {
    CHG_TRY(fill(d.de[k], E * D, 0.f, st));
    CHG_TRY(fill(d.da[k], A * D, 0.f, st));
    CHG_TRY(fill(d.dea[k], E * D, 0.f, st));
    CHG_TRY(fill(d.deb[k], B * D, 0.f, st));
  }

  for (int t = m.T - 1; t >= 0; --t) {
    const LayerOffsets& lo = L.layer[t];
    const LayerOffsets& lg = Lg.layer[t];
    const bool ang = lo.has_angle;
    const float *Wav = P + lo.av.W, *Wbe = P + lo.be.W, *Wan = P + lo.an.W;
    // inputs the modules read: under Eq. (10) the bond conv and the angle
    // update read v^{t+1}, and the angle update e^{t+1}
    const float* vbv = seq ? a.v[t + 1] : a.v[t];
    const float* vbt = seq ? d.v_t[t + 1] : d.v_t[t];
    const float* env = seq ? a.e[t + 1] : a.e[t];
    const float* ent = seq ? d.e_t[t + 1] : d.e_t[t];
    // output linears (bit 1 atom conv: dm = dv Wo^T; bit 2 bond conv:
    // dmu = de_b Wo^T) and their weight terms
    auto out_linears = [&](int which) -> int {
      if (which & 1) {
        CHG_TRY(gemm2(N, D, d.dm, D, d.dv, D, D, P + lo.av_Wo, D, 1, nullptr));
        cross(N, D, D, d.m[t][0], d.m[t][1], D, nullptr, d.dv, D, nullptr, lg.av_Wo, D);
        colsum(N, D, d.dv[1], D, nullptr, lg.av_bo);
      }
      if (which & 2) {
        if (B > 0) CHG_TRY(gemm2(B, D, d.dmu, D, d.de, D, D, P + lo.be_Wo, D, 1, g.bond_edge));
        cross(B, D, D, d.mu[t][0], d.mu[t][1], D, nullptr, d.de, D, g.bond_edge, lg.be_Wo, D);
        colsum(B, D, d.de[1], D, g.bond_edge, lg.be_bo);
      }
      return flush();
    };
    auto messages_bwd = [&](int which) -> int {
      if ((which & 1) && E > 0)
        KLAUNCH(st, "kd_msg_bwd", kd_bwd_atoms<<<dn_blocks(E * D), 256, 0, st>>>(E * D, D, a.edge_src, d.dm[0], d.dm[1],
                                                                                 a.ea, d.ea_t, d.pav[t][0], d.pav[t][1],
                                                                                 d.dpav[0], d.dpav[1], d.dea[0],
                                                                                 d.dea[1]));
      if ((which & 2) && B > 0)
        KLAUNCH(st, "kd_msg_bwd", kd_bwd_bonds<<<dn_blocks(B * D), 256, 0, st>>>(B * D, d.dmu[0], d.dmu[1], d.ss[t][0],
                                                                                 d.ss[t][1], a.eb, d.eb_t, d.deb[0],
                                                                                 d.deb[1], d.dss[0], d.dss[1]));
      if ((which & 2) && A > 0) {
        KLAUNCH(st, "kd_msg_bwd", kd_bwd_angles<<<dn_blocks(A * D), 256, 0, st>>>(A * D, D, a.ang_b1, a.ang_b2, d.dss[0],
                                                                                  d.dss[1], a.eb, d.eb_t, d.dpbe[0],
                                                                                  d.dpbe[1]));
        KLAUNCH(st, "kd_msg_bwd", kd_bwd_b2<<<dn_blocks(B * D), 256, 0, st>>>(B * D, D, a.bond_src, g.bond_ptr,
                                                                              g.angle_ptr, d.dss[0], d.dss[1],
                                                                              d.pbe[t][0], d.pbe[t][1], d.deb[0],
                                                                              d.deb[1]));
      }
      return CHGNET_OK;
    };
    auto gates_bwd = [&](int which) -> int {
      DnGates J{};
      const GatedOffsets* go[3] = {&lo.av, &lo.be, &lo.an};
      float* zs[3][2] = {{d.zav[t][0], d.zav[t][1]}, {d.zbe[t][0], d.zbe[t][1]}, {d.zan[t][0], d.zan[t][1]}};
      float* dp[3][2] = {{d.dpav[0], d.dpav[1]}, {d.dpbe[0], d.dpbe[1]}, {d.da[0], d.da[1]}};
      float* dz[3][2] = {{d.dzav[0], d.dzav[1]}, {d.dzbe[0], d.dzbe[1]}, {d.dzan[0], d.dzan[1]}};
      float* lnp[3] = {d.lnav, d.lnbe, d.lnan};
      for (int k = 0; k < 3; ++k) {
        if (!(which & (1 << k))) continue;
        DnGate& q = J.j[J.n++];
        q.rows = k == 0 ? E : A;
        q.zv = zs[k][0];
        q.zt = zs[k][1];
        q.gc = P + go[k]->g_c;
        q.bc = P + go[k]->b_c;
        q.gg = P + go[k]->g_g;
        q.bg = P + go[k]->b_g;
        q.dpv = dp[k][0];
        q.dpt = dp[k][1];
        q.dzv = dz[k][0];
        q.dzt = dz[k][1];
        q.lnp = lnp[k];
      }
      return gates(J, false);
    };
    // pre-activation gradients summed per atom (S blocks: 0, 1 atom conv v_i,
    // v_j; 2 bond-conv centre; 3 angle-update centre) and per bond (T blocks:
    // 0, 1 bond-conv first and second bond; 2, 3 angle update)
    auto dz_sums = [&](int which) -> int {
      const int q0 = (which & 1) ? 0 : (which & 2) ? 2 : 3;
      const int q1 = (which & 4) ? 4 : (which & 2) ? 3 : 2;
      if (N > 0 && q1 > q0)
        KLAUNCH(st, "kd_dz_sum", kd_dz_atoms<<<(unsigned)(N * (q1 - q0)), 256, 0, st>>>(
                                     (int)N, D, q0, q1 - q0, g.edge_ptr, g.edge_rev, g.bond_ptr, g.angle_ptr, d.dzav[0],
                                     d.dzav[1], d.dzbe[0], d.dzbe[1], d.dzan[0], d.dzan[1], d.S[0], d.S[1]));
      if (B > 0 && (which & 6))
        KLAUNCH(st, "kd_dz_sum", kd_dz_bonds<<<(unsigned)cdiv(B, 4), 256, 0, st>>>((int)B, D, (which >> 1) & 3,
                                                                                  g.angle_ptr, a.bond_src, g.bond_ptr,
                                                                                  a.ang_b2, d.dzbe[0], d.dzbe[1],
                                                                                  d.dzan[0], d.dzan[1], d.T[0], d.T[1]));
      return CHGNET_OK;
    };
    // input gradients of the modules in `which` (accumulated): atoms from S,
    // edges from dz_av, angles from dz_be, dz_an; then the bond rows of e
    // from T
    auto input_grads = [&](int which) -> int {
      std::vector<GemmProblem> ps;
      GemmProblem p = gp(N, D, d.dv[0], D);
      p.accumulate = 1;
      if (which & 1) {
        seg(p, d.S[0], 8 * D, 0, 2 * D, Wav, 2 * D, 1);
        seg(p, d.S[0], 8 * D, 2 * D, 2 * D, Wav + WB, 2 * D, 1);
      }
      if (which & 2) seg(p, d.S[0], 8 * D, 4 * D, 2 * D, Wbe, 2 * D, 1);
      if (which & 4) seg(p, d.S[0], 8 * D, 6 * D, 2 * D, Wan, 2 * D, 1);
      ps.push_back(p);
      ps.push_back(tangent_of(p, {d.S[1], d.S[1], d.S[1], d.S[1]}, d.dv[1], nullptr));
      if (which & 1) {
        p = gp(E, D, d.de[0], D);
        p.accumulate = 1;
        seg(p, d.dzav[0], 2 * D, 0, 2 * D, Wav + 2 * WB, 2 * D, 1);
        ps.push_back(p);
        ps.push_back(tangent_of(p, {d.dzav[1]}, d.de[1], nullptr));
      }
      if (which & 6) {
        p = gp(A, D, d.da[0], D);
        p.accumulate = 1;
        if (which & 2) seg(p, d.dzbe[0], 2 * D, 0, 2 * D, Wbe + 3 * WB, 2 * D, 1);
        if (which & 4) seg(p, d.dzan[0], 2 * D, 0, 2 * D, Wan + 3 * WB, 2 * D, 1);
        ps.push_back(p);
        ps.push_back(which == 4 ? tangent_of(p, {d.dzan[1]}, d.da[1], nullptr)
                                : tangent_of(p, {d.dzbe[1], d.dzan[1]}, d.da[1], nullptr));
      }
      CHG_TRY(run_gemms(ps, st, "kd_gemm"));
      if (which & 6) {
        ps.clear();
        p = gp(B, D, d.de[0], D);
        p.accumulate = 1;
        p.c_rows = g.bond_edge;
        if (which & 2) {
          seg(p, d.T[0], 8 * D, 0, 2 * D, Wbe + WB, 2 * D, 1);
          seg(p, d.T[0], 8 * D, 2 * D, 2 * D, Wbe + 2 * WB, 2 * D, 1);
        }
        if (which & 4) {
          seg(p, d.T[0], 8 * D, 4 * D, 2 * D, Wan + WB, 2 * D, 1);
          seg(p, d.T[0], 8 * D, 6 * D, 2 * D, Wan + 2 * WB, 2 * D, 1);
        }
        ps.push_back(p);
        ps.push_back(tangent_of(p, {d.T[1], d.T[1], d.T[1], d.T[1]}, d.de[1], nullptr));
        CHG_TRY(run_gemms(ps, st, "kd_gemm"));
      }
      return CHGNET_OK;
    };
    // weight terms of the gates, block by block: atom blocks over atoms
    // against S, bond blocks over bonds against T, edge and angle blocks over
    // their rows against dz
    auto gate_terms = [&](int gi, const float* const* dz, const float* lnp, const GatedOffsets& og) {
      const int64_t rows = gi == 0 ? E : A;
      if (gi == 0) {
        crossc(N, D, 2 * D, a.v[t], d.v_t[t], D, nullptr, d.S, 8 * D, 0, nullptr, og.W, 2 * D);
        crossc(N, D, 2 * D, a.v[t], d.v_t[t], D, nullptr, d.S, 8 * D, 2 * D, nullptr, og.W + WB, 2 * D);
        crossc(E, D, 2 * D, a.e[t], d.e_t[t], D, nullptr, dz, 2 * D, 0, nullptr, og.W + 2 * WB, 2 * D);
      } else {
        const int sc = gi == 1 ? 4 * D : 6 * D, tc = gi == 1 ? 0 : 4 * D;
        const float* ev = gi == 1 ? a.e[t] : env;
        const float* et = gi == 1 ? d.e_t[t] : ent;
        crossc(N, D, 2 * D, vbv, vbt, D, nullptr, d.S, 8 * D, sc, nullptr, og.W, 2 * D);
        crossc(B, D, 2 * D, ev, et, D, g.bond_edge, d.T, 8 * D, tc, nullptr, og.W + WB, 2 * D);
        crossc(B, D, 2 * D, ev, et, D, g.bond_edge, d.T, 8 * D, tc + 2 * D, nullptr, og.W + 2 * WB, 2 * D);
        crossc(A, D, 2 * D, a.a[t], d.a_t[t], D, nullptr, dz, 2 * D, 0, nullptr, og.W + 3 * WB, 2 * D);
      }
      colsum(rows, 2 * D, dz[1], 2 * D, nullptr, og.b);
      // LayerNorm scales and shifts: the column sums of the per-wavefront terms
      ts.push_back(split_out(tp(kDnGateWaves, 1, 4 * D, nullptr, 0, 0, nullptr, lnp, 4 * D, 0, nullptr, gB + og.g_c, D), D,
                             gB + og.b_c, gB + og.g_g, gB + og.b_g));
    };
    auto module_terms = [&](int which) -> int {
      if (which & 1) gate_terms(0, d.dzav, d.lnav, lg.av);
      if (which & 2) gate_terms(1, d.dzbe, d.lnbe, lg.be);
      if (which & 4) gate_terms(2, d.dzan, d.lnan, lg.an);
      return flush();
    };
    if (!seq) {
      const int all = ang ? 7 : 3;
      CHG_TRY(out_linears(3));
      CHG_TRY(messages_bwd(3));
      CHG_TRY(gates_bwd(all));
      CHG_TRY(dz_sums(all));
      CHG_TRY(input_grads(all));
      CHG_TRY(module_terms(all));
    } else {
      // Eq. (10) in reverse: the angle update (upstream da^{t+1}; gradients
      // into v^{t+1}, e^{t+1} and a^t), the bond conv (upstream de^{t+1};
      // into v^{t+1}, e^t, a^t), then the atom conv (upstream dv^{t+1})
      if (ang) {
        CHG_TRY(gates_bwd(4));
        CHG_TRY(dz_sums(4));
        CHG_TRY(input_grads(4));
        CHG_TRY(module_terms(4));
      }
      CHG_TRY(out_linears(2));
      CHG_TRY(messages_bwd(2));
      CHG_TRY(gates_bwd(2));
      CHG_TRY(dz_sums(2));
      CHG_TRY(input_grads(2));
      CHG_TRY(module_terms(2));
      CHG_TRY(out_linears(1));
      CHG_TRY(messages_bwd(1));
      CHG_TRY(gates_bwd(1));
      CHG_TRY(dz_sums(1));
      CHG_TRY(input_grads(1));
      CHG_TRY(module_terms(1));
    }
  }

  // embedding (Eq. 2) and sRBF frequencies
  // element table rows: g[Z_i - 1] += d v0_i (tangent), summed per element in atom order
  KLAUNCH(st, "kd_embed", k_embed_bwd_Z<<<94, 64 * kEmbZWaves, 0, st>>>((int)N, D, bt.Z, d.dv[1], gB + Lg.W_Z));
  cross(E, R, D, a.rbf_a, d.rbfa_t, R, nullptr, d.de, D, nullptr, Lg.W_e, 2 * D);
  colsum(E, D, d.de[1], D, nullptr, Lg.b_e0);
  cross(E, R, D, a.rbf_a, d.rbfa_t, R, nullptr, d.dea, D, nullptr, Lg.W_e + D, 2 * D);
  cross(B, R, D, a.rbf_b, d.rbfb_t, R, nullptr, d.deb, D, nullptr, Lg.W_eb, D);
  cross(A, K, D, a.ft, d.ft_t, K, nullptr, d.da, D, nullptr, Lg.W_th, D);
  colsum(A, D, d.da[1], D, nullptr, Lg.b_th);
  CHG_TRY(flush());
  if (E > 0) {
    std::vector<GemmProblem> ps;
    GemmProblem p = gp(E, R, d.drbfa[0], R);
    seg(p, d.de[0], D, 0, D, P + L.W_e, 2 * D, 1);
    seg(p, d.dea[0], D, 0, D, P + L.W_e + D, 2 * D, 1);
    ps.push_back(p);
    ps.push_back(tangent_of(p, {d.de[1], d.dea[1]}, d.drbfa[1], nullptr));
    if (B > 0) {
      p = gp(B, R, d.drbfb[0], R);
      seg(p, d.deb[0], D, 0, D, P + L.W_eb, D, 1);
      ps.push_back(p);
      ps.push_back(tangent_of(p, {d.deb[1]}, d.drbfb[1], nullptr));
    }
    CHG_TRY(run_gemms(ps, st, "kd_gemm"));
    KLAUNCH(st, "kd_embed", kd_freq<<<dn_blocks(E * R), 256, 0, st>>>(E * R, R, pe, inv_ca, nullptr, a.edge_len, d.ddot,
                                                                       P + L.f_a, d.drbfa[0], d.drbfa[1], d.fpa));
    colsum(E, R, d.fpa, R, nullptr, Lg.f_a);
    if (B > 0) {
      KLAUNCH(st, "kd_embed", kd_freq<<<dn_blocks(B * R), 256, 0, st>>>(B * R, R, pe, inv_cb, g.bond_edge, a.edge_len,
                                                                         d.ddot, P + L.f_b, d.drbfb[0], d.drbfb[1], d.fpb));
      colsum(B, R, d.fpb, R, nullptr, Lg.f_b);
    }
    CHG_TRY(flush());
  }
  KLAUNCH(st, "kd_add", kd_add<<<dn_blocks(Lg.total), 256, 0, st>>>(Lg.total, G, gB));
  return CHGNET_OK;
}
