// fp32 MFMA GEMMs for the per-atom, per-edge and per-angle linear layers.
//
// Each wavefront owns a 32x32 block of C built from four 16x16x4 fp32 MFMA
// tiles; a 256-thread workgroup covers 64x64, with the K dimension streamed
// through LDS in chunks of 16. Operand rows may be gathered through an index
// array (edge -> source atom, bond -> edge, angle -> bond), so the
// concatenated GatedMLP inputs of Eq. (4)-(6) never exist in memory: the
// products of their blocks are summed in the epilogue.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.hpp"
#include "gemm.hpp"

namespace chg {

typedef float v4f __attribute__((ext_vector_type(4)));

namespace {

__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + __expf(-x)); }

__global__ void __launch_bounds__(256) k_gemm(GemmBatch batch) {
  const GemmProblem& P = batch.p[blockIdx.z];
  const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  if (r0 >= P.M || c0 >= P.N) return;
  __shared__ float As[64][17];
  __shared__ float Bs[16][68];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = (wave >> 1) * 32, wc = (wave & 1) * 32;
  v4f acc[2][2];
  for (int a = 0; a < 2; ++a)
    for (int b = 0; b < 2; ++b) acc[a][b] = v4f{0.f, 0.f, 0.f, 0.f};
  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  const int grow = r0 + lrow;
  const bool rvalid = grow < P.M;
  const int64_t arow = rvalid ? (P.a_rows ? P.a_rows[grow] : grow) : 0;
  const int bk = tid >> 4, bc = (tid & 15) * 4;
  for (int s = 0; s < P.nseg; ++s) {
    const GemmSeg S = P.seg[s];
    const float* Arow = S.A + arow * S.lda + S.a_col;
    for (int k0 = 0; k0 < S.K; k0 += 16) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = k0 + lk + q;
        As[lrow][lk + q] = (rvalid && k < S.K) ? Arow[k] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = k0 + bk, n = c0 + bc + q;
        float v = 0.f;
        if (k < S.K && n < P.N) v = S.trans ? S.B[(int64_t)n * S.ldb + k] : S.B[(int64_t)k * S.ldb + n];
        Bs[bk][bc + q] = v;
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < 16; kk += 4) {
        const float a0 = As[wr + (lane & 15)][kk + (lane >> 4)];
        const float a1 = As[wr + 16 + (lane & 15)][kk + (lane >> 4)];
        const float b0 = Bs[kk + (lane >> 4)][wc + (lane & 15)];
        const float b1 = Bs[kk + (lane >> 4)][wc + 16 + (lane & 15)];
        acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0, acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b1, acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b0, acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1, acc[1][1], 0, 0, 0);
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int ti = 0; ti < 2; ++ti) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = r0 + wr + ti * 16 + 4 * (lane >> 4) + j;
      if (row >= P.M) continue;
#pragma unroll
      for (int tj = 0; tj < 2; ++tj) {
        const int col = c0 + wc + tj * 16 + (lane & 15);
        if (col >= P.N) continue;
        float v = acc[ti][tj][j];
        if (P.act == ACT_DSILU_MUL) {
          const float x = P.mul[(int64_t)row * P.mul_ld + col];
          const float sg = sigm(x);
          v *= sg * (1.0f + x * (1.0f - sg));
        }
        if (P.bias) v += P.bias[col];
        for (int q = 0; q < P.nadd; ++q) {
          const int64_t ar = P.add_rows[q] ? P.add_rows[q][row] : row;
          v += P.add[q][ar * P.add_ld[q] + col];
        }
        if (P.res) {
          const int64_t rr = P.res_rows ? P.res_rows[row] : row;
          v += P.res[rr * P.res_ld + col];
        }
        const int64_t cr = P.c_rows ? P.c_rows[row] : row;
        float* dst = P.C + cr * P.ldc + col;
        *dst = P.accumulate ? *dst + v : v;
        if (P.act == ACT_SILU_OUT) P.C2[(int64_t)row * P.ldc2 + col] = v * sigm(v);
      }
    }
  }
}

struct TnPlan {
  TnProblem p;
  int rpc;       // rows per chunk
  int nchunks;
  int tiles_n;   // tiles along n
  int tiles;     // total 64x64 tiles
  int64_t off;   // partial offset
};
struct TnLaunch {
  int n;
  TnPlan q[kMaxTnProblems];
};

__global__ void __launch_bounds__(256) k_tn(TnLaunch L, float* __restrict__ part) {
  const TnPlan& Q = L.q[blockIdx.z];
  const TnProblem& P = Q.p;
  const int chunk = blockIdx.x;
  if (chunk >= Q.nchunks || (int)blockIdx.y >= Q.tiles) return;
  const int m0 = (blockIdx.y / Q.tiles_n) * 64, n0 = (blockIdx.y % Q.tiles_n) * 64;
  const int rlo = chunk * Q.rpc;
  const int rhi = min(P.R, rlo + Q.rpc);
  __shared__ float Xs[16][68];
  __shared__ float Ys[16][68];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  v4f acc[2][2];
  for (int a = 0; a < 2; ++a)
    for (int b = 0; b < 2; ++b) acc[a][b] = v4f{0.f, 0.f, 0.f, 0.f};
  const int lr = tid >> 4, lc = (tid & 15) * 4;
  for (int r0 = rlo; r0 < rhi; r0 += 16) {
    const int r = r0 + lr;
    const bool rv = r < rhi;
    const int64_t xr = rv ? (P.x_rows ? P.x_rows[r] : r) : 0;
    const int64_t yr = rv ? (P.y_rows ? P.y_rows[r] : r) : 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int m = m0 + lc + q, n = n0 + lc + q;
      float xv = 0.f, yv = 0.f;
      if (rv && m < P.M) xv = P.X ? P.X[xr * P.ldx + P.x_col + m] : 1.0f;
      if (rv && n < P.N) yv = P.Y[yr * P.ldy + P.y_col + n];
      Xs[lr][lc + q] = xv;
      Ys[lr][lc + q] = yv;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; kk += 4) {
      const float a0 = Xs[kk + (lane >> 4)][wm + (lane & 15)];
      const float a1 = Xs[kk + (lane >> 4)][wm + 16 + (lane & 15)];
      const float b0 = Ys[kk + (lane >> 4)][wn + (lane & 15)];
      const float b1 = Ys[kk + (lane >> 4)][wn + 16 + (lane & 15)];
      acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1, acc[1][1], 0, 0, 0);
    }
    __syncthreads();
  }
  float* out = part + Q.off + (int64_t)chunk * P.M * P.N;
#pragma unroll
  for (int ti = 0; ti < 2; ++ti)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + wm + ti * 16 + 4 * (lane >> 4) + j;
      if (m >= P.M) continue;
#pragma unroll
      for (int tj = 0; tj < 2; ++tj) {
        const int n = n0 + wn + tj * 16 + (lane & 15);
        if (n < P.N) out[(int64_t)m * P.N + n] = acc[ti][tj][j];
      }
    }
}

// Ordered column sums of chunk partials: 16 wavefronts per block, wave w
// sums chunks w, w+16, ... (fp64), then the 16 partial sums are added in
// wave order. The result is independent of scheduling.
__device__ __forceinline__ double sum_chunks(const float* __restrict__ src, int nchunks, int64_t stride, int w) {
  double s0 = 0.0, s1 = 0.0;
  int c = w;
  for (; c + 16 < nchunks; c += 32) {
    s0 += (double)src[(int64_t)c * stride];
    s1 += (double)src[(int64_t)(c + 16) * stride];
  }
  if (c < nchunks) s0 += (double)src[(int64_t)c * stride];
  return s0 + s1;
}

__global__ void __launch_bounds__(1024) k_tn_reduce(TnLaunch L, const float* __restrict__ part) {
  __shared__ double red[16][64];
  const TnPlan& Q = L.q[blockIdx.y];
  const TnProblem& P = Q.p;
  const int64_t mn = (int64_t)P.M * P.N;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t k = (int64_t)blockIdx.x * 64 + lane;
  if ((int64_t)blockIdx.x * 64 >= mn) return;
  red[w][lane] = k < mn ? sum_chunks(part + Q.off + k, Q.nchunks, mn, w) : 0.0;
  __syncthreads();
  if (w == 0 && k < mn) {
    double s = 0.0;
    for (int q = 0; q < 16; ++q) s += red[q][lane];
    const int m = (int)(k / P.N), n = (int)(k % P.N);
    float* o = P.out + (int64_t)m * P.ld_out + n;
    *o = (float)((double)*o + s);
  }
}

__global__ void __launch_bounds__(1024) k_reduce_rows(const float* __restrict__ part, int nchunks, int64_t stride,
                                                      int count, float* __restrict__ out) {
  __shared__ double red[16][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k = blockIdx.x * 64 + lane;
  red[w][lane] = k < count ? sum_chunks(part + k, nchunks, stride, w) : 0.0;
  __syncthreads();
  if (w == 0 && k < count) {
    double s = 0.0;
    for (int q = 0; q < 16; ++q) s += red[q][lane];
    out[k] = (float)((double)out[k] + s);
  }
}

}  // namespace

int gemm_launch(const GemmBatch& b, hipStream_t st, const char* tag) {
  int gx = 0, gy = 0;
  for (int i = 0; i < b.n; ++i) {
    gx = std::max<int>(gx, (int)cdiv(b.p[i].M, 64));
    gy = std::max<int>(gy, (int)cdiv(b.p[i].N, 64));
  }
  if (b.n == 0 || gx == 0 || gy == 0) return CHGNET_OK;
  KLAUNCH(st, tag, k_gemm<<<dim3(gx, gy, b.n), 256, 0, st>>>(b));
  return CHGNET_OK;
}

int tn_launch(const TnBatch& b, float* part, int64_t part_cap, hipStream_t st, const char* tag) {
  TnLaunch L;
  L.n = b.n;
  int64_t off = 0;
  int gx = 0, gy = 0;
  const int64_t budget = part_cap / std::max(1, b.n);
  for (int i = 0; i < b.n; ++i) {
    TnPlan& q = L.q[i];
    q.p = b.p[i];
    const int tm = (int)cdiv(q.p.M, 64);
    q.tiles_n = (int)cdiv(q.p.N, 64);
    q.tiles = tm * q.tiles_n;
    const int64_t mn = (int64_t)q.p.M * q.p.N;
    int64_t nch = std::max<int64_t>(1, std::min<int64_t>(cdiv(q.p.R, 256), std::max(8, 512 / q.tiles)));
    nch = std::min<int64_t>(nch, 128);
    nch = std::min<int64_t>(nch, std::max<int64_t>(1, budget / std::max<int64_t>(1, mn)));
    int64_t rpc = cdiv(cdiv(q.p.R, nch), 16) * 16;
    if (rpc < 16) rpc = 16;
    q.rpc = (int)rpc;
    q.nchunks = q.p.R > 0 ? (int)cdiv(q.p.R, rpc) : 0;
    q.off = off;
    off += (int64_t)q.nchunks * mn;
    gx = std::max(gx, q.nchunks);
    gy = std::max(gy, q.tiles);
  }
  if (off > part_cap) return fail(CHGNET_EWORKSPACE, "split-K partial buffer too small");
  if (b.n == 0) return CHGNET_OK;
  if (gx > 0) {
    KLAUNCH(st, tag, k_tn<<<dim3(gx, gy, b.n), 256, 0, st>>>(L, part));
  }
  int64_t maxmn = 0;
  for (int i = 0; i < b.n; ++i) maxmn = std::max<int64_t>(maxmn, (int64_t)b.p[i].M * b.p[i].N);
  KLAUNCH(st, "k_tn_reduce", k_tn_reduce<<<dim3((unsigned)cdiv(maxmn, 64), b.n), 1024, 0, st>>>(L, part));
  return CHGNET_OK;
}

int reduce_rows_launch(const float* part, int nchunks, int64_t stride, int count, float* out, hipStream_t st) {
  if (count <= 0) return CHGNET_OK;
  KLAUNCH(st, "k_reduce_rows", k_reduce_rows<<<(unsigned)cdiv(count, 64), 1024, 0, st>>>(part, nchunks, stride, count, out));
  return CHGNET_OK;
}

}  // namespace chg
