// fp32 MFMA GEMMs for the per-atom, per-edge and per-angle linear layers.
//
// k_gemm: a 256-thread workgroup owns a 128 x 64 tile of C, each wavefront
// 32 rows x 64 columns as two 32x32 fp32 MFMA (32x32x2) accumulators, with
// the K dimension streamed through LDS in chunks of 32. k_gemm_w: direct-load
// 32 x 64 wave tiles with k split over wavefronts, for few rows or a long k.
// k_tn: split-K weight-gradient products X^T Y. Operand rows may be gathered
// through an index array (edge -> source atom, bond -> edge, angle -> bond),
// so the concatenated GatedMLP inputs of Eq. (4)-(6) never exist in memory:
// the products of their blocks are summed in the epilogue.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <string>

#include "common.hpp"
#include "gemm.hpp"

namespace chg {

typedef float v4f __attribute__((ext_vector_type(4)));

namespace {

__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + __expf(-x)); }

typedef float v16f __attribute__((ext_vector_type(16)));

// Load 4 consecutive floats p[k..k+3] of a row of length K (zero past K).
__device__ __forceinline__ float4 load4(const float* __restrict__ p, int k, int K, bool vec) {
  if (vec && k + 3 < K) return *reinterpret_cast<const float4*>(p + k);
  float4 v;
  v.x = k < K ? p[k] : 0.f;
  v.y = k + 1 < K ? p[k + 1] : 0.f;
  v.z = k + 2 < K ? p[k + 2] : 0.f;
  v.w = k + 3 < K ? p[k + 3] : 0.f;
  return v;
}

// NN product, 128 x BN tile per 256-thread block; wave w owns rows
// [32w, 32w + 32) and all BN columns as BN/32 tiles of 32x32 (fp32 MFMA
// 32x32x2). K is streamed through LDS in chunks of 32; the global loads of
// chunk c+1 are issued into registers before the MFMAs of chunk c.
// NADD gathered addends are summed in the epilogue; their row indices are
// staged in LDS once per block.
template <int BN>
struct GemmStage {
  float4 a[4];
  float4 b[BN / 32];
};

template <int BN>
__device__ __forceinline__ void gemm_fetch(const GemmProblem& P, const GemmSeg& S, int k0, int c0, int tid,
                                           const int64_t (&arow)[4], const bool (&aval)[4], GemmStage<BN>& g) {
  constexpr int KC = 32;
  const bool avec = ((S.lda | S.a_col) & 3) == 0 && ((uintptr_t)S.A & 15) == 0;
  const bool bvec = (S.ldb & 3) == 0 && ((uintptr_t)S.B & 15) == 0;
  (void)bvec;
  const int ak = (tid & 7) * 4;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    g.a[q] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (aval[q]) g.a[q] = load4(S.A + arow[q] * S.lda + S.a_col + k0, ak, S.K - k0, avec);
  }
  if (!S.trans) {
    // column strips: thread takes column n = tid % BN and 4 consecutive k
    constexpr int G = 256 / BN;  // k-groups per pass
    const int n = tid % BN, kg = tid / BN;
    const bool nv = c0 + n < P.N;
#pragma unroll
    for (int q = 0; q < BN / 32; ++q) {
      const int kb = k0 + 4 * (kg + G * q);
      const float* col = S.B + c0 + n;
      float4 v;
      v.x = (nv && kb + 0 < S.K) ? col[(int64_t)(kb + 0) * S.ldb] : 0.f;
      v.y = (nv && kb + 1 < S.K) ? col[(int64_t)(kb + 1) * S.ldb] : 0.f;
      v.z = (nv && kb + 2 < S.K) ? col[(int64_t)(kb + 2) * S.ldb] : 0.f;
      v.w = (nv && kb + 3 < S.K) ? col[(int64_t)(kb + 3) * S.ldb] : 0.f;
      g.b[q] = v;
    }
  } else {
#pragma unroll
    for (int q = 0; q < BN / 32; ++q) {
      const int idx = tid + 256 * q, n = idx / (KC / 4), kk = (idx % (KC / 4)) * 4;
      g.b[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (c0 + n < P.N) g.b[q] = load4(S.B + (int64_t)(c0 + n) * S.ldb + k0, kk, S.K - k0, bvec);
    }
  }
}

// Epilogue of one row and 4 consecutive columns: activation, bias,
// residual, optional accumulation, 16-byte stores when aligned.
__device__ __forceinline__ bool gemm_cvec(const GemmProblem& P) {
  return (P.ldc & 3) == 0 && ((uintptr_t)P.C & 15) == 0 &&
         (!P.res || ((P.res_ld & 3) == 0 && ((uintptr_t)P.res & 15) == 0)) &&
         (P.act != ACT_DSILU_MUL || ((P.mul_ld & 3) == 0 && ((uintptr_t)P.mul & 15) == 0)) &&
         (P.act != ACT_SILU_OUT || ((P.ldc2 & 3) == 0 && ((uintptr_t)P.C2 & 15) == 0));
}

__device__ __forceinline__ void gemm_store4(const GemmProblem& P, int row, int col, float4 sv, bool cvec) {
  if (row >= P.M || col >= P.N) return;
  float v[4] = {sv.x, sv.y, sv.z, sv.w};
  const int64_t rr = P.res ? (P.res_rows ? P.res_rows[row] : row) * (int64_t)P.res_ld : 0;
  const int64_t cr = (P.c_rows ? P.c_rows[row] : row) * (int64_t)P.ldc;
  if (cvec && col + 3 < P.N) {
    if (P.act == ACT_DSILU_MUL) {
      const float4 x4 = *reinterpret_cast<const float4*>(P.mul + (int64_t)row * P.mul_ld + col);
      const float xs[4] = {x4.x, x4.y, x4.z, x4.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float sg = sigm(xs[u]);
        v[u] *= sg * (1.0f + xs[u] * (1.0f - sg));
      }
    }
    if (P.bias)
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] += P.bias[col + u];
    if (P.res) {
      const float4 r4 = *reinterpret_cast<const float4*>(P.res + rr + col);
      v[0] += r4.x; v[1] += r4.y; v[2] += r4.z; v[3] += r4.w;
    }
    float4* dst = reinterpret_cast<float4*>(P.C + cr + col);
    if (P.accumulate) {
      const float4 o = *dst;
      v[0] += o.x; v[1] += o.y; v[2] += o.z; v[3] += o.w;
    }
    *dst = make_float4(v[0], v[1], v[2], v[3]);
    if (P.act == ACT_SILU_OUT)
      *reinterpret_cast<float4*>(P.C2 + (int64_t)row * P.ldc2 + col) =
          make_float4(v[0] * sigm(v[0]), v[1] * sigm(v[1]), v[2] * sigm(v[2]), v[3] * sigm(v[3]));
    return;
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int cc = col + u;
    if (cc >= P.N) break;
    float x = v[u];
    if (P.act == ACT_DSILU_MUL) {
      const float m = P.mul[(int64_t)row * P.mul_ld + cc];
      const float sg = sigm(m);
      x *= sg * (1.0f + m * (1.0f - sg));
    }
    if (P.bias) x += P.bias[cc];
    if (P.res) x += P.res[rr + cc];
    float* dst = P.C + cr + cc;
    *dst = P.accumulate ? *dst + x : x;
    if (P.act == ACT_SILU_OUT) P.C2[(int64_t)row * P.ldc2 + cc] = x * sigm(x);
  }
}

// ROLE only names the instantiation (0 other, 2 input gradients) so that
// profilers can tell the launches apart. OCC: wavefronts per SIMD the
// registers are sized for; at 4 the fragments of a chunk are read in two
// halves of 8 k-steps (126 VGPRs), for launches with a plain epilogue.
template <int BN, int ROLE, int OCC>
__global__ void __launch_bounds__(256, OCC == 4 ? 4 : 1) k_gemm(GemmBatch batch) {
  constexpr int BM = 128, KC = 32, NT = BN / 32, KP = KC + 4, SP = 64 + 4;
  const GemmProblem& P = batch.p[blockIdx.z];
  // Workgroups are dealt to the 8 XCDs round-robin by linear id (gridDim.x
  // is a multiple of 8). Renumber so that the column tiles of one row worker
  // share an XCD, and its A rows are fetched into one L2.
  int bx, by;
  {
    const int p = blockIdx.x + gridDim.x * blockIdx.y, j = p >> 3;
    by = j % gridDim.y;
    bx = 8 * (j / gridDim.y) + (p & 7);
  }
  const int c0 = by * BN;
  const int ntiles = (P.M + BM - 1) / BM;
  if (bx >= ntiles || c0 >= P.N) return;
  // Operand tiles are stored k-contiguous: As[row][k], Bs[col][k]. In MFMA
  // k-step i, lane half h = lane / 32 supplies k = 16 h + i, so each lane
  // reads its 16 A and B values of a chunk with four 16-byte LDS reads.
  // After the K loop the same LDS holds the output tile, 64 columns at a
  // time, so the epilogue writes whole rows with 16-byte stores. A block
  // walks row tiles bx, bx + gridDim.x, ...; the first chunk
  // of its next tile is fetched before the current tile's epilogue.
  constexpr int kOperand = BM * KP + BN * KP, kStage = 4 * 32 * SP;
  __shared__ __attribute__((aligned(16))) float smem[kOperand > kStage ? kOperand : kStage];
  float (*As)[KP] = reinterpret_cast<float (*)[KP]>(smem);
  float (*Bs)[KP] = reinterpret_cast<float (*)[KP]>(smem + BM * KP);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5;
  const int ar = tid >> 3, ak = (tid & 7) * 4;
  const bool cvec = gemm_cvec(P);
  int64_t arow[4];
  bool aval[4];
  auto set_rows = [&](int r0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = r0 + ar + 32 * q;
      aval[q] = r < P.M;
      arow[q] = aval[q] ? (P.a_rows ? P.a_rows[r] : r) : 0;
    }
  };
  GemmStage<BN> g;
  int tile = bx;
  set_rows(tile * BM);
  if (P.nseg > 0) gemm_fetch<BN>(P, P.seg[0], 0, c0, tid, arow, aval, g);
  while (tile < ntiles) {
    const int r0 = tile * BM;
    const int next = tile + gridDim.x;
    v16f acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[t][j] = 0.f;
    int s = 0, k0 = 0;
    while (s < P.nseg) {
      const bool trans = P.seg[s].trans;
#pragma unroll
      for (int q = 0; q < 4; ++q) *reinterpret_cast<float4*>(&As[ar + 32 * q][ak]) = g.a[q];
      if (!trans) {
        constexpr int G = 256 / BN;
#pragma unroll
        for (int q = 0; q < BN / 32; ++q)
          *reinterpret_cast<float4*>(&Bs[tid % BN][4 * (tid / BN + G * q)]) = g.b[q];
      } else {
#pragma unroll
        for (int q = 0; q < BN / 32; ++q) {
          const int idx = tid + 256 * q, n = idx / (KC / 4), kk = (idx % (KC / 4)) * 4;
          *reinterpret_cast<float4*>(&Bs[n][kk]) = g.b[q];
        }
      }
      __syncthreads();
      k0 += KC;
      if (k0 >= P.seg[s].K) {
        k0 = 0;
        ++s;
      }
      if (s < P.nseg) {
        gemm_fetch<BN>(P, P.seg[s], k0, c0, tid, arow, aval, g);
      } else if (next < ntiles) {
        set_rows(next * BM);
        gemm_fetch<BN>(P, P.seg[0], 0, c0, tid, arow, aval, g);
      }
      constexpr int HS = OCC >= 4 ? 2 : 1, KH = 16 / HS;  // fragment reads per chunk, k-steps each
#pragma unroll
      for (int hh = 0; hh < HS; ++hh) {
        float af[KH], bf[NT][KH];
        const float* ap = &As[32 * wave + (lane & 31)][16 * h + KH * hh];
#pragma unroll
        for (int q = 0; q < KH / 4; ++q) {
          const float4 v = *reinterpret_cast<const float4*>(ap + 4 * q);
          af[4 * q] = v.x; af[4 * q + 1] = v.y; af[4 * q + 2] = v.z; af[4 * q + 3] = v.w;
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const float* bp = &Bs[32 * t + (lane & 31)][16 * h + KH * hh];
#pragma unroll
          for (int q = 0; q < KH / 4; ++q) {
            const float4 v = *reinterpret_cast<const float4*>(bp + 4 * q);
            bf[t][4 * q] = v.x; bf[t][4 * q + 1] = v.y; bf[t][4 * q + 2] = v.z; bf[t][4 * q + 3] = v.w;
          }
        }
#pragma unroll
        for (int i = 0; i < KH; ++i)
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bf[t][i], acc[t], 0, 0, 0);
      }
      __syncthreads();
    }
    // ---- epilogue, 64 columns (two 32x32 tiles) at a time through LDS
    float* stg = smem + wave * 32 * SP;
#pragma unroll
    for (int half = 0; half < (NT + 1) / 2; ++half) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        if (2 * half + tt >= NT) break;
#pragma unroll
        for (int j = 0; j < 16; ++j)
          stg[(8 * (j >> 2) + 4 * h + (j & 3)) * SP + 32 * tt + (lane & 31)] = acc[2 * half + tt][j];
      }
      __syncthreads();
      const int cl = 4 * (lane & 15);
      const int col = c0 + 64 * half + cl;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int lr = (lane >> 4) + 4 * i;
        const float4 sv = *reinterpret_cast<const float4*>(stg + lr * SP + cl);
        gemm_store4(P, r0 + 32 * wave + lr, col, sv, cvec);
      }
      __syncthreads();
    }
    tile = next;
  }
}

// Direct-load GEMM for short or few row tiles: each wavefront owns a 32 x 64
// tile of C and streams its fragments straight from global memory (no LDS
// staging), k in groups of 8: in MFMA k-step i of a group, lane half h
// supplies k = 4h + i; lane c = lane % 32 holds output columns 2c + u of the
// tile (u < 2: two 32x32 tiles with interleaved columns), so B fragments are
// 8-byte row pieces (or 16-byte k runs when B is stored transposed). The
// WK wavefronts of a tile split its k groups into contiguous runs and their
// partial tiles are added in wave order in LDS before the shared epilogue.
// Rows, columns and k beyond the matrices are clamped into them and
// cancelled through a 0/1 mask on the B fragment (a clamped A entry is a
// finite operand entry times zero).
constexpr int kGwWaves = 8;
constexpr int kGwLd = 64 + 4;

template <int WK>
__global__ void __launch_bounds__(512, 2) k_gemm_w(GemmBatch batch) {
  __shared__ __attribute__((aligned(16))) float slot[kGwWaves * 32 * kGwLd];
  const GemmProblem& P = batch.p[blockIdx.z];
  constexpr int TPB = kGwWaves / WK;  // row tiles per block
  const int tid = threadIdx.x, lane = tid & 63, c = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tl = wave / WK, kp = wave % WK;
  const int r0 = (blockIdx.x * TPB + tl) * 32, n0 = blockIdx.y * 64;
  if ((int)blockIdx.x * TPB * 32 >= P.M || n0 >= P.N) return;  // uniform over the block
  int groups = 0;
  for (int s = 0; s < P.nseg; ++s) groups += (P.seg[s].K + 7) / 8;
  const int g_lo = kp * groups / WK, g_hi = (kp + 1) * groups / WK;
  // this lane's A row (clamped) and B columns (clamped)
  const int arow_i = min(r0 + c, P.M - 1);
  const int64_t arow = P.a_rows ? P.a_rows[arow_i] : arow_i;
  const int ncol0 = n0 + 2 * c;
  const int nc0 = min(ncol0, P.N - 1), nc1 = min(ncol0 + 1, P.N - 1);
  const float nm0 = ncol0 < P.N ? 1.f : 0.f, nm1 = ncol0 + 1 < P.N ? 1.f : 0.f;
  v16f acc[2];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[u][j] = 0.f;
  constexpr int NB = 4;  // register buffers: NB - 1 groups in flight ahead of the MFMAs
  float af[NB][4], bf[NB][4][2];
  // group g -> (segment, k0)
  auto locate = [&](int g, int& s, int& k0) {
    s = 0;
    int left = g;
    while (s + 1 < P.nseg && left >= (P.seg[s].K + 7) / 8) {
      left -= (P.seg[s].K + 7) / 8;
      ++s;
    }
    k0 = 8 * left;
  };
  auto fetch = [&](int g, int b) {
    int s, k0;
    locate(g, s, k0);
    const GemmSeg& S = P.seg[s];
    const int kb = k0 + 4 * h;
    const float* ap = S.A + arow * S.lda + S.a_col;
    // vector paths only where every lane's piece is inside (uniform tests)
    if (((S.lda | S.a_col | S.K) & 3) == 0 && ((uintptr_t)S.A & 15) == 0 && (S.K & 7) == 0) {
      const float4 t = *reinterpret_cast<const float4*>(ap + kb);
      af[b][0] = t.x; af[b][1] = t.y; af[b][2] = t.z; af[b][3] = t.w;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) af[b][i] = ap[min(kb + i, S.K - 1)];
    }
    float km[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) km[i] = kb + i < S.K ? 1.f : 0.f;
    if (!S.trans) {
      const bool bvec = (S.ldb & 1) == 0 && ((uintptr_t)S.B & 7) == 0 && n0 + 64 <= P.N;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float* bp = S.B + (int64_t)min(kb + i, S.K - 1) * S.ldb;
        if (bvec) {
          const float2 t = *reinterpret_cast<const float2*>(bp + ncol0);
          bf[b][i][0] = t.x * km[i];
          bf[b][i][1] = t.y * km[i];
        } else {
          bf[b][i][0] = bp[nc0] * (km[i] * nm0);
          bf[b][i][1] = bp[nc1] * (km[i] * nm1);
        }
      }
    } else {
      const bool bvec = (S.ldb & 3) == 0 && ((uintptr_t)S.B & 15) == 0 && (S.K & 7) == 0;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float* bp = S.B + (int64_t)(u ? nc1 : nc0) * S.ldb;
        const float m = u ? nm1 : nm0;
        if (bvec) {
          const float4 t = *reinterpret_cast<const float4*>(bp + kb);
          bf[b][0][u] = t.x * m; bf[b][1][u] = t.y * m; bf[b][2][u] = t.z * m; bf[b][3][u] = t.w * m;
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) bf[b][i][u] = bp[min(kb + i, S.K - 1)] * (km[i] * m);
        }
      }
    }
  };
  auto compute = [&](int b) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int u = 0; u < 2; ++u) acc[u] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[b][i], bf[b][i][u], acc[u], 0, 0, 0);
  };
  const int n = g_hi - g_lo;
#pragma unroll
  for (int j = 0; j < NB - 1; ++j)
    if (j < n) fetch(g_lo + j, j);
  for (int it = 0; it < n; it += NB) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (it + j + NB - 1 < n) fetch(g_lo + it + j + NB - 1, (j + NB - 1) % NB);
      if (it + j < n) compute(j);
    }
  }
  // partial tiles -> LDS, rows 8(j/4) + 4h + j%4, columns 2c + u
  float* my = slot + wave * 32 * kGwLd;
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int j = 0; j < 16; ++j) my[(8 * (j >> 2) + 4 * h + (j & 3)) * kGwLd + 2 * c + u] = acc[u][j];
  __syncthreads();
  // wave-ordered sum of each tile's WK partials, epilogue with row-contiguous
  // 4-column pieces: 32 rows x 16 pieces per tile
  const bool cvec = gemm_cvec(P);
  for (int q = tid; q < TPB * 32 * 16; q += 512) {
    const int t = q / (32 * 16), rr = (q / 16) % 32, cl = 4 * (q % 16);
    const float* base = slot + (t * WK) * 32 * kGwLd + rr * kGwLd + cl;
    float4 sum = *reinterpret_cast<const float4*>(base);
#pragma unroll
    for (int p = 1; p < WK; ++p) {
      const float4 v = *reinterpret_cast<const float4*>(base + p * 32 * kGwLd);
      sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
    }
    gemm_store4(P, (blockIdx.x * TPB + t) * 32 + rr, n0 + cl, sum, cvec);
  }
}

struct TnPlan {
  TnProblem p;
  int vx, vy;            // fragment widths: a wave tile is 32 vx x 32 vy
  int tiles_m, tiles_n;  // wave tiles per chunk (tiles_m = 0: column sums only)
  int rpc;               // rows per chunk (a multiple of 64: four wave ranges of 16-row groups)
  int nchunks;
  int block0;            // first block of this problem in the launch
  int has_bias;          // partials carry one more row: the column sums of Y
  float* bout;           // destination of the column sums (split like out)
  int bowidth;
  float* bouts[4];
  int64_t off;  // partial offset; a chunk's partial is (M + has_bias) x N
};
struct TnLaunch {
  int n;
  TnPlan q[kMaxTnProblems];
};

// Split-K X^T Y without LDS tiles: each wavefront streams its own row range
// and loads its MFMA fragments straight from global memory. In MFMA k-step i
// of a group of 2 KS rows, lane half h supplies row KS h + i; lane c = lane % 32
// holds columns vx c + v (v < vx) of the X row and vy c + u of the Y row, so
// wave tile v of X and u of Y are column-interleaved and the fragment loads
// are 4-, 8- or 16-byte vectors (vy = 4: 64 x 128 wave tiles, in a launch of
// their own at two blocks per compute unit). The next group's fragments are loaded while the
// current group's MFMAs run. The four wavefronts of a block take consecutive
// quarters of the block's rows; their tiles are added in wave order in LDS.
// A problem with a bias row also sums the Y columns (the bias gradient of a
// layer whose weight gradient is X^T Y).
// ROLE only names the instantiation (1: interaction-block weight gradients).
// reduction buffer: two wave tiles and four wavefronts' column sums
template <bool WIDE>
constexpr int tn_red_floats() { return WIDE ? 2 * 64 * 128 + 4 * 128 : 2 * 64 * 64 + 4 * 64; }
// Rows per split-K chunk at most: the eight output tiles of a chunk stream
// the same rows on one XCD, and a chunk of 2048 rows of 384 floats (3 MB)
// stays in that XCD's 4 MB L2 while they do (4480-row chunks measured 1.30
// ms per wide128 layer launch against 1.01 ms).
constexpr int kTnMaxChunkRows = 2048;
// rows of one wavefront's range (a quarter of a chunk): the size of its
// LDS row-index tables
constexpr int kTnWaveRows = kTnMaxChunkRows / 4;
// 64-row units of a launch (summed over its products and 64 x 64 wave tiles)
// from which it takes 64 x 128 wave tiles where N allows (enough work that
// 64 x 64 tiles would fill every block slot with kTnMaxChunkRows-row
// chunks). Measured per training step:
// wide128 -0.4 ms; triclinic40 (below the bound) 0.06 ms slower with them.
constexpr int kTnWideUnits = 3 * 256 * (kTnMaxChunkRows / 64);
// The bound in force: CHGNET_TN_WIDE_MIN_UNITS (a non-negative integer,
// read on every launch) overrides kTnWideUnits, so that the wide tiles can
// also be run, and checked, on small batches.
int64_t tn_wide_min_units() {
  const char* e = std::getenv("CHGNET_TN_WIDE_MIN_UNITS");
  if (e != nullptr && *e != 0) {
    char* end = nullptr;
    const long long v = std::strtoll(e, &end, 10);
    if (*end == 0 && v >= 0) return v;
  }
  return kTnWideUnits;
}

// RIDX: the problem gathers X or Y rows through an index array. The wave
// first copies its range's row indices to LDS (ridx: [2][kTnWaveRows], in the
// reduction buffer, which the block takes over once every wave is past its
// rows), so the fragment loads depend on no other global load and the loads
// of the groups ahead stay in flight.
template <int VX, int VY, bool XFULL, bool YFULL, bool HASX, bool RIDX>
__device__ __forceinline__ void tn_wave(const TnPlan& Q, int chunk, int m0, int n0, bool colsum, float* red,
                                        int* ridx, float* __restrict__ part) {
  // MFMA k-steps (row pairs) per register buffer: 2, or 1 where two-column
  // fragments are loaded one element at a time (partial or unaligned tiles,
  // not on the common shapes)
  constexpr int KS = ((VX == 2 && HASX && !XFULL) || (VY >= 2 && !YFULL)) ? 1 : 2;
  const TnProblem& P = Q.p;
  const int lane = threadIdx.x & 63, c = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar row range
  const int wr = Q.rpc / 4;
  const int rlo = chunk * Q.rpc + wave * wr;
  const int rhi = min(P.R, rlo + wr);
  const int xm = m0 + VX * c, yn = n0 + VY * c;
  v16f acc[VX][VY];
#pragma unroll
  for (int v = 0; v < VX; ++v)
#pragma unroll
    for (int u = 0; u < VY; ++u)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[v][u][j] = 0.f;
  float ysum[VY];
#pragma unroll
  for (int u = 0; u < VY; ++u) ysum[u] = 0.f;
  constexpr int NB = 4;  // register buffers: NB - 1 groups in flight ahead of the MFMAs
  float xf[NB][KS][VX], yf[NB][KS][VY];
  // Branch-free loads: rows and columns are clamped into the matrix. Columns
  // past M or N only reach outputs that are not stored; rows past the wave's
  // range are cancelled by a 0/1 mask on the Y values, applied when the
  // group is consumed, so that every load of a group is in flight at once.
  float rmask[NB][KS];
  if (RIDX) {
    for (int r = rlo + lane; r < rhi; r += 64) {
      ridx[r - rlo] = P.x_rows ? P.x_rows[r] : r;
      ridx[kTnWaveRows + r - rlo] = P.y_rows ? P.y_rows[r] : r;
    }
  }
  auto fetch = [&](int g, int b) {
    int xr[KS], yr[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      xr[i] = yr[i] = min(g + KS * h + i, rhi - 1);
      rmask[b][i] = g + KS * h + i < rhi ? 1.f : 0.f;
    }
    if (RIDX)
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        xr[i] = ridx[xr[i] - rlo];
        yr[i] = ridx[kTnWaveRows + yr[i] - rlo];
      }
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      if (HASX) {
        const float* xp = P.X + (int64_t)xr[i] * P.ldx + P.x_col;
        if (XFULL) {
          const float2 t = *reinterpret_cast<const float2*>(xp + xm);
          xf[b][i][0] = t.x;
          xf[b][i][VX - 1] = t.y;
        } else {
#pragma unroll
          for (int v = 0; v < VX; ++v) xf[b][i][v] = xp[min(xm + v, P.M - 1)];
        }
      }
      const float* yp = P.Y + (int64_t)yr[i] * P.ldy + P.y_col;
      if (YFULL && VY == 4) {
        const float4 t = *reinterpret_cast<const float4*>(yp + yn);
        yf[b][i][0] = t.x;
        yf[b][i][1 % VY] = t.y;
        yf[b][i][2 % VY] = t.z;
        yf[b][i][VY - 1] = t.w;
      } else if (YFULL) {
        const float2 t = *reinterpret_cast<const float2*>(yp + yn);
        yf[b][i][0] = t.x;
        yf[b][i][VY - 1] = t.y;
      } else {
#pragma unroll
        for (int u = 0; u < VY; ++u) yf[b][i][u] = yp[min(yn + u, P.N - 1)];
      }
    }
  };
  auto compute = [&](int b) {
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      float y[VY];
#pragma unroll
      for (int u = 0; u < VY; ++u) y[u] = yf[b][i][u] * rmask[b][i];
      if (HASX) {
#pragma unroll
        for (int v = 0; v < VX; ++v)
#pragma unroll
          for (int u = 0; u < VY; ++u)
            acc[v][u] = __builtin_amdgcn_mfma_f32_32x32x2f32(xf[b][i][v], y[u], acc[v][u], 0, 0, 0);
      }
      if (colsum) {
#pragma unroll
        for (int u = 0; u < VY; ++u) ysum[u] += y[u];
      }
    }
  };
  // a ring of NB register buffers with constant indices (NB groups per
  // iteration); a fixed trip count (rows past the range are masked) keeps
  // the accumulators in place
  constexpr int GRW = 2 * KS;  // rows per group (KS per lane half)
  const int iters = rhi > rlo ? (rhi - rlo + NB * GRW - 1) / (NB * GRW) : 0;
  if (iters > 0) {
#pragma unroll
    for (int b = 0; b < NB - 1; ++b) fetch(rlo + b * GRW, b);
  }
  for (int it = 0; it < iters; ++it) {
    const int g = rlo + it * NB * GRW;
    const bool more = it + 1 < iters;
    fetch(g + (NB - 1) * GRW, NB - 1);
    compute(0);
#pragma unroll
    for (int b = 1; b < NB; ++b) {
      if (more) fetch(g + (NB - 1 + b) * GRW, b - 1);
      compute(b);
    }
  }
  // the row-index tables share this LDS: every wavefront is past its rows
  if (RIDX) __syncthreads();
  constexpr int TILE = VX * VY * 16 * 64, CS = 32 * VY;  // a wave tile; a wavefront's column sums
  // column sums: the two lane halves hold different rows of the same column
  if (colsum) {
#pragma unroll
    for (int u = 0; u < VY; ++u) ysum[u] += __shfl_xor(ysum[u], 32);
    if (h == 0) {
#pragma unroll
      for (int u = 0; u < VY; ++u) red[2 * TILE + wave * CS + u * 32 + c] = ysum[u];
    }
  }
  // wave tiles added in the order (w0 + w1) + (w2 + w3)
  auto put = [&](float* dst) {
#pragma unroll
    for (int v = 0; v < VX; ++v)
#pragma unroll
      for (int u = 0; u < VY; ++u)
#pragma unroll
        for (int j = 0; j < 16; ++j) dst[((v * VY + u) * 16 + j) * 64 + lane] = acc[v][u][j];
  };
  auto add = [&](const float* src) {
#pragma unroll
    for (int v = 0; v < VX; ++v)
#pragma unroll
      for (int u = 0; u < VY; ++u)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[v][u][j] += src[((v * VY + u) * 16 + j) * 64 + lane];
  };
  if (wave == 1) put(red);
  if (wave == 3) put(red + TILE);
  __syncthreads();
  if (wave == 0) add(red);
  if (wave == 2) add(red + TILE);
  __syncthreads();
  if (wave == 2) put(red);
  __syncthreads();
  if (wave != 0) return;
  add(red);
  const int rows_out = P.M + Q.has_bias;
  float* out = part + Q.off + (int64_t)chunk * rows_out * P.N;
  if (HASX) {
#pragma unroll
    for (int v = 0; v < VX; ++v)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int m = m0 + VX * (8 * (j >> 2) + 4 * h + (j & 3)) + v;
        if (m >= P.M) continue;
#pragma unroll
        for (int u = 0; u < VY; ++u) {
          const int n = yn + u;
          if (n < P.N) out[(int64_t)m * P.N + n] = acc[v][u][j];
        }
      }
  }
  if (colsum && h == 0) {
    const float* ys = red + 2 * TILE;
#pragma unroll
    for (int u = 0; u < VY; ++u) {
      const int k = u * 32 + c;
      const float s = (ys[k] + ys[CS + k]) + (ys[2 * CS + k] + ys[3 * CS + k]);
      const int n = yn + u;
      if (n < P.N) out[(int64_t)P.M * P.N + n] = s;
    }
  }
}

template <bool RIDX>
__device__ __forceinline__ void tn_dispatch(const TnPlan& Q, int chunk, int m0, int n0, bool colsum, bool xf, bool yf,
                                            float* red, int* ridx, float* __restrict__ part) {
  if (Q.tiles_m == 0) {
    // column sums only
    if (yf) tn_wave<1, 2, false, true, false, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
    else if (Q.vy == 2) tn_wave<1, 2, false, false, false, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
    else tn_wave<1, 1, false, false, false, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
  } else if (Q.vx == 2 && Q.vy == 2) {
    if (xf && yf) tn_wave<2, 2, true, true, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
    else if (xf) tn_wave<2, 2, true, false, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
    else if (yf) tn_wave<2, 2, false, true, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
    else tn_wave<2, 2, false, false, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
  } else if (Q.vx == 2) {
    if (xf) tn_wave<2, 1, true, false, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
    else tn_wave<2, 1, false, false, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
  } else if (Q.vy == 2) {
    if (yf) tn_wave<1, 2, false, true, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
    else tn_wave<1, 2, false, false, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
  } else {
    tn_wave<1, 1, false, false, true, RIDX>(Q, chunk, m0, n0, colsum, red, ridx, part);
  }
}

// WIDE: the launch of the plans with 64 x 128 wave tiles (their blocks come
// first); b0 is the launch's first block.
template <int ROLE, bool WIDE>
__global__ void __launch_bounds__(256, WIDE ? 2 : 3) k_tn(TnLaunch L, int b0, float* __restrict__ part) {
  __shared__ float red[tn_red_floats<WIDE>()];
  static_assert(4 * 2 * kTnWaveRows <= tn_red_floats<false>(), "row-index tables fit in the reduction buffer");
  const int bid = b0 + (int)blockIdx.x;
  int k = 0;
  while (k + 1 < L.n && bid >= L.q[k + 1].block0) ++k;
  const TnPlan& Q = L.q[k];
  const int lb = bid - Q.block0;
  const int tiles = max(Q.tiles_m, 1) * Q.tiles_n;
  // The tiles of a row chunk sit 8 block indices apart, so that they run on
  // one XCD (blocks are dealt to the 8 XCDs in turn) and share its L2 for the
  // chunk's rows; chunks after the last full group of 8 keep consecutive tiles.
  const int grouped = (Q.nchunks / 8) * 8 * tiles;
  int chunk, tile;
  if (lb < grouped) {
    const int g = lb / (8 * tiles), rem = lb % (8 * tiles);
    tile = rem / 8;
    chunk = g * 8 + rem % 8;
  } else {
    chunk = (Q.nchunks / 8) * 8 + (lb - grouped) / tiles;
    tile = (lb - grouped) % tiles;
  }
  const int tm = tile / Q.tiles_n, tn = tile % Q.tiles_n;
  const int m0 = tm * 32 * Q.vx, n0 = tn * 32 * Q.vy;
  const bool colsum = Q.has_bias && tm == 0;
  // 8-byte fragment loads where the wave tile lies inside the matrix and
  // the rows are 8-byte aligned
  const TnProblem& P = Q.p;
  const bool xf = Q.vx == 2 && P.X && ((P.ldx | P.x_col) & 1) == 0 && ((uintptr_t)P.X & 7) == 0 && m0 + 64 <= P.M;
  int* ridx = reinterpret_cast<int*>(red) + (threadIdx.x >> 6) * 2 * kTnWaveRows;
  if constexpr (WIDE) {
    const bool yf = ((P.ldy | P.y_col) & 3) == 0 && ((uintptr_t)P.Y & 15) == 0 && n0 + 128 <= P.N;
    if (Q.tiles_m == 0) {
      // column sums only
      if (P.x_rows || P.y_rows) {
        if (yf) tn_wave<1, 4, false, true, false, true>(Q, chunk, m0, n0, colsum, red, ridx, part);
        else tn_wave<1, 4, false, false, false, true>(Q, chunk, m0, n0, colsum, red, ridx, part);
      } else {
        if (yf) tn_wave<1, 4, false, true, false, false>(Q, chunk, m0, n0, colsum, red, ridx, part);
        else tn_wave<1, 4, false, false, false, false>(Q, chunk, m0, n0, colsum, red, ridx, part);
      }
    } else if (P.x_rows || P.y_rows) {
      if (xf && yf) tn_wave<2, 4, true, true, true, true>(Q, chunk, m0, n0, colsum, red, ridx, part);
      else tn_wave<2, 4, false, false, true, true>(Q, chunk, m0, n0, colsum, red, ridx, part);
    } else {
      if (xf && yf) tn_wave<2, 4, true, true, true, false>(Q, chunk, m0, n0, colsum, red, ridx, part);
      else tn_wave<2, 4, false, false, true, false>(Q, chunk, m0, n0, colsum, red, ridx, part);
    }
  } else {
    const bool yf = Q.vy == 2 && ((P.ldy | P.y_col) & 1) == 0 && ((uintptr_t)P.Y & 7) == 0 && n0 + 64 <= P.N;
    if (P.x_rows || P.y_rows) tn_dispatch<true>(Q, chunk, m0, n0, colsum, xf, yf, red, ridx, part);
    else tn_dispatch<false>(Q, chunk, m0, n0, colsum, xf, yf, red, ridx, part);
  }
}

// Ordered column sums of chunk partials: 16 wavefronts per block, wave w
// sums chunks w, w+16, ... (fp64), then the 16 partial sums are added in
// wave order. The result is independent of scheduling.
__device__ __forceinline__ double sum_chunks(const float* __restrict__ src, int nchunks, int64_t stride, int w) {
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  int c = w;
  for (; c + 48 < nchunks; c += 64) {
    s0 += (double)src[(int64_t)c * stride];
    s1 += (double)src[(int64_t)(c + 16) * stride];
    s2 += (double)src[(int64_t)(c + 32) * stride];
    s3 += (double)src[(int64_t)(c + 48) * stride];
  }
  for (; c < nchunks; c += 16) s0 += (double)src[(int64_t)c * stride];
  return (s0 + s1) + (s2 + s3);
}

__global__ void __launch_bounds__(1024) k_tn_reduce(TnLaunch L, const float* __restrict__ part) {
  __shared__ double red[16][64];
  const TnPlan& Q = L.q[blockIdx.y];
  const TnProblem& P = Q.p;
  const int64_t mn = (int64_t)(P.M + Q.has_bias) * P.N;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t k = (int64_t)blockIdx.x * 64 + lane;
  if ((int64_t)blockIdx.x * 64 >= mn) return;
  red[w][lane] = k < mn ? sum_chunks(part + Q.off + k, Q.nchunks, mn, w) : 0.0;
  __syncthreads();
  if (w == 0 && k < mn) {
    double s = 0.0;
    for (int q = 0; q < 16; ++q) s += red[q][lane];
    const int m = (int)(k / P.N), n = (int)(k % P.N);
    float* o;
    if (m < P.M) {
      const int q = P.owidth > 0 ? n / P.owidth : 0;
      const int nn = P.owidth > 0 ? n - q * P.owidth : n;
      o = (q == 0 ? P.out : P.outs[q]) + (int64_t)m * P.ld_out + nn;
    } else {
      const int q = Q.bowidth > 0 ? n / Q.bowidth : 0;
      const int nn = Q.bowidth > 0 ? n - q * Q.bowidth : n;
      o = (q == 0 ? Q.bout : Q.bouts[q]) + nn;
    }
    *o = (float)((double)*o + s);
  }
}

// Ordered reduction of chunk partials, two launches. Level 1: block
// (x, g, job) sums the chunks of group g for 64 columns (4 wavefronts, fixed
// order, fp64) into part2[job][g]. Level 2: block (x, job) adds the groups in
// order (4 wavefronts x 8 groups, then the 4 wave sums in order).
__global__ void __launch_bounds__(256) k_reduce_rows1(ReduceJobs J, int groups_max, double* __restrict__ part2_all) {
  __shared__ double red[4][64];
  const ReduceJob& R = J.j[blockIdx.z];
  const int count = R.count, nchunks = R.nchunks;
  const int groups = max(1, min(groups_max, nchunks));
  const int per = (nchunks + groups - 1) / groups;
  if ((int)blockIdx.y >= groups || (int)blockIdx.x * 64 >= count) return;
  double* part2 = part2_all + (int64_t)blockIdx.z * groups_max * 8 * 128;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k = blockIdx.x * 64 + lane, g = blockIdx.y;
  const int c0 = g * per, c1 = min(nchunks, c0 + per);
  double s = 0.0;
  if (k < count)
    for (int c = c0 + w; c < c1; c += 4) s += (double)R.part[(int64_t)c * R.stride + k];
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && k < count) part2[(int64_t)g * count + k] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

__global__ void __launch_bounds__(256) k_reduce_rows2(ReduceJobs J, int groups_max, const double* __restrict__ part2_all) {
  __shared__ double red[4][64];
  const ReduceJob& R = J.j[blockIdx.y];
  const int count = R.count;
  const int groups = max(1, min(groups_max, R.nchunks));
  if ((int)blockIdx.x * 64 >= count) return;
  const double* part2 = part2_all + (int64_t)blockIdx.y * groups_max * 8 * 128;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k = blockIdx.x * 64 + lane;
  double v[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int q = w + 4 * u;
    v[u] = (k < count && q < groups) ? part2[(int64_t)q * count + k] : 0.0;
  }
  double t = 0.0;
#pragma unroll
  for (int u = 0; u < 8; ++u) t += v[u];
  red[w][lane] = t;
  __syncthreads();
  if (w == 0 && k < count) R.out[k] = (float)((double)R.out[k] + (((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane]));
}


// Linear + SiLU layers of the d = 128 readout MLPs (C = A W + b, C2 =
// silu(C), k = N = 128, more than 32768 rows): each wavefront of a 4-wave
// block owns 32 output columns and holds its B fragments (64 floats a lane)
// in registers for the whole launch (reloaded when the problem changes);
// blocks walk the 32-row tiles of the batch's problems. The A tile of tile
// i + 1 goes from registers to the other LDS buffer and the A loads of tile
// i + 2 are issued before the MFMAs of tile i; one block barrier per tile.
// The epilogue works from the accumulators: lane (h, c) holds column c of
// rows 8 (j / 4) + 4 h + j % 4, so each store writes two 128-byte row
// pieces. Measured on wide128: 0.27 -> 0.22 ms per head launch against the
// LDS-tiled GEMM (which re-reads the weights for every tile); with gathered
// residuals, scattered outputs or SiLU' factors it was slower and is not
// used for them.
struct SiluTiles {
  int tile0[kMaxGemmProblems + 1];
};
constexpr int kSiluRows = 32, kSiluK = 128, kSiluWaves = 4;

__global__ void __launch_bounds__(64 * kSiluWaves, 4) k_gemm_silu(GemmBatch batch, SiluTiles T) {
  constexpr int R = kSiluRows, K = kSiluK, NW = kSiluWaves, LD = K + 4, F = R * K / (64 * NW), TPR = K / F,
                KB = K / 32;
  static_assert(F % 4 == 0 && R * TPR == 64 * NW, "A tile split");
  __shared__ __attribute__((aligned(16))) float As[2][R * LD];
  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ntiles = T.tile0[batch.n];
  const int nt = (int)blockIdx.x < ntiles ? (ntiles - 1 - (int)blockIdx.x) / (int)gridDim.x + 1 : 0;
  if (nt == 0) return;
  auto prob_of = [&](int tile) {
    int k = 0;
    while (k + 1 < batch.n && tile >= T.tile0[k + 1]) ++k;
    return k;
  };
  auto tile_of = [&](int i) { return (int)blockIdx.x + i * (int)gridDim.x; };
  // A tile: thread -> row tid / TPR, F columns at F (tid % TPR); rows past M read as zero
  float4 av[F / 4];
  auto fetch = [&](int tile) {
    const int k = prob_of(tile);
    const GemmProblem& P = batch.p[k];
    const GemmSeg& S = P.seg[0];
    const int row = (tile - T.tile0[k]) * R + tid / TPR, ac = F * (tid % TPR);
#pragma unroll
    for (int q = 0; q < F / 4; ++q) av[q] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (row < P.M) {
      const int64_t ar = P.a_rows ? P.a_rows[row] : row;
      const float* src = S.A + ar * S.lda + S.a_col + ac;
#pragma unroll
      for (int q = 0; q < F / 4; ++q) av[q] = *reinterpret_cast<const float4*>(src + 4 * q);
    }
  };
  auto store = [&](float* X) {
    const int xr = tid / TPR, ac = F * (tid % TPR);
#pragma unroll
    for (int q = 0; q < F / 4; ++q) *reinterpret_cast<float4*>(&X[xr * LD + ac + 4 * q]) = av[q];
  };
  // B fragments: MFMA k-step e of k block kb takes k = 32 kb + 16 h + e
  float bfr[KB][16];
  int cur = -1;
  fetch(tile_of(0));
  store(As[0]);
  if (nt > 1) fetch(tile_of(1));
  __syncthreads();
  for (int i = 0; i < nt; ++i) {
    const int tile = tile_of(i);
    const int k = prob_of(tile);
    const GemmProblem& P = batch.p[k];
    const int col = 32 * wave + l32;
    if (k != cur) {
      cur = k;
      const GemmSeg& S = P.seg[0];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kk = 32 * kb + 16 * h + e;
          bfr[kb][e] = S.trans ? S.B[(int64_t)col * S.ldb + kk] : S.B[(int64_t)kk * S.ldb + col];
        }
    }
    if (i + 1 < nt) {
      store(As[(i + 1) & 1]);
      if (i + 2 < nt) fetch(tile_of(i + 2));
    }
    const float* X = As[i & 1];
    v16f acc;
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = 0.f;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      float af[16];
      const float* ap = &X[l32 * LD + 32 * kb + 16 * h];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = *reinterpret_cast<const float4*>(ap + 4 * q);
        af[4 * q] = v.x; af[4 * q + 1] = v.y; af[4 * q + 2] = v.z; af[4 * q + 3] = v.w;
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af[e], bfr[kb][e], acc, 0, 0, 0);
    }
    const int r0 = (tile - T.tile0[k]) * R;
    const float bias = P.bias ? P.bias[col] : 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int row = r0 + 8 * (j >> 2) + 4 * h + (j & 3);
      if (row < P.M) {
        const float x = acc[j] + bias;
        P.C[(int64_t)row * P.ldc + col] = x;
        P.C2[(int64_t)row * P.ldc2 + col] = x * sigm(x);
      }
    }
    __syncthreads();
  }
}

}  // namespace

int gemm_launch(const GemmBatch& b, hipStream_t st, const char* tag) {
  if (b.n == 0) return CHGNET_OK;
  {
    // the Linear + SiLU layers of the d = 128 heads (see k_gemm_silu)
    bool silu = true;
    int maxM = 0;
    SiluTiles T{};
    for (int i = 0; i < b.n && silu; ++i) {
      const GemmProblem& P = b.p[i];
      const GemmSeg& S = P.seg[0];
      silu = P.nseg == 1 && S.K == kSiluK && P.N == 32 * kSiluWaves && P.act == ACT_SILU_OUT && !P.res &&
             !P.c_rows && !P.accumulate && ((S.lda | S.a_col) & 3) == 0 && ((uintptr_t)S.A & 15) == 0;
      maxM = std::max(maxM, P.M);
      T.tile0[i + 1] = T.tile0[i] + (int)cdiv(std::max(P.M, 0), kSiluRows);
    }
    if (silu && maxM > 32768) {
      const unsigned grid = (unsigned)std::min(T.tile0[b.n], 4 * 256);
      KLAUNCH(st, tag, k_gemm_silu<<<grid, 64 * kSiluWaves, 0, st>>>(b, T));
      return CHGNET_OK;
    }
  }
  // 64-column tiles: a 128-column variant needs ~170 VGPRs (2 waves per
  // SIMD) and measured slower on every shape used here
  const int BN = 64;
  int gx = 0, gy = 0;
  for (int i = 0; i < b.n; ++i) {
    gx = std::max<int>(gx, (int)cdiv(b.p[i].M, 128));
    gy = std::max<int>(gy, (int)cdiv(b.p[i].N, BN));
  }
  if (gx == 0 || gy == 0) return CHGNET_OK;
  int maxM = 0, maxN = 0, maxK = 0;
  for (int i = 0; i < b.n; ++i) {
    maxM = std::max(maxM, b.p[i].M);
    maxN = std::max(maxN, b.p[i].N);
    int k = 0;
    for (int s = 0; s < b.p[i].nseg; ++s) k += b.p[i].seg[s].K;
    maxK = std::max(maxK, k);
  }
  if (maxM <= 32768 && (maxK >= 128 || maxM <= 4096)) {
    // few row tiles and a long k, or very few rows: direct-load wave tiles,
    // k split over 1-8 wavefronts so that the launch has about 2048 of them
    // (with k = 64 and ~10^4 rows the LDS-staged tiles below measured faster)
    int64_t tiles = 0;
    int maxg = 0;
    for (int i = 0; i < b.n; ++i) {
      tiles += cdiv(b.p[i].M, 32) * cdiv(b.p[i].N, 64);
      int g = 0;
      for (int s = 0; s < b.p[i].nseg; ++s) g += (int)cdiv(b.p[i].seg[s].K, 8);
      maxg = std::max(maxg, g);
    }
    int wk = 1;
    while (wk < kGwWaves && tiles * wk < 2048 && 2 * wk * 2 <= maxg) wk *= 2;
    const unsigned gyw = (unsigned)cdiv(maxN, 64);
    const unsigned gxw = (unsigned)cdiv(maxM, 32 * (kGwWaves / wk));
    const dim3 grid(gxw, gyw, b.n);
    if (wk == 1) KLAUNCH(st, tag, k_gemm_w<1><<<grid, 512, 0, st>>>(b));
    else if (wk == 2) KLAUNCH(st, tag, k_gemm_w<2><<<grid, 512, 0, st>>>(b));
    else if (wk == 4) KLAUNCH(st, tag, k_gemm_w<4><<<grid, 512, 0, st>>>(b));
    else KLAUNCH(st, tag, k_gemm_w<8><<<grid, 512, 0, st>>>(b));
    return CHGNET_OK;
  }
  // persistent row tiles: about 2048 blocks over the launch; row workers in
  // multiples of 8 (one per XCD, see k_gemm)
  const int per_problem = std::max(1, 2048 / (gy * b.n));
  const dim3 grid((unsigned)(cdiv(std::min(gx, per_problem), 8) * 8), gy, b.n);
  // four wavefronts per SIMD where no problem has an activation epilogue,
  // every segment is at least 128 deep and no problem has both more than
  // 65,536 rows and k > 128 (measured on wide128: the projection, update and
  // input-gradient launches 4-17 % faster; the SiLU / SiLU' launches of the
  // heads 17-25 % and the 31-deep embeddings 3 % slower; the Eq. 10 block's
  // edge and angle input gradients, k = 2d and 4d, 664 against 511 us)
  bool plain = true;
  for (int i = 0; i < b.n; ++i) {
    plain = plain && b.p[i].act == ACT_NONE;
    int k = 0;
    for (int s = 0; s < b.p[i].nseg; ++s) {
      plain = plain && b.p[i].seg[s].K >= 128;
      k += b.p[i].seg[s].K;
    }
    plain = plain && !(b.p[i].M > 65536 && k > 128);
  }
  const bool in_bwd = std::string(tag) == "gemm_in_bwd";
  if (in_bwd && plain) KLAUNCH(st, tag, k_gemm<64, 2, 4><<<grid, 256, 0, st>>>(b));
  else if (in_bwd) KLAUNCH(st, tag, k_gemm<64, 2, 3><<<grid, 256, 0, st>>>(b));
  else if (plain) KLAUNCH(st, tag, k_gemm<64, 0, 4><<<grid, 256, 0, st>>>(b));
  else KLAUNCH(st, tag, k_gemm<64, 0, 3><<<grid, 256, 0, st>>>(b));
  return CHGNET_OK;
}


int tn_launch(const TnBatch& b, float* part, int64_t part_cap, hipStream_t st, const char* tag) {
  if (b.n == 0) return CHGNET_OK;
  // A bias problem (X = ones, M = 1) becomes the column-sum row of a weight
  // problem over the same Y rows and columns, so Y is streamed once.
  TnLaunch L{};
  for (int i = 0; i < b.n; ++i) {
    const TnProblem& p = b.p[i];
    if (p.X == nullptr) continue;
    if (p.M <= 0 || p.N <= 0) return fail(CHGNET_EINVAL, "tn: empty output");
    TnPlan& q = L.q[L.n++];
    q = TnPlan{};
    q.p = p;
  }
  for (int i = 0; i < b.n; ++i) {
    const TnProblem& p = b.p[i];
    if (p.X != nullptr) continue;
    if (p.M != 1 || p.N <= 0) return fail(CHGNET_EINVAL, "tn: a problem without X must have one output row");
    TnPlan* host = nullptr;
    for (int j = 0; j < L.n && !host; ++j) {
      const TnProblem& w = L.q[j].p;
      if (!L.q[j].has_bias && w.X && w.R == p.R && w.N == p.N && w.Y == p.Y && w.ldy == p.ldy && w.y_col == p.y_col &&
          w.y_rows == p.y_rows)
        host = &L.q[j];
    }
    if (!host) {
      host = &L.q[L.n++];
      *host = TnPlan{};
      host->p = p;
      host->p.M = 0;
    }
    host->has_bias = 1;
    host->bout = p.out;
    host->bowidth = p.owidth;
    for (int q = 1; q < 4; ++q) host->bouts[q] = p.outs[q];
  }
  int64_t units = 0;
  for (int i = 0; i < L.n; ++i) {
    TnPlan& q = L.q[i];
    q.vx = q.p.M <= 32 ? 1 : 2;
    q.vy = q.p.N <= 32 ? 1 : 2;
    q.tiles_m = q.p.X ? (int)cdiv(q.p.M, 32 * q.vx) : 0;
    q.tiles_n = (int)cdiv(q.p.N, 32 * q.vy);
    units += cdiv(std::max(q.p.R, 0), 64) * std::max(q.tiles_m, 1) * q.tiles_n;
  }
  // 64 x 128 wave tiles (half the Y fragment loads and row-index reads per
  // MFMA; two 4-wave blocks per compute unit) for the large launches, and
  // the column sums of bias-only problems with them (no launch of 64 x 64
  // tiles is left for those)
  if (units >= tn_wide_min_units()) {
    units = 0;
    for (int i = 0; i < L.n; ++i) {
      TnPlan& q = L.q[i];
      if (q.p.N % 128 == 0 && (!q.p.X || q.p.M > 32)) {
        q.vy = 4;
        q.tiles_n = q.p.N / 128;
      }
      units += cdiv(std::max(q.p.R, 0), 64) * std::max(q.tiles_m, 1) * q.tiles_n;
    }
  }
  // about one block per resident slot (three 4-wave blocks per compute
  // unit): fewer, longer blocks measured faster than several rounds
  const int64_t per = std::max<int64_t>(1, cdiv(units, 3 * 256));
  const int rpc = (int)std::min<int64_t>(64 * per, kTnMaxChunkRows);
  // the wide plans first: their blocks are the first launch's
  std::stable_partition(L.q, L.q + L.n, [](const TnPlan& q) { return q.vy == 4; });
  int64_t off = 0, blocks = 0, maxmn = 0, wide_blocks = 0;
  for (int i = 0; i < L.n; ++i) {
    TnPlan& q = L.q[i];
    q.rpc = rpc;
    q.nchunks = q.p.R > 0 ? (int)cdiv(q.p.R, rpc) : 0;
    q.block0 = (int)blocks;
    q.off = off;
    const int64_t mn = (int64_t)(q.p.M + q.has_bias) * q.p.N;
    off += (int64_t)q.nchunks * mn;
    blocks += (int64_t)q.nchunks * std::max(q.tiles_m, 1) * q.tiles_n;
    maxmn = std::max(maxmn, mn);
    if (q.vy == 4) wide_blocks = blocks;
  }
  if (off > part_cap) return fail(CHGNET_EWORKSPACE, "split-K partial buffer too small");
  if (blocks > 0x7fffffff) return fail(CHGNET_EINVAL, "tn: too many blocks");
  if (blocks > 0) {
    // the wide and the 64 x 64 plans' launches are timed as one under `tag`
    const bool in = std::string(tag) == "tn_in";
    const unsigned wb = (unsigned)wide_blocks, nb = (unsigned)(blocks - wide_blocks);
    KLAUNCH(st, tag, {
      if (wb > 0 && in) k_tn<1, true><<<wb, 256, 0, st>>>(L, 0, part);
      if (wb > 0 && !in) k_tn<0, true><<<wb, 256, 0, st>>>(L, 0, part);
      if (nb > 0 && in) k_tn<1, false><<<nb, 256, 0, st>>>(L, (int)wb, part);
      if (nb > 0 && !in) k_tn<0, false><<<nb, 256, 0, st>>>(L, (int)wb, part);
    });
    KLAUNCH(st, "k_tn_reduce", k_tn_reduce<<<dim3((unsigned)cdiv(maxmn, 64), L.n), 1024, 0, st>>>(L, part));
  }
  return CHGNET_OK;
}

int reduce_rows_multi(const ReduceJobs& J, double* scratch, hipStream_t st) {
  if (J.n == 0) return CHGNET_OK;
  int maxc = 0, maxg = 1;
  for (int i = 0; i < J.n; ++i) {
    if (J.j[i].count > 8 * 128) return fail(CHGNET_EINVAL, "reduce: count too large");
    maxc = std::max(maxc, J.j[i].count);
    maxg = std::max(maxg, std::min(32, J.j[i].nchunks));
  }
  if (maxc == 0) return CHGNET_OK;
  KLAUNCH(st, "k_reduce_rows1", k_reduce_rows1<<<dim3((unsigned)cdiv(maxc, 64), maxg, J.n), 256, 0, st>>>(J, 32, scratch));
  KLAUNCH(st, "k_reduce_rows2", k_reduce_rows2<<<dim3((unsigned)cdiv(maxc, 64), J.n), 256, 0, st>>>(J, 32, scratch));
  return CHGNET_OK;
}

int reduce_rows_launch(const float* part, int nchunks, int64_t stride, int count, float* out, double* scratch,
                       hipStream_t st) {
  ReduceJobs J{};
  J.n = 1;
  J.j[0] = ReduceJob{part, nchunks, stride, count, out};
  return reduce_rows_multi(J, scratch, st);
}

}  // namespace chg
