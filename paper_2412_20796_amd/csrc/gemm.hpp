// fp32 MFMA GEMMs with gathered operands and fused epilogues (gfx950).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace chg {

// One K-segment of an NN product: rows of A (gathered by the problem's
// a_rows) times B. B element (k, n) = trans ? B[n*ldb + k] : B[k*ldb + n].
struct GemmSeg {
  const float* A;
  int lda;
  int a_col;  // first column of A used by this segment
  int K;
  const float* B;
  int ldb;
  int trans;
};

enum GemmAct { ACT_NONE = 0, ACT_SILU_OUT = 1, ACT_DSILU_MUL = 2 };

// C[c_rows(r), c] (+)= sum_seg A[a_rows(r), a_col + k] B(k, c) + bias[c]
//                      + res[res_rows(r), c]
// ACT_SILU_OUT: also C2[r, c] = silu(value).
// ACT_DSILU_MUL: value *= silu'(mul[r, c]) before bias/adds (backward of an
//                activation; use without bias/adds/res).
struct GemmProblem {
  int M, N;
  const int* a_rows;
  int nseg;
  GemmSeg seg[4];
  const float* bias;
  const float* res;
  int res_ld;
  const int* res_rows;
  float* C;
  int ldc;
  const int* c_rows;
  int accumulate;
  int act;
  float* C2;
  int ldc2;
  const float* mul;
  int mul_ld;
};

constexpr int kMaxGemmProblems = 6;
struct GemmBatch {
  int n;
  GemmProblem p[kMaxGemmProblems];
};

int gemm_launch(const GemmBatch& b, hipStream_t st, const char* tag);

// dW[m, n] (+)= sum_r X[x_rows(r), x_col + m] * Y[y_rows(r), y_col + n]
// over r in [0, R); X == nullptr means a single column of ones (M = 1, the
// bias gradient). Deterministic: per-chunk partials, then an ordered fp64 sum.
struct TnProblem {
  int R, M, N;
  const float* X;
  int ldx, x_col;
  const int* x_rows;
  const float* Y;
  int ldy, y_col;
  const int* y_rows;
  float* out;  // out[m * ld_out + n] += result
  int ld_out;
  // optional column split: columns [q*owidth, (q+1)*owidth) go to outs[q]
  // (outs[0] unused: out), owidth = 0 means a single output
  int owidth;
  float* outs[4];
};

constexpr int kMaxTnProblems = 16;
struct TnBatch {
  int n;
  TnProblem p[kMaxTnProblems];
};

// part: scratch of part_cap floats.
int tn_launch(const TnBatch& b, float* part, int64_t part_cap, hipStream_t st, const char* tag);

struct ReduceJob {
  const float* part;
  int nchunks;
  int64_t stride;
  int count;
  float* out;
};
constexpr int kMaxReduceJobs = 20;
struct ReduceJobs {
  int n;
  ReduceJob j[kMaxReduceJobs];
};
// Up to kMaxReduceJobs independent reductions in two launches (32 ordered
// group sums, then their ordered sum); scratch: n * 32 * 1024 doubles.
int reduce_rows_multi(const ReduceJobs& J, double* scratch, hipStream_t st);

// out[k] += sum_c part[c*stride + k] (k < count), in a fixed order, in fp64.
// scratch: 32 * count doubles.
int reduce_rows_launch(const float* part, int nchunks, int64_t stride, int count, float* out, double* scratch,
                       hipStream_t st);

}  // namespace chg
