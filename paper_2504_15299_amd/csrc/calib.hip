// Calibration-aware MWQ (Sec. 3.3.1: Eq. 3 and Eq. 5 minimise the output
// error ||WX - W^X||^2 over calibration activations X; Algorithm 1 quantizes
// the weights block by block and moves each block's quantization error onto
// the columns not yet quantized through H^c, the Cholesky factor of the
// inverse of H = 2 X X^T + lambda I).  Setup work, not on the timed path.
//
// Factor (binary64): U = upper-triangular factor with H^-1 = U^T U.  With J
// the order-reversing permutation, J H J = L L^T (lower Cholesky factor L)
// gives H = V V^T with V = J L J upper triangular, so H^-1 = V^-T V^-1 and
// U = V^-1 = J L^-1 J: one Cholesky factorization and one triangular
// inverse.  Both are blocked in 64 x 64 tiles; every tile product sums in a
// fixed order, so the factor is deterministic.
//
// Calibrated pack (binary32): the integer codes are decided exactly as the
// plain pack decides them (same per-group rules, same arithmetic, no FMA
// contraction), on targets that the compensation has moved; the
// compensation E = D U_BB^-1, T_F -= E U_BF is written as fmaf chains in
// ascending index order, one chain per element, so the GPU reproduces the
// CPU definition of the algorithm bit for bit.  Rows are independent: the
// update of a row's later columns uses only that row's block error.
#pragma clang fp contract(off)

#include "internal.h"

namespace d2moe {
namespace {

constexpr int FT = 64;  // factor tile

// ---- factor ----------------------------------------------------------------

__global__ void info_init_kernel(int32_t* info) { *info = 0; }

// Lower tiles of Hr = J H J, H[a][b] = 2 sum_t X[t][a] X[t][b] + lambda [a == b].
__global__ __launch_bounds__(256) void hessian_kernel(const float* __restrict__ X, int tokens,
                                                      int n, double lambda, double* __restrict__ A) {
  const int ti = blockIdx.y, tj = blockIdx.x;
  if (tj > ti) return;
  __shared__ double xa[16][FT], xb[16][FT];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  double acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0;
  for (int t0 = 0; t0 < tokens; t0 += 16) {
    for (int idx = threadIdx.x; idx < 16 * FT; idx += 256) {
      const int tt = idx / FT, c = idx % FT, t = t0 + tt;
      const int fa = n - 1 - (ti * FT + c), fb = n - 1 - (tj * FT + c);
      xa[tt][c] = t < tokens ? (double)X[(size_t)t * n + fa] : 0.0;
      xb[tt][c] = t < tokens ? (double)X[(size_t)t * n + fb] : 0.0;
    }
    __syncthreads();
#pragma unroll 4
    for (int tt = 0; tt < 16; ++tt) {
      double a[4], b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = xa[tt][ty * 4 + r];
#pragma unroll
      for (int c = 0; c < 4; ++c) b[c] = xb[tt][tx * 4 + c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fma(a[r], b[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i = ti * FT + ty * 4 + r, j = tj * FT + tx * 4 + c;
      A[(size_t)i * n + j] = 2.0 * acc[r][c] + (i == j ? lambda : 0.0);
    }
}

// Cholesky factorization of diagonal tile k (its trailing updates from the
// tiles left of it are already applied).  A non-positive pivot records its
// 1-based column in *info (first failure wins) and continues with pivot 1.
__global__ __launch_bounds__(256) void potrf_diag_kernel(double* __restrict__ A, int n, int k,
                                                         int32_t* __restrict__ info) {
  __shared__ double a[FT][FT + 1];
  const size_t base = (size_t)k * FT;
  for (int idx = threadIdx.x; idx < FT * FT; idx += 256) {
    const int r = idx / FT, c = idx % FT;
    a[r][c] = c <= r ? A[(base + r) * n + base + c] : 0.0;
  }
  __syncthreads();
  for (int j = 0; j < FT; ++j) {
    if (threadIdx.x == 0) {
      double d = a[j][j];
      if (!(d > 0.0)) {
        atomicCAS(info, 0, (int32_t)(base + j + 1));
        d = 1.0;
      }
      a[j][j] = sqrt(d);
    }
    __syncthreads();
    const double djj = a[j][j];
    for (int r = j + 1 + (int)threadIdx.x; r < FT; r += 256) a[r][j] = a[r][j] / djj;
    __syncthreads();
    for (int idx = threadIdx.x; idx < FT * FT; idx += 256) {
      const int r = idx / FT, c = idx % FT;
      if (c > j && r >= c) a[r][c] = fma(-a[r][j], a[c][j], a[r][c]);
    }
    __syncthreads();
  }
  for (int idx = threadIdx.x; idx < FT * FT; idx += 256) {
    const int r = idx / FT, c = idx % FT;
    A[(base + r) * n + base + c] = c <= r ? a[r][c] : 0.0;
  }
}

// Panel tiles below diagonal tile k: A[i][k] <- A[i][k] L_kk^-T (one lane
// per tile row, forward substitution in ascending column order).
__global__ __launch_bounds__(64) void trsm_kernel(double* __restrict__ A, int n, int k) {
  __shared__ double l[FT][FT + 1], b[FT][FT + 1];
  const size_t bk = (size_t)k * FT, bi = (size_t)(k + 1 + blockIdx.x) * FT;
  for (int idx = threadIdx.x; idx < FT * FT; idx += 64) {
    const int r = idx / FT, c = idx % FT;
    l[r][c] = A[(bk + r) * n + bk + c];
    b[r][c] = A[(bi + r) * n + bk + c];
  }
  __syncthreads();
  const int r = threadIdx.x;
  for (int j = 0; j < FT; ++j) {
    double v = b[r][j];
    for (int m = 0; m < j; ++m) v = fma(-b[r][m], l[j][m], v);
    b[r][j] = v / l[j][j];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < FT * FT; idx += 64) {
    const int rr = idx / FT, c = idx % FT;
    A[(bi + rr) * n + bk + c] = b[rr][c];
  }
}

// Trailing update of the lower tiles (i, j), k < j <= i:
// A[i][j] -= A[i][k] A[j][k]^T.
__global__ __launch_bounds__(256) void chol_update_kernel(double* __restrict__ A, int n, int k) {
  const int i = k + 1 + blockIdx.y, j = k + 1 + blockIdx.x;
  if (j > i) return;
  __shared__ double pa[FT][FT + 1], pb[FT][FT + 1];
  const size_t bk = (size_t)k * FT, bi = (size_t)i * FT, bj = (size_t)j * FT;
  for (int idx = threadIdx.x; idx < FT * FT; idx += 256) {
    const int r = idx / FT, c = idx % FT;
    pa[r][c] = A[(bi + r) * n + bk + c];
    pb[r][c] = A[(bj + r) * n + bk + c];
  }
  __syncthreads();
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  double acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0;
  for (int m = 0; m < FT; ++m) {
    double a[4], b[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) a[r] = pa[ty * 4 + r][m];
#pragma unroll
    for (int c = 0; c < 4; ++c) b[c] = pb[tx * 4 + c][m];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[r][c] = fma(a[r], b[c], acc[r][c]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const size_t o = (bi + ty * 4 + r) * n + bj + tx * 4 + c;
      A[o] = A[o] - acc[r][c];
    }
}

// Inverse of every lower-triangular diagonal tile: M_kk = L_kk^-1 (one lane
// per column, forward substitution).
__global__ __launch_bounds__(64) void trinv_diag_kernel(const double* __restrict__ L,
                                                        double* __restrict__ M, int n) {
  __shared__ double l[FT][FT + 1], y[FT][FT + 1];
  const size_t bk = (size_t)blockIdx.x * FT;
  for (int idx = threadIdx.x; idx < FT * FT; idx += 64) {
    const int r = idx / FT, c = idx % FT;
    l[r][c] = L[(bk + r) * n + bk + c];
  }
  __syncthreads();
  const int c = threadIdx.x;
  for (int r = 0; r < FT; ++r) {
    double v = r == c ? 1.0 : 0.0;
    for (int m = c; m < r; ++m) v = fma(-l[r][m], y[m][c], v);
    y[r][c] = r < c ? 0.0 : v / l[r][r];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < FT * FT; idx += 64) {
    const int r = idx / FT, cc = idx % FT;
    M[(bk + r) * n + bk + cc] = y[r][cc];
  }
}

// Block row i of M = L^-1 below the diagonal: for tile column k < i
// (workgroup k), M[i][k] = -M_ii (sum_{m=k}^{i-1} L[i][m] M[m][k]).
__global__ __launch_bounds__(256) void trinv_row_kernel(const double* __restrict__ L,
                                                        double* __restrict__ M, int n, int i) {
  const int k = blockIdx.x;
  __shared__ double pa[FT][FT + 1], pb[FT][FT + 1];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const size_t bi = (size_t)i * FT, bk = (size_t)k * FT;
  double acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0;
  for (int m = k; m < i; ++m) {
    const size_t bm = (size_t)m * FT;
    for (int idx = threadIdx.x; idx < FT * FT; idx += 256) {
      const int r = idx / FT, c = idx % FT;
      pa[r][c] = L[(bi + r) * n + bm + c];
      pb[r][c] = M[(bm + r) * n + bk + c];
    }
    __syncthreads();
    for (int q = 0; q < FT; ++q) {
      double a[4], b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = pa[ty * 4 + r][q];
#pragma unroll
      for (int c = 0; c < 4; ++c) b[c] = pb[q][tx * 4 + c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fma(a[r], b[c], acc[r][c]);
    }
    __syncthreads();
  }
  // T in pb, M_ii in pa; then M[i][k] = -M_ii T
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) pb[ty * 4 + r][tx * 4 + c] = acc[r][c];
  for (int idx = threadIdx.x; idx < FT * FT; idx += 256) {
    const int r = idx / FT, c = idx % FT;
    pa[r][c] = M[(bi + r) * n + bi + c];
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0;
  for (int q = 0; q < FT; ++q) {
    double a[4], b[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) a[r] = pa[ty * 4 + r][q];
#pragma unroll
    for (int c = 0; c < 4; ++c) b[c] = pb[q][tx * 4 + c];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[r][c] = fma(a[r], b[c], acc[r][c]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) M[(bi + ty * 4 + r) * n + bk + tx * 4 + c] = -acc[r][c];
}

// U[a][b] = M[n-1-a][n-1-b] rounded to binary32 on and above the diagonal.
__global__ __launch_bounds__(256) void reverse_round_kernel(const double* __restrict__ M,
                                                            float* __restrict__ U, int n) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)n * n) return;
  const int a = (int)(idx / n), b = (int)(idx % n);
  U[idx] = b >= a ? (float)M[(size_t)(n - 1 - a) * n + (n - 1 - b)] : 0.0f;
}

// ---- calibrated pack ---------------------------------------------------------

__global__ __launch_bounds__(256) void copy_rows_kernel(const float* __restrict__ src,
                                                        float* __restrict__ dst, size_t count) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < count) dst[i] = src[i];
}

constexpr int kMaxGamma = 128;  // compensation block size: 64 or 128 columns

// One lane per row: quantize block [b0, b0 + gamma) of level `lev` from the
// row's current targets T, write its codes into the packed layout, update
// the row's residual chain R, and solve E = D U_BB^-1 for its block error D.
//   W: the expert's original rows [N][h]; T, R: [N][h]; E: [N][gamma].
template <int G>
__global__ __launch_bounds__(64) void calib_quant_kernel(
    const float* __restrict__ W, const float* __restrict__ T, float* __restrict__ R,
    const float* __restrict__ U, float* __restrict__ E, MwqView m, uint32_t* __restrict__ planes,
    uint16_t* __restrict__ scales, uint8_t* __restrict__ zeros, int e, int lev, int b0,
    int gamma) {
  __shared__ float de[kMaxGamma * 64];  // lane-private columns: de[j * 64 + lane]
  const int lane = threadIdx.x;
  const int n = blockIdx.x * 64 + lane;
  if (n >= m.rows) return;  // no barrier below: the LDS columns are lane-private
  const int h = m.cols, BR = 2048 / G;
  const int rb = n / BR, i = n % BR;
  const int qmax = (1 << m.b_min) - 1;
  const float* t = T + (size_t)n * h;
  const float* w = W + (size_t)n * h;
  float* rr = R + (size_t)n * h;
  for (int c0 = b0; c0 < b0 + gamma; c0 += G) {
    const int kb = c0 / G;
    const size_t blk = m.block(e, rb, kb);
    if (lev == 0) {
      float mn = 0.0f, mx = 0.0f;
      for (int k = 0; k < G; ++k) {
        const float v = t[c0 + k];
        if (v < mn) mn = v;
        if (v > mx) mx = v;
      }
      const float range = mx - mn;
      uint16_t s_h = f2h(range / (float)qmax);
      float s1 = h2f(s_h);
      if (!(s1 > 0.0f) || __builtin_isinf(s1)) {
        s_h = 0x3c00u;
        s1 = 1.0f;
      }
      float zf = rintf(-mn / s1);
      zf = zf < 0.0f ? 0.0f : zf;
      zf = zf > (float)qmax ? (float)qmax : zf;
      const int z = (int)zf;
      zeros[m.zero_idx(blk, i)] = (uint8_t)z;
      scales[m.scale_idx(blk, 0, i)] = s_h;
      for (int sub = 0; sub < G / 32; ++sub) {
        uint32_t words[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int j = 0; j < 32; ++j) {
          const int k = c0 + sub * 32 + j;
          const float v = t[k];
          float qf = rintf(v / s1 + (float)z);
          qf = qf < 0.0f ? 0.0f : qf;
          qf = qf > (float)qmax ? (float)qmax : qf;
          const int q = (int)qf;
          const float what = (float)(q - z) * s1;
          de[(k - b0) * 64 + lane] = v - what;
          rr[k] = w[k] - what;
          for (int p = 0; p < 8; ++p)
            if (p < m.b_min) words[p] |= (uint32_t)((q >> p) & 1) << j;
        }
        for (int p = 0; p < m.b_min; ++p)
          planes[m.plane_word(blk, p, sub * BR + i)] = words[p];
      }
    } else {
      float acc = 0.0f;
      for (int k = 0; k < G; ++k) acc = acc + fabsf(t[c0 + k]);
      const uint16_t sb_h = f2h(acc / (float)G);
      const float sb = h2f(sb_h);
      scales[m.scale_idx(blk, lev, i)] = sb_h;
      const int p = m.b_min + lev - 1;
      for (int sub = 0; sub < G / 32; ++sub) {
        uint32_t word = 0;
        for (int j = 0; j < 32; ++j) {
          const int k = c0 + sub * 32 + j;
          const float v = t[k];
          const bool pos = v >= 0.0f;  // -0.0 >= 0: sign +1
          word |= (uint32_t)pos << j;
          de[(k - b0) * 64 + lane] = pos ? (v - sb) : (v + sb);
          rr[k] = pos ? (rr[k] - sb) : (rr[k] + sb);
        }
        planes[m.plane_word(blk, p, sub * BR + i)] = word;
      }
    }
  }
  // E = D U_BB^-1, forward substitution in ascending order
  for (int j = 0; j < gamma; ++j) {
    float v = de[j * 64 + lane];
    for (int q = 0; q < j; ++q)
      v = fmaf(-de[q * 64 + lane], U[(size_t)(b0 + q) * h + (b0 + j)], v);
    v = v / U[(size_t)(b0 + j) * h + (b0 + j)];
    de[j * 64 + lane] = v;
    E[(size_t)n * gamma + j] = v;
  }
}

// T[n][f] -= sum_j E[n][j] U[b0 + j][f] for the columns f >= b0 + gamma, as
// one fmaf chain per element in ascending j.  Tile: 64 rows x 32 columns,
// 4 x 4 per thread (128 threads).
constexpr int kUpdCols = 32;
__global__ __launch_bounds__(128) void calib_update_kernel(float* __restrict__ T,
                                                           const float* __restrict__ U,
                                                           const float* __restrict__ E, int N,
                                                           int h, int b0, int gamma) {
  __shared__ float es[64 * (kMaxGamma + 1)];   // [64][gamma + 1]
  __shared__ float us[kMaxGamma * kUpdCols];   // [gamma][32]
  const int n0 = blockIdx.y * 64;
  const int f0 = b0 + gamma + blockIdx.x * kUpdCols;
  for (int idx = threadIdx.x; idx < 64 * gamma; idx += 128) {
    const int r = idx / gamma, j = idx % gamma;
    es[r * (gamma + 1) + j] = n0 + r < N ? E[(size_t)(n0 + r) * gamma + j] : 0.0f;
  }
  for (int idx = threadIdx.x; idx < gamma * kUpdCols; idx += 128) {
    const int j = idx / kUpdCols, c = idx % kUpdCols;
    us[j * kUpdCols + c] = U[(size_t)(b0 + j) * h + f0 + c];
  }
  __syncthreads();
  const int tx = threadIdx.x % 8, ty = threadIdx.x / 8;
  float acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int n = n0 + ty * 4 + r;
      acc[r][c] = n < N ? T[(size_t)n * h + f0 + tx * 4 + c] : 0.0f;
    }
  for (int j = 0; j < gamma; ++j) {
    float ev[4], uv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) ev[r] = es[(ty * 4 + r) * (gamma + 1) + j];
#pragma unroll
    for (int c = 0; c < 4; ++c) uv[c] = us[j * kUpdCols + tx * 4 + c];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(-ev[r], uv[c], acc[r][c]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int n = n0 + ty * 4 + r;
    if (n < N)
#pragma unroll
      for (int c = 0; c < 4; ++c) T[(size_t)n * h + f0 + tx * 4 + c] = acc[r][c];
  }
}

}  // namespace

size_t calib_factor_workspace(int n) { return (size_t)2 * n * n * sizeof(double); }

hipError_t launch_calib_factor(const float* X, int tokens, int n, double lambda, float* U,
                               void* ws, int32_t* info, hipStream_t s) {
  double* A = (double*)ws;
  double* M = A + (size_t)n * n;
  const int nb = n / FT;
  info_init_kernel<<<1, 1, 0, s>>>(info);
  hessian_kernel<<<dim3(nb, nb), 256, 0, s>>>(X, tokens, n, lambda, A);
  for (int k = 0; k < nb; ++k) {
    potrf_diag_kernel<<<1, 256, 0, s>>>(A, n, k, info);
    if (k + 1 < nb) {
      trsm_kernel<<<nb - k - 1, 64, 0, s>>>(A, n, k);
      chol_update_kernel<<<dim3(nb - k - 1, nb - k - 1), 256, 0, s>>>(A, n, k);
    }
  }
  trinv_diag_kernel<<<nb, 64, 0, s>>>(A, M, n);
  for (int i = 1; i < nb; ++i) trinv_row_kernel<<<i, 256, 0, s>>>(A, M, n, i);
  const size_t total = (size_t)n * n;
  reverse_round_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(M, U, n);
  return hipGetLastError();
}

size_t calib_pack_workspace(int rows, int cols, int gamma) {
  return ((size_t)2 * rows * cols + (size_t)rows * gamma) * sizeof(float);
}

hipError_t launch_pack_calibrated(const float* W, const float* U, int gamma,
                                  const d2moe_mwq* out, void* ws, hipStream_t s) {
  const MwqView m = view_of(out);
  const int N = m.rows, h = m.cols;
  float* T = (float*)ws;
  float* R = T + (size_t)N * h;
  float* E = R + (size_t)N * h;
  const size_t count = (size_t)N * h;
  const unsigned cgrid = (unsigned)((count + 255) / 256);
  const int rgrid = (N + 63) / 64;
  for (int e = 0; e < m.E; ++e) {
    const float* We = W + (size_t)e * count;
    for (int lev = 0; lev < m.levels(); ++lev) {
      copy_rows_kernel<<<cgrid, 256, 0, s>>>(lev == 0 ? We : R, T, count);
      for (int b0 = 0; b0 < h; b0 += gamma) {
        if (m.group == 64)
          calib_quant_kernel<64><<<rgrid, 64, 0, s>>>(We, T, R, U, E, m, out->planes,
                                                      out->scales, out->zeros, e, lev, b0, gamma);
        else
          calib_quant_kernel<128><<<rgrid, 64, 0, s>>>(We, T, R, U, E, m, out->planes,
                                                       out->scales, out->zeros, e, lev, b0, gamma);
        if (b0 + gamma < h)
          calib_update_kernel<<<dim3((h - b0 - gamma) / kUpdCols, rgrid), 128, 0, s>>>(
              T, U, E, N, h, b0, gamma);
      }
    }
  }
  return hipGetLastError();
}

}  // namespace d2moe
