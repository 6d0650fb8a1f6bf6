// MWQ quantize + bit-plane pack (Sec. 3.3.1: Eq. 2 asymmetric base level,
// Eq. 4-5 binary residual levels, Algorithm 1 with X = I) and the debug
// unpack hook.
//
// The packed codes are integers decided by binary32 arithmetic, so this file
// is compiled without FMA contraction and every step runs in the same order
// as the specification in d2moe.h: one lane owns one (row, group) and walks its
// group sequentially.  Setup work, not on the timed path.
#pragma clang fp contract(off)

#include "internal.h"

namespace d2moe {
namespace {

constexpr int kPackRows = 64;  // rows (lanes) per workgroup

// One workgroup = 64 consecutive rows x one group of one expert.  The group's
// weights are staged in LDS (row stride group+1 floats: conflict-free column
// walks), then each lane quantizes its row sequentially.
template <int G>
__global__ __launch_bounds__(kPackRows) void pack_kernel(const float* __restrict__ W,
                                                         MwqView m, uint32_t* __restrict__ planes,
                                                         uint16_t* __restrict__ scales,
                                                         uint8_t* __restrict__ zeros) {
  __shared__ float R[kPackRows * (G + 1)];
  const int e = blockIdx.z, kb = blockIdx.y;
  const int n0 = blockIdx.x * kPackRows;
  const int lane = threadIdx.x;
  const int nrows = min(kPackRows, m.rows - n0);

  // cooperative, coalesced staging of W[e][n0 .. n0+63][kb*G .. +G]
  const float* src = W + ((size_t)e * m.rows + n0) * m.cols + (size_t)kb * G;
  for (int idx = lane; idx < nrows * G; idx += kPackRows) {
    const int r = idx / G, c = idx % G;
    R[r * (G + 1) + c] = src[(size_t)r * m.cols + c];
  }
  __syncthreads();
  if (lane >= nrows) return;

  const int n = n0 + lane;
  const int BR = 2048 / G;
  const int rb = n / BR, i = n % BR;
  const size_t blk = m.block(e, rb, kb);
  const int qmax = (1 << m.b_min) - 1;
  float* r = R + lane * (G + 1);

  // base level: min-max range including 0
  float mn = 0.0f, mx = 0.0f;
  for (int k = 0; k < G; ++k) {
    const float v = r[k];
    if (v < mn) mn = v;
    if (v > mx) mx = v;
  }
  const float range = mx - mn;
  const float s_raw = range / (float)qmax;
  uint16_t s_h = f2h(s_raw);
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

  // base codes -> planes 0 .. b_min-1; residual kept in LDS
  for (int sub = 0; sub < G / 32; ++sub) {
    uint32_t words[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int j = 0; j < 32; ++j) {
      const int k = sub * 32 + j;
      const float v = r[k];
      float qf = rintf(v / s1 + (float)z);
      qf = qf < 0.0f ? 0.0f : qf;
      qf = qf > (float)qmax ? (float)qmax : qf;
      const int q = (int)qf;
      const float what = (float)(q - z) * s1;
      r[k] = v - what;
      for (int p = 0; p < 8; ++p)
        if (p < m.b_min) words[p] |= (uint32_t)((q >> p) & 1) << j;
    }
    const int w = sub * BR + i;
    for (int p = 0; p < m.b_min; ++p) planes[m.plane_word(blk, p, w)] = words[p];
  }

  // residual levels: one sign plane + one scale per added bit
  for (int lev = 1; lev < m.levels(); ++lev) {
    float acc = 0.0f;
    for (int k = 0; k < G; ++k) acc = acc + fabsf(r[k]);
    const float s_mean = acc / (float)G;
    const uint16_t sb_h = f2h(s_mean);
    const float sb = h2f(sb_h);
    scales[m.scale_idx(blk, lev, i)] = sb_h;
    const int p = m.b_min + lev - 1;
    for (int sub = 0; sub < G / 32; ++sub) {
      uint32_t word = 0;
      for (int j = 0; j < 32; ++j) {
        const int k = sub * 32 + j;
        const float v = r[k];
        const bool pos = v >= 0.0f;
        word |= (uint32_t)pos << j;
        r[k] = pos ? (v - sb) : (v + sb);
      }
      planes[m.plane_word(blk, p, sub * BR + i)] = word;
    }
  }
}

// Element-wise unpack through the canonical addressing.
__global__ void debug_unpack_kernel(MwqView m, int e, int bits, uint8_t* __restrict__ q1,
                                    int8_t* __restrict__ signs) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)m.rows * m.cols;
  if (idx >= total) return;
  const int n = (int)(idx / m.cols), k = (int)(idx % m.cols);
  const int BR = m.BR();
  const size_t blk = m.block(e, n / BR, k / m.group);
  const int w = ((k % m.group) / 32) * BR + n % BR;
  const int bit = k % 32;
  int q = 0;
  for (int p = 0; p < m.b_min; ++p) q |= (int)((m.planes[m.plane_word(blk, p, w)] >> bit) & 1u) << p;
  q1[idx] = (uint8_t)q;
  for (int p = m.b_min; p < bits; ++p) {
    const int s = (int)((m.planes[m.plane_word(blk, p, w)] >> bit) & 1u);
    signs[(size_t)(p - m.b_min) * total + idx] = s ? (int8_t)1 : (int8_t)-1;
  }
}

}  // namespace

hipError_t launch_pack(const float* W, const d2moe_mwq* out, hipStream_t s) {
  MwqView m = view_of(out);
  dim3 grid((m.rows + kPackRows - 1) / kPackRows, m.cols / m.group, m.E);
  if (m.group == 64)
    pack_kernel<64><<<grid, kPackRows, 0, s>>>(W, m, out->planes, out->scales, out->zeros);
  else
    pack_kernel<128><<<grid, kPackRows, 0, s>>>(W, m, out->planes, out->scales, out->zeros);
  return hipGetLastError();
}

hipError_t launch_debug_unpack(const d2moe_mwq* w, int expert, int bits, uint8_t* q1,
                               int8_t* signs, hipStream_t s) {
  MwqView m = view_of(w);
  const size_t total = (size_t)m.rows * m.cols;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  debug_unpack_kernel<<<blocks, 256, 0, s>>>(m, expert, bits, q1, signs);
  return hipGetLastError();
}

}  // namespace d2moe
